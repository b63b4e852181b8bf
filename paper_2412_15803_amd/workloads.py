"""Seeded synthetic workloads for the 4-bit decode linears.

This module only *generates inputs* (shapes, seeded fp32 weights, fp16
activations, raw packed words for structured tests).  It holds none of the
quantization or GEMV arithmetic, so both the HIP library's tests and the CPU
oracle can consume the same inputs without sharing any of the method.

Shapes stand in for the paper's 1-8B decoder models (Sec. 1; Table 1 runs
Llama-3.1-8B and Phi-3.5-mini, 4-bit): a Llama-3.2-3B-like layer (hidden
3072, 24 query / 8 kv heads of 128, intermediate 8192, vocabulary 128256) and
a Llama-3.1-8B-like layer (hidden 4096, 32 / 8 heads, intermediate 14336).
No trained weights are used: W ~ N(0, 0.02^2) in fp32, x ~ N(0, 1) in fp16.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

WEIGHT_STD = 0.02


@dataclass(frozen=True)
class Linear:
    name: str
    n: int  # output features (rows of W)
    k: int  # input features (columns of W)


# One decoder layer's linears, fused the way decode engines run them.
LLAMA3B_LAYER = (
    Linear("qkv", 5120, 3072),        # (24 + 2*8) heads * 128
    Linear("o", 3072, 3072),
    Linear("gate_up", 16384, 3072),   # 2 * 8192
    Linear("down", 3072, 8192),
)
LLAMA3B_LAYERS = 28
LLAMA3B_LM_HEAD = Linear("lm_head", 128256, 3072)

LLAMA8B_LAYER = (
    Linear("qkv", 6144, 4096),        # (32 + 2*8) heads * 128
    Linear("o", 4096, 4096),
    Linear("gate_up", 28672, 4096),   # 2 * 14336
    Linear("down", 4096, 14336),
)

SMALL_GEMV = Linear("gemv_512", 512, 512)

# Tensor-parallel shard shapes (one GPU's share at TP=8 of the 8B layer);
# used only as extra narrow/short shapes in the parity tests.
LLAMA8B_TP8_SHARDS = (
    Linear("gate_up_tp8", 3584, 4096),
    Linear("down_tp8", 4096, 1792),
)


def decode_step_linears(base_seed: int = 1234):
    """The 3B-class decode step: 28 x (qkv, o, gate_up, down) + lm_head.

    Returns a list of (Linear, weight_seed, x_seed) in execution order.
    """
    out = []
    for layer in range(LLAMA3B_LAYERS):
        for lid, lin in enumerate(LLAMA3B_LAYER):
            ws = base_seed + 10 * layer + lid
            out.append((Linear(f"l{layer}.{lin.name}", lin.n, lin.k), ws, ws + 100_000))
    ws = base_seed + 999
    out.append((LLAMA3B_LM_HEAD, ws, ws + 100_000))
    return out


def decode_step_linears_8b(base_seed: int = 4321):
    """The 8B-class step: 32 x (qkv, o, gate_up, down) + lm_head 128256x4096.

    Returns a list of (Linear, weight_seed, x_seed) in execution order.
    """
    out = []
    for layer in range(32):
        for lid, lin in enumerate(LLAMA8B_LAYER):
            ws = base_seed + 10 * layer + lid
            out.append((Linear(f"l{layer}.{lin.name}", lin.n, lin.k), ws, ws + 100_000))
    ws = base_seed + 999
    out.append((Linear("lm_head", 128256, 4096), ws, ws + 100_000))
    return out


def ideal_bytes(n: int, k: int, m: int) -> int:
    """Bytes a decode linear must move at least once: packed 4-bit codes,
    fp16 group scales, fp16 x and fp16 y."""
    return n * k // 2 + n * (k // 32) * 2 + 2 * m * k + 2 * m * n


# ----------------------------------------------------------------- host side

def weights_host(seed: int, n: int, k: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.standard_normal((n, k), dtype=np.float32) * np.float32(WEIGHT_STD)


def x_host(seed: int, m: int, k: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.standard_normal((m, k), dtype=np.float32).astype(np.float16)


def random_words_host(seed: int, n: int, k: int) -> np.ndarray:
    """Uniformly random packed words [N, K/8] (every 4-bit code equally likely)."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, 2**32, size=(n, k // 8), dtype=np.uint64).astype(np.uint32)


def constant_scales_host(n: int, k: int, bits: int) -> np.ndarray:
    return np.full((n, k // 32), bits, dtype=np.uint16)


def random_scales_host(seed: int, n: int, k: int, lo: float = 1e-4, hi: float = 1e-2) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.uniform(lo, hi, size=(n, k // 32)).astype(np.float16).view(np.uint16)


def pow2_scales_host(seed: int, n: int, k: int, lo_exp: int = -10, hi_exp: int = -6) -> np.ndarray:
    """fp16 scale bits 2^e, e drawn per (row, group) from [lo_exp, hi_exp]:
    every scaled code is exact in fp16, so sums of small-integer x stay
    exact while each group still has its own scale."""
    rng = np.random.default_rng(seed)
    e = rng.integers(lo_exp, hi_exp + 1, size=(n, k // 32))
    return np.ldexp(np.ones_like(e, dtype=np.float64), e).astype(np.float16).view(np.uint16)


def small_int_x_host(seed: int, m: int, k: int, lim: int = 4) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(-lim, lim + 1, size=(m, k)).astype(np.float16)


def one_hot_x_host(m: int, k: int, cols) -> np.ndarray:
    x = np.zeros((m, k), dtype=np.float16)
    for i, c in enumerate(cols):
        x[i, c] = 1.0
    return x


# --------------------------------------------------------------- device side

def weights_device(seed: int, n: int, k: int, device="cuda"):
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(seed)
    w = torch.randn((n, k), generator=g, device=device, dtype=torch.float32)
    return w.mul_(WEIGHT_STD)


def x_device(seed: int, m: int, k: int, device="cuda"):
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randn((m, k), generator=g, device=device, dtype=torch.float32).to(torch.float16)
