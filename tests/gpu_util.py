"""Helpers for the GPU parity tests: move seeded inputs to the device, call the
HIP library through its C-ABI binding, bring results back as NumPy."""

from __future__ import annotations

import sys

import numpy as np

DEV = "cuda:0"


def announce(msg: str) -> None:
    print(f"\n[gpu] {msg}", flush=True)
    sys.stdout.flush()


def require_gpu():
    import pytest
    import torch

    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a visible GPU")


def to_dev(a: np.ndarray):
    import torch

    a = np.ascontiguousarray(a)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    elif a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(DEV)


def to_host(t, dtype) -> np.ndarray:
    return t.detach().cpu().numpy().view(dtype)


def gpu_pack(w_dev):
    import torch

    from paper_2412_15803_amd import wq

    n, k = w_dev.shape
    packed = torch.empty((n, k // 8), dtype=torch.int32, device=w_dev.device)
    scales = torch.empty((n, k // 32), dtype=torch.float16, device=w_dev.device)
    wq.wq_pack(w_dev, packed, scales)
    return packed, scales


def gpu_gemv(packed, scales, x):
    import torch

    from paper_2412_15803_amd import wq

    m = x.shape[0]
    n = packed.shape[0]
    y = torch.full((m, n), float("nan"), dtype=torch.float16, device=x.device)
    wq.wq_gemv(packed, scales, x, y)
    return y


def sample_rows(n: int, count: int, seed: int) -> np.ndarray:
    """Sorted distinct rows: the first and last few rows plus random ones."""
    if n <= count:
        return np.arange(n)
    rng = np.random.default_rng(seed)
    edge = [0, 1, 2, n // 2, n - 3, n - 2, n - 1]
    rest = rng.choice(n, size=count, replace=False)
    return np.unique(np.concatenate([edge, rest]))
