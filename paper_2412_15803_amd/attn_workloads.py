"""Seeded synthetic inputs for decode attention over a paged KV cache.

Only inputs are made here (query vectors, key/value pages, block tables and
sequence lengths); none of the attention arithmetic lives in this module, so
the HIP library's tests and the CPU oracle consume the same inputs without
sharing any of the method.

Shapes follow the decoder classes of the linears: a 3B-class layer has 24
query heads and 8 kv heads of 128, an 8B-class layer 32 and 8.  Keys, values
and queries are N(0, 1) in fp16 (the scale of normalised, rotated
activations); pages of 16 tokens are handed out in a random order, as in a
cache that has served and freed many sequences.  Entries of a block table
past a sequence's last page hold -1.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

HEAD_DIM = 128
PAGE_SIZE = 16


@dataclass(frozen=True)
class AttnShape:
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int = HEAD_DIM


LLAMA3B_ATTN = AttnShape("attn_3b", 24, 8)
LLAMA8B_ATTN = AttnShape("attn_8b", 32, 8)


def default_scale(head_dim: int) -> float:
    return float(1.0 / np.sqrt(head_dim))


def pages_needed(seq_lens, page_size: int) -> int:
    return int(sum((int(n) + page_size - 1) // page_size for n in seq_lens))


def attention_bytes(seq_lens, num_q_heads: int, num_kv_heads: int, head_dim: int,
                    page_size: int = PAGE_SIZE) -> int:
    """Bytes a decode-attention call must move at least once: every cached
    key and value of every sequence (fp16), the fp16 queries and outputs,
    the used block-table entries and the lengths (int32)."""
    tokens = int(sum(int(n) for n in seq_lens))
    num_seqs = len(seq_lens)
    return (2 * tokens * num_kv_heads * head_dim * 2
            + 2 * num_seqs * num_q_heads * head_dim * 2
            + 4 * pages_needed(seq_lens, page_size) + 4 * num_seqs)


# ----------------------------------------------------------------- host side

def block_table_host(seed: int, seq_lens, page_size: int, extra_pages: int = 0,
                     max_pages_per_seq: int | None = None):
    """Random distinct physical pages for every sequence.

    Returns (block_table int32 [S, max_pages_per_seq], num_pages)."""
    need = [(int(n) + page_size - 1) // page_size for n in seq_lens]
    width = max(need + [1]) if max_pages_per_seq is None else max_pages_per_seq
    if width < max(need + [0]):
        raise ValueError("max_pages_per_seq too small for the longest sequence")
    num_pages = sum(need) + extra_pages
    rng = np.random.default_rng(seed)
    order = rng.permutation(max(num_pages, 1)).astype(np.int32)
    table = np.full((len(seq_lens), width), -1, dtype=np.int32)
    at = 0
    for s, n in enumerate(need):
        table[s, :n] = order[at:at + n]
        at += n
    return table, max(num_pages, 1)


def kv_cache_host(seed: int, num_pages: int, num_kv_heads: int, page_size: int, head_dim: int):
    """(k_cache, v_cache), each fp16 [num_pages, num_kv_heads, page_size, head_dim]."""
    rng = np.random.default_rng(seed)
    shape = (num_pages, num_kv_heads, page_size, head_dim)
    k = rng.standard_normal(shape, dtype=np.float32).astype(np.float16)
    v = rng.standard_normal(shape, dtype=np.float32).astype(np.float16)
    return k, v


def q_host(seed: int, num_seqs: int, num_q_heads: int, head_dim: int):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((num_seqs, num_q_heads, head_dim), dtype=np.float32).astype(np.float16)


# --------------------------------------------------------------- device side

def kv_cache_device(seed: int, num_pages: int, num_kv_heads: int, page_size: int, head_dim: int,
                    device="cuda"):
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(seed)
    shape = (num_pages, num_kv_heads, page_size, head_dim)
    k = torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(torch.float16)
    v = torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(torch.float16)
    return k, v


def q_device(seed: int, num_seqs: int, num_q_heads: int, head_dim: int, device="cuda"):
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randn((num_seqs, num_q_heads, head_dim), generator=g, device=device,
                       dtype=torch.float32).to(torch.float16)
