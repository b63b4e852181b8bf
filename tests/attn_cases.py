"""Structured inputs for the decode-attention tests (oracle pins and GPU
parity): random caches, caches with a known answer, and rearrangements that
must not change the answer.  Built on the seeded generators of
paper_2412_15803_amd.attn_workloads; no attention arithmetic here.

Addressing used throughout: token t of sequence s sits in slot t % P of page
block_table[s][t // P]; a cache is [pages, kv_heads, P, head_dim].
"""

from __future__ import annotations

from typing import NamedTuple

import numpy as np

from paper_2412_15803_amd import attn_workloads as aw


class AttnCase(NamedTuple):
    q: np.ndarray            # fp16 [S, HQ, D]
    k_cache: np.ndarray      # fp16 [pages, HKV, P, D]
    v_cache: np.ndarray      # fp16 [pages, HKV, P, D]
    block_table: np.ndarray  # int32 [S, max_pages]
    seq_lens: np.ndarray     # int32 [S]
    scale: float


def random_case(seed, hq, hkv, d, page, lens, extra_pages=0, max_pages=None):
    table, num_pages = aw.block_table_host(seed, lens, page, extra_pages, max_pages)
    k, v = aw.kv_cache_host(seed + 1, num_pages, hkv, page, d)
    q = aw.q_host(seed + 2, len(lens), hq, d)
    return AttnCase(q, k, v, table, np.asarray(lens, dtype=np.int32), aw.default_scale(d))


def _token_addr(case, s, t):
    page = case.block_table[s][t // case.k_cache.shape[2]]
    return int(page), t % case.k_cache.shape[2]


def logical_keys(case, s):
    """[L, HKV, D] keys of sequence s, page by page in table order."""
    return _logical(case.k_cache, case, s)


def logical_values(case, s):
    return _logical(case.v_cache, case, s)


def _logical(cache, case, s):
    length = int(case.seq_lens[s])
    page = cache.shape[2]
    parts = []
    for i in range((length + page - 1) // page):
        blk = cache[case.block_table[s][i]]            # [HKV, P, D]
        parts.append(np.transpose(blk, (1, 0, 2)))     # [P, HKV, D]
    if not parts:
        return np.zeros((0,) + (cache.shape[1], cache.shape[3]), dtype=cache.dtype)
    return np.concatenate(parts, axis=0)[:length]


def integer_values_case(seed, hq, hkv, d, page, lens, extra_pages=2):
    """Keys in {-4..4}, values in {-8..8} (exact in fp16 and in every fp32
    sum of up to 2^20 of them), queries N(0, 1/4)."""
    base = random_case(seed, hq, hkv, d, page, lens, extra_pages)
    rng = np.random.default_rng(seed + 3)
    k = rng.integers(-4, 5, size=base.k_cache.shape).astype(np.float16)
    v = rng.integers(-8, 9, size=base.v_cache.shape).astype(np.float16)
    q = (base.q.astype(np.float32) * 0.5).astype(np.float16)
    return base._replace(q=q, k_cache=k, v_cache=v)


def one_hot_case(seed, hq, hkv, d, page, lens, big=200.0, extra_pages=3, max_pages=None):
    """Every query head h of sequence s has a single coordinate i_h set; the
    kv group's keys are zero along i_h except at one target token, where the
    score is `big` (natural-log units).  All other scores of the head are 0,
    so with big >= 104 every other weight is exactly 0 even in fp32 and the
    output is exactly the target's value vector.

    Returns (case, targets) with targets[s][h] the target token."""
    case = random_case(seed, hq, hkv, d, page, lens, extra_pages, max_pages)
    q = np.zeros_like(case.q)
    k = case.k_cache.copy()
    rng = np.random.default_rng(seed + 7)
    g = hq // hkv
    amp = np.float16(np.sqrt(big / case.scale))
    targets = []
    for s, length in enumerate(case.seq_lens):
        length = int(length)
        tg = [0] * hq
        if length == 0:
            targets.append(tg)
            continue
        for kvh in range(hkv):
            dims = rng.choice(d, size=g, replace=False)
            # clear the chosen coordinates for every token of this sequence
            for t in range(length):
                p, slot = _token_addr(case, s, t)
                k[p, kvh, slot, dims] = 0
            for j in range(g):
                h = kvh * g + j
                tgt = int(rng.integers(0, length))
                tg[h] = tgt
                q[s, h, dims[j]] = amp
                p, slot = _token_addr(case, s, tgt)
                k[p, kvh, slot, dims[j]] = amp
        targets.append(tg)
    return case._replace(q=q, k_cache=k), targets


def two_token_case(d, i, c, k0, k1, seed):
    """One sequence of two tokens, one query and one kv head; q = c e_i and
    the keys' coordinate i is k0 and k1."""
    case = random_case(seed, 1, 1, d, 4, (2,), extra_pages=1)
    q = np.zeros_like(case.q)
    q[0, 0, i] = c
    k = case.k_cache.copy()
    p, slot = _token_addr(case, 0, 0)
    k[p, 0, slot, i] = k0
    p, slot = _token_addr(case, 0, 1)
    k[p, 0, slot, i] = k1
    return case._replace(q=q, k_cache=k)


def dense_single_head_case(vals, page, seed):
    """One sequence, one head of width 1 whose values are `vals`."""
    vals = np.asarray(vals, dtype=np.float16)
    case = random_case(seed, 1, 1, 1, page, (len(vals),), extra_pages=2)
    v = case.v_cache.copy()
    for t, val in enumerate(vals):
        p, slot = _token_addr(case, 0, t)
        v[p, 0, slot, 0] = val
    return case._replace(v_cache=v)


def select_sequences(case, idx):
    idx = list(idx)
    return case._replace(q=case.q[idx], block_table=case.block_table[idx], seq_lens=case.seq_lens[idx])


def shuffle_physical_pages(case, seed):
    """Move page p to physical slot perm[p] and rewrite the table."""
    n = case.k_cache.shape[0]
    perm = np.random.default_rng(seed).permutation(n)
    k = np.empty_like(case.k_cache)
    v = np.empty_like(case.v_cache)
    k[perm] = case.k_cache
    v[perm] = case.v_cache
    table = np.where(case.block_table >= 0, perm[np.maximum(case.block_table, 0)], -1).astype(np.int32)
    return case._replace(k_cache=k, v_cache=v, block_table=table)


def reverse_tokens(case):
    """Store every sequence's tokens in reverse order (same pages)."""
    k = case.k_cache.copy()
    v = case.v_cache.copy()
    for s, length in enumerate(case.seq_lens):
        length = int(length)
        lk, lv = logical_keys(case, s), logical_values(case, s)
        for t in range(length):
            p, slot = _token_addr(case, s, length - 1 - t)
            k[p, :, slot, :] = lk[t]
            v[p, :, slot, :] = lv[t]
    return case._replace(k_cache=k, v_cache=v)


def shift_keys(case, coord, delta):
    k = case.k_cache.astype(np.float32)
    k[..., coord] += np.float32(delta)
    k16 = k.astype(np.float16)
    assert np.array_equal(k16.astype(np.float32), k), "shifted keys must stay exact in fp16"
    return case._replace(k_cache=k16)
