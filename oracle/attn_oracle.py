"""CPU oracle for decode-step attention over a paged KV cache.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

What is computed (Sec. 2.2: the engine keeps each sequence's keys and values
in a paged KV cache; Sec. 2.3: PagedAttention-style kernels run the attention
of a decoding step over it).  The paper gives no formula; this is the
textbook scaled dot-product softmax attention of one new query token per
sequence, with grouped-query heads as in the Llama-class models of Table 1:

  * the cache holds `num_pages` pages of `page_size` tokens; K and V are
    [num_pages][num_kv_heads][page_size][head_dim] arrays;
  * token t (0 <= t < L_s) of sequence s is slot t % page_size of physical
    page block_table[s][t // page_size];
  * query head h reads kv head h // G, G = num_q_heads / num_kv_heads;
  * a_t = scale * <q[s,h], K_t>,  w_t = exp(a_t) / sum_u exp(a_u),
    o[s,h] = sum_t w_t V_t;
  * an empty sequence (L_s = 0) has the zero vector as output.

Everything is in float64 (products of fp16 values are exact there), with the
row maximum subtracted before exp so that large scores do not overflow.  The
fp16 result is the float64 result rounded once.
"""

from __future__ import annotations

import numpy as np

# Tolerance for a result computed with fp32 arithmetic (any summation order,
# any split of the sequence), measured against W = sum_t w_t |V_t[d]|:
#   * both sides round to fp16 once: together at most 2^-10 |o| <= 2^-10 W;
#   * an fp32 score (a D-term dot product, then one multiply by an fp32
#     constant) is off by at most (D + 2) 2^-24 S in log units, with
#     S = max_t scale * sum_d |q_d K_t,d|, so each weight is off by a factor
#     within 1 +- eps, eps <= (D + 2) 2^-24 S, and the output by <= 2 eps W;
#   * fp32 sums of p_t V_t and of p_t (a few hundred terms deep in any order
#     the kernels use): well below 1e-4 W.
# With D = 128 the total stays below 2e-3 W while S <= 60, the precondition
# the tests check (random N(0, 1) inputs give S of about 10).  The absolute
# term covers fp16 subnormals.
ATTN_REL_TOL = 2e-3
ATTN_ABS_TOL = 1e-6
ATTN_MAX_SCORE_BOUND = 60.0


def _check_inputs(q, k_cache, v_cache, block_table, seq_lens):
    q = np.asarray(q)
    k_cache = np.asarray(k_cache)
    v_cache = np.asarray(v_cache)
    block_table = np.asarray(block_table)
    seq_lens = np.asarray(seq_lens)
    for name, a in (("q", q), ("k_cache", k_cache), ("v_cache", v_cache)):
        if a.dtype != np.float16:
            raise TypeError(f"{name} must be float16")
    if q.ndim != 3:
        raise ValueError("q must be [num_seqs, num_q_heads, head_dim]")
    if k_cache.ndim != 4 or k_cache.shape != v_cache.shape:
        raise ValueError("k_cache and v_cache must both be [pages, kv_heads, page_size, head_dim]")
    num_seqs, hq, d = q.shape
    num_pages, hkv, page_size, d2 = k_cache.shape
    if d2 != d:
        raise ValueError("head_dim of q and of the cache differ")
    if hkv < 1 or hq % hkv != 0:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    if block_table.ndim != 2 or block_table.shape[0] != num_seqs:
        raise ValueError("block_table must be [num_seqs, max_pages_per_seq]")
    if seq_lens.shape != (num_seqs,):
        raise ValueError("seq_lens must be [num_seqs]")
    max_pages = block_table.shape[1]
    for s in range(num_seqs):
        length = int(seq_lens[s])
        if length < 0 or length > max_pages * page_size:
            raise ValueError(f"sequence {s}: length {length} outside [0, {max_pages * page_size}]")
        used = block_table[s, : (length + page_size - 1) // page_size]
        if np.any(used < 0) or np.any(used >= num_pages):
            raise ValueError(f"sequence {s}: block table names a page outside [0, {num_pages})")
        if not np.all(np.isfinite(q[s])):
            raise ValueError("q must be finite")
    return q, k_cache, v_cache, block_table, seq_lens


def sequence_kv(cache: np.ndarray, table_row: np.ndarray, length: int, page_size: int) -> np.ndarray:
    """Logical [length, kv_heads, head_dim] view of one sequence's keys or
    values: token t is slot t % page_size of page table_row[t // page_size]."""
    t = np.arange(length)
    pages = table_row[t // page_size]
    slots = t % page_size
    return cache[pages, :, slots, :]


def decode_attention_f64(q, k_cache, v_cache, block_table, seq_lens, scale: float):
    """Return (o64, wabs, smax):

    o64[s, h, :]   the float64 attention output (see the module docstring);
    wabs[s, h, :]  sum_t w_t |V_t| per dimension, the scale of the tolerance;
    smax[s, h]     max_t scale * sum_d |q_d K_t,d|, which the tolerance
                   derivation assumes to stay below ATTN_MAX_SCORE_BOUND.
    """
    q, k_cache, v_cache, block_table, seq_lens = _check_inputs(q, k_cache, v_cache, block_table, seq_lens)
    num_seqs, hq, d = q.shape
    hkv, page_size = k_cache.shape[1], k_cache.shape[2]
    group = hq // hkv
    o64 = np.zeros((num_seqs, hq, d), dtype=np.float64)
    wabs = np.zeros((num_seqs, hq, d), dtype=np.float64)
    smax = np.zeros((num_seqs, hq), dtype=np.float64)
    for s in range(num_seqs):
        length = int(seq_lens[s])
        if length == 0:
            continue
        keys = sequence_kv(k_cache, block_table[s], length, page_size).astype(np.float64)
        values = sequence_kv(v_cache, block_table[s], length, page_size).astype(np.float64)
        for h in range(hq):
            kvh = h // group
            kk = keys[:, kvh, :]                      # [L, D]
            vv = values[:, kvh, :]                    # [L, D]
            qq = q[s, h].astype(np.float64)           # [D]
            a = scale * (kk @ qq)                     # scores, [L]
            e = np.exp(a - np.max(a))
            w = e / np.sum(e)                         # softmax weights
            o64[s, h] = w @ vv
            wabs[s, h] = w @ np.abs(vv)
            smax[s, h] = abs(scale) * np.max(np.abs(kk) @ np.abs(qq))
    return o64, wabs, smax


def decode_attention(q, k_cache, v_cache, block_table, seq_lens, scale: float) -> np.ndarray:
    """fp16 output [num_seqs, num_q_heads, head_dim]: the float64 result
    rounded once to binary16 (round to nearest even)."""
    o64, _, _ = decode_attention_f64(q, k_cache, v_cache, block_table, seq_lens, scale)
    return o64.astype(np.float16)


def attn_tol_bound(wabs: np.ndarray) -> np.ndarray:
    """Per-element bound on |o_gpu - o_ref| for an fp32 computation."""
    return ATTN_REL_TOL * np.asarray(wabs, dtype=np.float64) + ATTN_ABS_TOL


def attn_within_tolerance(o_gpu, o_ref, wabs) -> np.ndarray:
    """Element-wise pass mask; NaN or infinite GPU values never pass."""
    a = np.asarray(o_gpu).astype(np.float64)
    b = np.asarray(o_ref).astype(np.float64)
    diff = np.abs(a - b)
    return np.isfinite(a) & (diff <= attn_tol_bound(wabs))
