"""Pins for the paged decode-attention oracle: closed forms, invariants, a
library routine on a dense copy, and hand-worked rounding cases.

Every pin takes an oracle namespace `orc` (oracle.attn_oracle, or a copy with
a planted mistake) and raises when it does not hold.  The expected values come
from constructions whose answer is known without the softmax formula (uniform
weights, a single dominant key, two keys and the logistic function), from
torch's own scaled_dot_product_attention on a dense copy of the keys and
values that the test lays out itself, or from exact rational arithmetic.
"""

from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

import attn_cases


def _run(orc, case, scale=None):
    scale = case.scale if scale is None else scale
    return orc.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                    case.seq_lens, scale)


def _run16(orc, case, scale=None):
    scale = case.scale if scale is None else scale
    return orc.decode_attention(case.q, case.k_cache, case.v_cache, case.block_table,
                                case.seq_lens, scale)


# ----------------------------------------------------------- library routine

def pin_matches_torch_sdpa(orc):
    """A dense copy of each sequence (pages concatenated in table order,
    built here page by page) through torch's float64 scaled-dot-product
    attention with grouped-query heads gives the same outputs."""
    import torch
    import torch.nn.functional as F

    for seed, (hq, hkv, d, page, lens) in enumerate([
        (6, 2, 16, 4, (7, 13, 1)),
        (8, 8, 32, 16, (40,)),
        (4, 1, 8, 8, (17, 64)),
    ]):
        case = attn_cases.random_case(100 + seed, hq, hkv, d, page, lens, extra_pages=5)
        o64, _, _ = _run(orc, case)
        for s, length in enumerate(lens):
            npg = (length + page - 1) // page
            kd = np.concatenate([case.k_cache[case.block_table[s, i]] for i in range(npg)], axis=1)[:, :length]
            vd = np.concatenate([case.v_cache[case.block_table[s, i]] for i in range(npg)], axis=1)[:, :length]
            qt = torch.from_numpy(case.q[s].astype(np.float64))[None, :, None, :]
            kt = torch.from_numpy(kd.astype(np.float64))[None]
            vt = torch.from_numpy(vd.astype(np.float64))[None]
            ref = F.scaled_dot_product_attention(qt, kt, vt, scale=case.scale, enable_gqa=True)
            ref = ref[0, :, 0, :].numpy()
            assert np.allclose(o64[s], ref, rtol=0, atol=1e-12), (seed, s, np.max(np.abs(o64[s] - ref)))


# ---------------------------------------------------------------- closed forms

def pin_uniform_weights_give_the_mean(orc):
    """q = 0 (or scale = 0) makes every weight 1/L: o is the exact mean of
    the values, compared as rationals and after one fp16 rounding."""
    case = attn_cases.integer_values_case(7, hq=4, hkv=2, d=8, page=4, lens=(1, 5, 12, 16))
    for variant in ("zero_q", "zero_scale"):
        if variant == "zero_q":
            c = case._replace(q=np.zeros_like(case.q))
            o64, wabs, _ = _run(orc, c)
            o16 = _run16(orc, c)
        else:
            o64, wabs, _ = _run(orc, case, scale=0.0)
            o16 = _run16(orc, case, scale=0.0)
        for s, length in enumerate(case.seq_lens):
            vals = attn_cases.logical_values(case, s)          # [L, HKV, D] ints
            for h in range(case.q.shape[1]):
                kvh = h // (case.q.shape[1] // case.k_cache.shape[1])
                for dd in range(case.q.shape[2]):
                    col = [int(v) for v in vals[:, kvh, dd]]
                    mean = Fraction(sum(col), int(length))
                    amean = Fraction(sum(abs(v) for v in col), int(length))
                    # 1/L is inexact in float64 for L = 5 or 12: allow its rounding
                    assert abs(Fraction(o64[s, h, dd]) - mean) <= Fraction(1, 2**44), (variant, s, h, dd)
                    assert abs(Fraction(wabs[s, h, dd]) - amean) <= Fraction(1, 2**44), (variant, s, h, dd)
                    # these means are never fp16 halfway cases, so one rounding decides
                    assert o16[s, h, dd] == np.float16(float(mean)), (variant, s, h, dd)


def pin_single_dominant_key_selects_its_value(orc):
    """Each query head picks out one token whose score exceeds every other
    by hundreds: its output is exactly that token's value vector.  Different
    heads of one kv group pick different tokens, so the head-to-kv-head map,
    the page lookup and the slot inside the page are all checked."""
    for big in (64.0, 2048.0):     # the second makes exp overflow unless shifted
        case, targets = attn_cases.one_hot_case(11, hq=6, hkv=2, d=16, page=4, lens=(9, 23), big=big)
        o16 = _run16(orc, case)
        o64, _, _ = _run(orc, case)
        for s in range(len(case.seq_lens)):
            vals = attn_cases.logical_values(case, s)
            for h in range(case.q.shape[1]):
                kvh = h // 3
                want = vals[targets[s][h], kvh]
                assert np.array_equal(o16[s, h], want), (big, s, h)
                assert np.all(np.isfinite(o64[s, h]))


def pin_two_keys_follow_the_logistic(orc):
    """With two tokens o = v0 + (v1 - v0) * sigma(a1 - a0), sigma(x) =
    (1 + tanh(x / 2)) / 2, where the scores a_t = scale * c * k_t[i] are set
    up along one coordinate i of q."""
    d, c, i = 8, 3.0, 5
    scale = 0.25
    for k0, k1 in ((1.0, 2.0), (-0.5, 0.75), (4.0, -4.0), (0.0, 0.0)):
        case = attn_cases.two_token_case(d=d, i=i, c=c, k0=k0, k1=k1, seed=5)
        o64, _, _ = _run(orc, case, scale=scale)
        x = scale * c * (k1 - k0)
        sig = (1.0 + math.tanh(x / 2.0)) / 2.0
        vals = attn_cases.logical_values(case, 0).astype(np.float64)
        want = vals[0, 0] + (vals[1, 0] - vals[0, 0]) * sig
        assert np.allclose(o64[0, 0], want, rtol=1e-14, atol=1e-15), (k0, k1)


def pin_single_token_is_its_value(orc):
    case = attn_cases.random_case(3, 4, 4, 16, 8, (1, 1), extra_pages=3)
    o16 = _run16(orc, case)
    for s in range(2):
        vals = attn_cases.logical_values(case, s)
        for h in range(4):
            assert np.array_equal(o16[s, h], vals[0, h]), (s, h)


def pin_empty_sequence_is_zero(orc):
    case = attn_cases.random_case(4, 4, 2, 16, 4, (0, 9, 0), extra_pages=2)
    o64, wabs, _ = _run(orc, case)
    assert np.all(o64[0] == 0) and np.all(o64[2] == 0)
    assert np.all(wabs[0] == 0)
    ref = _run(orc, attn_cases.select_sequences(case, [1]))[0]
    assert np.array_equal(o64[1], ref[0])


def pin_direct_fp16_rounding(orc):
    """The fp16 result is rounded once from float64.  Uniform weights over
    2^15 tokens whose values average to 1 + 2^-11 + 2^-25: just above the
    halfway point between fp16 1.0 and 1 + 2^-10, so the correct result is
    1 + 2^-10 (an fp32 intermediate would land on the tie and give 1.0)."""
    n = 1 << 15
    high = (n >> 1) + 1                      # tokens holding 1 + 2^-10
    vals = np.ones(n, dtype=np.float16)
    vals[:high] = np.float16(1.0 + 2.0 ** -10)
    case = attn_cases.dense_single_head_case(vals, page=1024, seed=9)
    o16 = _run16(orc, case, scale=0.0)
    assert o16.view(np.uint16)[0, 0, 0] == 0x3C01, hex(int(o16.view(np.uint16)[0, 0, 0]))


# ------------------------------------------------------------------ invariants

def pin_physical_page_order_is_irrelevant(orc):
    """Moving pages to other physical slots (and updating the table) does
    not change a single bit of the float64 result."""
    case = attn_cases.random_case(21, 6, 2, 16, 4, (11, 30), extra_pages=7)
    moved = attn_cases.shuffle_physical_pages(case, seed=22)
    a, _, _ = _run(orc, case)
    b, _, _ = _run(orc, moved)
    assert np.array_equal(a, b)


def pin_token_order_is_irrelevant(orc):
    """Attention over a set of (key, value) pairs does not depend on their
    order: reversing the tokens of a sequence changes only rounding."""
    case = attn_cases.random_case(31, 4, 2, 16, 4, (13, 29), extra_pages=3)
    rev = attn_cases.reverse_tokens(case)
    a, _, _ = _run(orc, case)
    b, _, _ = _run(orc, rev)
    assert np.allclose(a, b, rtol=0, atol=1e-13)


def pin_common_score_shift_is_irrelevant(orc):
    """Adding the same vector u to every key adds scale * <q, u> to every
    score of a head and leaves the weights unchanged."""
    case = attn_cases.integer_values_case(41, hq=4, hkv=2, d=8, page=4, lens=(6, 10))
    shifted = attn_cases.shift_keys(case, coord=2, delta=4.0)
    a, _, _ = _run(orc, case)
    b, _, _ = _run(orc, shifted)
    assert np.allclose(a, b, rtol=0, atol=1e-12)
    # and the shift is not a no-op on the scores themselves
    assert not np.array_equal(case.k_cache, shifted.k_cache)


def pin_output_is_a_convex_combination(orc):
    case = attn_cases.random_case(51, 8, 2, 32, 16, (1, 17, 100), extra_pages=4)
    o64, wabs, _ = _run(orc, case)
    for s, length in enumerate(case.seq_lens):
        vals = attn_cases.logical_values(case, s).astype(np.float64)
        for h in range(8):
            col = vals[:, h // 4, :]
            assert np.all(o64[s, h] >= col.min(axis=0) - 1e-12)
            assert np.all(o64[s, h] <= col.max(axis=0) + 1e-12)
            assert np.all(wabs[s, h] >= np.abs(o64[s, h]) - 1e-12)
            assert np.all(wabs[s, h] <= np.abs(col).max(axis=0) + 1e-12)


def pin_score_bound_closed_form(orc):
    """smax[s, h] = |scale| * max_t sum_d |q_d K_t,d|, worked by hand on a
    case where it differs from the largest signed score, from the largest
    |signed score| and from the same bound without |scale|.

    Pages of 2 tokens, sequence 0 of 3 tokens in pages [1, 0] (so token 2
    is slot 0 of page 0; slot 1 of page 0 holds an unused key of 9s), one
    empty sequence, 4 query heads on 2 kv heads, scale = -1/2.
      kv head 0: K_0 = (-1,-1,2,1), K_1 = (-2,1,0,1), K_2 = (0,0,4,0)
      kv head 1: K_0 = (1,1,1,1),   K_1 = (-3,0,0,0), K_2 = (0,-1,0,0)
      q_0 = (1,-2,0,3)  on kv 0: sum|qK| = 6, 7, 0 -> 7  (signed 4, -1, 0)
      q_1 = (0,0,1,0)   on kv 0: sum|qK| = 2, 0, 4 -> 4
      q_2 = (1,-2,0,3)  on kv 1: sum|qK| = 6, 3, 2 -> 6  (on kv 0 it would be 7)
      q_3 = (-1,0,0,0)  on kv 1: sum|qK| = 1, 3, 0 -> 3  (signed -1, 3, 0)
    so smax = (3.5, 2, 3, 1.5) for sequence 0 and 0 for the empty one."""
    d, page = 4, 2
    k = np.zeros((2, 2, page, d), dtype=np.float16)
    keys = {0: [(-1, -1, 2, 1), (-2, 1, 0, 1), (0, 0, 4, 0)],
            1: [(1, 1, 1, 1), (-3, 0, 0, 0), (0, -1, 0, 0)]}
    where = [(1, 0), (1, 1), (0, 0)]           # (page, slot) of tokens 0, 1, 2
    for kvh, rows in keys.items():
        for (pg, sl), row in zip(where, rows):
            k[pg, kvh, sl] = row
    k[0, :, 1] = 9.0                           # the unused slot
    v = np.ones_like(k)
    q = np.zeros((2, 4, d), dtype=np.float16)
    q[0] = [(1, -2, 0, 3), (0, 0, 1, 0), (1, -2, 0, 3), (-1, 0, 0, 0)]
    q[1] = q[0]
    table = np.array([[1, 0], [-1, -1]], dtype=np.int32)
    lens = np.array([3, 0], dtype=np.int32)
    _, _, smax = orc.decode_attention_f64(q, k, v, table, lens, -0.5)
    assert np.array_equal(smax, np.array([[3.5, 2.0, 3.0, 1.5], [0.0, 0.0, 0.0, 0.0]])), smax


# --------------------------------------------------------------- tolerance

def pin_tolerance_scale(orc):
    """At |o| = sum_t w_t |V_t| = 1 (all values 1), one fp16 ulp of error
    passes and three do not; NaN never passes."""
    one = np.float16(1.0)
    up1 = np.nextafter(one, np.float16(2))
    up3 = np.nextafter(np.nextafter(up1, np.float16(2)), np.float16(2))
    wabs = np.ones(3)
    ok = orc.attn_within_tolerance(np.array([up1, up3, np.float16(np.nan)]), np.array([one, one, one]), wabs)
    assert list(ok) == [True, False, False]
    # and the bound is taken against the weighted absolute values
    case = attn_cases.integer_values_case(61, hq=2, hkv=1, d=4, page=4, lens=(8,))
    case = case._replace(q=np.zeros_like(case.q))
    _, wabs, _ = _run(orc, case)
    vals = attn_cases.logical_values(case, 0).astype(np.float64)
    assert np.allclose(wabs[0, 0], np.abs(vals[:, 0, :]).mean(axis=0), rtol=0, atol=1e-15)


def pin_rejects_invalid_tables(orc):
    case = attn_cases.random_case(71, 2, 1, 8, 4, (9,), extra_pages=0)
    bad = case.block_table.copy()
    bad[0, 2] = case.k_cache.shape[0]
    for bt, lens in ((bad, case.seq_lens), (case.block_table, np.array([case.block_table.shape[1] * 4 + 1]))):
        try:
            orc.decode_attention_f64(case.q, case.k_cache, case.v_cache, bt, lens, case.scale)
        except ValueError:
            continue
        raise AssertionError("invalid table or length accepted")


ALL_PINS = [
    pin_matches_torch_sdpa,
    pin_uniform_weights_give_the_mean,
    pin_single_dominant_key_selects_its_value,
    pin_two_keys_follow_the_logistic,
    pin_single_token_is_its_value,
    pin_empty_sequence_is_zero,
    pin_direct_fp16_rounding,
    pin_physical_page_order_is_irrelevant,
    pin_token_order_is_irrelevant,
    pin_common_score_shift_is_irrelevant,
    pin_output_is_a_convex_combination,
    pin_tolerance_scale,
    pin_score_bound_closed_form,
    pin_rejects_invalid_tables,
]
