"""Pins for the CPU oracle: checks against hand-derived values, closed forms,
invariants and exact-rational brute force.

Every pin takes an oracle namespace `orc` (the real `oracle` package, or a
copy with a planted mistake) and raises AssertionError when it does not hold.
None of them re-types the oracle's formulas: the expected values come from
the fixtures under tests/golden/ (derived by hand), from closed forms, or from
the exact-arithmetic helpers in tests/exact.py.
"""

from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np

import exact

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _group_from_case(case):
    w = np.zeros(32, dtype=np.float32)
    for idx, hx in case["nonzero"].items():
        w[int(idx)] = exact.fp32_from_hex(hx)
    return w


# ------------------------------------------------------------------ packing

def pin_unpack_every_code_every_position(orc):
    """Each code 0..15 at each of the 8 positions of a word, built through the
    byte layout, is read back at element 8j+i and dequantizes to q - 8."""
    k = 64
    for pos in range(8):
        for code in range(16):
            codes = np.full((1, k), 8, dtype=np.int64)
            word = 5  # somewhere in the middle of the row
            codes[0, 8 * word + pos] = code
            codes[0, 8 * 2 + (7 - pos)] = 15 - code  # a second marker elsewhere
            packed = exact.pack_codes_bytes_2d(codes)
            scales = np.full((1, k // 32), 0x3C00, dtype=np.uint16)  # 1.0
            q, s16 = orc.unpack(packed, scales, 1, k)
            assert np.array_equal(q.astype(np.int64), codes), (pos, code)
            w_hat = orc.dequant(packed, scales, 1, k)
            assert np.array_equal(w_hat, (codes - 8).astype(np.float32)), (pos, code)


def pin_golden_quantize_groups(orc):
    """Hand-worked groups: ties to even, the stored fp16 scale as divisor,
    zero/underflowing/subnormal scales and the clamp."""
    for case in _load("quantize_groups.json")["cases"]:
        w = _group_from_case(case)[None, :]
        packed, scales = orc.quantize_pack(w)
        want_codes = np.array(case["codes"], dtype=np.int64)[None, :]
        want_packed = exact.pack_codes_bytes_2d(want_codes)
        assert int(scales[0, 0]) == int(case["scale_bits"], 16), case["name"]
        assert np.array_equal(packed, want_packed), case["name"]


def pin_golden_groups_in_any_row_and_group(orc):
    """The hand-worked groups placed at shuffled (row, group) slots of a larger
    matrix give the same scale and words there (no cross-group or cross-row
    leakage, right scale index)."""
    cases = _load("quantize_groups.json")["cases"]
    n, g = 4, 3
    slots = [(r, c) for r in range(n) for c in range(g)]
    order = np.random.default_rng(1).permutation(len(slots))
    w = np.zeros((n, 32 * g), dtype=np.float32)
    placed = []
    for case, si in zip(cases, order):
        r, c = slots[si]
        w[r, 32 * c:32 * c + 32] = _group_from_case(case)
        placed.append((r, c, case))
    packed, scales = orc.quantize_pack(w)
    for r, c, case in placed:
        assert int(scales[r, c]) == int(case["scale_bits"], 16), case["name"]
        want = exact.pack_codes_bytes(case["codes"])
        assert np.array_equal(packed[r, 4 * c:4 * c + 4], want), case["name"]


def pin_roundtrip_codes(orc):
    """Codes whose group holds a +-7 code and no 0 code, with a normal scale,
    survive dequantize -> quantize unchanged: max|w_hat| = 7*s16 so the
    recomputed scale is s16 again and each w_hat/s16 is the integer q - 8."""
    rng = np.random.default_rng(7)
    n, k = 6, 256
    codes = rng.integers(1, 16, size=(n, k))
    for r in range(n):
        for g in range(k // 32):
            codes[r, 32 * g + rng.integers(0, 32)] = rng.choice([1, 15])
    packed = exact.pack_codes_bytes_2d(codes)
    s = rng.uniform(2.0**-13, 2.0**3, size=(n, k // 32)).astype(np.float16)
    scales = s.view(np.uint16)
    w_hat = orc.dequant(packed, scales, n, k)
    p2, s2 = orc.quantize_pack(w_hat)
    assert np.array_equal(s2, scales)
    assert np.array_equal(p2, packed)


def pin_quantize_matches_exact_rationals(orc, seed=11, n=4, k=128):
    """Random groups (several magnitudes) against quantization carried out in
    exact rationals with IEEE rounding implemented from its definition."""
    rng = np.random.default_rng(seed)
    w = rng.standard_normal((n, k), dtype=np.float32) * np.float32(0.02)
    w[1] *= np.float32(3e-6)      # scales in the fp16 subnormal range
    w[2] *= np.float32(1e3)
    packed, scales = orc.quantize_pack(w)
    for r in range(n):
        for g in range(k // 32):
            bits, codes = exact.quantize_group_exact(w[r, 32 * g:32 * g + 32])
            assert int(scales[r, g]) == bits, (r, g)
            assert np.array_equal(packed[r, 4 * g:4 * g + 4], exact.pack_codes_bytes(codes)), (r, g)


def pin_quantization_error_bound(orc):
    """For groups with a normal stored scale: |w - w_hat| <= s16/2 (plus the
    fp32 division's rounding), and the group's max-magnitude element gets a
    code of 1 or 15."""
    rng = np.random.default_rng(3)
    n, k = 32, 512
    w = rng.standard_normal((n, k), dtype=np.float32) * np.float32(0.02)
    packed, scales = orc.quantize_pack(w)
    w_hat = orc.dequant(packed, scales, n, k)
    s16 = scales.view(np.float16).astype(np.float64)
    assert np.all(s16 >= 2.0**-14)
    per_elem = np.repeat(s16, 32, axis=1)
    err = np.abs(w.astype(np.float64) - w_hat.astype(np.float64))
    assert np.all(err <= per_elem * (0.5 + 8 * 2.0**-24))
    q, _ = orc.unpack(packed, scales, n, k)
    wg = np.abs(w.reshape(n, k // 32, 32))
    qg = q.reshape(n, k // 32, 32).astype(np.int64)
    at_max = np.take_along_axis(qg, np.argmax(wg, axis=2)[..., None], axis=2)[..., 0]
    assert np.all((at_max == 1) | (at_max == 15))


def pin_pack_deterministic_and_row_independent(orc):
    rng = np.random.default_rng(5)
    w = rng.standard_normal((20, 96), dtype=np.float32) * np.float32(0.02)
    p1, s1 = orc.quantize_pack(w)
    p2, s2 = orc.quantize_pack(w.copy())
    assert np.array_equal(p1, p2) and np.array_equal(s1, s2)
    rows = [0, 7, 19]
    p3, s3 = orc.quantize_pack(np.ascontiguousarray(w[rows]))
    assert np.array_equal(p3, p1[rows]) and np.array_equal(s3, s1[rows])


# --------------------------------------------------------------------- GEMV

def _case_arrays(case, k=32):
    codes = np.full((1, k), 8, dtype=np.int64)
    for idx, c in case["codes"].items():
        codes[0, int(idx)] = c
    x_bits = np.zeros((1, k), dtype=np.uint16)
    for idx, b in case["x_bits"].items():
        x_bits[0, int(idx)] = int(b, 16)
    packed = exact.pack_codes_bytes_2d(codes)
    scales = np.full((1, k // 32), int(case["scale_bits"], 16), dtype=np.uint16)
    return packed, scales, x_bits.view(np.float16)


def pin_golden_gemv(orc):
    for case in _load("gemv_cases.json")["cases"]:
        packed, scales, x = _case_arrays(case)
        y = orc.gemv(packed, scales, x, 1, 32)
        assert int(y.view(np.uint16)[0, 0]) == int(case["y_bits"], 16), case["name"]


def pin_gemv_one_hot(orc):
    """x = e_j returns fp16(w_hat[:, j]) exactly, for random codes and scales."""
    rng = np.random.default_rng(9)
    n, k = 8, 96
    codes = rng.integers(0, 16, size=(n, k))
    packed = exact.pack_codes_bytes_2d(codes)
    scales = rng.uniform(1e-3, 0.5, size=(n, k // 32)).astype(np.float16).view(np.uint16)
    cols = [0, 1, 31, 32, 47, 95]
    x = np.zeros((len(cols), k), dtype=np.float16)
    for i, c in enumerate(cols):
        x[i, c] = 1.0
    y = orc.gemv(packed, scales, x, n, k).view(np.uint16)
    for i, c in enumerate(cols):
        for r in range(n):
            want = exact.round_fp16(exact.fp16_to_fraction(int(scales[r, c // 32])) * (int(codes[r, c]) - 8))
            assert int(y[i, r]) == exact.fraction_to_fp16_bits(want), (i, r)


def pin_gemv_all_zero_and_all_max_codes(orc):
    """Codes all 0 dequantize to -8*s: with x = 1, y = fp16(-256 * sum_g s_g).
    Codes all 15 with one scale s and x = 1: y = fp16(7 * s * K)."""
    rng = np.random.default_rng(13)
    n, k = 4, 160
    scales = rng.uniform(1e-3, 1e-1, size=(n, k // 32)).astype(np.float16).view(np.uint16)
    packed = np.zeros((n, k // 8), dtype=np.uint32)
    x = np.ones((1, k), dtype=np.float16)
    y = orc.gemv(packed, scales, x, n, k).view(np.uint16)
    for r in range(n):
        total = sum((exact.fp16_to_fraction(int(b)) for b in scales[r]), Fraction(0)) * -256
        assert int(y[0, r]) == exact.fraction_to_fp16_bits(exact.round_fp16(total)), r
    s_bits = 0x2A3D  # an fp16 value with a full significand
    packed15 = exact.pack_codes_bytes_2d(np.full((n, k), 15))
    scales15 = np.full((n, k // 32), s_bits, dtype=np.uint16)
    y15 = orc.gemv(packed15, scales15, x, n, k).view(np.uint16)
    want = exact.fraction_to_fp16_bits(exact.round_fp16(7 * exact.fp16_to_fraction(s_bits) * k))
    assert np.all(y15 == want)


def pin_gemv_linearity(orc):
    """y64(a*x1 + b*x2) == a*y64(x1) + b*y64(x2) exactly, for powers of two
    a, b and small-integer x (every sum is then exact in fp64)."""
    rng = np.random.default_rng(17)
    n, k = 6, 128
    codes = rng.integers(0, 16, size=(n, k))
    packed = exact.pack_codes_bytes_2d(codes)
    scales = (2.0 ** rng.integers(-8, 0, size=(n, k // 32))).astype(np.float16).view(np.uint16)
    x1 = rng.integers(-8, 9, size=(1, k)).astype(np.float16)
    x2 = rng.integers(-8, 9, size=(1, k)).astype(np.float16)
    for a, b in [(1.0, 1.0), (2.0, -0.5), (-4.0, 0.25)]:
        xc = (np.float16(a) * x1 + np.float16(b) * x2).astype(np.float16)
        lhs = orc.gemv_f64(packed, scales, xc, n, k)
        rhs = a * orc.gemv_f64(packed, scales, x1, n, k) + b * orc.gemv_f64(packed, scales, x2, n, k)
        assert np.array_equal(lhs, rhs)


def pin_gemv_brute_force(orc):
    """Tiny random cases against the exact rational sum rounded once to fp16."""
    rng = np.random.default_rng(21)
    for (n, k, m) in [(1, 32, 1), (3, 32, 2), (4, 64, 3), (2, 64, 1)]:
        codes = rng.integers(0, 16, size=(n, k))
        packed = exact.pack_codes_bytes_2d(codes)
        scales = rng.uniform(1e-4, 0.2, size=(n, k // 32)).astype(np.float16).view(np.uint16)
        x = rng.standard_normal((m, k)).astype(np.float16)
        y = orc.gemv(packed, scales, x, n, k).view(np.uint16)
        want = exact.exact_gemv_fp16_bits(codes.tolist(), scales.tolist(), x.view(np.uint16).tolist())
        assert np.array_equal(y, np.array(want, dtype=np.uint16)), (n, k, m)


def pin_gemv_integer_exact(orc):
    """Every scale 2^-6 and x in {-4..4}: the result is an exact multiple of
    2^-6, equal to the integer sum of (q-8)*x times 2^-6."""
    rng = np.random.default_rng(23)
    n, k, m = 5, 256, 3
    codes = rng.integers(0, 16, size=(n, k))
    packed = exact.pack_codes_bytes_2d(codes)
    scales = np.full((n, k // 32), 0x2400, dtype=np.uint16)
    x = rng.integers(-4, 5, size=(m, k))
    y = orc.gemv_f64(packed, scales, x.astype(np.float16), n, k)
    want = (x @ (codes - 8).T).astype(np.float64) * 2.0**-6
    assert np.array_equal(y, want)


def pin_tolerance(orc):
    """The bound is 1e-3 * sum|w_hat x| + 1e-5: for x = e_j it is
    1e-3*|w_hat[n, j]| + 1e-5; for x = 0 it is exactly 1e-5.  Signed zeros
    compare equal, NaN never passes."""
    n, k = 2, 64
    codes = np.full((n, k), 8)
    codes[0, 3] = 1    # -7
    codes[1, 3] = 12   # +4
    packed = exact.pack_codes_bytes_2d(codes)
    scales = np.full((n, k // 32), 0x3800, dtype=np.uint16)  # 0.5
    x = np.zeros((2, k), dtype=np.float16)
    x[0, 3] = 1.0
    b = orc.tol_bound(packed, scales, x, n, k)
    assert b[0, 0] == 1e-3 * 3.5 + 1e-5 and b[0, 1] == 1e-3 * 2.0 + 1e-5
    assert b[1, 0] == 1e-5 and b[1, 1] == 1e-5
    ok = orc.within_tolerance(np.array([-0.0, np.nan, 1.0]), np.array([0.0, 0.0, 1.0 + 2e-5]), np.array([0.0, 1.0, 1e-5]))
    assert list(ok) == [True, False, False]


ALL_PINS = [
    pin_unpack_every_code_every_position,
    pin_golden_quantize_groups,
    pin_golden_groups_in_any_row_and_group,
    pin_roundtrip_codes,
    pin_quantize_matches_exact_rationals,
    pin_quantization_error_bound,
    pin_pack_deterministic_and_row_independent,
    pin_golden_gemv,
    pin_gemv_one_hot,
    pin_gemv_all_zero_and_all_max_codes,
    pin_gemv_linearity,
    pin_gemv_brute_force,
    pin_gemv_integer_exact,
    pin_tolerance,
]
