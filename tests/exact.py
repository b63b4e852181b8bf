"""Exact-arithmetic helpers used to pin the oracle.

Written independently of the oracle: IEEE binary rounding is implemented here
from its definition on exact rationals (fractions.Fraction), and the 4-bit
packing is expressed at the byte level (byte t of a row holds element 2t in
its low nibble and element 2t+1 in its high nibble) instead of the oracle's
shift-per-word formulation.
"""

from __future__ import annotations

import struct
from fractions import Fraction

import numpy as np

INF = float("inf")


def _round_half_even_int(v: Fraction) -> int:
    fl = v.numerator // v.denominator
    rem = v - fl
    if rem > Fraction(1, 2):
        return fl + 1
    if rem < Fraction(1, 2):
        return fl
    return fl if fl % 2 == 0 else fl + 1


def round_half_even(v: Fraction) -> int:
    """Nearest integer, ties to even."""
    return _round_half_even_int(Fraction(v))


def round_binary(v: Fraction, p: int, emin: int, emax: int):
    """Round exact v to the binary format with p-bit significand (incl. hidden
    bit), minimum normal exponent emin, maximum exponent emax.  Ties to even.
    Returns a Fraction, or +-inf on overflow."""
    v = Fraction(v)
    if v == 0:
        return Fraction(0)
    sign = -1 if v < 0 else 1
    a = abs(v)
    e = 0
    while a >= Fraction(2) ** (e + 1):
        e += 1
    while a < Fraction(2) ** e:
        e -= 1
    e = max(e, emin)
    quantum = Fraction(2) ** (e - (p - 1))
    n = _round_half_even_int(a / quantum)
    r = n * quantum
    max_finite = (2 - Fraction(2) ** (1 - p)) * Fraction(2) ** emax
    if r > max_finite:
        return sign * INF
    return sign * r


def round_fp16(v: Fraction):
    return round_binary(v, 11, -14, 15)


def round_fp32(v: Fraction):
    return round_binary(v, 24, -126, 127)


def fp16_to_fraction(bits: int) -> Fraction:
    """Exact value of an IEEE binary16 bit pattern (finite only)."""
    sign = -1 if bits & 0x8000 else 1
    exp = (bits >> 10) & 0x1F
    man = bits & 0x3FF
    assert exp != 0x1F, "non-finite fp16"
    if exp == 0:
        return sign * Fraction(man, 2**24)
    return sign * (1 + Fraction(man, 1024)) * Fraction(2) ** (exp - 15)


def fraction_to_fp16_bits(v) -> int:
    """Bit pattern of an exactly representable fp16 value (or +-inf)."""
    if v == INF:
        return 0x7C00
    if v == -INF:
        return 0xFC00
    v = Fraction(v)
    if v == 0:
        return 0
    sign = 0x8000 if v < 0 else 0
    a = abs(v)
    if a < Fraction(2) ** -14:
        man = a * 2**24
        assert man.denominator == 1 and man < 1024
        return sign | int(man)
    e = 0
    while a >= Fraction(2) ** (e + 1):
        e += 1
    while a < Fraction(2) ** e:
        e -= 1
    man = (a / Fraction(2) ** e - 1) * 1024
    assert man.denominator == 1, "not representable in fp16"
    return sign | ((e + 15) << 10) | int(man)


def f32(v) -> Fraction:
    """Exact value of a Python/NumPy float after conversion to fp32."""
    return Fraction(float(np.float32(v)))


def fp32_from_hex(s: str) -> np.float32:
    """Parse a C99 hex-float string and check it is exactly an fp32 value."""
    d = float.fromhex(s)
    f = np.float32(d)
    assert float(f) == d, f"{s} is not exactly representable in fp32"
    return f


def pack_codes_bytes(codes_row) -> np.ndarray:
    """Pack one row of 4-bit codes through the byte layout and reinterpret the
    little-endian bytes as uint32 words."""
    codes_row = [int(c) for c in codes_row]
    assert len(codes_row) % 8 == 0
    raw = bytearray()
    for t in range(len(codes_row) // 2):
        lo, hi = codes_row[2 * t], codes_row[2 * t + 1]
        assert 0 <= lo < 16 and 0 <= hi < 16
        raw.append(lo | (hi << 4))
    nwords = len(raw) // 4
    return np.array(struct.unpack("<%dI" % nwords, bytes(raw)), dtype=np.uint32)


def pack_codes_bytes_2d(codes) -> np.ndarray:
    codes = np.asarray(codes)
    return np.stack([pack_codes_bytes(r) for r in codes])


def quantize_group_exact(ws):
    """Reference quantization of one 32-element group in exact arithmetic:
    amax, fp32(amax / 7), fp16 of that, fp32(w / s16), round half even, +8,
    clamp [0, 15].  Returns (scale_bits, codes)."""
    wf = [Fraction(float(np.float32(w))) for w in ws]
    amax = max(abs(w) for w in wf)
    s32 = round_fp32(amax / 7)
    s16 = round_fp16(s32)
    bits = fraction_to_fp16_bits(s16)
    if s16 == 0:
        return bits, [8] * len(wf)
    codes = []
    for w in wf:
        r = round_fp32(w / s16)
        q = round_half_even(r) + 8
        codes.append(min(15, max(0, q)))
    return bits, codes


def exact_gemv_fp16_bits(codes, scale_bits, x_bits):
    """y bits = fp16(sum_k s16*(q-8)*x) with the sum done in exact rationals and
    a single exact rounding.  codes [N][K] ints, scale_bits [N][K/32] ints,
    x_bits [M][K] ints (fp16 bit patterns)."""
    n = len(codes)
    k = len(codes[0])
    m = len(x_bits)
    xs = [[fp16_to_fraction(b) for b in row] for row in x_bits]
    out = [[0] * n for _ in range(m)]
    for r in range(n):
        w_hat = [fp16_to_fraction(scale_bits[r][kk // 32]) * (codes[r][kk] - 8) for kk in range(k)]
        for mi in range(m):
            total = sum((w_hat[kk] * xs[mi][kk] for kk in range(k)), Fraction(0))
            out[mi][r] = fraction_to_fp16_bits(round_fp16(total))
    return out


def dequant_reference(packed, scale_bits, n: int, k: int) -> np.ndarray:
    """float64 w_hat [N, K] read through the byte layout: byte t of a row
    holds element 2t in its low nibble and 2t + 1 in its high nibble; each
    code q means (q - 8) times its group's fp16 scale."""
    raw = np.ascontiguousarray(np.asarray(packed, dtype=np.uint32)).view(np.uint8).reshape(n, k // 2)
    codes = np.empty((n, k), dtype=np.int64)
    codes[:, 0::2] = raw & 0xF
    codes[:, 1::2] = raw >> 4
    s = np.asarray(scale_bits, dtype=np.uint16).view(np.float16).astype(np.float64)
    return (codes - 8).astype(np.float64) * np.repeat(s, 32, axis=1)
