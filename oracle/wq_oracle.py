"""CPU oracle for 4-bit group-quantized decode linears (y = x . dequant(W)^T).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the tests, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code, tables or helpers with the HIP
library; both sides only receive the same seeded inputs.

What it computes
----------------
The paper (WebLLM, Sec. 1 and Sec. 3 / Table 1) decodes token by token with
"4-bit quantized" 1-8B models whose converted weights are produced ahead of
time (Sec. 2.3); the decode-step linear layers stream every weight once per
token.  The paper does not spell out the weight format, so this oracle fixes
one reading of it and every step below follows that reading:

* W is [N, K] (output x input, row-major); K is cut into groups of 32
  consecutive elements of one row.
* Per group: a = max|w| (exact), scale s32 = a / 7 as an IEEE fp32 division,
  stored scale s16 = fp16(s32) rounded to nearest-even with subnormals kept.
* Per element: if s16 == 0 the code is q = 8; otherwise r = w / fp32(s16)
  (IEEE fp32 division, i.e. the *stored* scale is the divisor) and
  q = clamp(round_half_even(r) + 8, 0, 15).
* Packing: eight 4-bit codes per little-endian uint32; element 8j+i of a row
  sits in bits [4i, 4i+4) of word j.  Scales are stored as fp16 bit patterns
  [N, K/32].
* Dequantization: w_hat = fp32(s16) * (q - 8), exact in fp32.
* GEMV: y[m, n] = sum_k w_hat[n, k] * x[m, k] with x in fp16, every product
  exact in fp64, the sum in fp64, and ONE rounding fp64 -> fp16 at the end.
* Tolerance for a GPU result: |y_gpu - y_ref| <= 1e-3 * sum_k |w_hat x| + 1e-5.

Every function is written for clarity, not speed; vectorisation is only over
independent elements and never changes a rounded result.
"""

from __future__ import annotations

import numpy as np

GROUP = 32          # elements per quantization group along K
CODES_PER_WORD = 8  # 4-bit codes per uint32 word
ZERO_CODE = 8       # the code that dequantizes to 0 (symmetric offset)
QMAX_CODE = 15
SCALE_DIVISOR = 7   # largest |q - 8| produced for a group's max element
REL_TOL = 1e-3
ABS_TOL = 1e-5


def _check_group(group: int) -> None:
    if group != GROUP:
        raise ValueError(f"only group={GROUP} is defined, got {group}")


def quantize_pack(w: np.ndarray, group: int = GROUP):
    """Quantize fp32 W[N, K] to packed uint32 [N, K/8] and fp16 scale bits [N, K/32].

    Follows the 4-bit weight conversion step (Sec. 2.3: converted weights made
    ahead of time; Table 1: 4-bit quantized models) in the reading given in
    the module docstring: scale from the group's max magnitude, division by
    the stored fp16 scale, round-half-even, +8 offset, clamp, nibble packing.
    """
    _check_group(group)
    w = np.asarray(w)
    if w.dtype != np.float32:
        raise TypeError("W must be float32")
    if w.ndim != 2:
        raise ValueError("W must be 2-D [N, K]")
    n, k = w.shape
    if k % group != 0:
        raise ValueError("K must be a multiple of the group size")
    if not np.all(np.isfinite(w)):
        raise ValueError("W must be finite")
    ngroups = k // group
    wg = w.reshape(n, ngroups, group)

    # Step 1: per-group maximum magnitude (exact).
    amax = np.max(np.abs(wg), axis=2)
    # Step 2: fp32 scale a / 7 (IEEE division), then fp16 round-to-nearest-even.
    s32 = (amax / np.float32(SCALE_DIVISOR)).astype(np.float32)
    s16 = s32.astype(np.float16)
    divisor = s16.astype(np.float32)

    # Step 3: codes.  A zero stored scale gives the zero code everywhere.
    q = np.full((n, ngroups, group), ZERO_CODE, dtype=np.int64)
    nonzero = divisor != 0
    r = (wg[nonzero] / divisor[nonzero][:, None]).astype(np.float32)
    rounded = np.rint(r).astype(np.int64)          # round half to even
    q[nonzero] = np.clip(rounded + ZERO_CODE, 0, QMAX_CODE)
    q = q.reshape(n, k)

    # Step 4: pack eight codes per word, element 8j+i in bits [4i, 4i+4).
    packed = np.zeros((n, k // CODES_PER_WORD), dtype=np.uint32)
    for i in range(CODES_PER_WORD):
        packed |= q[:, i::CODES_PER_WORD].astype(np.uint32) << np.uint32(4 * i)
    return packed, s16.view(np.uint16).copy()


def unpack(packed: np.ndarray, scales: np.ndarray, n: int, k: int, group: int = GROUP):
    """Return (codes uint8 [N, K], stored scales float16 [N, K/32]).

    Inverse of the packing step of `quantize_pack` (same reading of the
    4-bit format of Sec. 2.3 / Table 1).
    """
    _check_group(group)
    packed = np.asarray(packed, dtype=np.uint32)
    scales = np.asarray(scales, dtype=np.uint16)
    if packed.shape != (n, k // CODES_PER_WORD) or scales.shape != (n, k // group):
        raise ValueError("packed/scales shape mismatch")
    q = np.empty((n, k), dtype=np.uint8)
    for i in range(CODES_PER_WORD):
        q[:, i::CODES_PER_WORD] = (packed >> np.uint32(4 * i)) & np.uint32(0xF)
    return q, scales.view(np.float16)


def dequant(packed: np.ndarray, scales: np.ndarray, n: int, k: int, group: int = GROUP):
    """w_hat[N, K] = fp32(s16) * (q - 8), exact in fp32 (Sec. 2.3 reading)."""
    q, s16 = unpack(packed, scales, n, k, group)
    per_element_scale = np.repeat(s16.astype(np.float32), group, axis=1)
    return (q.astype(np.float32) - np.float32(ZERO_CODE)) * per_element_scale


def gemv_f64(packed, scales, x, n: int, k: int, group: int = GROUP, row_chunk: int = 2048):
    """Unrounded y64[M, N] = sum_k w_hat[n, k] * x[m, k] in fp64.

    The decode-step linear layer (Sec. 1 and Table 1: token-by-token decoding
    with 4-bit weights) is a plain matrix-vector product with the
    dequantized weights.  Each product is exact in fp64 (at most 15 + 11
    significant bits); the sum is an fp64 sum.  Rows are processed in chunks
    only to bound memory.
    """
    x = np.asarray(x)
    if x.dtype != np.float16:
        raise TypeError("x must be float16")
    if x.ndim != 2 or x.shape[1] != k:
        raise ValueError("x must be [M, K]")
    m = x.shape[0]
    x64 = x.astype(np.float64)
    y64 = np.empty((m, n), dtype=np.float64)
    for r0 in range(0, n, row_chunk):
        r1 = min(n, r0 + row_chunk)
        w_hat = dequant(packed[r0:r1], scales[r0:r1], r1 - r0, k, group).astype(np.float64)
        for mi in range(m):
            y64[mi, r0:r1] = np.sum(w_hat * x64[mi][None, :], axis=1)
    return y64


def gemv(packed, scales, x, n: int, k: int, group: int = GROUP):
    """y[M, N] in fp16: the fp64 result rounded ONCE, directly, to fp16."""
    return gemv_f64(packed, scales, x, n, k, group).astype(np.float16)


def tol_bound(packed, scales, x, n: int, k: int, group: int = GROUP, row_chunk: int = 2048):
    """Allowed |y_gpu - y_ref| per element: 1e-3 * sum_k |w_hat x| + 1e-5 (fp64)."""
    x64 = np.abs(np.asarray(x, dtype=np.float16).astype(np.float64))
    m = x64.shape[0]
    out = np.empty((m, n), dtype=np.float64)
    for r0 in range(0, n, row_chunk):
        r1 = min(n, r0 + row_chunk)
        w_abs = np.abs(dequant(packed[r0:r1], scales[r0:r1], r1 - r0, k, group).astype(np.float64))
        for mi in range(m):
            out[mi, r0:r1] = np.sum(w_abs * x64[mi][None, :], axis=1)
    return REL_TOL * out + ABS_TOL


def within_tolerance(y_test, y_ref, bound):
    """Boolean mask: |f64(y_test) - f64(y_ref)| <= bound.  +0 and -0 compare
    equal, equal infinities compare equal, any NaN fails."""
    a = np.asarray(y_test).astype(np.float64)
    b = np.asarray(y_ref).astype(np.float64)
    with np.errstate(invalid="ignore"):
        diff = np.abs(a - b)
    return (a == b) | (np.isfinite(diff) & (diff <= bound))
