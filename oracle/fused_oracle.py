"""CPU oracle for the operations fused around the decode linears of a layer.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

The paper's compiler fuses kernels at the graph level (Sec. 2.3); in the
Llama-class decoders of Table 1 the elementwise work that sits next to the
decode linears is RMS normalisation before the QKV and gate/up projections,
the SiLU-gated product before the down projection, the residual additions
after the O and down projections, and the choice of the next token from the
final logits.  The paper writes none of them down; these are their textbook
definitions, in float64, each fp16 result rounded once:

  * RMSNorm:  x_eff[k] = x[k] / sqrt(mean_j x[j]^2 + eps) * g[k]
  * SiLU-mul: for x of length 2K, x_eff[k] = silu(x[k]) * x[K + k],
              silu(a) = a / (1 + exp(-a))
  * x_eff is the fp16 input of the linear (the rounded prologue result);
  * residual: y[n] = sum_k w_hat[n, k] x_eff[k] + r[n], rounded once;
  * argmax:   the smallest index n of the largest y[n] (fp16 values).
"""

from __future__ import annotations

import numpy as np

from . import wq_oracle

PRO_NONE = 0
PRO_RMSNORM = 1
PRO_SILU_MUL = 2

# Tolerance of a fused linear computed in fp32, against
# V = sum_k |w_hat[n, k] x_eff[k]| + |r[n]|:
#   * the plain linear's own bound (1e-3 of sum |w_hat x| + 1e-5, both
#     roundings of y included; adding r in fp32 before the one rounding
#     adds at most 2^-24 |r|);
#   * the prologue: the fp32 value before its fp16 rounding is within a few
#     2^-24 of the exact one, so the two sides' x_eff differ by at most one
#     fp16 ulp (2^-10 |x_eff|), which moves y by at most 2^-10 sum |w_hat x_eff|;
#   * y's rounding now covers |r| too: 2^-10 |r| for the two sides together.
# 2e-3 V + 1e-5 covers the sum.
FUSED_REL_TOL = 2e-3
FUSED_ABS_TOL = 1e-5


def _f16(a, name):
    a = np.asarray(a)
    if a.dtype != np.float16:
        raise TypeError(f"{name} must be float16")
    return a


def rmsnorm_f64(x, g, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g in float64, for 1-D fp16 x and g."""
    x = _f16(x, "x").astype(np.float64)
    g = _f16(g, "norm weight").astype(np.float64)
    if x.ndim != 1 or g.shape != x.shape:
        raise ValueError("x and the norm weight must be 1-D of one length")
    if not (eps >= 0.0 and np.isfinite(eps)):
        raise ValueError("eps must be finite and >= 0")
    ms = np.mean(x * x)
    if ms + eps == 0.0:
        raise ValueError("RMSNorm of a zero vector with eps = 0 is undefined")
    return x / np.sqrt(ms + eps) * g


def silu_mul_f64(x) -> np.ndarray:
    """silu(x[:K]) * x[K:] in float64 for 1-D fp16 x of even length 2K."""
    x = _f16(x, "x").astype(np.float64)
    if x.ndim != 1 or x.shape[0] % 2 != 0:
        raise ValueError("x must be 1-D of even length")
    k = x.shape[0] // 2
    a, b = x[:k], x[k:]
    return a / (1.0 + np.exp(-a)) * b


def prologue(x, kind: int, g=None, eps: float = 0.0) -> np.ndarray:
    """The linear's fp16 input x_eff for prologue `kind`."""
    if kind == PRO_NONE:
        return _f16(x, "x").copy()
    if kind == PRO_RMSNORM:
        return rmsnorm_f64(x, g, eps).astype(np.float16)
    if kind == PRO_SILU_MUL:
        return silu_mul_f64(x).astype(np.float16)
    raise ValueError(f"unknown prologue {kind}")


def fused_linear_f64(packed, scales, x, n: int, k: int, kind: int = PRO_NONE, g=None, eps: float = 0.0,
                     residual=None):
    """Return (y64 [N], x_eff [K] fp16): the linear applied to the prologue's
    output, plus the residual, before the output rounding."""
    x_eff = prologue(x, kind, g, eps)
    if x_eff.shape != (k,):
        raise ValueError(f"the prologue gives {x_eff.shape[0]} inputs, the linear takes {k}")
    y64 = wq_oracle.gemv_f64(packed, scales, x_eff[None, :], n, k)[0]
    if residual is not None:
        r = _f16(residual, "residual")
        if r.shape != (n,):
            raise ValueError("residual must be [N]")
        y64 = y64 + r.astype(np.float64)
    return y64, x_eff


def fused_linear(packed, scales, x, n: int, k: int, kind: int = PRO_NONE, g=None, eps: float = 0.0,
                 residual=None) -> np.ndarray:
    """fp16 y [N], rounded once from float64."""
    return fused_linear_f64(packed, scales, x, n, k, kind, g, eps, residual)[0].astype(np.float16)


def fused_tol_bound(packed, scales, x_eff, n: int, k: int, residual=None) -> np.ndarray:
    """Per-row bound on |y_gpu - y_ref| for an fp32 computation."""
    w_abs = np.abs(wq_oracle.dequant(packed, scales, n, k).astype(np.float64))
    v = w_abs @ np.abs(np.asarray(x_eff, dtype=np.float16).astype(np.float64))
    if residual is not None:
        v = v + np.abs(np.asarray(residual, dtype=np.float16).astype(np.float64))
    return FUSED_REL_TOL * v + FUSED_ABS_TOL


def fused_within_tolerance(y_gpu, y_ref, bound) -> np.ndarray:
    a = np.asarray(y_gpu).astype(np.float64)
    b = np.asarray(y_ref).astype(np.float64)
    return np.isfinite(a) & (np.abs(a - b) <= bound)


def argmax_first(y) -> int:
    """Smallest index of the largest value of a 1-D fp16 vector (no NaN)."""
    y = _f16(y, "logits")
    if y.ndim != 1 or y.shape[0] == 0:
        raise ValueError("logits must be a non-empty 1-D vector")
    if np.any(np.isnan(y)):
        raise ValueError("logits must not contain NaN")
    best = 0
    for i in range(1, y.shape[0]):
        if y[i] > y[best]:
            best = i
    return best
