"""Pins for the fused-operation oracle (RMSNorm, SiLU-mul, residual, argmax):
torch's float64 library routines, closed forms, identities and hand-worked
rounding cases.  Every pin takes an oracle namespace `orc` (oracle.fused_oracle
or a copy with a planted mistake) and raises when it does not hold.
"""

from __future__ import annotations

import numpy as np

import exact
from paper_2412_15803_amd import workloads as wl


def _rng(seed):
    return np.random.default_rng(seed)


def _h(a):
    return np.asarray(a, dtype=np.float64).astype(np.float16)


# ------------------------------------------------------------------- RMSNorm

def pin_rmsnorm_matches_torch(orc):
    import torch
    import torch.nn.functional as F

    for seed, k, eps in ((1, 64, 1e-5), (2, 3072, 1e-6), (3, 96, 0.0), (4, 5, 0.5)):
        rng = _rng(seed)
        x = _h(rng.standard_normal(k) * 3)
        g = _h(rng.uniform(0.5, 1.5, k))
        got = orc.rmsnorm_f64(x, g, eps)
        ref = F.rms_norm(torch.from_numpy(x.astype(np.float64)), (k,), torch.from_numpy(g.astype(np.float64)),
                         eps=eps).numpy()
        assert np.allclose(got, ref, rtol=1e-13, atol=0), (seed, np.max(np.abs(got - ref)))


def pin_rmsnorm_closed_forms(orc):
    """A vector of one magnitude c (eps = 0) normalises to +-g exactly; a
    one-hot c e_i gives sqrt(K) sign(c) g_i at i and 0 elsewhere."""
    k = 48
    g = _h(np.arange(1, k + 1) / 8.0)
    signs = np.where(np.arange(k) % 3 == 0, -1.0, 1.0)
    for c in (0.25, 3.0, 1000.0):
        x = _h(signs * c)
        assert np.array_equal(orc.rmsnorm_f64(x, g, 0.0), signs * g.astype(np.float64))
    for i, c in ((0, 2.0), (17, -0.5)):
        x = np.zeros(k, dtype=np.float16)
        x[i] = c
        got = orc.rmsnorm_f64(x, g, 0.0)
        want = np.zeros(k)
        want[i] = np.sqrt(k) * np.sign(c) * float(g[i])
        assert np.allclose(got, want, rtol=1e-15, atol=0)
    # eps inside the root: c e_0 with eps = c^2 (K - 1) / K gives mean + eps = c^2
    c = 2.0
    x = np.zeros(k, dtype=np.float16)
    x[0] = c
    got = orc.rmsnorm_f64(x, g, c * c * (k - 1) / k)
    assert np.isclose(got[0], float(g[0]), rtol=1e-15)


def pin_rmsnorm_scale_invariance(orc):
    rng = _rng(5)
    # magnitudes in [1/4, 4]: scaled by 2^-3 .. 2^4 they stay normal fp16 values
    x = _h(rng.choice([-1.0, 1.0], 256) * rng.uniform(0.25, 4.0, 256))
    g = _h(rng.uniform(0.5, 1.5, 256))
    base = orc.rmsnorm_f64(x, g, 0.0)
    for j in (-3, 4):
        assert np.array_equal(orc.rmsnorm_f64(_h(x.astype(np.float64) * 2.0 ** j), g, 0.0), base)


# ------------------------------------------------------------------ SiLU-mul

def pin_silu_mul_matches_torch(orc):
    import torch
    import torch.nn.functional as F

    rng = _rng(6)
    x = _h(rng.standard_normal(2 * 500) * 4)
    got = orc.silu_mul_f64(x)
    t = torch.from_numpy(x.astype(np.float64))
    ref = (F.silu(t[:500]) * t[500:]).numpy()
    assert np.allclose(got, ref, rtol=1e-14, atol=1e-300)


def pin_silu_identities(orc):
    """silu(0) = 0; silu(a) - silu(-a) = a; silu(a) -> a for large a and
    -> 0 for large -a; the up half is the second half of x."""
    a = np.array([0.0, 0.5, 1.0, 3.0, -2.0, 30.0, -30.0], dtype=np.float16)
    ones = np.ones_like(a)
    s = orc.silu_mul_f64(np.concatenate([a, ones]))
    s_neg = orc.silu_mul_f64(np.concatenate([-a, ones]))
    assert s[0] == 0.0
    assert np.allclose(s - s_neg, a.astype(np.float64), rtol=1e-15, atol=1e-15)
    assert abs(s[5] - 30.0) < 1e-11 and abs(s[6]) < 1e-11
    up = np.array([2.0, 0.0, -1.0, 0.0, 4.0, 1.0, 0.0], dtype=np.float16)
    s2 = orc.silu_mul_f64(np.concatenate([a, up]))
    assert np.allclose(s2, s * up.astype(np.float64), rtol=1e-15, atol=0)


# ------------------------------------------------------------ linear + residual

def _two_group_linear():
    """N = 1, K = 64: w_hat[0] = 1 (scale 1, code 9), w_hat[32] = 2^-11
    (scale 2^-12, code 10), every other code 8."""
    codes = np.full((1, 64), 8, dtype=np.int64)
    codes[0, 0] = 9
    codes[0, 32] = 10
    packed = exact.pack_codes_bytes_2d(codes)
    scales = np.array([[0x3C00, 0x0C00]], dtype=np.uint16)   # 1.0, 2^-12
    return packed, scales


def pin_residual_single_rounding(orc):
    """w_hat . x = 1 + 2^-11 is halfway between fp16 1 and 1 + 2^-10; the
    residual 2^-20 lifts it above, so the once-rounded result is 1 + 2^-10
    (rounding the linear first would give 1.0 and then 1.0 again)."""
    packed, scales = _two_group_linear()
    x = np.zeros(64, dtype=np.float16)
    x[0] = 1.0
    x[32] = 1.0
    r = np.array([2.0 ** -20], dtype=np.float16)
    y = orc.fused_linear(packed, scales, x, 1, 64, orc.PRO_NONE, residual=r)
    assert y.view(np.uint16)[0] == 0x3C01, hex(int(y.view(np.uint16)[0]))
    y0 = orc.fused_linear(packed, scales, x, 1, 64, orc.PRO_NONE)
    assert y0.view(np.uint16)[0] == 0x3C00


def pin_residual_is_added(orc):
    rng = _rng(8)
    n, k = 40, 96
    packed = wl.random_words_host(9, n, k)
    scales = wl.random_scales_host(10, n, k)
    x = _h(rng.standard_normal(k))
    r = _h(rng.standard_normal(n) * 5)
    y_plain, _ = orc.fused_linear_f64(packed, scales, x, n, k)
    y_res, _ = orc.fused_linear_f64(packed, scales, x, n, k, residual=r)
    assert np.array_equal(y_res, y_plain + r.astype(np.float64))


def pin_prologue_feeds_the_linear(orc):
    """The linear sees exactly the rounded prologue output."""
    rng = _rng(11)
    n, k = 24, 64
    packed = wl.random_words_host(12, n, k)
    scales = wl.random_scales_host(13, n, k)
    x = _h(rng.standard_normal(k) * 2)
    g = _h(rng.uniform(0.5, 1.5, k))
    y, x_eff = orc.fused_linear_f64(packed, scales, x, n, k, orc.PRO_RMSNORM, g=g, eps=1e-5)
    assert np.array_equal(x_eff, orc.rmsnorm_f64(x, g, 1e-5).astype(np.float16))
    # against a plain dot product with the dequantized weights
    w_hat = exact.dequant_reference(packed, scales, n, k)
    assert np.allclose(y, w_hat @ x_eff.astype(np.float64), rtol=1e-13, atol=1e-13)
    xg = _h(rng.standard_normal(2 * k))
    y2, x2 = orc.fused_linear_f64(packed, scales, xg, n, k, orc.PRO_SILU_MUL)
    assert np.array_equal(x2, orc.silu_mul_f64(xg).astype(np.float16))
    assert np.allclose(y2, w_hat @ x2.astype(np.float64), rtol=1e-13, atol=1e-13)


def pin_fused_tolerance_scale(orc):
    """With V = 1, two fp16 ulps of error pass and three do not; the bound
    counts |r|."""
    packed, scales = _two_group_linear()
    x = np.zeros(64, dtype=np.float16)
    x[0] = 1.0
    b = orc.fused_tol_bound(packed, scales, x, 1, 64)
    one = np.float16(1.0)
    up2 = np.float16(1.0 + 2 * 2.0 ** -10)
    up3 = np.float16(1.0 + 3 * 2.0 ** -10)
    assert orc.fused_within_tolerance(np.array([up2]), np.array([one]), b)[0]
    assert not orc.fused_within_tolerance(np.array([up3]), np.array([one]), b)[0]
    assert not orc.fused_within_tolerance(np.array([np.float16(np.nan)]), np.array([one]), b)[0]
    br = orc.fused_tol_bound(packed, scales, x, 1, 64, residual=np.array([np.float16(-3.0)]))
    assert np.isclose(br[0] - b[0], orc.FUSED_REL_TOL * 3.0)


# -------------------------------------------------------------------- argmax

def pin_argmax(orc):
    y = np.array([1.0, 3.0, -2.0, 3.0, 0.5], dtype=np.float16)
    assert orc.argmax_first(y) == 1                       # first of two equal maxima
    assert orc.argmax_first(np.array([-5.0, -1.0, -1.0], dtype=np.float16)) == 1
    assert orc.argmax_first(np.array([0.0, -0.0], dtype=np.float16)) == 0
    assert orc.argmax_first(np.array([-0.0, 0.0], dtype=np.float16)) == 0
    assert orc.argmax_first(np.array([7.0], dtype=np.float16)) == 0
    z = np.full(1000, -np.inf, dtype=np.float16)
    z[999] = np.float16(-65504)
    assert orc.argmax_first(z) == 999
    rng = _rng(14)
    r = _h(rng.standard_normal(5000))
    assert orc.argmax_first(r) == int(np.flatnonzero(r == r.max())[0])


def pin_rejects_bad_inputs(orc):
    for call in (
        lambda: orc.rmsnorm_f64(np.zeros(8, np.float16), np.ones(8, np.float16), 0.0),
        lambda: orc.rmsnorm_f64(np.ones(8, np.float16), np.ones(8, np.float16), -1.0),
        lambda: orc.silu_mul_f64(np.ones(7, np.float16)),
        lambda: orc.argmax_first(np.array([1.0, np.nan], np.float16)),
    ):
        try:
            call()
        except ValueError:
            continue
        raise AssertionError("invalid input accepted")


ALL_PINS = [
    pin_rmsnorm_matches_torch,
    pin_rmsnorm_closed_forms,
    pin_rmsnorm_scale_invariance,
    pin_silu_mul_matches_torch,
    pin_silu_identities,
    pin_residual_single_rounding,
    pin_residual_is_added,
    pin_prologue_feeds_the_linear,
    pin_fused_tolerance_scale,
    pin_argmax,
    pin_rejects_bad_inputs,
]
