"""GPU parity of the fused decode linears (RMSNorm / SiLU-mul prologues,
residual epilogue, argmax of the logits) through the C ABI, against the CPU
oracle.

Random inputs are compared within the oracle's derived fp32 bound; inputs
whose prologue result and dot products are exact in any order are compared
bit for bit, including a whole chain of dependent linears ending in argmax.
"""

from __future__ import annotations

import numpy as np
import pytest

from gpu_util import announce, require_gpu, sample_rows, to_dev
from oracle import fused_oracle as fo
from paper_2412_15803_amd import workloads as wl

pytestmark = pytest.mark.gpu

PRO = {"none": fo.PRO_NONE, "rmsnorm": fo.PRO_RMSNORM, "silu": fo.PRO_SILU_MUL}


def _h(a):
    return np.asarray(a, dtype=np.float64).astype(np.float16)


def run_chain(descs, argmax=False):
    """descs: list of dicts of host arrays (packed, scales, x, norm, residual,
    prologue, eps) where x / residual may instead be ("y", j) to read linear
    j's output.  Runs one wq_fused_linears call; returns (ys, argmax)."""
    import torch

    from paper_2412_15803_amd import wq

    require_gpu()
    ys, lins = [], []
    for d in descs:
        n = d["packed"].shape[0]
        ys.append(torch.full((n,), float("nan"), dtype=torch.float16, device="cuda:0"))
    for i, d in enumerate(descs):
        x = ys[d["x"][1]] if isinstance(d["x"], tuple) else to_dev(d["x"]).view(torch.float16)
        if isinstance(d.get("x"), tuple) and d["x"][2:]:
            x = x[d["x"][2]:d["x"][3]]
        lin = {"packed_w": to_dev(d["packed"]), "scales": to_dev(d["scales"]).view(torch.float16),
               "x": x, "y": ys[i], "prologue": d.get("prologue", fo.PRO_NONE), "eps": d.get("eps", 0.0)}
        if d.get("norm") is not None:
            lin["norm_weight"] = to_dev(d["norm"]).view(torch.float16)
        r = d.get("residual")
        if r is not None:
            lin["residual"] = ys[r[1]] if isinstance(r, tuple) else to_dev(r).view(torch.float16)
        if d.get("in_place"):
            ys[i].copy_(lin["residual"])
            lin["residual"] = ys[i]
        lins.append(lin)
    am = torch.full((1,), -7, dtype=torch.int32, device="cuda:0") if argmax else None
    wq.wq_fused_linears(lins, argmax=am)
    torch.cuda.synchronize()
    out = [y.cpu().numpy() for y in ys]
    return out, (int(am.cpu().item()) if argmax else None)


def random_linear(seed, n, k):
    return wl.random_words_host(seed, n, k), wl.random_scales_host(seed + 1, n, k)


def oracle_linear(d, x, residual):
    n, k = d["packed"].shape[0], d["packed"].shape[1] * 8
    y64, x_eff = fo.fused_linear_f64(d["packed"], d["scales"], x, n, k, d.get("prologue", fo.PRO_NONE),
                                     d.get("norm"), d.get("eps", 0.0), residual)
    return y64.astype(np.float16), fo.fused_tol_bound(d["packed"], d["scales"], x_eff, n, k, residual)


# (label, N, K, prologue, residual?)
SHAPES = [
    ("3B qkv rmsnorm", 5120, 3072, "rmsnorm", False),
    ("3B o residual", 3072, 3072, "none", True),
    ("3B gate_up rmsnorm", 16384, 3072, "rmsnorm", False),
    ("3B down silu residual", 3072, 8192, "silu", True),
    ("8B qkv rmsnorm", 6144, 4096, "rmsnorm", False),
    ("8B down silu residual", 4096, 14336, "silu", True),
    ("K max silu", 257, 16384, "silu", True),
    ("ragged rmsnorm residual", 1000, 96, "rmsnorm", True),
    ("tiny silu", 33, 32, "silu", False),
    ("odd groups rmsnorm", 129, 32 * 7, "rmsnorm", True),
    ("lpr32 gpl5 silu", 700, 32 * 160, "silu", False),
    ("lpr16 gpl3 rmsnorm", 90, 32 * 48, "rmsnorm", True),
    ("plain residual", 4096, 4096, "none", True),
]


@pytest.mark.parametrize("label,n,k,pro,res", SHAPES, ids=[s[0] for s in SHAPES])
def test_fused_linear_within_tolerance(label, n, k, pro, res):
    announce(f"fused {label} N={n} K={k}")
    rng = np.random.default_rng(n * 7 + k)
    packed, scales = random_linear(n + k, n, k)
    d = {"packed": packed, "scales": scales, "prologue": PRO[pro], "eps": 1e-5}
    if pro == "silu":
        d["x"] = _h(np.concatenate([rng.standard_normal(k) * 2.0, rng.standard_normal(k)]))
    else:
        d["x"] = _h(rng.standard_normal(k))
    if pro == "rmsnorm":
        d["norm"] = _h(rng.uniform(0.5, 1.5, k))
    d["residual"] = _h(rng.standard_normal(n) * 4) if res else None
    (y,), _ = run_chain([d])
    ref, bound = oracle_linear(d, d["x"], d["residual"])
    ok = fo.fused_within_tolerance(y, ref, bound)
    assert ok.all(), f"{label}: {np.count_nonzero(~ok)} rows out of tolerance, first {np.flatnonzero(~ok)[:5]}"


def test_fused_lm_head_rmsnorm_argmax():
    """The final projection: RMSNorm -> 128256 x 3072 logits -> argmax.  The
    logits are checked against the oracle on sampled rows, and the argmax is
    the first maximum of the returned logits."""
    announce("fused lm_head 128256x3072 + argmax")
    n, k = 128256, 3072
    rng = np.random.default_rng(11)
    packed, scales = random_linear(12, n, k)
    d = {"packed": packed, "scales": scales, "prologue": fo.PRO_RMSNORM, "eps": 1e-5,
         "x": _h(rng.standard_normal(k)), "norm": _h(rng.uniform(0.5, 1.5, k))}
    (y,), am = run_chain([d], argmax=True)
    assert am == int(np.flatnonzero(y == y.max())[0])
    rows = sample_rows(n, 512, 13)
    sub = {"packed": packed[rows], "scales": scales[rows], "prologue": fo.PRO_RMSNORM, "eps": 1e-5,
           "x": d["x"], "norm": d["norm"]}
    ref, bound = oracle_linear(sub, d["x"], None)
    assert fo.fused_within_tolerance(y[rows], ref, bound).all()


# ------------------------------------------------------------- bit-exact

def _int_linear(seed, n, k, scale_bits=0x2400):  # 2^-6
    return wl.random_words_host(seed, n, k), np.full((n, k // 32), scale_bits, dtype=np.uint16)


@pytest.mark.parametrize("n,k", [(3072, 3072), (1000, 96), (129, 32 * 7), (257, 16384)])
def test_fused_rmsnorm_exact(n, k):
    """x of one magnitude (a power of two) with eps = 0 normalises to +-g
    exactly; with integer g, scales 2^-6 and an integer residual every sum is
    exact in fp32, so y matches bit for bit."""
    announce(f"fused rmsnorm exact N={n} K={k}")
    rng = np.random.default_rng(k)
    packed, scales = _int_linear(k + 1, n, k)
    x = _h(rng.choice([-1.0, 1.0], k) * 8.0)
    g = _h(rng.integers(-4, 5, k))
    r = _h(rng.integers(-64, 65, n))
    d = {"packed": packed, "scales": scales, "prologue": fo.PRO_RMSNORM, "eps": 0.0, "x": x, "norm": g,
         "residual": r}
    (y,), _ = run_chain([d])
    ref = fo.fused_linear(packed, scales, x, n, k, fo.PRO_RMSNORM, g, 0.0, r)
    assert np.array_equal(y.view(np.uint16), ref.view(np.uint16))


@pytest.mark.parametrize("n,k", [(3072, 8192), (4096, 14336), (33, 32), (700, 32 * 160)])
def test_fused_silu_exact(n, k):
    """Gates of 0 or 32 give silu exactly 0 or 32 in fp32 (exp(-32) vanishes
    next to 1); with integer up values the products and every dot product
    are exact."""
    announce(f"fused silu exact N={n} K={k}")
    rng = np.random.default_rng(k + 3)
    packed, scales = _int_linear(k + 2, n, k)
    gate = _h(rng.choice([0.0, 32.0], k))
    up = _h(rng.integers(-4, 5, k))
    d = {"packed": packed, "scales": scales, "prologue": fo.PRO_SILU_MUL, "x": np.concatenate([gate, up])}
    (y,), _ = run_chain([d])
    ref = fo.fused_linear(packed, scales, d["x"], n, k, fo.PRO_SILU_MUL)
    assert np.array_equal(y.view(np.uint16), ref.view(np.uint16))


def test_fused_in_place_residual_matches_separate():
    announce("fused in-place residual")
    rng = np.random.default_rng(21)
    n, k = 3072, 3072
    packed, scales = random_linear(22, n, k)
    base = {"packed": packed, "scales": scales, "x": _h(rng.standard_normal(k)),
            "residual": _h(rng.standard_normal(n))}
    (a,), _ = run_chain([base])
    (b,), _ = run_chain([dict(base, in_place=True)])
    assert np.array_equal(a.view(np.uint16), b.view(np.uint16))


def _exact_chain(seed):
    """A dependent chain in which every value is exact: one-hot x -> gate/up
    values in {0, 32} and {-8..7} -> SiLU-mul -> down + residual (in place)
    -> a plain projection whose logits have deliberate ties -> argmax."""
    rng = np.random.default_rng(seed)
    hidden, inter, vocab = 256, 256, 4096
    # gate/up: 2*inter rows over `hidden`; x = e_j picks column j.  Bounds that
    # keep every fp32 sum exact: |x_eff| <= 64, |down sum| <= 256 * 64 / 8 =
    # 2048, |logit sums| <= 256 * 2080 / 8 < 2^18 (multiples of 2^-6).
    codes = np.full((2 * inter, hidden), 8, dtype=np.int64)
    j = 77
    codes[:inter, j] = rng.choice([8, 12], inter)             # gate: 0 or 4 * scale 8 = 32
    codes[inter:, j] = rng.integers(6, 11, inter)             # up: -2..2 at scale 1
    import exact

    gu_packed = exact.pack_codes_bytes_2d(codes)
    gu_scales = np.concatenate([np.full((inter, hidden // 32), 0x4800, np.uint16),    # 8.0
                                np.full((inter, hidden // 32), 0x3C00, np.uint16)])   # 1.0
    x = np.zeros(hidden, dtype=np.float16)
    x[j] = 1.0
    down_packed, down_scales = _int_linear(seed + 1, hidden, inter)
    h0 = _h(rng.integers(-32, 33, hidden))
    # logits: rows repeat in pairs, so every maximum is tied with its twin
    half_packed, half_scales = _int_linear(seed + 2, vocab // 2, hidden)
    lm_packed = np.repeat(half_packed, 2, axis=0)
    lm_scales = np.repeat(half_scales, 2, axis=0)
    descs = [
        {"packed": gu_packed, "scales": gu_scales, "x": x},
        {"packed": down_packed, "scales": down_scales, "x": ("y", 0), "prologue": fo.PRO_SILU_MUL,
         "residual": h0, "in_place": True},
        {"packed": lm_packed, "scales": lm_scales, "x": ("y", 1)},
    ]
    return descs, (gu_packed, gu_scales, x, down_packed, down_scales, h0, lm_packed, lm_scales, hidden, inter, vocab)


def test_fused_exact_chain_with_argmax():
    announce("fused exact dependent chain + argmax")
    descs, (gp, gs, x, dp, ds, h0, lp, ls, hidden, inter, vocab) = _exact_chain(31)
    (y_gu, h1, logits), am = run_chain(descs, argmax=True)
    r_gu = fo.fused_linear(gp, gs, x, 2 * inter, hidden)
    r_h1 = fo.fused_linear(dp, ds, r_gu, hidden, inter, fo.PRO_SILU_MUL, residual=h0)
    r_lg = fo.fused_linear(lp, ls, r_h1, vocab, hidden)
    assert np.array_equal(y_gu.view(np.uint16), r_gu.view(np.uint16))
    assert np.array_equal(h1.view(np.uint16), r_h1.view(np.uint16))
    assert np.array_equal(logits.view(np.uint16), r_lg.view(np.uint16))
    assert am == fo.argmax_first(r_lg)
    assert am % 2 == 0, "ties must resolve to the smaller index"


def test_fused_chain_equals_separate_calls():
    """One call running a dependent chain gives the same bits as one call
    per linear (with every linear reading the previous one's output)."""
    announce("fused chain vs separate calls")
    rng = np.random.default_rng(41)
    hid, inter = 3072, 8192
    qkv_p, qkv_s = random_linear(42, 5120, hid)
    o_p, o_s = random_linear(43, hid, hid)
    gu_p, gu_s = random_linear(44, 2 * inter, hid)
    dn_p, dn_s = random_linear(45, hid, inter)
    h = _h(rng.standard_normal(hid))
    g1, g2 = _h(rng.uniform(0.5, 1.5, hid)), _h(rng.uniform(0.5, 1.5, hid))
    descs = [
        {"packed": qkv_p, "scales": qkv_s, "x": h, "prologue": fo.PRO_RMSNORM, "norm": g1, "eps": 1e-5},
        {"packed": o_p, "scales": o_s, "x": ("y", 0, 0, hid), "residual": h},
        {"packed": gu_p, "scales": gu_s, "x": ("y", 1), "prologue": fo.PRO_RMSNORM, "norm": g2, "eps": 1e-5},
        {"packed": dn_p, "scales": dn_s, "x": ("y", 2), "prologue": fo.PRO_SILU_MUL, "residual": ("y", 1)},
    ]
    chain, _ = run_chain(descs)
    prev = []
    for i, d in enumerate(descs):
        di = dict(d)
        if isinstance(d["x"], tuple):
            src = prev[d["x"][1]]
            di["x"] = src[d["x"][2]:d["x"][3]] if len(d["x"]) > 2 else src
        if isinstance(d.get("residual"), tuple):
            di["residual"] = prev[d["residual"][1]]
        (y,), _ = run_chain([di])
        prev.append(y)
        assert np.array_equal(y.view(np.uint16), chain[i].view(np.uint16)), i
    # and the first linear of the chain against the oracle
    ref, bound = oracle_linear(descs[0], h, None)
    assert fo.fused_within_tolerance(chain[0], ref, bound).all()


def _argmax_through_residual(logits, offset):
    """A linear with x = 0 and the logits as its residual returns exactly the
    logits (0 + r, rounded once); its y starts `offset` elements into a
    buffer, so the argmax kernel also sees unaligned vectors."""
    import torch

    from paper_2412_15803_amd import wq

    require_gpu()
    n = logits.shape[0]
    packed, scales = random_linear(5 + n, n, 32)
    x = torch.zeros(32, dtype=torch.float16, device="cuda:0")
    buf = torch.full((n + offset,), float("nan"), dtype=torch.float16, device="cuda:0")
    y = buf[offset:]
    am = torch.full((1,), -7, dtype=torch.int32, device="cuda:0")
    lin = {"packed_w": to_dev(packed), "scales": to_dev(scales).view(torch.float16), "x": x, "y": y,
           "residual": to_dev(logits).view(torch.float16)}
    wq.wq_fused_linears([lin], argmax=am)
    torch.cuda.synchronize()
    got_y = y.cpu().numpy()
    assert np.array_equal(got_y.view(np.uint16), logits.view(np.uint16)) or \
        np.array_equal(np.isnan(got_y), np.isnan(logits)), "residual pass-through changed the logits"
    return int(am.cpu().item())


def _first_max_ignoring_nan(v):
    ok = ~np.isnan(v.astype(np.float32))
    if not ok.any():
        return -1
    m = v[ok].max()
    return int(np.flatnonzero(ok & (v == m))[0])


@pytest.mark.parametrize("n", [1, 7, 8, 9, 17, 33, 1000, 16384 + 3, 128256])
@pytest.mark.parametrize("offset", [0, 1, 5])
def test_fused_argmax_edge_cases(n, offset):
    announce(f"argmax n={n} offset={offset}")
    rng = np.random.default_rng(n + offset)
    base = _h(rng.standard_normal(n))
    cases = [base]
    tie = base.copy()
    top = np.float16(9.0)
    idx = sorted(set(int(i) for i in rng.integers(0, n, 3)))
    tie[idx] = top                                   # equal maxima: the first must win
    cases.append(tie)
    neg = np.full(n, -np.inf, dtype=np.float16)      # all -inf: index 0
    cases.append(neg)
    if n > 2:
        with_nan = base.copy()
        with_nan[rng.integers(0, n, max(1, n // 4))] = np.nan
        with_nan[0] = np.nan
        cases.append(with_nan)
    cases.append(np.full(n, np.nan, dtype=np.float16))   # nothing to choose: -1
    for c in cases:
        got = _argmax_through_residual(c, offset)
        assert got == _first_max_ignoring_nan(c), (n, offset, got)
        if not np.isnan(c.astype(np.float32)).any():
            assert got == fo.argmax_first(c)


def test_fused_argmax_nan_and_neg_inf_mix():
    """-inf as the largest value behind vectors of NaN, and a maximum that
    appears again in a later vector and in the scalar tail."""
    announce("argmax NaN / -inf mix")
    n = 8 * 1024 * 3 + 5
    v = np.full(n, np.nan, dtype=np.float16)
    v[8 * 1024 * 2 + 3] = -np.inf
    v[8 * 1024 * 2 + 9] = -np.inf
    assert _argmax_through_residual(v, 0) == 8 * 1024 * 2 + 3
    w = _h(np.random.default_rng(3).standard_normal(n))
    w[[40, 8 * 1024 + 40, n - 1]] = np.float16(50.0)
    for off in (0, 3):
        assert _argmax_through_residual(w, off) == 40
