"""The persistent dependent-chain path of wq_fused_linears (one cooperative
launch per chain, grid-wide barriers between linears; WQ_FUSED_PERSISTENT=1)
on the GPU, through
the C ABI: bit for bit the same outputs as the per-linear path (one launch
per linear, the default), over 3B-class layers with attention's
place taken by the qkv slice, long random chains of every compiled shape,
repeated and interleaved calls, and the error path of its bounded waits
(forced from the host with a one-tick time limit: every wave still ends)."""

from __future__ import annotations

import numpy as np
import pytest

from gpu_util import announce, require_gpu
from oracle import fused_oracle as fo
from test_gpu_fused import _h, oracle_linear, random_linear, run_chain

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


def _both_paths(descs, monkeypatch, argmax=False):
    from paper_2412_15803_amd import wq

    monkeypatch.setenv("WQ_FUSED_PERSISTENT", "1")
    persistent = run_chain(descs, argmax)
    wq.wq_fused_check()
    monkeypatch.setenv("WQ_FUSED_PERSISTENT", "0")
    per_linear = run_chain(descs, argmax)
    monkeypatch.delenv("WQ_FUSED_PERSISTENT", raising=False)
    return persistent, per_linear


def _same(a, b, what):
    bad = np.flatnonzero(a.view(np.uint16) != b.view(np.uint16))
    assert bad.size == 0, f"{what}: {bad.size} outputs differ, first {bad[:5].tolist()}"


def _layers_3b(seed, layers, vocab):
    """`layers` 3B-class layers (qkv, o + residual, gate_up, down + residual,
    RMSNorm prologues, the o projection reading the first 3072 qkv outputs)
    and a final RMSNorm projection of `vocab` rows."""
    rng = np.random.default_rng(seed)
    hid, inter = 3072, 8192
    h = _h(rng.standard_normal(hid))
    descs = []
    for l in range(layers):
        b = len(descs)
        src = ("y", b - 1) if b else h
        qp, qs = random_linear(seed + 10 * l + 1, 5120, hid)
        op, os_ = random_linear(seed + 10 * l + 2, hid, hid)
        gp, gs = random_linear(seed + 10 * l + 3, 2 * inter, hid)
        dp, ds = random_linear(seed + 10 * l + 4, hid, inter)
        descs += [
            {"packed": qp, "scales": qs, "x": src, "prologue": fo.PRO_RMSNORM, "eps": 1e-5,
             "norm": _h(rng.uniform(0.5, 1.5, hid))},
            {"packed": op, "scales": os_, "x": ("y", b, 0, hid), "residual": src},
            {"packed": gp, "scales": gs, "x": ("y", b + 1), "prologue": fo.PRO_RMSNORM, "eps": 1e-5,
             "norm": _h(rng.uniform(0.5, 1.5, hid))},
            {"packed": dp, "scales": ds, "x": ("y", b + 2), "prologue": fo.PRO_SILU_MUL, "residual": ("y", b + 1)},
        ]
    lp, ls = random_linear(seed + 999, vocab, hid)
    descs.append({"packed": lp, "scales": ls, "x": ("y", len(descs) - 1), "prologue": fo.PRO_RMSNORM, "eps": 1e-5,
                  "norm": _h(rng.uniform(0.5, 1.5, hid))})
    return descs


def test_persistent_3b_layers_match_per_linear_path(monkeypatch):
    announce("persistent chain: 3 layers of 3B shapes + 32000-row head, argmax")
    descs = _layers_3b(500, 3, 32000)
    (ys_p, am_p), (ys_l, am_l) = _both_paths(descs, monkeypatch, argmax=True)
    for i, (a, b) in enumerate(zip(ys_p, ys_l)):
        assert np.isfinite(a.astype(np.float64)).all(), f"linear {i} not finite"
        _same(a, b, f"linear {i}")
    assert am_p == am_l
    # and the first linear against the oracle
    ref, bound = oracle_linear(descs[0], descs[0]["x"], None)
    assert fo.fused_within_tolerance(ys_p[0], ref, bound).all()


# K values whose rows take each compiled narrow shape: 64 lanes x 1..4 groups,
# 32 lanes x 1 or 3, 16 lanes x 1 or 3 (and ragged rows below a cover).
NARROW_K = [32 * g for g in (1, 2, 3, 5, 12, 16, 32, 48, 64, 96, 128, 192, 256, 250, 100)]


@pytest.mark.parametrize("seed", [1, 2])
def test_persistent_random_chains_match_per_linear_path(seed, monkeypatch):
    """Forty dependent linears of random widths over every narrow shape,
    random prologues and residuals; consecutive linears share the previous
    output as x (or its first K entries)."""
    rng = np.random.default_rng(7000 + seed)
    dims = [int(rng.choice(NARROW_K))]
    descs = []
    x0 = None
    for i in range(40):
        k = dims[-1]
        pro = int(rng.choice([fo.PRO_NONE, fo.PRO_RMSNORM, fo.PRO_SILU_MUL]))
        n_out = int(rng.choice(NARROW_K))
        n = 2 * n_out if rng.random() < 0.3 else n_out
        if pro == fo.PRO_SILU_MUL:
            # x holds [gate; up] of the previous output: the previous linear is 2K wide
            pass
        p, s = random_linear(seed * 1000 + i, n, k)
        if i == 0:
            x0 = _h(rng.standard_normal(2 * k if pro == fo.PRO_SILU_MUL else k))
            x = x0
        else:
            prev_n = descs[-1]["packed"].shape[0]
            need = 2 * k if pro == fo.PRO_SILU_MUL else k
            if prev_n < need:
                pro = fo.PRO_NONE
                need = k
            if prev_n < need:
                x = _h(rng.standard_normal(k))
            else:
                x = ("y", i - 1, 0, need)
        d = {"packed": p, "scales": s, "x": x, "prologue": pro, "eps": 1e-5}
        if pro == fo.PRO_RMSNORM:
            d["norm"] = _h(rng.uniform(0.5, 1.5, k))
        if rng.random() < 0.4:
            d["residual"] = _h(rng.standard_normal(n))
        descs.append(d)
        dims.append(n_out if n == n_out else n // 2)
    announce(f"persistent random chain seed={seed}")
    (ys_p, _), (ys_l, _) = _both_paths(descs, monkeypatch)
    for i, (a, b) in enumerate(zip(ys_p, ys_l)):
        _same(a, b, f"seed {seed} linear {i} ({descs[i]['packed'].shape[0]}x{descs[i]['packed'].shape[1] * 8})")


def test_persistent_repeated_and_interleaved_calls(monkeypatch):
    """The generation numbers continue across launches: the same chain five
    times, interleaved with another chain, gives the same bits every time."""
    from paper_2412_15803_amd import wq

    a = _layers_3b(600, 1, 4096)
    b = _layers_3b(700, 2, 8192)
    announce("persistent repeated and interleaved chains")
    monkeypatch.setenv("WQ_FUSED_PERSISTENT", "1")
    first_a, first_b = run_chain(a)[0], run_chain(b)[0]
    for rep in range(4):
        for descs, ref, tag in ((a, first_a, "a"), (b, first_b, "b")):
            ys, _ = run_chain(descs)
            for i, (x, y) in enumerate(zip(ys, ref)):
                _same(x, y, f"chain {tag} rep {rep} linear {i}")
    wq.wq_fused_check()


def test_persistent_timeout_reports_error_and_recovers(monkeypatch):
    """With the per-wait limit forced to one clock tick from the host, the
    waits between workgroups run out: every wave still ends, and
    wq_fused_check reports WQ_ERR_HIP.  The next call with the normal limit
    gives the right outputs and a clean check."""
    from paper_2412_15803_amd import wq

    descs = _layers_3b(800, 2, 4096)
    announce("persistent chain with a one-tick wait limit")
    monkeypatch.setenv("WQ_FUSED_PERSISTENT", "1")
    monkeypatch.setenv("WQ_CHAIN_TIMEOUT_TICKS", "1")
    run_chain(descs)
    with pytest.raises(wq.WQError) as info:
        wq.wq_fused_check()
    assert info.value.status == wq.WQ_ERR_HIP
    wq.wq_fused_check()  # the condition was cleared by the first check
    monkeypatch.delenv("WQ_CHAIN_TIMEOUT_TICKS")
    announce("persistent chain after the timeout")
    (ys_p, _), (ys_l, _) = _both_paths(descs, monkeypatch)
    for i, (x, y) in enumerate(zip(ys_p, ys_l)):
        _same(x, y, f"after timeout linear {i}")


def _in_place_layers(seed, layers, vocab):
    """The bench's buffer pattern: one residual stream h updated in place by
    o and down (residual = y = h), qkv and gate_up outputs reused by every
    layer, RMSNorm weights per layer; returns a function running the chain
    from a fresh copy of h0 and returning every buffer and the argmax."""
    import torch

    from paper_2412_15803_amd import wq

    g = torch.Generator(device="cuda:0")
    g.manual_seed(seed)
    hid, inter = 3072, 8192
    dev = "cuda:0"

    def rnd(shape, lo=None):
        t = torch.rand(shape, generator=g, device=dev) + 0.5 if lo else torch.randn(shape, generator=g, device=dev)
        return t.to(torch.float16)

    def lin(n, k):
        p = torch.randint(-2**31, 2**31 - 1, (n, k // 8), dtype=torch.int32, device=dev, generator=g)
        s = (torch.rand((n, k // 32), device=dev, generator=g) * 0.01 + 0.001).to(torch.float16)
        return p, s

    h0 = rnd(hid)
    h = torch.empty(hid, dtype=torch.float16, device=dev)
    qkv = torch.empty(5120, dtype=torch.float16, device=dev)
    gu = torch.empty(2 * inter, dtype=torch.float16, device=dev)
    logits = torch.empty(vocab, dtype=torch.float16, device=dev)
    token = torch.empty(1, dtype=torch.int32, device=dev)
    R, S = wq.PROLOGUE_RMSNORM, wq.PROLOGUE_SILU_MUL
    chain = []
    for _ in range(layers):
        (qp, qs), (op, os_), (gp, gs), (dp, ds) = lin(5120, hid), lin(hid, hid), lin(2 * inter, hid), lin(hid, inter)
        chain += [dict(packed_w=qp, scales=qs, x=h, y=qkv, prologue=R, norm_weight=rnd(hid, True), eps=1e-5),
                  dict(packed_w=op, scales=os_, x=qkv[:hid], y=h, residual=h),
                  dict(packed_w=gp, scales=gs, x=h, y=gu, prologue=R, norm_weight=rnd(hid, True), eps=1e-5),
                  dict(packed_w=dp, scales=ds, x=gu, y=h, prologue=S, residual=h)]
    lp, ls = lin(vocab, hid)
    chain.append(dict(packed_w=lp, scales=ls, x=h, y=logits, prologue=R, norm_weight=rnd(hid, True), eps=1e-5))
    arr = wq.make_fused_array(chain)

    def run():
        h.copy_(h0)
        for t in (qkv, gu, logits):
            t.fill_(float("nan"))
        wq.wq_fused_linears(chain, argmax=token, _array=arr)
        torch.cuda.synchronize()
        return [t.cpu().numpy().copy() for t in (h, qkv, gu, logits)], int(token.item())

    return run


def test_persistent_in_place_residual_stream_matches(monkeypatch):
    """Outputs written over inputs that other workgroups still read in the
    same launch (h is read by qkv's and gate_up's prologues and updated in
    place by o and down): the persistent chain writes the caller's buffers
    only after the whole chain, and must match the per-linear path."""
    from paper_2412_15803_amd import wq

    run = _in_place_layers(900, 3, 16000)
    announce("persistent chain over an in-place residual stream")
    monkeypatch.setenv("WQ_FUSED_PERSISTENT", "1")
    bufs_p, tok_p = run()
    wq.wq_fused_check()
    bufs_p2, tok_p2 = run()
    monkeypatch.setenv("WQ_FUSED_PERSISTENT", "0")
    bufs_l, tok_l = run()
    monkeypatch.delenv("WQ_FUSED_PERSISTENT", raising=False)
    for name, a, a2, b in zip(("h", "qkv", "gate_up", "logits"), bufs_p, bufs_p2, bufs_l):
        assert np.isfinite(b.astype(np.float64)).all(), name
        _same(a, b, f"in place: {name}")
        _same(a2, b, f"in place, second call: {name}")
    assert tok_p == tok_l == tok_p2
