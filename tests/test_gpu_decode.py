"""wq_decode_linears on the GPU: the grouped batch-1 kernel (M = 1,
K <= 16384), the grouped matrix-core kernel (2 <= M <= 64) and the
per-linear fallback, against the CPU oracle.

Outputs are pre-filled with NaN and every row is checked, so a tile that is
never computed shows up.  Integer-valued data (unit scales, codes in
{7, 8, 9}, x in {-1, 0, 1}) keeps every partial sum an exact integer in
fp32, so results are unique and compared bit for bit, also along chains of
dependent linears.
"""

import numpy as np
import pytest

import oracle
from gpu_util import announce, require_gpu, to_dev, to_host
from paper_2412_15803_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


def int_linear(rng, n, k, p_nonzero=1 / 8):
    """Packed words and unit scales for codes in {7, 8, 9}."""
    p = p_nonzero / 2
    codes = rng.choice([7, 8, 9], size=(n, k), p=[p, 1 - 2 * p, p])
    packed = np.zeros((n, k // 8), dtype=np.uint32)
    for b in range(8):
        packed |= codes[:, b::8].astype(np.uint32) << np.uint32(4 * b)
    return packed, wl.constant_scales_host(n, k, 0x3C00)


def nan_out(m, n):
    import torch

    return torch.full((m, n), float("nan"), dtype=torch.float16, device="cuda")


def run(lins, m=1, stream=None):
    import torch

    from paper_2412_15803_amd import wq

    wq.wq_decode_linears(lins, m=m, stream=stream)
    torch.cuda.synchronize()


def check_exact(y_dev, y_ref, what):
    yh = to_host(y_dev, np.float16)
    bad = np.argwhere(yh.view(np.uint16) != y_ref.view(np.uint16))
    assert bad.size == 0, f"{what}: {len(bad)} mismatches, first {bad[:4].tolist()}"


def test_independent_linears_mixed_k_bit_exact():
    """Independent linears of every groups-per-lane class (K from 32 to
    16384), ragged row counts, one call."""
    rng = np.random.default_rng(1)
    shapes = [(37, 32), (1000, 512), (513, 2048), (300, 3072), (129, 4096), (77, 6144), (64, 8192),
              (50, 10240), (33, 14336), (17, 16384), (4097, 3072)]
    announce("decode independent mixed K")
    host, lins = [], []
    for n, k in shapes:
        p, s = int_linear(rng, n, k, 1 / 4)
        x = rng.integers(-1, 2, size=(1, k)).astype(np.float16)
        host.append((p, s, x))
        lins.append((to_dev(p), to_dev(s), to_dev(x), nan_out(1, n)))
    run(lins)
    for (p, s, x), (_, _, _, y), (n, k) in zip(host, lins, shapes):
        check_exact(y, oracle.gemv(p, s, x, n, k), f"{n}x{k}")


def test_small_k_only_uses_narrow_kernel_bit_exact():
    rng = np.random.default_rng(2)
    shapes = [(5120, 3072), (3072, 3072), (16384, 3072), (3072, 8192)]
    announce("decode 3B layer shapes, integer data")
    host, lins = [], []
    for n, k in shapes:
        p, s = int_linear(rng, n, k)
        x = rng.integers(-1, 2, size=(1, k)).astype(np.float16)
        host.append((p, s, x))
        lins.append((to_dev(p), to_dev(s), to_dev(x), nan_out(1, n)))
    run(lins)
    for (p, s, x), (_, _, _, y), (n, k) in zip(host, lins, shapes):
        check_exact(y, oracle.gemv(p, s, x, n, k), f"{n}x{k}")


# Largest |y| a bounded chain may reach: every value along the chain is then
# an integer exact in fp16, and every fp32 partial sum (at most K * 2048 <
# 2^24 in magnitude for K <= 8192) is an exact integer in any order.
CHAIN_LIMIT = 2048


def bounded_chain(rng, dims, x0, p_nonzero):
    """Unit-scale layers with codes in {7, 8, 9} for a chain x -> y -> ...,
    built one layer at a time from the exact integer outputs of the previous
    one: a row whose output would leave [-CHAIN_LIMIT, CHAIN_LIMIT] (for any
    batch row) has random nonzero codes set back to 8 until it does not.
    Returns the layers and the exact outputs of every layer (int64)."""
    layers, outs, x = [], [], x0.astype(np.int64)
    for i in range(len(dims) - 1):
        n, k = dims[i + 1], dims[i]
        p = p_nonzero / 2
        codes = rng.choice([7, 8, 9], size=(n, k), p=[p, 1 - 2 * p, p]).astype(np.int64)
        while True:
            y = x @ (codes - 8).T                            # [M, N], exact
            bad = np.flatnonzero(np.abs(y).max(axis=0) > CHAIN_LIMIT)
            if bad.size == 0:
                break
            # drop about half of each offending row's nonzero codes
            drop = (rng.random((bad.size, k)) < 0.5) & (codes[bad] != 8)
            codes[bad] = np.where(drop, 8, codes[bad])
        packed = np.zeros((n, k // 8), dtype=np.uint32)
        for b in range(8):
            packed |= codes[:, b::8].astype(np.uint32) << np.uint32(4 * b)
        layers.append((packed, wl.constant_scales_host(n, k, 0x3C00)))
        outs.append(y)
        x = y
    return layers, outs


def check_chain_reference(ref, exact, what):
    """The oracle's outputs along a bounded chain are finite, equal the exact
    integers the chain was built from, and are mostly nonzero (so the bit
    comparison is not one of NaN or zero patterns)."""
    assert np.all(np.isfinite(ref)), f"{what}: oracle output not finite"
    assert np.array_equal(ref.astype(np.float64), exact.astype(np.float64)), f"{what}: oracle differs from the exact sums"
    assert np.count_nonzero(exact) >= exact.size // 4, f"{what}: mostly zero"


def test_long_dependency_chain_bit_exact():
    """x of linear i+1 is y of linear i for 40 linears of varying widths;
    every output stays a finite integer of at most CHAIN_LIMIT in magnitude,
    so each of the 40 comparisons is of exact, mostly nonzero values."""
    rng = np.random.default_rng(3)
    dims = [int(d) for d in rng.choice([256, 512, 1024, 2048, 3072], size=41)]
    x0 = rng.integers(-8, 9, size=(1, dims[0])).astype(np.float16)
    layers, exact = bounded_chain(rng, dims, x0, 1 / 16)
    announce("decode 40-linear chain")
    lins, x = [], to_dev(x0)
    for p, s in layers:
        y = nan_out(1, p.shape[0])
        lins.append((to_dev(p), to_dev(s), x, y))
        x = y
    run(lins)
    xr = x0
    for i, ((p, s), lin, ex) in enumerate(zip(layers, lins, exact)):
        xr = oracle.gemv(p, s, xr, p.shape[0], p.shape[1] * 8)
        check_chain_reference(xr, ex, f"chain linear {i}")
        check_exact(lin[3], xr, f"chain linear {i}")


def test_write_after_read_and_three_way_conflicts():
    """Linear 2 overwrites linear 0's input (write-after-read) and reads
    linear 1's output; linear 4 conflicts with three earlier linears, which
    switches the whole call to strict ordering."""
    import torch

    rng = np.random.default_rng(4)
    k = n = 1024
    L = [int_linear(rng, n, k, 1 / 16) for _ in range(5)]
    xa = rng.integers(-1, 2, size=(1, k)).astype(np.float16)
    buf_a = to_dev(xa)                # x of 0 and 1, overwritten by 2
    y0, y1, y3 = nan_out(1, n), nan_out(1, n), nan_out(1, n)
    big = torch.full((1, 3 * n), float("nan"), dtype=torch.float16, device="cuda")
    y4 = big[:, :n]                    # written by 4; 4 reads a view spanning y0-like data
    announce("decode WAR + 3-way conflicts")
    lins = [
        (to_dev(L[0][0]), to_dev(L[0][1]), buf_a, y0),
        (to_dev(L[1][0]), to_dev(L[1][1]), buf_a, y1),
        (to_dev(L[2][0]), to_dev(L[2][1]), y1, buf_a),   # reads y1, overwrites x of 0 and 1
        (to_dev(L[3][0]), to_dev(L[3][1]), buf_a, y3),   # reads the new buf_a
        (to_dev(L[4][0]), to_dev(L[4][1]), y3, y4),
    ]
    run(lins)
    r0 = oracle.gemv(L[0][0], L[0][1], xa, n, k)
    r1 = oracle.gemv(L[1][0], L[1][1], xa, n, k)
    r2 = oracle.gemv(L[2][0], L[2][1], r1, n, k)
    r3 = oracle.gemv(L[3][0], L[3][1], r2, n, k)
    r4 = oracle.gemv(L[4][0], L[4][1], r3, n, k)
    check_exact(y0, r0, "0")
    check_exact(y1, r1, "1")
    check_exact(buf_a, r2, "2 (overwrote the shared input)")
    check_exact(y3, r3, "3")
    check_exact(y4, r4, "4")

    # Three conflicts for one linear: it reads y3 and overwrites y0 and y1.
    rng2 = np.random.default_rng(5)
    L5 = int_linear(rng2, 2 * n, k, 1 / 16)
    both = torch.full((1, 2 * n), float("nan"), dtype=torch.float16, device="cuda")
    lins2 = [
        (to_dev(L[0][0]), to_dev(L[0][1]), buf_a, both[:, :n]),
        (to_dev(L[1][0]), to_dev(L[1][1]), buf_a, both[:, n:]),
        (to_dev(L[3][0]), to_dev(L[3][1]), buf_a, y3),
        (to_dev(L5[0]), to_dev(L5[1]), y3, both),
    ]
    xb = to_host(buf_a, np.float16)
    run(lins2)
    r3b = oracle.gemv(L[3][0], L[3][1], xb, n, k)
    check_exact(y3, r3b, "3b")
    check_exact(both, oracle.gemv(L5[0], L5[1], r3b, 2 * n, k), "5 (three conflicts)")


def test_repeated_and_alternating_calls():
    """Counters reset between launches; switching descriptor lists re-uploads
    the table; two streams each get their own workspace."""
    import torch

    rng = np.random.default_rng(6)
    setA = [int_linear(rng, n, 2048, 1 / 8) for n in (700, 1300, 64)]
    setB = [int_linear(rng, n, 3072, 1 / 8) for n in (2000, 96)]
    xA = rng.integers(-1, 2, size=(1, 2048)).astype(np.float16)
    xB = rng.integers(-1, 2, size=(1, 3072)).astype(np.float16)
    dA, dB = to_dev(xA), to_dev(xB)
    linsA = [(to_dev(p), to_dev(s), dA, nan_out(1, p.shape[0])) for p, s in setA]
    linsB = [(to_dev(p), to_dev(s), dB, nan_out(1, p.shape[0])) for p, s in setB]
    refA = [oracle.gemv(p, s, xA, p.shape[0], 2048) for p, s in setA]
    refB = [oracle.gemv(p, s, xB, p.shape[0], 3072) for p, s in setB]
    announce("decode repeated / alternating / two streams")
    for rep in range(3):
        for lins, refs in ((linsA, refA), (linsB, refB)):
            for lin in lins:
                lin[3].fill_(float("nan"))
            run(lins)
            for lin, r in zip(lins, refs):
                check_exact(lin[3], r, f"rep {rep}")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for lin in linsA + linsB:
        lin[3].fill_(float("nan"))
    torch.cuda.synchronize()
    from paper_2412_15803_amd import wq

    wq.wq_decode_linears(linsA, m=1, stream=s1)
    wq.wq_decode_linears(linsB, m=1, stream=s2)
    torch.cuda.synchronize()
    for lin, r in zip(linsA + linsB, refA + refB):
        check_exact(lin[3], r, "two streams")


def test_many_linears_grow_workspace():
    rng = np.random.default_rng(7)
    count = 300
    shapes = [(int(rng.integers(1, 200)), int(rng.choice([32, 64, 256, 1024]))) for _ in range(count)]
    announce(f"decode {count} small linears")
    host, lins = [], []
    for n, k in shapes:
        p, s = int_linear(rng, n, k, 1 / 4)
        x = rng.integers(-1, 2, size=(1, k)).astype(np.float16)
        host.append((p, s, x))
        lins.append((to_dev(p), to_dev(s), to_dev(x), nan_out(1, n)))
    run(lins)
    for (p, s, x), lin, (n, k) in zip(host, lins, shapes):
        check_exact(lin[3], oracle.gemv(p, s, x, n, k), f"{n}x{k}")


def test_fallback_paths_small_batch_and_long_k():
    """A two-linear chain at M = 4 (two grouped launches) and K > 16384 at
    M = 1 (one launch per linear), still in order."""
    rng = np.random.default_rng(8)
    announce("decode fallback M=4 chain and K=16416")
    m = 4
    a = int_linear(rng, 512, 1024, 1 / 16)
    b = int_linear(rng, 256, 512, 1 / 16)
    x0 = rng.integers(-1, 2, size=(m, 1024)).astype(np.float16)
    ya, yb = nan_out(m, 512), nan_out(m, 256)
    run([(to_dev(a[0]), to_dev(a[1]), to_dev(x0), ya), (to_dev(b[0]), to_dev(b[1]), ya, yb)], m=m)
    ra = oracle.gemv(a[0], a[1], x0, 512, 1024)
    check_exact(ya, ra, "M=4 first")
    check_exact(yb, oracle.gemv(b[0], b[1], ra, 256, 512), "M=4 second")
    c = int_linear(rng, 100, 16416, 1 / 16)
    xc = rng.integers(-1, 2, size=(1, 16416)).astype(np.float16)
    yc = nan_out(1, 100)
    run([(to_dev(c[0]), to_dev(c[1]), to_dev(xc), yc)])
    check_exact(yc, oracle.gemv(c[0], c[1], xc, 100, 16416), "K=16416")


def test_decode_matches_single_gemv_random_data():
    """On random fp data the persistent kernel gives the same bits as
    wq_gemv for each linear (same per-row arithmetic), and both are within
    tolerance of the oracle."""
    import torch

    from paper_2412_15803_amd import wq

    rng = np.random.default_rng(9)
    shapes = [(5120, 3072), (3072, 8192), (6144, 4096), (4096, 14336)]
    announce("decode vs gemv, random data")
    lins, singles, host = [], [], []
    for i, (n, k) in enumerate(shapes):
        p, s = wl.random_words_host(50 + i, n, k), wl.random_scales_host(70 + i, n, k)
        x = wl.x_host(60 + i, 1, k)
        host.append((p, s, x))
        dp, ds, dx = to_dev(p), to_dev(s), to_dev(x)
        lins.append((dp, ds, dx, nan_out(1, n)))
        y1 = nan_out(1, n)
        wq.wq_gemv(dp, ds, dx, y1)
        singles.append(y1)
    run(lins)
    for (p, s, x), lin, y1, (n, k) in zip(host, lins, singles, shapes):
        assert torch.equal(lin[3].view(torch.int16), y1.view(torch.int16)), f"{n}x{k}"
        ok = oracle.within_tolerance(to_host(lin[3], np.float16), oracle.gemv(p, s, x, n, k),
                                     oracle.tol_bound(p, s, x, n, k))
        assert ok.all(), f"{n}x{k}"


@pytest.mark.parametrize("m", [2, 4, 16, 17, 33])
def test_small_batch_independent_linears_bit_exact(m):
    """Independent linears of mixed K (a group count that is not a multiple
    of 4, the 8B shapes' widths, K = 14336) and ragged N in one grouped
    matrix-core launch per 16 batch rows; every row checked."""
    rng = np.random.default_rng(100 + m)
    shapes = [(300, 1056), (4096, 4096), (1000, 14336), (37, 800), (6144, 4096), (257, 2080)]
    announce(f"decode small batch M={m}, {len(shapes)} independent linears")
    host, lins = [], []
    for n, k in shapes:
        p, s = int_linear(rng, n, k, 1 / 8)
        x = rng.integers(-1, 2, size=(m, k)).astype(np.float16)
        host.append((p, s, x))
        lins.append((to_dev(p), to_dev(s), to_dev(x), nan_out(m, n)))
    run(lins, m=m)
    for (p, s, x), lin, (n, k) in zip(host, lins, shapes):
        check_exact(lin[3], oracle.gemv(p, s, x, n, k), f"M={m} {n}x{k}")


@pytest.mark.parametrize("m", [3, 8, 16])
def test_small_batch_pow2_scales_bit_exact(m):
    """Grouped matrix-core launch with a power-of-two scale per (row, group):
    any mix-up of which lane applies which group's scale changes the bits.
    Even and odd group counts per row (the two scale load paths)."""
    shapes = [(300, 1056), (520, 4096), (77, 3104), (131, 14336), (1000, 2080)]
    announce(f"decode small batch M={m}, power-of-two scales")
    host, lins = [], []
    for i, (n, k) in enumerate(shapes):
        p = wl.random_words_host(400 + i, n, k)
        s = wl.pow2_scales_host(500 + i, n, k)
        x = wl.small_int_x_host(600 + i, m, k, lim=3)
        host.append((p, s, x))
        lins.append((to_dev(p), to_dev(s), to_dev(x), nan_out(m, n)))
    run(lins, m=m)
    for (p, s, x), lin, (n, k) in zip(host, lins, shapes):
        check_exact(lin[3], oracle.gemv(p, s, x, n, k), f"M={m} {n}x{k}")


@pytest.mark.parametrize("m", [2, 3, 5])
def test_small_batch_3b_layer_bit_exact(m):
    """The 3B layer's four linears (96-group rows walked in 32-group tiles,
    and the 256-group down projection) in one grouped vector launch; every
    row checked."""
    rng = np.random.default_rng(500 + m)
    shapes = [(lin.n, lin.k) for lin in wl.LLAMA3B_LAYER]
    announce(f"decode small batch M={m}, 3B layer")
    host, lins = [], []
    for n, k in shapes:
        p, s = int_linear(rng, n, k, 1 / 4)
        x = rng.integers(-1, 2, size=(m, k)).astype(np.float16)
        host.append((p, s, x))
        lins.append((to_dev(p), to_dev(s), to_dev(x), nan_out(m, n)))
    run(lins, m=m)
    for (p, s, x), lin, (n, k) in zip(host, lins, shapes):
        check_exact(lin[3], oracle.gemv(p, s, x, n, k), f"M={m} {n}x{k}")


@pytest.mark.parametrize("m", [4, 16])
def test_small_batch_dependency_chain_bit_exact(m):
    """x of linear i+1 is y of linear i for 12 linears: every linear is its
    own grouped launch, in stream order."""
    rng = np.random.default_rng(200 + m)
    dims = [int(d) for d in rng.choice([256, 512, 1024, 2048], size=13)]
    x0 = rng.integers(-8, 9, size=(m, dims[0])).astype(np.float16)
    layers, exact = bounded_chain(rng, dims, x0, 1 / 16)
    announce(f"decode small batch M={m}, 12-linear chain")
    lins, x = [], to_dev(x0)
    for p, s in layers:
        y = nan_out(m, p.shape[0])
        lins.append((to_dev(p), to_dev(s), x, y))
        x = y
    run(lins, m=m)
    xr = x0
    for i, ((p, s), lin, ex) in enumerate(zip(layers, lins, exact)):
        xr = oracle.gemv(p, s, xr, p.shape[0], p.shape[1] * 8)
        check_chain_reference(xr, ex, f"M={m} chain linear {i}")
        check_exact(lin[3], xr, f"M={m} chain linear {i}")


@pytest.mark.parametrize("m", [4, 16])
def test_small_batch_decode_random_data_tolerance(m):
    """Random codes, scales and x on the 8B layer's shapes: every output of
    the grouped launch within tolerance of the oracle (sampled rows)."""
    shapes = [(6144, 4096), (4096, 4096), (28672, 4096), (4096, 14336)]
    announce(f"decode small batch M={m}, 8B layer, random data")
    host, lins = [], []
    for i, (n, k) in enumerate(shapes):
        p, s = wl.random_words_host(300 + i, n, k), wl.random_scales_host(310 + i, n, k)
        x = wl.x_host(320 + i + m, m, k)
        host.append((p, s, x))
        lins.append((to_dev(p), to_dev(s), to_dev(x), nan_out(m, n)))
    run(lins, m=m)
    for (p, s, x), lin, (n, k) in zip(host, lins, shapes):
        rows = np.sort(np.random.default_rng(n + k).choice(n, size=min(n, 256), replace=False))
        pr, sr = np.ascontiguousarray(p[rows]), np.ascontiguousarray(s[rows])
        y = to_host(lin[3], np.float16)[:, rows]
        ok = oracle.within_tolerance(y, oracle.gemv(pr, sr, x, len(rows), k), oracle.tol_bound(pr, sr, x, len(rows), k))
        assert ok.all(), f"M={m} {n}x{k}: {(~ok).sum()} outside tolerance"


@pytest.mark.parametrize("m", [3, 6, 8, 16])
def test_small_batch_both_paths_bit_exact(m, monkeypatch):
    """From M = 3 on the matrix cores are the default; the vector kernel
    (forced through WQ_SMALL_BATCH_VECTOR, read by the library at every call)
    must give the same exact results, single GEMV and decode step alike."""
    from paper_2412_15803_amd import wq

    rng = np.random.default_rng(400 + m)
    shapes = [(4096, 4096), (1000, 14336), (257, 2080)]
    host, data = [], []
    for n, k in shapes:
        p, s = int_linear(rng, n, k, 1 / 8)
        x = rng.integers(-1, 2, size=(m, k)).astype(np.float16)
        host.append((p, s, x))
        data.append((to_dev(p), to_dev(s), to_dev(x)))
    for vector in (False, True):
        if vector:
            monkeypatch.setenv("WQ_SMALL_BATCH_VECTOR", "1")
        else:
            monkeypatch.delenv("WQ_SMALL_BATCH_VECTOR", raising=False)
        announce(f"small batch M={m} {'vector' if vector else 'matrix-core'} path")
        lins = [(p, s, x, nan_out(m, n)) for (p, s, x), (n, k) in zip(data, shapes)]
        run(lins, m=m)
        for (p, s, x), lin, (n, k) in zip(host, lins, shapes):
            ref = oracle.gemv(p, s, x, n, k)
            check_exact(lin[3], ref, f"decode M={m} {n}x{k} vector={vector}")
            y1 = nan_out(m, n)
            wq.wq_gemv(lin[0], lin[1], lin[2], y1)
            check_exact(y1, ref, f"gemv M={m} {n}x{k} vector={vector}")
    monkeypatch.delenv("WQ_SMALL_BATCH_VECTOR", raising=False)


@pytest.mark.parametrize("m", [1, 3, 4, 8, 16])
def test_decode_random_linear_sets_bit_exact(m):
    """A seeded set of 12 independent linears of random N and K in one call
    (the grouped kernels' plans: mixed classes, ragged row runs, balanced
    wave ranges), integer-exact inputs, every output checked."""
    rng = np.random.default_rng(7000 + m)
    shapes = [(int(rng.integers(1, 3000)), 32 * int(rng.integers(1, 449))) for _ in range(12)]
    announce(f"decode random set M={m} shapes={shapes}")
    host, lins = [], []
    for n, k in shapes:
        p = wl.random_words_host(int(rng.integers(1 << 30)), n, k)
        s = wl.constant_scales_host(n, k, 0x2400)
        x = wl.small_int_x_host(int(rng.integers(1 << 30)), m, k)
        host.append((p, s, x))
        lins.append((to_dev(p), to_dev(s), to_dev(x), nan_out(m, n)))
    run(lins, m=m)
    for (p, s, x), lin, (n, k) in zip(host, lins, shapes):
        check_exact(lin[3], oracle.gemv(p, s, x, n, k), f"M={m} {n}x{k}")


# ------------------------------------------------------- plans and capture

def _int_set(rng, shapes, m):
    host, lins = [], []
    for n, k in shapes:
        p, s = int_linear(rng, n, k, 1 / 4)
        x = rng.integers(-1, 2, size=(m, k)).astype(np.float16)
        host.append((p, s, x))
        lins.append((to_dev(p), to_dev(s), to_dev(x), nan_out(m, n)))
    return host, lins


def _check_set(host, lins, what):
    for (p, s, x), lin in zip(host, lins):
        n, k = p.shape[0], p.shape[1] * 8
        check_exact(lin[3], oracle.gemv(p, s, x, n, k), f"{what} {n}x{k}")


# Reusable plan buffers the library keeps per stream (include/wq.h).
RESIDENT_PLANS = 32


def test_alternating_lists_stay_correct():
    """Two descriptor lists used alternately on one stream (both plans stay
    resident), then more lists than the resident plans kept per stream, then
    the first two again: every call's outputs exact."""
    rng = np.random.default_rng(801)
    sets = [_int_set(rng, [(int(rng.integers(1, 700)), 32 * int(rng.integers(1, 130))) for _ in range(3)], 1)
            for _ in range(2)]
    sets += [_int_set(rng, [(int(rng.integers(1, 300)), 32 * int(rng.integers(1, 50)))], 1)
             for _ in range(RESIDENT_PLANS + 4)]
    announce("decode alternating lists")
    order = [0, 1, 0, 1, 0] + list(range(2, len(sets))) + [0, 1]
    for i in order:
        host, lins = sets[i]
        for lin in lins:
            lin[3].fill_(float("nan"))
        run(lins)
        _check_set(host, lins, f"list {i}")


def test_capture_needs_a_resident_plan():
    """Capturing a call whose plan is not on the device yet is refused
    (WQ_ERR_UNSUPPORTED, nothing recorded); after one eager call on the same
    stream the capture records only launches, and the graph still replays
    correctly after more than the resident-plan count of other lists has
    passed through that stream."""
    import torch

    from paper_2412_15803_amd import wq

    rng = np.random.default_rng(802)
    host, lins = _int_set(rng, [(5120, 3072), (3072, 3072), (16384, 3072), (3072, 8192)], 1)
    others = [_int_set(rng, [(int(rng.integers(1, 300)), 32 * int(rng.integers(1, 50)))], 1)
              for _ in range(RESIDENT_PLANS + 4)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    # the stream's workspace exists before capture (its set-up is not a
    # capture-safe operation), but this list's plan is not in it
    wq.wq_decode_linears(others[0][1], stream=s)
    s.synchronize()
    announce("decode capture of a new list")
    g0 = torch.cuda.CUDAGraph()
    status = None
    with torch.cuda.graph(g0, stream=s):
        try:
            wq.wq_decode_linears(lins, stream=s)
        except wq.WQError as e:
            status = e.status
    assert status == wq.WQ_ERR_UNSUPPORTED
    del g0
    announce("decode capture of a resident list")
    wq.wq_decode_linears(lins, stream=s)
    s.synchronize()
    _check_set(host, lins, "eager")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        wq.wq_decode_linears(lins, stream=s)
    for rep in range(3):
        for oh, ol in others:
            with torch.cuda.stream(s):
                wq.wq_decode_linears(ol, stream=s)
        s.synchronize()
        for oh, ol in others:
            _check_set(oh, ol, f"other list, round {rep}")
        for lin in lins:
            lin[3].fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _check_set(host, lins, f"replay {rep}")
    del g
