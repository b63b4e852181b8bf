"""Parity of the HIP library (through its C ABI) with the CPU oracle.

Bit-exact: packing (codes and scale bits) on every input; the GEMV on inputs
where the exact result is unique (one-hot x, integer-valued data whose fp32
partial sums are exact in any order).  Otherwise the GEMV must satisfy, per
element, |y_gpu - y_ref| <= 1e-3 * sum_k |w_hat x| + 1e-5.  Full-size shapes
are compared on sampled rows, which the oracle computes one by one; the
launch configuration is the one used at that size everywhere else.
"""

import json
import os

import numpy as np
import pytest

import oracle
from gpu_util import announce, gpu_gemv, gpu_pack, require_gpu, sample_rows, to_dev, to_host
from paper_2412_15803_amd import workloads as wl

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

SHAPES_3B = [(lin.n, lin.k) for lin in wl.LLAMA3B_LAYER]
SHAPES_8B = [(lin.n, lin.k) for lin in wl.LLAMA8B_LAYER]
SHAPES_TP = [(lin.n, lin.k) for lin in wl.LLAMA8B_TP8_SHARDS]
# Ragged and boundary shapes: K/32 not a multiple of 64, N not a multiple of
# the rows per step, one group per row, the largest tuned K and one past it.
SHAPES_EDGE = [(1, 32), (3, 64), (37, 800), (4097, 3104), (257, 2080), (5, 16384), (7, 16416), (1000, 1056)]


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


# ------------------------------------------------------------------- pack

def _check_pack(w_host, rows=None, label=""):
    announce(f"pack {label} shape={w_host.shape}")
    packed, scales = gpu_pack(to_dev(w_host))
    p = to_host(packed, np.uint32)
    s = to_host(scales, np.uint16)
    if rows is None:
        rp, rs = oracle.quantize_pack(w_host)
        assert np.array_equal(s, rs), "scale bits differ"
        assert np.array_equal(p, rp), "packed words differ"
    else:
        rp, rs = oracle.quantize_pack(np.ascontiguousarray(w_host[rows]))
        assert np.array_equal(s[rows], rs), "scale bits differ"
        assert np.array_equal(p[rows], rp), "packed words differ"


def test_pack_small_config_bit_exact():
    _check_pack(wl.weights_host(1, 512, 512), label="512x512")


def test_pack_golden_groups_bit_exact():
    cases = json.load(open(os.path.join(GOLDEN, "quantize_groups.json")))["cases"]
    w = np.zeros((len(cases), 32), dtype=np.float32)
    for i, c in enumerate(cases):
        for idx, hx in c["nonzero"].items():
            w[i, int(idx)] = np.float32(float.fromhex(hx))
    announce("pack golden groups")
    packed, scales = gpu_pack(to_dev(w))
    p = to_host(packed, np.uint32)
    s = to_host(scales, np.uint16)
    for i, c in enumerate(cases):
        assert int(s[i, 0]) == int(c["scale_bits"], 16), c["name"]
        codes = [(int(p[i, j // 8]) >> (4 * (j % 8))) & 0xF for j in range(32)]
        assert codes == c["codes"], c["name"]


def test_pack_ties_tiny_and_large_magnitudes_bit_exact():
    rng = np.random.default_rng(31)
    n, k = 96, 800
    w = rng.standard_normal((n, k), dtype=np.float32) * np.float32(0.02)
    # Exact ties: w = s * (j + 1/2) in groups whose max is 7 s (s a power of 2).
    for r in range(0, 16):
        s = np.float32(2.0 ** rng.integers(-10, 2))
        g = rng.integers(0, k // 32)
        vals = (rng.integers(-7, 7, size=32) + np.float32(0.5)) * s
        vals[rng.integers(0, 32)] = 7 * s * rng.choice([-1, 1])
        w[r, 32 * g:32 * g + 32] = vals.astype(np.float32)
    w[16:24] *= np.float32(3e-6)   # fp16 subnormal and zero scales
    w[24:28] *= np.float32(1e-9)   # scales that underflow to 0
    w[28:32] = 0.0                 # all-zero rows
    w[32:40] *= np.float32(3e3)    # large scales
    w[40:48] = np.abs(w[40:48])    # one-signed groups
    _check_pack(w, label="ties/magnitudes")


@pytest.mark.parametrize("n,k", SHAPES_3B + SHAPES_EDGE, ids=lambda v: str(v))
def test_pack_shapes_bit_exact(n, k):
    w = wl.weights_host(100 + n + k, n, k)
    rows = None if n * k <= 4_000_000 else sample_rows(n, 256, n + k)
    _check_pack(w, rows, label=f"{n}x{k}")


def test_pack_largest_linear_sampled_bit_exact():
    n, k = 28672, 4096
    w = wl.weights_host(7, n, k)
    _check_pack(w, sample_rows(n, 512, 3), label="8B gate_up")


# ------------------------------------------------------------------- GEMV

def _gemv_case(packed_h, scales_h, x_h, rows, exact, label):
    n = packed_h.shape[0]
    k = packed_h.shape[1] * 8
    m = x_h.shape[0]
    announce(f"gemv {label} N={n} K={k} M={m} exact={exact}")
    y = to_host(gpu_gemv(to_dev(packed_h), to_dev(scales_h), to_dev(x_h)), np.float16)
    if rows is None:
        rows = np.arange(n)
    pr, sr = np.ascontiguousarray(packed_h[rows]), np.ascontiguousarray(scales_h[rows])
    y_ref = oracle.gemv(pr, sr, x_h, len(rows), k)
    y_gpu = y[:, rows]
    if exact:
        bad = np.argwhere(y_gpu.view(np.uint16) != y_ref.view(np.uint16))
        assert bad.size == 0, f"{len(bad)} mismatches, first {bad[:5].tolist()} gpu={y_gpu[tuple(bad[0])]} ref={y_ref[tuple(bad[0])]}"
    else:
        bound = oracle.tol_bound(pr, sr, x_h, len(rows), k)
        ok = oracle.within_tolerance(y_gpu, y_ref, bound)
        bad = np.argwhere(~ok)
        assert bad.size == 0, f"{len(bad)} outside tolerance, first {bad[:5].tolist()}"
    return y


def _random_packed(seed, n, k):
    return wl.random_words_host(seed, n, k), wl.random_scales_host(seed + 1, n, k)


def test_gemv_small_config_tolerance():
    n = k = 512
    w = wl.weights_host(1, n, k)
    x = wl.x_host(2, 1, k)
    # oracle inputs come from the oracle's own packing of the same W
    rp, rs = oracle.quantize_pack(w)
    announce("gemv 512x512 random")
    packed, scales = gpu_pack(to_dev(w))
    y = to_host(gpu_gemv(packed, scales, to_dev(x)), np.float16)
    y_ref = oracle.gemv(rp, rs, x, n, k)
    assert np.all(oracle.within_tolerance(y, y_ref, oracle.tol_bound(rp, rs, x, n, k)))


@pytest.mark.parametrize("n,k", [(512, 512), (5120, 3072), (3072, 8192), (4096, 14336), (37, 800), (7, 16416)],
                         ids=lambda v: str(v))
@pytest.mark.parametrize("m", [1, 4, 16])
def test_gemv_one_hot_bit_exact(n, k, m):
    p, s = _random_packed(n * 7 + k, n, k)
    rng = np.random.default_rng(n + k + m)
    cols = rng.choice(k, size=m, replace=False)
    cols[0] = k - 1
    x = wl.one_hot_x_host(m, k, cols)
    _gemv_case(p, s, x, sample_rows(n, 512, 5), True, "one-hot")


INT_SHAPES = SHAPES_3B + SHAPES_8B + SHAPES_TP + SHAPES_EDGE + [(wl.LLAMA3B_LM_HEAD.n, wl.LLAMA3B_LM_HEAD.k)]


@pytest.mark.parametrize("n,k", INT_SHAPES, ids=lambda v: str(v))
def test_gemv_integer_exact_m1(n, k):
    """Every scale 2^-6 and x in {-4..4}: every partial sum is a multiple of
    2^-6 of magnitude at most 8*4*K*2^-6 (below 2^24 units for K <= 2^17), so
    fp32 accumulation is exact in any order and the result is unique."""
    p = wl.random_words_host(n + k, n, k)
    s = wl.constant_scales_host(n, k, 0x2400)
    x = wl.small_int_x_host(n * 3 + k, 1, k)
    _gemv_case(p, s, x, sample_rows(n, 512, 9), True, "integer-exact")


# Batch-1 single-linear launches of about 1024 waves: a last wave with one
# row or one partial step, a wave count just past 1024, and rows that fit
# one step of the widest shapes.
M1_LAUNCH_EDGES = [(2049, 3072), (1025, 4096), (2047, 8192), (3, 14336), (65, 96), (1024 * 6 + 5, 3072)]


@pytest.mark.parametrize("n,k", M1_LAUNCH_EDGES, ids=lambda v: str(v))
def test_gemv_integer_exact_m1_launch_edges(n, k):
    p = wl.random_words_host(n * 11 + k, n, k)
    s = wl.constant_scales_host(n, k, 0x2400)
    x = wl.small_int_x_host(n * 5 + k, 1, k)
    _gemv_case(p, s, x, None, True, "integer-exact launch edge")


@pytest.mark.parametrize("n,k", SHAPES_8B + SHAPES_EDGE[2:5], ids=lambda v: str(v))
@pytest.mark.parametrize("m", [2, 4, 8, 16])
def test_gemv_integer_exact_small_batch(n, k, m):
    p = wl.random_words_host(n + k + m, n, k)
    s = wl.constant_scales_host(n, k, 0x2400)
    x = wl.small_int_x_host(n * 3 + k + m, m, k)
    _gemv_case(p, s, x, sample_rows(n, 256, 11), True, "integer-exact")


def _use_path(monkeypatch, path):
    """'vector' forces the vector small-batch kernel (the library reads
    WQ_SMALL_BATCH_VECTOR at every call); 'default' takes the library's
    choice (the vector kernel at M = 2, the matrix cores from M = 3)."""
    if path == "vector":
        monkeypatch.setenv("WQ_SMALL_BATCH_VECTOR", "1")
    else:
        monkeypatch.delenv("WQ_SMALL_BATCH_VECTOR", raising=False)


# Group counts that the vector small-batch kernel walks in 32-group tiles
# with two row sets per wave (96 and 160 groups: an odd multiple of 32; 1, 2,
# 31 and 32 groups: below one 64-group tile), and the 3B layer's widths.
SHAPES_32_GROUP_TILES = SHAPES_3B + [(1, 32), (3, 64), (33, 992), (8, 1024), (1000, 5120)]


@pytest.mark.parametrize("path", ["vector", "default"])
@pytest.mark.parametrize("n,k", SHAPES_32_GROUP_TILES, ids=lambda v: str(v))
@pytest.mark.parametrize("m", [2, 3, 4, 7])
def test_gemv_integer_exact_small_batch_32_group_tiles(n, k, m, path, monkeypatch):
    _use_path(monkeypatch, path)
    p = wl.random_words_host(5 * n + k + m, n, k)
    s = wl.constant_scales_host(n, k, 0x2400)
    x = wl.small_int_x_host(n + 7 * k + m, m, k)
    _gemv_case(p, s, x, sample_rows(n, 256, 19), True, "integer-exact")


# Single linears with few row runs: the vector kernel splits each run's K
# tiles over 2 or 4 waves of a block and sums their partials in LDS.  Ragged
# N (last run of one row), uneven tile shares (5 tiles over 4 waves) and
# several tiles per wave.
SHAPES_K_SPLIT = [(37, 8192), (1001, 5120), (5, 16384), (3, 4096)]


@pytest.mark.parametrize("path", ["vector", "default"])
@pytest.mark.parametrize("n,k", SHAPES_K_SPLIT, ids=lambda v: str(v))
@pytest.mark.parametrize("m", [2, 3, 5, 7])
def test_gemv_integer_exact_small_batch_k_split(n, k, m, path, monkeypatch):
    _use_path(monkeypatch, path)
    p = wl.random_words_host(11 * n + k + m, n, k)
    s = wl.constant_scales_host(n, k, 0x2400)
    x = wl.small_int_x_host(3 * n + 5 * k + m, m, k)
    _gemv_case(p, s, x, None, True, "integer-exact K split")


def _random_small_batch_shapes(count, seed):
    """Seeded (N, K, M) draws across the vector kernel's launch shapes: 64- and
    32-group tiles, K split over 1, 2 or 4 waves, ragged row runs, M 2..7."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        n = int(rng.choice([int(rng.integers(1, 64)), int(rng.integers(64, 1200)), int(rng.integers(1200, 6000))]))
        k = 32 * int(rng.integers(1, 513))
        m = int(rng.integers(2, 8))
        out.append((n, k, m))
    return out


def _random_shapes(count, seed, ms):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        n = int(rng.choice([int(rng.integers(1, 64)), int(rng.integers(64, 1200)), int(rng.integers(1200, 6000))]))
        k = 32 * int(rng.integers(1, 513))
        out.append((n, k, int(rng.choice(ms))))
    return out


@pytest.mark.parametrize("n,k,m", _random_shapes(16, 2025, [1]) + _random_shapes(16, 2026, list(range(8, 17))),
                         ids=lambda v: str(v))
def test_gemv_integer_exact_random_shapes_m1_and_matrix_cores(n, k, m):
    """Seeded shapes for the batch-1 kernels (every lanes-per-row and
    groups-per-lane class, ragged N) and the matrix-core kernel (M 8..16)."""
    p = wl.random_words_host(n * 5 + k * 7 + m, n, k)
    s = wl.constant_scales_host(n, k, 0x2400)
    x = wl.small_int_x_host(n + 3 * k + 19 * m, m, k)
    _gemv_case(p, s, x, None, True, "integer-exact random shape")


@pytest.mark.parametrize("n,k,m", [(16, 32, 8), (40, 96, 16), (257, 544, 9), (300, 1056, 16), (1000, 2080, 12),
                                   (520, 4096, 16), (131, 14336, 8), (77, 3104, 13), (64, 256, 3), (999, 4096, 5),
                                   (200, 8192, 7)], ids=lambda v: str(v))
def test_gemv_pow2_scales_matrix_cores_bit_exact(n, k, m):
    """A power-of-two scale per (row, group) and small-integer x keep every
    sum exact, so any mix-up of which lane applies which group's scale
    changes the bits.  Even and odd numbers of groups per row (the two scale
    load paths), one to several waves per block, ragged N."""
    p = wl.random_words_host(n * 11 + k + m, n, k)
    s = wl.pow2_scales_host(n + 5 * k + m, n, k)
    x = wl.small_int_x_host(2 * n + k + 3 * m, m, k, lim=3)
    _gemv_case(p, s, x, None, True, "power-of-two scales")


# Batches past 16 rows run on the matrix cores in chunks of 16 rows.  On a
# one-tile launch with at least 32 steps of K, a last chunk of at most 8 rows
# splits K over eight waves per block and the chunks before it over four.
@pytest.mark.parametrize("n,k,m", [(300, 4096, 20), (4096, 4096, 24), (131, 14336, 40), (1000, 8192, 56)],
                         ids=lambda v: str(v))
def test_gemv_integer_exact_matrix_core_chunks(n, k, m):
    p = wl.random_words_host(n * 13 + k + m, n, k)
    s = wl.constant_scales_host(n, k, 0x2400)
    x = wl.small_int_x_host(n + 11 * k + m, m, k)
    _gemv_case(p, s, x, sample_rows(n, 256, 23), True, "integer-exact chunked batch")


@pytest.mark.parametrize("path", ["vector", "default"])
@pytest.mark.parametrize("n,k,m", _random_small_batch_shapes(24, 2024), ids=lambda v: str(v))
def test_gemv_integer_exact_small_batch_random_shapes(n, k, m, path, monkeypatch):
    _use_path(monkeypatch, path)
    p = wl.random_words_host(n * 7 + k * 3 + m, n, k)
    s = wl.constant_scales_host(n, k, 0x2400)
    x = wl.small_int_x_host(n + k + 17 * m, m, k)
    _gemv_case(p, s, x, None, True, "integer-exact random shape")


@pytest.mark.parametrize("m", [4, 16])
def test_gemv_integer_exact_small_batch_3b_lm_head(m):
    """The 3B LM head on the vector kernel (M=4) and on the matrix cores with
    2-step chunks (M=16, the launch used for very tall linears)."""
    n, k = wl.LLAMA3B_LM_HEAD.n, wl.LLAMA3B_LM_HEAD.k
    p = wl.random_words_host(23, n, k)
    s = wl.constant_scales_host(n, k, 0x2400)
    x = wl.small_int_x_host(29 + m, m, k)
    _gemv_case(p, s, x, sample_rows(n, 512, 31), True, "integer-exact LM head")


@pytest.mark.parametrize("n,k", SHAPES_3B + SHAPES_8B + SHAPES_TP + SHAPES_EDGE, ids=lambda v: str(v))
def test_gemv_random_weights_tolerance_m1(n, k):
    w = wl.weights_host(1000 + n + k, n, k)
    x = wl.x_host(2000 + n + k, 1, k)
    rows = sample_rows(n, 512, 13)
    rp, rs = oracle.quantize_pack(np.ascontiguousarray(w[rows]))
    announce(f"gemv random N={n} K={k}")
    packed, scales = gpu_pack(to_dev(w))
    y = to_host(gpu_gemv(packed, scales, to_dev(x)), np.float16)[:, rows]
    y_ref = oracle.gemv(rp, rs, x, len(rows), k)
    ok = oracle.within_tolerance(y, y_ref, oracle.tol_bound(rp, rs, x, len(rows), k))
    assert ok.all(), f"{(~ok).sum()} outside tolerance"


@pytest.mark.parametrize("n,k", SHAPES_8B, ids=lambda v: str(v))
@pytest.mark.parametrize("m", [4, 8, 16])
def test_gemv_random_weights_tolerance_small_batch(n, k, m):
    w = wl.weights_host(3000 + n + k, n, k)
    x = wl.x_host(4000 + n + k + m, m, k)
    rows = sample_rows(n, 256, 17)
    rp, rs = oracle.quantize_pack(np.ascontiguousarray(w[rows]))
    announce(f"gemv random N={n} K={k} M={m}")
    packed, scales = gpu_pack(to_dev(w))
    y = to_host(gpu_gemv(packed, scales, to_dev(x)), np.float16)[:, rows]
    y_ref = oracle.gemv(rp, rs, x, len(rows), k)
    ok = oracle.within_tolerance(y, y_ref, oracle.tol_bound(rp, rs, x, len(rows), k))
    assert ok.all(), f"{(~ok).sum()} outside tolerance"


@pytest.mark.parametrize("m", [3, 5, 17, 33])
def test_gemv_odd_batch_sizes(m):
    n, k = 300, 1056
    w = wl.weights_host(5000 + m, n, k)
    x = wl.x_host(6000 + m, m, k)
    rp, rs = oracle.quantize_pack(w)
    announce(f"gemv M={m}")
    packed, scales = gpu_pack(to_dev(w))
    y = to_host(gpu_gemv(packed, scales, to_dev(x)), np.float16)
    y_ref = oracle.gemv(rp, rs, x, n, k)
    assert oracle.within_tolerance(y, y_ref, oracle.tol_bound(rp, rs, x, n, k)).all()


def test_gemv_largest_batch():
    m, n, k = 65535, 3, 64
    p, s = _random_packed(77, n, k)
    x = wl.small_int_x_host(78, m, k)
    s = wl.constant_scales_host(n, k, 0x2400)
    _gemv_case(p, s, x, None, True, "M=65535")


def test_gemv_all_zero_codes_closed_form():
    """Codes 0 everywhere dequantize to -8*s; with x = 1 every output is
    fp16(-256 * sum of the row's scales)."""
    n, k = 1024, 4096
    p = np.zeros((n, k // 8), dtype=np.uint32)
    s = wl.random_scales_host(5, n, k)
    x = np.ones((1, k), dtype=np.float16)
    _gemv_case(p, s, x, sample_rows(n, 256, 1), False, "all-zero codes")


def test_gemv_deterministic_and_stream():
    import torch

    from paper_2412_15803_amd import wq

    n, k = 5120, 3072
    w = wl.weights_host(8, n, k)
    x = wl.x_host(9, 1, k)
    announce("gemv determinism / side stream")
    packed, scales = gpu_pack(to_dev(w))
    xd = to_dev(x)
    y1 = gpu_gemv(packed, scales, xd)
    side = torch.cuda.Stream()
    y2 = torch.empty_like(y1)
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        wq.wq_gemv(packed, scales, xd, y2)
    side.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


def test_gemv_invalid_call_leaves_output_untouched():
    import torch

    from paper_2412_15803_amd import wq

    announce("gemv invalid args")
    # K = 48 is not a multiple of the group size: the library refuses it.
    packed = torch.zeros((64, 6), dtype=torch.int32, device="cuda")
    scales = torch.zeros((64, 1), dtype=torch.float16, device="cuda")
    x = torch.zeros((1, 48), dtype=torch.float16, device="cuda")
    y = torch.full((1, 64), 3.0, dtype=torch.float16, device="cuda")
    with pytest.raises(wq.WQError) as e:
        wq.wq_gemv(packed, scales, x, y)
    assert e.value.status == wq.WQ_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert bool((y == 3.0).all())


# ----------------------------------------------------------- decode step

def test_decode_linears_dependency_chain_bit_exact():
    """Linears chained through their outputs (x of linear i+1 is y of linear
    i, plus one skip connection).  With unit scales, codes in {7, 8, 9} and
    x in {-1, 0, 1} every partial sum is an integer below 2^24, so each
    output is the exact sum rounded once: bit-exact along the whole chain.
    Codes are mostly 8 (zero) so magnitudes stay below the fp16 range."""
    import torch

    from paper_2412_15803_amd import wq

    rng = np.random.default_rng(41)
    dims = [512, 768, 1024, 512, 640]
    k0 = dims[0]
    x0 = rng.integers(-1, 2, size=(1, k0)).astype(np.float16)
    layers = []
    for i in range(len(dims) - 1):
        k, n = dims[i], dims[i + 1]
        codes = rng.choice([7, 8, 9], size=(n, k), p=[1 / 16, 7 / 8, 1 / 16])
        packed = np.zeros((n, k // 8), dtype=np.uint32)
        for b in range(8):
            packed |= codes[:, b::8].astype(np.uint32) << np.uint32(4 * b)
        layers.append((packed, wl.constant_scales_host(n, k, 0x3C00)))
    # one extra linear reading the output of linear 0 again (a skip)
    n_skip = 256
    codes = rng.choice([7, 8, 9], size=(n_skip, dims[1]), p=[1 / 16, 7 / 8, 1 / 16])
    pk = np.zeros((n_skip, dims[1] // 8), dtype=np.uint32)
    for b in range(8):
        pk |= codes[:, b::8].astype(np.uint32) << np.uint32(4 * b)
    skip = (pk, wl.constant_scales_host(n_skip, dims[1], 0x3C00))

    announce("decode_linears chain")
    xs = [to_dev(x0)]
    ys = []
    lin = []
    for (p, s) in layers:
        y = torch.full((1, p.shape[0]), float("nan"), dtype=torch.float16, device="cuda")
        lin.append((to_dev(p), to_dev(s), xs[-1], y))
        ys.append(y)
        xs.append(y)
    y_skip = torch.full((1, n_skip), float("nan"), dtype=torch.float16, device="cuda")
    lin.append((to_dev(skip[0]), to_dev(skip[1]), ys[0], y_skip))
    wq.wq_decode_linears(lin, m=1)
    torch.cuda.synchronize()

    x_ref = x0
    outs = []
    for (p, s) in layers:
        y_ref = oracle.gemv(p, s, x_ref, p.shape[0], p.shape[1] * 8)
        outs.append(y_ref)
        x_ref = y_ref
    y_skip_ref = oracle.gemv(skip[0], skip[1], outs[0], n_skip, dims[1])
    for i, (yd, yr) in enumerate(zip(ys + [y_skip], outs + [y_skip_ref])):
        yh = to_host(yd, np.float16)
        assert np.array_equal(yh.view(np.uint16), yr.view(np.uint16)), f"linear {i}"


def test_decode_step_3b_sampled():
    """The full 3B-class decode step (28 layers + lm_head, 113 linears) with
    weights generated on the device per linear; every linear is checked on
    sampled rows: packing bit-exact and outputs within tolerance."""
    import torch

    from paper_2412_15803_amd import wq

    plan = wl.decode_step_linears(base_seed=1234)
    announce(f"decode step: building {len(plan)} linears")
    lins, checks = [], []
    for idx, (lin, ws, xs) in enumerate(plan):
        w = wl.weights_device(ws, lin.n, lin.k)
        packed, scales = gpu_pack(w)
        rows = sample_rows(lin.n, 24, idx)
        w_rows = w[torch.from_numpy(rows).to(w.device)].cpu().numpy()
        del w
        x = wl.x_device(xs, 1, lin.k)
        y = torch.full((1, lin.n), float("nan"), dtype=torch.float16, device="cuda")
        lins.append((packed, scales, x, y))
        checks.append((lin, rows, w_rows))
    announce("decode step: running wq_decode_linears")
    wq.wq_decode_linears(lins, m=1)
    torch.cuda.synchronize()
    for (packed, scales, x, y), (lin, rows, w_rows) in zip(lins, checks):
        rp, rs = oracle.quantize_pack(w_rows)
        ri = torch.from_numpy(rows).to("cuda")
        assert np.array_equal(to_host(packed[ri], np.uint32), rp), lin.name
        assert np.array_equal(to_host(scales[ri], np.uint16), rs), lin.name
        xh = to_host(x, np.float16)
        y_ref = oracle.gemv(rp, rs, xh, len(rows), lin.k)
        yg = to_host(y, np.float16)[:, rows]
        ok = oracle.within_tolerance(yg, y_ref, oracle.tol_bound(rp, rs, xh, len(rows), lin.k))
        assert ok.all(), lin.name


@pytest.mark.parametrize("m", [1, 8])
def test_decode_step_8b_sampled(m):
    """The 8B-class decode step (32 layers + lm_head, 129 linears, K up to
    14336) in one wq_decode_linears call at M = 1 (batch-1 grouped kernel)
    and M = 8 (matrix-core grouped kernel), weights generated on the device
    and packed by the library; every linear checked on sampled rows."""
    import torch

    from paper_2412_15803_amd import wq

    plan = wl.decode_step_linears_8b()
    announce(f"8B decode step M={m}: building {len(plan)} linears")
    lins, checks = [], []
    for idx, (lin, ws, xs) in enumerate(plan):
        w = wl.weights_device(ws, lin.n, lin.k)
        packed, scales = gpu_pack(w)
        rows = sample_rows(lin.n, 16, 1000 + idx)
        w_rows = w[torch.from_numpy(rows).to(w.device)].cpu().numpy()
        del w
        x = wl.x_device(xs, m, lin.k)
        y = torch.full((m, lin.n), float("nan"), dtype=torch.float16, device="cuda")
        lins.append((packed, scales, x, y))
        checks.append((lin, rows, w_rows))
    announce(f"8B decode step M={m}: running wq_decode_linears")
    wq.wq_decode_linears(lins, m=m)
    torch.cuda.synchronize()
    for (packed, scales, x, y), (lin, rows, w_rows) in zip(lins, checks):
        rp, rs = oracle.quantize_pack(w_rows)
        xh = to_host(x, np.float16)
        y_ref = oracle.gemv(rp, rs, xh, len(rows), lin.k)
        y_gpu = to_host(y, np.float16)[:, rows]
        ok = oracle.within_tolerance(y_gpu, y_ref, oracle.tol_bound(rp, rs, xh, len(rows), lin.k))
        assert ok.all(), f"{lin.name}: {(~ok).sum()} outside tolerance"
