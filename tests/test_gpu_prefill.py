"""GPU parity of the prefill GEMM (wq_gemv with more than 64 rows of x: the
tiled matrix-core kernel) against the CPU oracle.

Integer-exact inputs (scales 2^-6, x in {-4..4}) make every product and
partial sum exact in fp32 and every scaled weight exact in fp16, so those
cases are compared bit for bit; random inputs are compared within the GEMV
tolerance.  Ragged M, N and K (including K with a half-stage tail) cover the
tile edges; full prompt-sized shapes are checked on sampled rows and columns.
"""

from __future__ import annotations

import numpy as np
import pytest

import oracle
from gpu_util import announce, gpu_gemv, sample_rows, to_dev, to_host
from paper_2412_15803_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _run(packed, scales, x, rows_m=None, rows_n=None, exact=False, label=""):
    m, k = x.shape
    n = packed.shape[0]
    announce(f"prefill {label} M={m} N={n} K={k} exact={exact}")
    y = to_host(gpu_gemv(to_dev(packed), to_dev(scales), to_dev(x)), np.float16)
    rows_m = np.arange(m) if rows_m is None else rows_m
    rows_n = np.arange(n) if rows_n is None else rows_n
    pr, sr = np.ascontiguousarray(packed[rows_n]), np.ascontiguousarray(scales[rows_n])
    xs = np.ascontiguousarray(x[rows_m])
    ref = oracle.gemv(pr, sr, xs, len(rows_n), k)
    got = y[np.ix_(rows_m, rows_n)]
    if exact:
        bad = np.argwhere(got.view(np.uint16) != ref.view(np.uint16))
        assert bad.size == 0, f"{len(bad)} mismatches, first {bad[:5].tolist()}"
    else:
        ok = oracle.within_tolerance(got, ref, oracle.tol_bound(pr, sr, xs, len(rows_n), k))
        assert ok.all(), f"{np.count_nonzero(~ok)} outside tolerance, first {np.argwhere(~ok)[:5].tolist()}"
    return y


EXACT_SHAPES = [
    (65, 64, 64),        # one row past the small-batch range, one tile
    (128, 128, 64),      # exactly one tile, one stage
    (129, 130, 96),      # ragged M and N, K with a half stage
    (300, 1000, 3072),
    (1000, 33, 32),      # a single group
    (256, 257, 4128),    # K % 64 == 32
    (777, 5120, 3072),   # 3B qkv shape
]


@pytest.mark.parametrize("m,n,k", EXACT_SHAPES, ids=[f"M{m}_N{n}_K{k}" for m, n, k in EXACT_SHAPES])
def test_prefill_integer_exact(m, n, k):
    packed = wl.random_words_host(m + n + k, n, k)
    scales = wl.constant_scales_host(n, k, 0x2400)
    x = wl.small_int_x_host(m * 3 + k, m, k)
    _run(packed, scales, x, exact=True, label="integer-exact")


RANDOM_SHAPES = [(65, 3072, 3072), (200, 1000, 8192), (1024, 3072, 3072), (130, 4096, 14336)]


@pytest.mark.parametrize("m,n,k", RANDOM_SHAPES, ids=[f"M{m}_N{n}_K{k}" for m, n, k in RANDOM_SHAPES])
def test_prefill_random_tolerance(m, n, k):
    packed = wl.random_words_host(7 * m + n, n, k)
    scales = wl.random_scales_host(11 * k + m, n, k)
    x = wl.x_host(13 * m + k, m, k)
    rows_n = sample_rows(n, 384, m + n)
    _run(packed, scales, x, rows_n=rows_n, label="random")


@pytest.mark.parametrize("m,n,k", [(2048, 16384, 3072), (512, 28672, 4096), (4096, 3072, 8192)],
                         ids=["3B_gate_up_M2048", "8B_gate_up_M512", "3B_down_M4096"])
def test_prefill_prompt_shapes_sampled(m, n, k):
    """Prompt-sized shapes of the decoder layers, in the configuration bench.py
    times: every output computed, sampled rows of x and of W compared."""
    packed = wl.random_words_host(m + 3 * n, n, k)
    scales = wl.random_scales_host(m + 5 * n, n, k)
    x = wl.x_host(m + 7 * k, m, k)
    _run(packed, scales, x, rows_m=sample_rows(m, 48, m), rows_n=sample_rows(n, 256, n), label="prompt")


def test_prefill_quantized_weights_from_pack():
    """End to end: fp32 weights packed on the device, then a prefill GEMM."""
    from gpu_util import gpu_pack

    m, n, k = 300, 640, 1024
    w = wl.weights_host(91, n, k)
    x = wl.x_host(92, m, k)
    announce(f"prefill after wq_pack M={m} N={n} K={k}")
    packed, scales = gpu_pack(to_dev(w))
    y = to_host(gpu_gemv(packed, scales, to_dev(x)), np.float16)
    rp, rs = oracle.quantize_pack(w)
    ref = oracle.gemv(rp, rs, x, n, k)
    assert oracle.within_tolerance(y, ref, oracle.tol_bound(rp, rs, x, n, k)).all()


def test_prefill_decode_linears_chain_bit_exact():
    """wq_decode_linears at M = 96 (one launch per linear) with the second
    linear reading the first one's output."""
    import torch

    from paper_2412_15803_amd import wq

    announce("prefill decode_linears chain M=96")
    m, n1, k1, n2 = 96, 256, 128, 64
    p1 = wl.random_words_host(1, n1, k1)
    s1 = wl.constant_scales_host(n1, k1, 0x2000)  # 2^-7
    p2 = wl.random_words_host(2, n2, n1)
    s2 = wl.constant_scales_host(n2, n1, 0x2000)
    x = wl.small_int_x_host(3, m, k1, lim=2)
    xd = to_dev(x)
    y1 = torch.empty((m, n1), dtype=torch.float16, device=xd.device)
    y2 = torch.empty((m, n2), dtype=torch.float16, device=xd.device)
    lins = [(to_dev(p1), to_dev(s1), xd, y1), (to_dev(p2), to_dev(s2), y1, y2)]
    wq.wq_decode_linears(lins, m=m)
    torch.cuda.synchronize()
    r1 = oracle.gemv(p1, s1, x, n1, k1)
    r2 = oracle.gemv(p2, s2, r1, n2, n1)
    assert np.array_equal(to_host(y1, np.float16).view(np.uint16), r1.view(np.uint16))
    assert np.array_equal(to_host(y2, np.float16).view(np.uint16), r2.view(np.uint16))
