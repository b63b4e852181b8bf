"""GPU parity of decode attention over a paged KV cache (HIP kernels through
the C ABI) against the CPU oracle.

Random inputs are compared within the oracle's fp32 tolerance; inputs whose
answer is unique in any summation order (one dominant key, uniform weights
over integer values) are compared bit for bit, as are rearrangements of the
same cache that must not change the result.
"""

from __future__ import annotations

import numpy as np
import pytest

import attn_cases
from gpu_util import announce, require_gpu, to_dev
from oracle import attn_oracle

pytestmark = pytest.mark.gpu


def gpu_attention(case, max_seq_len=None, workspace=None):
    import torch

    from paper_2412_15803_amd import wq

    require_gpu()
    if max_seq_len is None:
        max_seq_len = int(max(case.seq_lens)) if len(case.seq_lens) else 0
    q = to_dev(case.q)
    k = to_dev(case.k_cache)
    v = to_dev(case.v_cache)
    # Widen the table (with -1, never read) so that it can hold max_seq_len.
    page = case.k_cache.shape[2]
    width = max(case.block_table.shape[1], -(-max_seq_len // page), 1)
    host_table = np.full((case.block_table.shape[0], width), -1, dtype=np.int32)
    host_table[:, :case.block_table.shape[1]] = case.block_table
    table = torch.from_numpy(host_table).to(q.device)
    lens = torch.from_numpy(np.ascontiguousarray(case.seq_lens.astype(np.int32))).to(q.device)
    out = torch.full(case.q.shape, float("nan"), dtype=torch.float16, device=q.device)
    wq.paged_attention(q.view(torch.float16), k.view(torch.float16), v.view(torch.float16), table, lens,
                       out, case.scale, max_seq_len, workspace=workspace)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def check_tolerance(case, got, label):
    o64, wabs, smax = attn_oracle.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                                       case.seq_lens, case.scale)
    assert np.all(smax <= attn_oracle.ATTN_MAX_SCORE_BOUND), "inputs outside the tolerance's range"
    ref = o64.astype(np.float16)
    ok = attn_oracle.attn_within_tolerance(got, ref, wabs)
    if not np.all(ok):
        bad = np.argwhere(~ok)
        s, h, d = bad[0]
        raise AssertionError(f"{label}: {len(bad)} elements out of tolerance, first at {tuple(bad[0])}: "
                             f"gpu {got[s, h, d]!r} ref {ref[s, h, d]!r} bound "
                             f"{attn_oracle.attn_tol_bound(wabs)[s, h, d]:.3g}")
    return ref


# (num_q_heads, num_kv_heads, page_size, seq_lens, max_seq_len or None)
RANDOM_CASES = [
    (24, 8, 16, (1,), None),
    (24, 8, 16, (15,), None),
    (24, 8, 16, (16,), None),
    (24, 8, 16, (17,), None),
    (24, 8, 16, (64,), None),
    (24, 8, 16, (65,), None),
    (24, 8, 16, (100,), None),
    (24, 8, 16, (1000,), None),
    (24, 8, 16, (4096,), None),
    (24, 8, 16, (4097,), None),
    (32, 8, 16, (33, 2048, 0, 5), None),
    (32, 8, 16, (300, 7), 5000),
    (8, 8, 16, (777,), None),
    (16, 8, 32, (513,), None),
    (40, 8, 16, (129,), None),
    (48, 8, 16, (200,), None),
    (56, 8, 16, (95,), None),
    (64, 8, 16, (1500,), None),
    (8, 1, 16, (2000,), None),
    (4, 2, 1, (70,), None),
    (4, 2, 2, (131,), None),
    (6, 2, 4, (99,), None),
    (6, 2, 8, (257,), None),
    (24, 8, 64, (1000,), None),
    (24, 8, 256, (3000,), None),
    (24, 8, 1024, (2500,), None),
    (24, 8, 16, tuple(range(1, 40)), None),
    # chunks (multiples of 64 tokens) that start inside a page
    (24, 8, 256, (20000,), None),
    (8, 8, 128, (10000,), None),
    (32, 8, 16, (8192,) * 4, None),
    # many sequences: chunks of 512 and 4096 tokens (long per-wave loops,
    # page lists longer than the workgroup)
    (8, 8, 1, tuple(range(2000, 2000 + 16 * 61, 61)), 4096),
    (32, 8, 16, tuple(int(x) for x in np.random.default_rng(3).integers(1, 8193, size=64)), 8192),
]


@pytest.mark.parametrize("hq,hkv,page,lens,max_len", RANDOM_CASES,
                         ids=[f"hq{c[0]}_kv{c[1]}_p{c[2]}_L{'-'.join(map(str, c[3][:4]))}"
                              f"{'...' if len(c[3]) > 4 else ''}_m{c[4]}" for c in RANDOM_CASES])
def test_attention_random_within_tolerance(hq, hkv, page, lens, max_len):
    seed = 1000 + hq * 7 + page + len(lens) + sum(lens) % 97
    announce(f"attention random hq={hq} hkv={hkv} page={page} lens={lens[:6]} max={max_len} seed={seed}")
    case = attn_cases.random_case(seed, hq, hkv, 128, page, lens, extra_pages=5)
    got = gpu_attention(case, max_seq_len=max_len)
    check_tolerance(case, got, f"hq={hq} hkv={hkv} page={page}")


@pytest.mark.parametrize("hq,hkv,page,lens", [
    (24, 8, 16, (1, 16, 17, 64, 100)),
    (24, 8, 16, (4097,)),
    (32, 8, 16, (9000, 3)),
    (64, 8, 4, (333,)),
    (8, 1, 32, (1200,)),
    (6, 2, 1, (90,)),
])
def test_attention_one_hot_bit_exact(hq, hkv, page, lens):
    """Each head's output is exactly one cached value vector: this checks
    the page lookup, the slot inside the page, the head-to-kv-head map and
    the merge of chunks bit for bit."""
    announce(f"attention one-hot hq={hq} hkv={hkv} page={page} lens={lens}")
    case, targets = attn_cases.one_hot_case(77 + page, hq, hkv, 128, page, lens, big=200.0)
    got = gpu_attention(case)
    g = hq // hkv
    for s in range(len(lens)):
        vals = attn_cases.logical_values(case, s)
        for h in range(hq):
            want = vals[targets[s][h], h // g]
            assert np.array_equal(got[s, h].view(np.uint16), want.view(np.uint16)), (s, h, targets[s][h])
    assert np.array_equal(got, attn_oracle.decode_attention(case.q, case.k_cache, case.v_cache,
                                                            case.block_table, case.seq_lens, case.scale))


@pytest.mark.parametrize("lens,page", [((64,), 16), ((1024, 256), 16), ((4096,), 16), ((16384,), 32),
                                       ((2, 4, 8, 128), 4)])
def test_attention_uniform_weights_bit_exact(lens, page):
    """q = 0 gives weights 1/L; with integer values and L a power of two the
    mean is exact in fp32 in any order, so the GPU output equals the oracle's
    bit for bit."""
    announce(f"attention uniform lens={lens} page={page}")
    case = attn_cases.integer_values_case(31, 24, 8, 128, page, lens)
    case = case._replace(q=np.zeros_like(case.q))
    got = gpu_attention(case)
    ref = attn_oracle.decode_attention(case.q, case.k_cache, case.v_cache, case.block_table, case.seq_lens,
                                       case.scale)
    assert np.array_equal(got.view(np.uint16), ref.view(np.uint16))


def test_attention_zero_scale_bit_exact():
    announce("attention scale=0")
    case = attn_cases.integer_values_case(32, 32, 8, 128, 16, (512, 2048))
    case = case._replace(scale=0.0)
    got = gpu_attention(case)
    ref = attn_oracle.decode_attention(case.q, case.k_cache, case.v_cache, case.block_table, case.seq_lens, 0.0)
    assert np.array_equal(got.view(np.uint16), ref.view(np.uint16))


def test_attention_physical_layout_does_not_change_bits():
    """The same sequences stored in other physical pages give identical
    bits (the kernel's arithmetic depends only on logical positions)."""
    announce("attention page permutation")
    case = attn_cases.random_case(41, 24, 8, 128, 16, (1000, 4097, 31), extra_pages=20)
    moved = attn_cases.shuffle_physical_pages(case, seed=42)
    a = gpu_attention(case)
    b = gpu_attention(moved)
    assert np.array_equal(a.view(np.uint16), b.view(np.uint16))
    check_tolerance(case, a, "page permutation")


def test_attention_repeatable_and_max_len_independent():
    """Repeated calls give the same bits; a looser max_seq_len changes the
    launch (more chunk slots) but not a value when the chunk length stays."""
    announce("attention repeat")
    case = attn_cases.random_case(51, 32, 8, 128, 16, (3000, 500), extra_pages=3)
    a = gpu_attention(case)
    b = gpu_attention(case)
    assert np.array_equal(a.view(np.uint16), b.view(np.uint16))
    c = gpu_attention(case, max_seq_len=3500)
    assert np.array_equal(a.view(np.uint16), c.view(np.uint16))


def test_attention_empty_sequences_are_zero():
    announce("attention empty sequences")
    case = attn_cases.random_case(61, 24, 8, 128, 16, (0, 37, 0), extra_pages=2)
    for max_len in (37, 4096):
        got = gpu_attention(case, max_seq_len=max_len)
        assert np.all(got[0] == 0) and np.all(got[2] == 0)
        check_tolerance(case, got, "empty")
    only_empty = attn_cases.select_sequences(case, [0])
    assert np.all(gpu_attention(only_empty, max_seq_len=0) == 0)


@pytest.mark.parametrize("max_len", [100, 5000])
def test_attention_invalid_tables_give_nan(max_len):
    """A used block-table entry outside the cache, a length above
    max_seq_len and a negative length make that sequence's output NaN; the
    other sequences are unchanged."""
    announce(f"attention invalid inputs max_len={max_len}")
    case = attn_cases.random_case(71, 24, 8, 128, 16, (90, 60, 80, 70), extra_pages=2, max_pages=400)
    clean = gpu_attention(case, max_seq_len=max_len)
    table = case.block_table.copy()
    table[0, 3] = case.k_cache.shape[0]          # one past the last page
    table[2, 0] = -5
    lens = case.seq_lens.copy()
    lens[1] = max_len + 1                        # above max_seq_len
    lens[3] = -1
    bad = case._replace(block_table=table, seq_lens=lens)
    got = gpu_attention(bad, max_seq_len=max_len)
    for s in range(4):
        assert np.all(np.isnan(got[s].astype(np.float32))), s
    # a bad entry past the used pages is never read
    table2 = case.block_table.copy()
    table2[0, 6:] = 1 << 30
    ok = gpu_attention(case._replace(block_table=table2), max_seq_len=max_len)
    assert np.array_equal(ok.view(np.uint16), clean.view(np.uint16))


@pytest.mark.parametrize("hq,lens", [(24, (4096,)), (32, (3000, 7, 5000, 64)), (24, (2048,) * 16)])
def test_attention_xcd_placement_bit_identical(hq, lens, monkeypatch):
    """Placing every chunk of a (sequence, kv head) pair on one XCD only
    moves work between workgroups: each chunk still covers the same tokens
    and the merge folds the chunks in the same order, so the outputs are
    the same bits with the placement on and off (8 kv heads: the pairs
    divide evenly over the XCDs, and the sequences are split)."""
    announce(f"attention XCD placement hq={hq} lens={lens[:4]}")
    case = attn_cases.random_case(120 + hq + len(lens), hq, 8, 128, 16, lens, extra_pages=3)
    monkeypatch.setenv("WQ_ATTN_XCD_LOCAL", "1")
    on = gpu_attention(case)
    monkeypatch.setenv("WQ_ATTN_XCD_LOCAL", "0")
    off = gpu_attention(case)
    assert np.array_equal(on.view(np.uint16), off.view(np.uint16))
    check_tolerance(case, on, "XCD placement")


def test_attention_shared_workspace_across_shapes():
    """One workspace serves consecutive calls of different shapes."""
    import torch

    from paper_2412_15803_amd import wq

    announce("attention shared workspace")
    big = wq.paged_attention_workspace_size(4, 32, 8, 128, 8192)
    ws = torch.empty(big, dtype=torch.uint8, device="cuda:0")
    for seed, (hq, lens) in enumerate([(32, (8192, 100, 5, 4000)), (24, (2000,)), (32, (7, 7000))]):
        case = attn_cases.random_case(80 + seed, hq, 8, 128, 16, lens, extra_pages=1)
        got = gpu_attention(case, max_seq_len=8192, workspace=ws)
        check_tolerance(case, got, f"shared workspace {seed}")


@pytest.mark.parametrize("name,hq,ctx", [("3b_ctx4096", 24, 4096), ("3b_ctx32768", 24, 32768),
                                         ("8b_ctx32768", 32, 32768)])
def test_attention_decode_shapes_full(name, hq, ctx):
    """The benchmarked decode-attention shapes (one sequence, 8 kv heads,
    pages of 16), every output element against the oracle."""
    announce(f"attention full shape {name}")
    case = attn_cases.random_case(90 + hq, hq, 8, 128, 16, (ctx,), extra_pages=64)
    got = gpu_attention(case)
    check_tolerance(case, got, name)


def test_attention_batch_of_sequences_full():
    """A decode batch of 16 sequences of mixed lengths (the multi-sequence
    launch configuration), every element against the oracle."""
    announce("attention batch of 16")
    rng = np.random.default_rng(5)
    lens = tuple(int(x) for x in rng.integers(1, 4096, size=16))
    case = attn_cases.random_case(95, 32, 8, 128, 16, lens, extra_pages=10)
    got = gpu_attention(case, max_seq_len=4096)
    check_tolerance(case, got, "batch 16")
