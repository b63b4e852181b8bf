"""The C-ABI library on the CPU: it loads, exports every function declared in
the headers under include/, and rejects invalid arguments on the host before any HIP call
(no GPU needed: these calls never reach the device)."""

import ctypes
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))
                 if f.endswith(".h"))


@pytest.fixture(scope="module")
def L():
    from paper_2412_15803_amd import wq

    if not os.path.exists(wq.LIB_PATH):
        from paper_2412_15803_amd import build

        build.build(verbose=False)
    return wq.lib()


def declared_functions():
    src = "".join(open(h).read() for h in HEADERS)
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(wq_[a-z_]+)\s*\(", src)))


def test_header_declares_expected_entry_points():
    from paper_2412_15803_amd import wq

    assert declared_functions() == sorted(wq.EXPORTED)


def test_every_declared_symbol_is_exported(L):
    from paper_2412_15803_amd import wq

    out = subprocess.run(["nm", "-D", "--defined-only", wq.LIB_PATH], capture_output=True, text=True, check=True).stdout
    dyn = set(line.split()[-1] for line in out.splitlines() if line.strip())
    for name in declared_functions():
        assert name in dyn, name
        assert hasattr(L, name)


def test_status_strings(L):
    names = {0: b"WQ_OK", 1: b"WQ_ERR_INVALID_ARG", 2: b"WQ_ERR_UNSUPPORTED", 3: b"WQ_ERR_MISALIGNED", 4: b"WQ_ERR_HIP"}
    for code, name in names.items():
        assert L.wq_status_string(code) == name
    for code in (-1, 5, 1000):
        assert L.wq_status_string(code) == b"WQ_UNKNOWN_STATUS"
    assert L.wq_version() == 100


# Fake, well-aligned, non-overlapping "device" addresses: validation fails
# before anything would dereference them.
P, S, X, Y, W = 0x100000, 0x200000, 0x300000, 0x400000, 0x500000
vp = ctypes.c_void_p


def gemv(L, p=P, s=S, x=X, y=Y, n=64, k=64, m=1, g=32):
    return L.wq_gemv(vp(p), vp(s), vp(x), vp(y), n, k, m, g, None)


@pytest.mark.parametrize(
    "kwargs,status,needle",
    [
        (dict(p=0), 1, "null"),
        (dict(s=0), 1, "null"),
        (dict(x=0), 1, "null"),
        (dict(y=0), 1, "null"),
        (dict(n=0), 1, "positive"),
        (dict(n=-5), 1, "positive"),
        (dict(k=0), 1, "positive"),
        (dict(m=0), 1, "M must be"),
        (dict(m=65536), 1, "M must be"),
        (dict(g=64), 2, "group"),
        (dict(g=0), 2, "group"),
        (dict(k=48), 2, "multiple of 32"),
        (dict(n=2**31), 1, "too large"),
        (dict(p=P + 8), 3, "packed_w"),
        (dict(x=X + 4), 3, "x must be"),
        (dict(s=S + 1), 3, "scales"),
        (dict(y=Y + 1), 3, "y must be"),
        (dict(y=X + 64), 1, "overlaps"),
        (dict(y=P + 16), 1, "overlaps"),
        (dict(y=S + 2), 1, "overlaps"),
    ],
)
def test_gemv_rejects(L, kwargs, status, needle):
    st = gemv(L, **kwargs)
    assert st == status
    assert needle in L.wq_last_error_message().decode()


def pack(L, w=W, p=P, s=S, n=64, k=64, g=32):
    return L.wq_pack(vp(w), vp(p), vp(s), n, k, g, None)


@pytest.mark.parametrize(
    "kwargs,status",
    [
        (dict(w=0), 1), (dict(p=0), 1), (dict(s=0), 1),
        (dict(n=0), 1), (dict(k=-32), 1), (dict(g=16), 2), (dict(k=40), 2),
        (dict(w=W + 4), 3), (dict(p=P + 4), 3), (dict(s=S + 1), 3),
        (dict(p=W + 256), 1), (dict(s=W), 1), (dict(s=P + 16), 1),
        (dict(n=2**40, k=2**20), 1),
    ],
)
def test_pack_rejects(L, kwargs, status):
    assert pack(L, **kwargs) == status


def _linears(n_lin, override=None):
    from paper_2412_15803_amd.wq import WqLinear

    arr = (WqLinear * n_lin)()
    for i in range(n_lin):
        base = 0x10000000 * (i + 1)
        arr[i].packed_w, arr[i].scales, arr[i].x, arr[i].y = base, base + 0x1000000, base + 0x2000000, base + 0x3000000
        arr[i].N, arr[i].K = 64, 64
    for (i, field), val in (override or {}).items():
        setattr(arr[i], field, val)
    return arr


def test_decode_linears_rejects(L):
    from paper_2412_15803_amd.wq import WqLinear

    arr = _linears(3)
    assert L.wq_decode_linears(None, 3, 1, 32, None) == 1
    assert L.wq_decode_linears(arr, 0, 1, 32, None) == 1
    assert L.wq_decode_linears(arr, 65537, 1, 32, None) == 1
    assert L.wq_decode_linears(arr, 3, 0, 32, None) == 1
    assert L.wq_decode_linears(arr, 3, 1, 64, None) == 2
    bad = _linears(3, {(2, "K"): 40})
    assert L.wq_decode_linears(bad, 3, 1, 32, None) == 2
    assert "linear 2" in L.wq_last_error_message().decode()
    bad = _linears(3, {(1, "x"): 0x20000000 + 0x2000000 + 2})
    assert L.wq_decode_linears(bad, 3, 1, 32, None) == 3
    assert "linear 1" in L.wq_last_error_message().decode()
    # y of linear 0 lands on the scales of linear 2
    bad = _linears(3, {(0, "y"): 0x30000000 + 0x1000000 + 64})
    assert L.wq_decode_linears(bad, 3, 1, 32, None) == 1
    assert "overlaps" in L.wq_last_error_message().decode()
    # y of linear 1 is allowed to be the x of linear 2 (a dependency chain)
    ok = _linears(3, {(1, "y"): 0x30000000 + 0x2000000})
    assert isinstance(ok[0], WqLinear)
    # ...which passes validation, so the (GPU-less) call only fails at HIP time
    # or, on a GPU host, is never attempted here.


def test_decode_linears_noalloc_rejects(L):
    arr = _linears(3)
    assert L.wq_decode_linears_noalloc(None, 3, 1, 32, None) == 1
    assert L.wq_decode_linears_noalloc(arr, 0, 1, 32, None) == 1
    assert L.wq_decode_linears_noalloc(_linears(1025), 1025, 1, 32, None) == 1
    assert "WQ_NOALLOC_MAX_LINEARS" in L.wq_last_error_message().decode()
    assert L.wq_decode_linears_noalloc(arr, 3, 1, 64, None) == 2
    assert L.wq_decode_linears_noalloc(arr, 3, 0, 32, None) == 1
    bad = _linears(3, {(1, "x"): 0x20000000 + 0x2000000 + 8})
    assert L.wq_decode_linears_noalloc(bad, 3, 1, 32, None) == 3
    assert "linear 1" in L.wq_last_error_message().decode()
    clash = _linears(3, {(2, "y"): 0x10000000 + 64})
    assert L.wq_decode_linears_noalloc(clash, 3, 1, 32, None) == 1
    assert "overlaps packed_w or scales" in L.wq_last_error_message().decode()


def test_stream_read_rejects(L):
    assert L.wq_stream_read(None, 1 << 20, vp(S), None) == 1
    assert L.wq_stream_read(vp(P), 1 << 20, None, None) == 1
    assert L.wq_stream_read(vp(P), 0, vp(S), None) == 1
    assert L.wq_stream_read(vp(P), 1000, vp(S), None) == 1
    assert L.wq_stream_read(vp(P + 8), 1 << 20, vp(S), None) == 3
    assert L.wq_stream_read(vp(P), 1 << 20, vp(S + 2), None) == 3


def _no_device_visible():
    """True only where no GPU can be reached: no KFD device node and no
    render node.  The test below hands the library fake device addresses,
    which on a GPU host would be dereferenced, so it must never run there."""
    if os.path.exists("/dev/kfd"):
        return False
    dri = "/dev/dri"
    return not (os.path.isdir(dri) and any(n.startswith("renderD") for n in os.listdir(dri)))


@pytest.mark.skipif(not _no_device_visible(), reason="only safe and meaningful on a host without a GPU")
def test_valid_calls_without_device_report_hip_error():
    """Valid arguments reach the HIP runtime, which has no device here: every
    entry point returns WQ_ERR_HIP with the runtime's message (in a child
    process, so nothing in this one touches a GPU runtime)."""
    code = """
import ctypes
from paper_2412_15803_amd import wq
from test_abi import _linears, _fused, attention
L = wq.lib()
vp = ctypes.c_void_p
res = {
    "gemv": L.wq_gemv(vp(0x100000), vp(0x200000), vp(0x300000), vp(0x400000), 64, 64, 1, 32, None),
    "gemv_m4": L.wq_gemv(vp(0x100000), vp(0x200000), vp(0x300000), vp(0x400000), 64, 64, 4, 32, None),
    "pack": L.wq_pack(vp(0x500000), vp(0x100000), vp(0x200000), 64, 64, 32, None),
    "decode": L.wq_decode_linears(_linears(3), 3, 1, 32, None),
    "decode_m8": L.wq_decode_linears(_linears(3), 3, 8, 32, None),
    "decode_noalloc": L.wq_decode_linears_noalloc(_linears(3), 3, 1, 32, None),
    "decode_noalloc_m4": L.wq_decode_linears_noalloc(_linears(3), 3, 4, 32, None),
    "fused": L.wq_fused_linears(_fused(2), 2, None, 32, None),
    "attention": attention(L),
    "stream_read": L.wq_stream_read(vp(0x100000), 1 << 20, vp(0x200000), None),
    "fused_check": L.wq_fused_check(None),
}
for name, st in res.items():
    print(name, st, L.wq_last_error_message().decode() if st else "")
"""
    env = dict(os.environ, PYTHONPATH=os.pathsep.join([ROOT, os.path.join(ROOT, "tests")]))
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=120,
                         env=env)
    assert out.returncode == 0, out.stderr
    lines = out.stdout.strip().splitlines()
    assert len(lines) == 11, out.stdout
    for line in lines:
        name, st = line.split()[:2]
        assert st == "4", line


def test_binding_refuses_host_tensors():
    import torch

    from paper_2412_15803_amd import wq

    w = torch.zeros(4, 32)
    with pytest.raises(ValueError, match="device tensor"):
        wq.wq_pack(w, torch.zeros(4, 4, dtype=torch.int32), torch.zeros(4, 1, dtype=torch.float16))


# ------------------------------------------------------- paged attention

QA, KA, VA, TA, LA, OA, WA = (0x1000000 * i for i in range(1, 8))


def attention(L, q=QA, k=KA, v=VA, t=TA, lens=LA, o=OA, seqs=1, hq=24, hkv=8, d=128, page=16, pages=256,
              max_pages=256, max_len=4096, scale=0.088, ws=WA, ws_bytes=1 << 24):
    return L.wq_paged_attention(vp(q), vp(k), vp(v), vp(t), vp(lens), vp(o), seqs, hq, hkv, d, page, pages,
                                max_pages, max_len, scale, vp(ws), ws_bytes, None)


def workspace_bytes(L, seqs, hq, hkv, d, max_len):
    out = ctypes.c_size_t(12345)
    st = L.wq_paged_attention_workspace_size(seqs, hq, hkv, d, max_len, ctypes.byref(out))
    return st, out.value


@pytest.mark.parametrize(
    "kwargs,status,needle",
    [
        (dict(q=0), 1, "null"), (dict(k=0), 1, "null"), (dict(v=0), 1, "null"),
        (dict(t=0), 1, "null"), (dict(lens=0), 1, "null"), (dict(o=0), 1, "null"),
        (dict(seqs=0), 1, "num_seqs"), (dict(seqs=(1 << 20) + 1), 1, "num_seqs"),
        (dict(hkv=0), 1, "num_kv_heads"), (dict(hkv=257, hq=257), 1, "num_kv_heads"),
        (dict(hq=20), 1, "multiple"), (dict(hq=72), 2, "query heads per kv head"),
        (dict(d=64), 2, "head_dim"), (dict(page=12), 2, "page_size"), (dict(page=2048), 2, "page_size"),
        (dict(page=0), 2, "page_size"), (dict(pages=0), 1, "num_pages"), (dict(max_pages=0), 1, "max_pages"),
        (dict(max_len=-1), 1, "max_seq_len"), (dict(max_len=(1 << 22) + 1, max_pages=1 << 20), 1, "max_seq_len"),
        (dict(max_len=4097), 1, "exceeds"), (dict(scale=float("inf")), 1, "scale"),
        (dict(scale=float("nan")), 1, "scale"),
        (dict(q=QA + 8), 3, "16-byte"), (dict(o=OA + 2), 3, "16-byte"), (dict(k=KA + 4), 3, "16-byte"),
        (dict(v=VA + 8), 3, "16-byte"), (dict(t=TA + 2), 3, "4-byte"), (dict(lens=LA + 1), 3, "4-byte"),
        (dict(ws=0), 1, "workspace"), (dict(ws_bytes=1000), 1, "workspace"), (dict(ws=WA + 4), 3, "workspace"),
        (dict(o=QA + 64), 1, "out overlaps"), (dict(o=KA + 4096), 1, "out overlaps"),
        (dict(o=LA), 1, "out overlaps"), (dict(ws=TA), 1, "workspace overlaps"),
        (dict(o=WA + 256), 1, "out overlaps the workspace"),
    ],
)
def test_attention_rejects(L, kwargs, status, needle):
    st = attention(L, **kwargs)
    assert st == status, L.wq_last_error_message()
    assert needle in L.wq_last_error_message().decode()


def test_attention_workspace_size(L):
    # one sequence of 4096 tokens, 8 kv heads: 64 chunks of 64 tokens, so
    # per query head 64 x (128 floats + (m, l))
    assert workspace_bytes(L, 1, 24, 8, 128, 4096) == (0, 24 * 64 * (128 * 4 + 8))
    # a short sequence is not split: no workspace
    assert workspace_bytes(L, 1, 24, 8, 128, 64) == (0, 0)
    assert workspace_bytes(L, 1, 24, 8, 128, 0) == (0, 0)
    # more sequences: longer chunks keep the launch near 512 workgroups
    st, n = workspace_bytes(L, 16, 32, 8, 128, 4096)
    assert st == 0 and n == 16 * 32 * 4 * (128 * 4 + 8)
    # enough sequences to fill the chip: no split, no workspace
    assert workspace_bytes(L, 64, 32, 8, 128, 4096) == (0, 0)
    assert workspace_bytes(L, 1, 24, 8, 64, 4096)[0] == 2
    assert L.wq_paged_attention_workspace_size(1, 24, 8, 128, 4096, None) == 1
    # the call accepts exactly the reported size and no less
    n = workspace_bytes(L, 1, 24, 8, 128, 4096)[1]
    assert attention(L, ws_bytes=n - 1) == 1


# ------------------------------------------------------- fused linears

def _fused(n_lin, override=None):
    from paper_2412_15803_amd.wq import WqFusedLinear

    arr = (WqFusedLinear * n_lin)()
    for i in range(n_lin):
        base = 0x10000000 * (i + 1)
        arr[i].packed_w, arr[i].scales = base, base + 0x1000000
        arr[i].x, arr[i].y = base + 0x2000000, base + 0x3000000
        arr[i].norm_weight, arr[i].residual = base + 0x4000000, None
        arr[i].N, arr[i].K, arr[i].prologue, arr[i].eps = 64, 64, 1, 1e-5
    for (i, field), val in (override or {}).items():
        setattr(arr[i], field, val)
    return arr


@pytest.mark.parametrize(
    "override,status,needle",
    [
        ({(0, "x"): None}, 1, "null"),
        ({(1, "norm_weight"): None}, 1, "norm_weight"),
        ({(1, "prologue"): 3}, 1, "prologue"),
        ({(0, "eps"): -1.0}, 1, "eps"),
        ({(0, "eps"): float("inf")}, 1, "eps"),
        ({(0, "N"): 0}, 1, "positive"),
        ({(0, "K"): 48}, 2, "multiple of 32"),
        ({(0, "K"): 16416}, 2, "multiple of 32"),
        ({(0, "x"): 0x12000008}, 3, "16-byte"),
        ({(0, "norm_weight"): 0x14000002}, 3, "16-byte"),
        ({(0, "y"): 0x13000001}, 3, "2-byte"),
        ({(0, "residual"): 0x15000001}, 3, "2-byte"),
        ({(0, "y"): 0x12000000 + 64}, 1, "y overlaps x"),
        ({(0, "y"): 0x14000000 + 16}, 1, "norm_weight"),
        ({(0, "residual"): 0x13000000 + 2}, 1, "residual overlaps y"),
        ({(1, "y"): 0x10000000 + 64}, 1, "overlaps packed_w or scales"),
        # SILU_MUL reads 2K entries of x: y right after the first K overlaps
        ({(0, "prologue"): 2, (0, "y"): 0x12000000 + 128}, 1, "y overlaps x"),
    ],
)
def test_fused_rejects(L, override, status, needle):
    arr = _fused(2, override)
    st = L.wq_fused_linears(arr, 2, None, 32, None)
    assert st == status, L.wq_last_error_message()
    assert needle in L.wq_last_error_message().decode()


def test_fused_rejects_call_level(L):
    arr = _fused(2)
    assert L.wq_fused_linears(None, 2, None, 32, None) == 1
    assert L.wq_fused_linears(arr, 0, None, 32, None) == 1
    assert L.wq_fused_linears(arr, 2, None, 64, None) == 2
    assert L.wq_fused_linears(arr, 2, vp(0x30000002), 32, None) == 3
    # argmax inside an array of the chain (the second linear's y)
    assert L.wq_fused_linears(arr, 2, vp(0x20000000 + 0x3000000 + 8), 32, None) == 1
    assert "argmax overlaps" in L.wq_last_error_message().decode()
    # residual equal to y (an in-place add) is accepted by validation
    ok = _fused(1, {(0, "residual"): 0x13000000})
    assert ok[0].residual == ok[0].y
