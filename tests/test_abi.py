"""The C-ABI library on the CPU: it loads, exports every function declared in
include/wq.h, and rejects invalid arguments on the host before any HIP call
(no GPU needed: these calls never reach the device)."""

import ctypes
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wq.h")


@pytest.fixture(scope="module")
def L():
    from paper_2412_15803_amd import wq

    if not os.path.exists(wq.LIB_PATH):
        from paper_2412_15803_amd import build

        build.build(verbose=False)
    return wq.lib()


def declared_functions():
    src = open(HEADER).read()
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


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="only meaningful on a host without a GPU")
def test_valid_call_without_device_reports_hip_error():
    # In a child process, so nothing here touches a GPU runtime.
    code = (
        "import ctypes; from paper_2412_15803_amd import wq; L = wq.lib();"
        "st = L.wq_gemv(ctypes.c_void_p(0x100000), ctypes.c_void_p(0x200000), ctypes.c_void_p(0x300000),"
        " ctypes.c_void_p(0x400000), 64, 64, 1, 32, None);"
        "print(st, L.wq_last_error_message().decode())"
    )
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    assert out.stdout.split()[0] == "4"
    assert "HIP error" in out.stdout


def test_binding_refuses_host_tensors():
    import torch

    from paper_2412_15803_amd import wq

    w = torch.zeros(4, 32)
    with pytest.raises(ValueError, match="device tensor"):
        wq.wq_pack(w, torch.zeros(4, 4, dtype=torch.int32), torch.zeros(4, 1, dtype=torch.float16))
