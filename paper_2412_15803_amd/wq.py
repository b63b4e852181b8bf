"""Thin ctypes binding of the C ABI in include/wq.h, include/wq_attention.h,
include/wq_fused.h and include/wq_probe.h.

Only argument marshalling happens here: torch tensors are turned into device
pointers and sizes, the current HIP stream is passed through, and non-OK
status codes become WQError.  Every step of the computation runs in the HIP
library; if the library is not built this module raises instead of falling
back to anything else.
"""

from __future__ import annotations

import ctypes
import os

# The in-tree build.  WQ_LIBRARY names another build of the same library to
# load instead (the host-sanitizer test loads one built with AddressSanitizer
# on its host code).
LIB_PATH = os.environ.get("WQ_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib", "libwq.so")

WQ_OK = 0
WQ_ERR_INVALID_ARG = 1
WQ_ERR_UNSUPPORTED = 2
WQ_ERR_MISALIGNED = 3
WQ_ERR_HIP = 4

GROUP = 32

# Every function declared in the headers under include/.
EXPORTED = ("wq_status_string", "wq_last_error_message", "wq_version", "wq_pack", "wq_gemv",
            "wq_decode_linears", "wq_decode_linears_noalloc", "wq_paged_attention_workspace_size",
            "wq_paged_attention", "wq_fused_linears", "wq_fused_check", "wq_stream_read")

# Limits of wq_decode_linears_noalloc (include/wq.h).
NOALLOC_MAX_LINEARS = 1024
NOALLOC_SCRATCH_BYTES = 131072

PROLOGUE_NONE = 0
PROLOGUE_RMSNORM = 1
PROLOGUE_SILU_MUL = 2


class WqLinear(ctypes.Structure):
    _fields_ = [
        ("packed_w", ctypes.c_void_p),
        ("scales", ctypes.c_void_p),
        ("x", ctypes.c_void_p),
        ("y", ctypes.c_void_p),
        ("N", ctypes.c_int64),
        ("K", ctypes.c_int64),
    ]


class WqFusedLinear(ctypes.Structure):
    _fields_ = [
        ("packed_w", ctypes.c_void_p),
        ("scales", ctypes.c_void_p),
        ("x", ctypes.c_void_p),
        ("y", ctypes.c_void_p),
        ("norm_weight", ctypes.c_void_p),
        ("residual", ctypes.c_void_p),
        ("N", ctypes.c_int64),
        ("K", ctypes.c_int64),
        ("prologue", ctypes.c_int32),
        ("eps", ctypes.c_float),
    ]


class WQError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """Load libwq.so (once) and declare the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"HIP library not built: {LIB_PATH} is missing "
                           "(run `python -m paper_2412_15803_amd.build`)")
    L = ctypes.CDLL(LIB_PATH)
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    L.wq_status_string.argtypes = [ctypes.c_int]
    L.wq_status_string.restype = ctypes.c_char_p
    L.wq_last_error_message.argtypes = []
    L.wq_last_error_message.restype = ctypes.c_char_p
    L.wq_version.argtypes = []
    L.wq_version.restype = ctypes.c_int
    L.wq_pack.argtypes = [vp, vp, vp, i64, i64, i64, vp]
    L.wq_pack.restype = ctypes.c_int
    L.wq_gemv.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, vp]
    L.wq_gemv.restype = ctypes.c_int
    L.wq_decode_linears.argtypes = [ctypes.POINTER(WqLinear), i64, i64, i64, vp]
    L.wq_decode_linears.restype = ctypes.c_int
    L.wq_decode_linears_noalloc.argtypes = [ctypes.POINTER(WqLinear), i64, i64, i64, vp]
    L.wq_decode_linears_noalloc.restype = ctypes.c_int
    L.wq_paged_attention_workspace_size.argtypes = [i64, i64, i64, i64, i64, ctypes.POINTER(ctypes.c_size_t)]
    L.wq_paged_attention_workspace_size.restype = ctypes.c_int
    L.wq_paged_attention.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i64, i64,
                                     ctypes.c_float, vp, ctypes.c_size_t, vp]
    L.wq_paged_attention.restype = ctypes.c_int
    L.wq_fused_linears.argtypes = [ctypes.POINTER(WqFusedLinear), i64, vp, i64, vp]
    L.wq_fused_linears.restype = ctypes.c_int
    L.wq_fused_check.argtypes = [vp]
    L.wq_fused_check.restype = ctypes.c_int
    L.wq_stream_read.argtypes = [vp, i64, vp, vp]
    L.wq_stream_read.restype = ctypes.c_int
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().wq_status_string(int(status)).decode()


def last_error_message() -> str:
    return lib().wq_last_error_message().decode()


def _check(status: int) -> None:
    if status != WQ_OK:
        raise WQError(status, last_error_message())


# ------------------------------------------------------------- marshalling

def _dev_tensor(t, name, dtypes, shape):
    import torch

    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor (got {t.device})")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous (row-major)")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream, device):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream)


def _word_dtypes():
    import torch

    return (torch.int32, torch.uint32)


def _half_dtypes():
    import torch

    return (torch.float16, torch.int16, torch.uint16)


def wq_pack(w, packed_w, scales, group: int = GROUP, stream=None) -> None:
    """Quantize fp32 w [N, K] into packed_w [N, K/8] (int32/uint32 words) and
    scales [N, K/32] (fp16), both preallocated on the same device."""
    import torch

    if w.dim() != 2:
        raise ValueError("w must be 2-D [N, K]")
    n, k = w.shape
    pw = _dev_tensor(w, "w", (torch.float32,), (n, k))
    pp = _dev_tensor(packed_w, "packed_w", _word_dtypes(), (n, k // 8))
    ps = _dev_tensor(scales, "scales", _half_dtypes(), (n, k // group if group else 0))
    _check(lib().wq_pack(pw, pp, ps, n, k, group, _stream(stream, w.device)))


def wq_gemv(packed_w, scales, x, y, group: int = GROUP, stream=None) -> None:
    """y [M, N] = x [M, K] . dequant(packed_w, scales)^T (fp16 in, fp16 out)."""
    if x.dim() != 2 or packed_w.dim() != 2:
        raise ValueError("x must be [M, K] and packed_w [N, K/8]")
    m, k = x.shape
    n = packed_w.shape[0]
    pp = _dev_tensor(packed_w, "packed_w", _word_dtypes(), (n, k // 8))
    ps = _dev_tensor(scales, "scales", _half_dtypes(), (n, k // group if group else 0))
    px = _dev_tensor(x, "x", _half_dtypes(), (m, k))
    py = _dev_tensor(y, "y", _half_dtypes(), (m, n))
    _check(lib().wq_gemv(pp, ps, px, py, n, k, m, group, _stream(stream, x.device)))


def make_linear_array(linears, m: int, group: int = GROUP):
    """Marshal a sequence of (packed_w, scales, x, y) tensor tuples into a
    ctypes wq_linear array."""
    arr = (WqLinear * len(linears))()
    for i, (packed_w, scales, x, y) in enumerate(linears):
        if x.dim() != 2 or x.shape[0] != m:
            raise ValueError(f"linear {i}: x must be [M={m}, K]")
        k = x.shape[1]
        n = packed_w.shape[0]
        arr[i].packed_w = _dev_tensor(packed_w, f"linears[{i}].packed_w", _word_dtypes(), (n, k // 8)).value
        arr[i].scales = _dev_tensor(scales, f"linears[{i}].scales", _half_dtypes(), (n, k // group if group else 0)).value
        arr[i].x = _dev_tensor(x, f"linears[{i}].x", _half_dtypes(), (m, k)).value
        arr[i].y = _dev_tensor(y, f"linears[{i}].y", _half_dtypes(), (m, n)).value
        arr[i].N = n
        arr[i].K = k
    return arr


def wq_decode_linears(linears, m: int = 1, group: int = GROUP, stream=None, _array=None) -> None:
    """Run a decode step's linears in order on one stream.  `linears` is a
    sequence of (packed_w, scales, x, y) tuples; a prebuilt array from
    make_linear_array may be passed as _array to skip re-marshalling."""
    arr = _array if _array is not None else make_linear_array(linears, m, group)
    device = linears[0][2].device
    _check(lib().wq_decode_linears(arr, len(arr), m, group, _stream(stream, device)))


def wq_decode_linears_noalloc(linears, m: int = 1, group: int = GROUP, stream=None, _array=None) -> None:
    """wq_decode_linears through the entry point that allocates nothing (its
    plan lives in the library's fixed per-device array; see include/wq.h)."""
    arr = _array if _array is not None else make_linear_array(linears, m, group)
    device = linears[0][2].device
    _check(lib().wq_decode_linears_noalloc(arr, len(arr), m, group, _stream(stream, device)))


# ------------------------------------------------------- paged attention

def paged_attention_workspace_size(num_seqs: int, num_q_heads: int, num_kv_heads: int,
                                   head_dim: int, max_seq_len: int) -> int:
    """Bytes of device workspace wq_paged_attention needs (0: none)."""
    out = ctypes.c_size_t(0)
    _check(lib().wq_paged_attention_workspace_size(num_seqs, num_q_heads, num_kv_heads, head_dim,
                                                   max_seq_len, ctypes.byref(out)))
    return int(out.value)


def paged_workspace(q, max_seq_len: int, num_kv_heads: int):
    """A device workspace (uint8 tensor, or None) sized for these shapes."""
    import torch

    num_seqs, hq, d = q.shape
    n = paged_attention_workspace_size(num_seqs, hq, num_kv_heads, d, max_seq_len)
    return torch.empty(n, dtype=torch.uint8, device=q.device) if n else None


def paged_attention(q, k_cache, v_cache, block_table, seq_lens, out, scale: float, max_seq_len: int,
                    workspace=None, stream=None) -> None:
    """out [S, HQ, D] = decode attention of q [S, HQ, D] over the paged
    caches [pages, HKV, P, D] (fp16), block_table [S, max_pages] and
    seq_lens [S] (int32), all on one device.  `workspace` is a uint8 device
    tensor from paged_workspace (allocated here when omitted)."""
    import torch

    if q.dim() != 3 or k_cache.dim() != 4:
        raise ValueError("q must be [S, HQ, D] and the caches [pages, HKV, P, D]")
    num_seqs, hq, d = q.shape
    num_pages, hkv, page, d2 = k_cache.shape
    max_pages = block_table.shape[1] if block_table.dim() == 2 else 0
    pq = _dev_tensor(q, "q", _half_dtypes(), (num_seqs, hq, d))
    pk = _dev_tensor(k_cache, "k_cache", _half_dtypes(), (num_pages, hkv, page, d2))
    pv = _dev_tensor(v_cache, "v_cache", _half_dtypes(), (num_pages, hkv, page, d2))
    pt = _dev_tensor(block_table, "block_table", (torch.int32,), (num_seqs, max_pages))
    pl = _dev_tensor(seq_lens, "seq_lens", (torch.int32,), (num_seqs,))
    po = _dev_tensor(out, "out", _half_dtypes(), (num_seqs, hq, d))
    if workspace is None:
        workspace = paged_workspace(q, max_seq_len, hkv)
    if workspace is not None:
        if workspace.device != q.device or workspace.dtype != torch.uint8 or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous uint8 tensor on the device of q")
        pw, nw = ctypes.c_void_p(workspace.data_ptr()), workspace.numel()
    else:
        pw, nw = None, 0
    _check(lib().wq_paged_attention(pq, pk, pv, pt, pl, po, num_seqs, hq, hkv, d, page, num_pages,
                                    max_pages, max_seq_len, float(scale), pw, nw,
                                    _stream(stream, q.device)))


# ------------------------------------------------------- fused decode chain

def make_fused_array(linears, group: int = GROUP):
    """Marshal dicts with keys packed_w, scales, x, y (tensors) and optional
    prologue (PROLOGUE_*), norm_weight, eps, residual into a ctypes
    wq_fused_linear array.  x is [K] ([2K] for PROLOGUE_SILU_MUL), y and
    residual [N], norm_weight [K]; 1-D or [1, n] tensors are accepted."""
    arr = (WqFusedLinear * len(linears))()
    for i, d in enumerate(linears):
        packed_w, scales, x, y = d["packed_w"], d["scales"], d["x"], d["y"]
        pro = int(d.get("prologue", PROLOGUE_NONE))
        n = packed_w.shape[0]
        k = packed_w.shape[1] * 8
        xk = 2 * k if pro == PROLOGUE_SILU_MUL else k
        arr[i].packed_w = _dev_tensor(packed_w, f"linears[{i}].packed_w", _word_dtypes(), (n, k // 8)).value
        arr[i].scales = _dev_tensor(scales, f"linears[{i}].scales", _half_dtypes(), (n, k // group)).value
        arr[i].x = _dev_tensor(x.reshape(-1), f"linears[{i}].x", _half_dtypes(), (xk,)).value
        arr[i].y = _dev_tensor(y.reshape(-1), f"linears[{i}].y", _half_dtypes(), (n,)).value
        norm = d.get("norm_weight")
        arr[i].norm_weight = _dev_tensor(norm, f"linears[{i}].norm_weight", _half_dtypes(), (k,)).value \
            if norm is not None else None
        res = d.get("residual")
        arr[i].residual = _dev_tensor(res.reshape(-1), f"linears[{i}].residual", _half_dtypes(), (n,)).value \
            if res is not None else None
        arr[i].N = n
        arr[i].K = k
        arr[i].prologue = pro
        arr[i].eps = float(d.get("eps", 0.0))
    return arr


def wq_fused_linears(linears, argmax=None, group: int = GROUP, stream=None, _array=None) -> None:
    """Run a chain of fused linears in order (see make_fused_array); when
    `argmax` (a device int32 tensor of one element) is given, the index of
    the largest element of the last linear's y is written to it."""
    import torch

    arr = _array if _array is not None else make_fused_array(linears, group)
    device = linears[0]["x"].device
    pa = _dev_tensor(argmax.reshape(-1), "argmax", (torch.int32,), (1,)) if argmax is not None else None
    _check(lib().wq_fused_linears(arr, len(arr), pa, group, _stream(stream, device)))


def wq_fused_check(device=None, stream=None) -> None:
    """Synchronize the stream and raise WQError if a persistent chain on the
    device gave up since the last check (a bounded wait ran out)."""
    import torch

    device = torch.device("cuda", torch.cuda.current_device()) if device is None else device
    _check(lib().wq_fused_check(_stream(stream, device)))


# ------------------------------------------------------- measurement probe

def stream_read(buf, sink, stream=None) -> None:
    """Read the whole device tensor `buf` once (wq_stream_read); `sink` is a
    device int32/uint32 tensor of at least 1024 elements."""
    import torch

    if buf.device.type != "cuda" or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous device tensor")
    nbytes = buf.numel() * buf.element_size()
    if sink.device != buf.device or sink.dtype not in (torch.int32, torch.uint32) or sink.numel() < 1024:
        raise ValueError("sink must be a device int32 tensor of at least 1024 elements")
    _check(lib().wq_stream_read(ctypes.c_void_p(buf.data_ptr()), nbytes, ctypes.c_void_p(sink.data_ptr()),
                                _stream(stream, buf.device)))
