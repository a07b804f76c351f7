"""ctypes binding for libxgemm (include/xgemm.h).

Argument marshalling only: every entry point forwards to the HIP library with
the same name, and all arithmetic runs in its kernels.  Torch tensors are used
for device memory and streams; ``gemm`` reads their pointers, strides and the
current stream and calls ``xgemm_run``.  There is no fallback path: if
``libxgemm.so`` is missing the import of this module fails.
"""
from __future__ import annotations

import ctypes
import os
import re

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "libxgemm.so")
_HEADER = os.path.join(os.path.dirname(_PKG), "include", "xgemm.h")

XGEMM_BF16 = 0
XGEMM_FP16 = 1

XGEMM_OK = 0
XGEMM_ERR_INVALID_ARG = 1
XGEMM_ERR_UNSUPPORTED = 2
XGEMM_ERR_ALLOC = 3
XGEMM_ERR_HIP = 4

XGEMM_TILE_256x256 = 0
XGEMM_TILE_256x128 = 1
XGEMM_TILE_128x128 = 2
XGEMM_TILE_COUNT = 3

XGEMM_KERNEL_GENERAL = 0
XGEMM_KERNEL_PIPELINED = 1
XGEMM_KERNEL_PERSISTENT = 2


class xgemm_config(ctypes.Structure):
    _fields_ = [("tile", ctypes.c_int32), ("split_k", ctypes.c_int32),
                ("group_m", ctypes.c_int32), ("stream_k", ctypes.c_int32)]

    def __repr__(self):
        return "xgemm_config(tile=%d, split_k=%d, group_m=%d, stream_k=%d)" % (
            self.tile, self.split_k, self.group_m, self.stream_k)


XGEMM_BAND_NONE = 0
XGEMM_BAND_COLUMNS = 1
XGEMM_BAND_ROWS = 2


class xgemm_band(ctypes.Structure):
    _fields_ = [("axis", ctypes.c_int32), ("reserved", ctypes.c_int32), ("extent", ctypes.c_int64),
                ("body", xgemm_config), ("band", xgemm_config)]

    def __repr__(self):
        return "xgemm_band(axis=%d, extent=%d, body=%r, band=%r)" % (self.axis, self.extent, self.body, self.band)


XGEMM_TRACE_LDS_LOAD = 0
XGEMM_TRACE_LDS_READ = 1
XGEMM_TRACE_WAIT_VM = 2
XGEMM_TRACE_WAIT_LGKM = 3
XGEMM_TRACE_BARRIER = 4
XGEMM_TRACE_STORE = 5
XGEMM_TRACE_LDS_WRITE = 6
XGEMM_TRACE_LOAD = 7


class xgemv_config(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int32), ("unroll", ctypes.c_int32), ("split_k", ctypes.c_int32)]

    def __init__(self, rows=2, unroll=4, split_k=1):
        super().__init__(rows, unroll, split_k)

    def __repr__(self):
        return "xgemv_config(rows=%d, unroll=%d, split_k=%d)" % (self.rows, self.unroll, self.split_k)


class xgemm_trace_event(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("arg", ctypes.c_int32), ("lds", ctypes.c_int64),
                ("addr", ctypes.c_int64)]


class xgemm_trace_info(ctypes.Structure):
    _fields_ = [("segments", ctypes.c_int32), ("family", ctypes.c_int32), ("reduce", ctypes.c_int32),
                ("threads", ctypes.c_int32), ("lds_bytes", ctypes.c_int32), ("split", ctypes.c_int32),
                ("grid", ctypes.c_int64), ("workspace_bytes", ctypes.c_int64),
                ("tile_base", ctypes.c_int32), ("tile_count", ctypes.c_int32),
                ("packed", ctypes.c_int32), ("k", ctypes.c_int32), ("lda", ctypes.c_int64), ("ldb", ctypes.c_int64),
                ("a_offset", ctypes.c_int64), ("b_offset", ctypes.c_int64), ("data_offset", ctypes.c_int64),
                ("dp_rounds", ctypes.c_int32), ("sk_tiles", ctypes.c_int32), ("kt", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class XgemmError(RuntimeError):
    def __init__(self, status: int, detail: str = ""):
        self.status = status
        msg = "xgemm error %d (%s)" % (status, xgemm_strerror(status))
        if detail:
            msg += ": " + detail
        super().__init__(msg)


# torch ships its own HIP runtime with the same soname as the system one.  It
# must be loaded first so that libxgemm.so binds to it: one runtime per
# process, so that torch's device memory and streams are valid here.
import torch  # noqa: E402,F401

if not os.path.exists(_LIB_PATH):
    raise ImportError("libxgemm.so is not built (%s); run __graft_entry__.build() or "
                      "python -m paper_2609_16389_amd.build" % _LIB_PATH)

lib = ctypes.CDLL(_LIB_PATH)

_i64, _i32, _p = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
_handle_t = ctypes.c_void_p

lib.xgemm_create.argtypes = [ctypes.POINTER(_handle_t)]
lib.xgemm_create.restype = _i32
lib.xgemm_destroy.argtypes = [_handle_t]
lib.xgemm_destroy.restype = _i32
lib.xgemm_set_workspace_limit.argtypes = [_handle_t, ctypes.c_size_t]
lib.xgemm_set_workspace_limit.restype = _i32
lib.xgemm_set_persistent.argtypes = [_handle_t, _i32]
lib.xgemm_set_persistent.restype = _i32
lib.xgemm_run.argtypes = [_handle_t, _i64, _i64, _i64, _p, _i64, _p, _i64, _p, _i64, _i32, _p]
lib.xgemm_run.restype = _i32
lib.xgemm_run_noalloc.argtypes = [_handle_t, _i64, _i64, _i64, _p, _i64, _p, _i64, _p, _i64, _i32, _p]
lib.xgemm_run_noalloc.restype = _i32
lib.xgemm_run_config.argtypes = [_handle_t, _i64, _i64, _i64, _p, _i64, _p, _i64, _p, _i64, _i32, _p,
                                 ctypes.POINTER(xgemm_config)]
lib.xgemm_run_config.restype = _i32
lib.xgemm_run_strided_batched.argtypes = [_handle_t, _i64, _i64, _i64, _i64, _p, _i64, _i64, _p, _i64, _i64,
                                          _p, _i64, _i64, _i32, _p]
lib.xgemm_run_strided_batched.restype = _i32
lib.xgemm_select_config.argtypes = [_i64, _i64, _i64, _i32, _i32, ctypes.POINTER(xgemm_config)]
lib.xgemm_select_config.restype = _i32
lib.xgemm_select_band.argtypes = [_i64, _i64, _i64, _i32, _i32, ctypes.POINTER(xgemm_band)]
lib.xgemm_select_plan.argtypes = [_i64, _i64, _i64, _i32, _i32, _i32, ctypes.POINTER(xgemm_band)]
lib.xgemm_select_plan.restype = _i32
lib.xgemm_select_band.restype = _i32
lib.xgemm_tile_info.argtypes = [_i32] + [ctypes.POINTER(ctypes.c_int)] * 4
lib.xgemm_tile_info.restype = _i32
lib.xgemm_kernel_family.argtypes = [_i64, _i64, _i64, _p, _i64, _p, _i64, ctypes.POINTER(xgemm_config)]
lib.xgemm_kernel_family.restype = _i32
lib.xgemm_workspace_bytes.argtypes = [_i64, _i64, _i64, _i32, ctypes.POINTER(xgemm_config)]
lib.xgemm_workspace_bytes.restype = ctypes.c_size_t
lib.xgemm_trace_plan.argtypes = [_i64, _i64, _i64, _p, _i64, _p, _i64, _p, _i64, ctypes.POINTER(xgemm_config),
                                 _i32, _i32, ctypes.POINTER(xgemm_trace_info)]
lib.xgemm_trace_plan.restype = _i32
lib.xgemm_trace_workgroup.argtypes = [_i64, _i64, _i64, _p, _i64, _p, _i64, _p, _i64, _p,
                                      ctypes.POINTER(xgemm_config), _i32, _i32, _i64, _i32, _p, _i64, _p]
lib.xgemm_trace_workgroup.restype = _i32
lib.xgemv_run.argtypes = [_handle_t, _i64, _i64, _p, _i64, _p, _p, _p]
lib.xgemv_run.restype = _i32
lib.xgemv_run_config.argtypes = [_handle_t, _i64, _i64, _p, _i64, _p, _p, _p, ctypes.POINTER(xgemv_config)]
lib.xgemv_run_config.restype = _i32
lib.xgemv_select_config.argtypes = [_i64, _i64, _i32, ctypes.POINTER(xgemv_config)]
lib.xgemv_select_config.restype = _i32
lib.xgemv_trace_workgroup.argtypes = [_i64, _i64, _p, _i64, _p, _p, _p, ctypes.POINTER(xgemv_config), _i64, _p,
                                      _i64, _p]
lib.xgemv_trace_workgroup.restype = _i32
lib.xgemm_strerror.argtypes = [_i32]
lib.xgemm_strerror.restype = ctypes.c_char_p
lib.xgemm_last_error.argtypes = [_handle_t]
lib.xgemm_last_error.restype = ctypes.c_char_p


def header_functions(path: str = _HEADER):
    """Names of the functions include/xgemm.h declares."""
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(xgem[mv]_[a-z_]+)\s*\(", text)))


# ---------------------------------------------------------------------------
# same-name wrappers (raw status codes, as the C ABI)
# ---------------------------------------------------------------------------

def xgemm_create() -> int:
    """Returns a handle (an int address); raises XgemmError on failure."""
    h = _handle_t()
    rc = lib.xgemm_create(ctypes.byref(h))
    if rc != XGEMM_OK:
        raise XgemmError(rc)
    return h.value


def xgemm_destroy(h) -> int:
    return lib.xgemm_destroy(h)


def xgemm_set_workspace_limit(h, nbytes) -> int:
    return lib.xgemm_set_workspace_limit(h, nbytes)


def xgemm_set_persistent(h, enable) -> int:
    return lib.xgemm_set_persistent(h, enable)


def xgemm_run(h, M, N, K, A, lda, B, ldb, C, ldc, dtype, stream) -> int:
    return lib.xgemm_run(h, M, N, K, A, lda, B, ldb, C, ldc, dtype, stream)


def xgemm_run_noalloc(h, M, N, K, A, lda, B, ldb, C, ldc, dtype, stream) -> int:
    return lib.xgemm_run_noalloc(h, M, N, K, A, lda, B, ldb, C, ldc, dtype, stream)


XGEMM_NOALLOC_SCRATCH_BYTES = 64 << 20


def xgemm_run_config(h, M, N, K, A, lda, B, ldb, C, ldc, dtype, stream, cfg) -> int:
    return lib.xgemm_run_config(h, M, N, K, A, lda, B, ldb, C, ldc, dtype, stream,
                                ctypes.byref(cfg) if cfg is not None else None)


def xgemm_run_strided_batched(h, batch, M, N, K, A, lda, stride_a, B, ldb, stride_b, C, ldc, stride_c,
                              dtype, stream) -> int:
    return lib.xgemm_run_strided_batched(h, batch, M, N, K, A, lda, stride_a, B, ldb, stride_b, C, ldc, stride_c,
                                         dtype, stream)


def xgemm_select_config(M, N, K, dtype, cu_count) -> xgemm_config:
    cfg = xgemm_config()
    rc = lib.xgemm_select_config(M, N, K, dtype, cu_count, ctypes.byref(cfg))
    if rc != XGEMM_OK:
        raise XgemmError(rc)
    return cfg


def xgemm_select_band(M, N, K, dtype, cu_count) -> xgemm_band:
    out = xgemm_band()
    rc = lib.xgemm_select_band(M, N, K, dtype, cu_count, ctypes.byref(out))
    if rc != XGEMM_OK:
        raise XgemmError(rc)
    return out


def xgemm_select_plan(M, N, K, dtype, cu_count, persistent) -> xgemm_band:
    out = xgemm_band()
    rc = lib.xgemm_select_plan(M, N, K, dtype, cu_count, persistent, ctypes.byref(out))
    if rc != XGEMM_OK:
        raise XgemmError(rc)
    return out


def xgemm_tile_info(tile):
    vals = [ctypes.c_int() for _ in range(4)]
    rc = lib.xgemm_tile_info(tile, *[ctypes.byref(v) for v in vals])
    if rc != XGEMM_OK:
        raise XgemmError(rc)
    return tuple(v.value for v in vals)  # (bm, bn, bk, threads)


def xgemm_kernel_family(M, N, K, A, lda, B, ldb, cfg) -> int:
    return lib.xgemm_kernel_family(M, N, K, A, lda, B, ldb, ctypes.byref(cfg))


def xgemm_workspace_bytes(M, N, K, cu_count, cfg) -> int:
    return int(lib.xgemm_workspace_bytes(M, N, K, cu_count, ctypes.byref(cfg)))


def xgemm_trace_plan(M, N, K, A, lda, B, ldb, C, ldc, cfg, cu_count, segment) -> xgemm_trace_info:
    """Launch `segment` of the plan for these arguments; raises XgemmError."""
    info = xgemm_trace_info()
    rc = lib.xgemm_trace_plan(M, N, K, A, lda, B, ldb, C, ldc, ctypes.byref(cfg), cu_count, segment,
                              ctypes.byref(info))
    if rc != XGEMM_OK:
        raise XgemmError(rc)
    return info


# numpy layout of xgemm_trace_event
TRACE_EVENT_DTYPE = [("op", "<i4"), ("arg", "<i4"), ("lds", "<i8"), ("addr", "<i8")]


def xgemm_trace_workgroup(M, N, K, A, lda, B, ldb, C, ldc, W, cfg, cu_count, segment, block, threads,
                          capacity=None, schedule=0):
    """Events of every thread of one workgroup: a list of `threads` numpy
    record arrays (fields op, arg, lds, addr).  `threads` must be the
    launch's thread count (xgemm_trace_plan's info.threads), since the
    library writes that many counts.  `schedule` picks which piece of a
    persistent kernel's split tile counts in first (0: its last K steps).
    Raises XgemmError."""
    import numpy as np
    if threads != xgemm_trace_plan(M, N, K, A, lda, B, ldb, C, ldc, cfg, cu_count, segment).threads:
        raise XgemmError(XGEMM_ERR_INVALID_ARG, "threads is not the launch's thread count")
    counts = np.zeros(threads, dtype=np.int64)
    cptr = counts.ctypes.data_as(ctypes.c_void_p)
    if capacity is None:
        rc = lib.xgemm_trace_workgroup(M, N, K, A, lda, B, ldb, C, ldc, W, ctypes.byref(cfg), cu_count,
                                       segment, block, schedule, None, 0, cptr)
        if rc != XGEMM_OK:
            raise XgemmError(rc)
        capacity = int(counts.max())
    out = np.zeros((threads, max(capacity, 1)), dtype=TRACE_EVENT_DTYPE)
    rc = lib.xgemm_trace_workgroup(M, N, K, A, lda, B, ldb, C, ldc, W, ctypes.byref(cfg), cu_count, segment,
                                   block, schedule, out.ctypes.data_as(ctypes.c_void_p), out.shape[1], cptr)
    if rc != XGEMM_OK:
        raise XgemmError(rc)
    if int(counts.max()) > out.shape[1]:
        return xgemm_trace_workgroup(M, N, K, A, lda, B, ldb, C, ldc, W, cfg, cu_count, segment, block,
                                     threads, int(counts.max()), schedule)
    return [out[t, :counts[t]] for t in range(threads)]


def xgemv_run(h, M, K, A, lda, x, y, stream) -> int:
    return lib.xgemv_run(h, M, K, A, lda, x, y, stream)


def xgemv_run_config(h, M, K, A, lda, x, y, stream, cfg) -> int:
    return lib.xgemv_run_config(h, M, K, A, lda, x, y, stream, ctypes.byref(cfg) if cfg is not None else None)


def xgemv_select_config(M, K, cu_count) -> xgemv_config:
    out = xgemv_config()
    rc = lib.xgemv_select_config(M, K, cu_count, ctypes.byref(out))
    if rc != XGEMM_OK:
        raise XgemmError(rc)
    return out


def xgemm_strerror(status: int) -> str:
    return lib.xgemm_strerror(status).decode()


def xgemm_last_error(h) -> str:
    return lib.xgemm_last_error(h).decode()


# ---------------------------------------------------------------------------
# torch convenience layer (marshalling only)
# ---------------------------------------------------------------------------

_handles = {}


def _stream_ptr(stream) -> int:
    """The hipStream_t address of a torch stream, a raw address or None (the
    null stream)."""
    if stream is None:
        return 0
    return int(getattr(stream, "cuda_stream", stream) or 0)


def handle(device_index: int | None = None, stream=None):
    """The handle this module owns for (device, stream), created on first use.

    A handle's workspace (split-k partials, operand copies) belongs to one
    stream at a time: the library orders calls that share it across streams
    after each other, so one handle per stream is what lets calls on
    different streams run concurrently.  ``stream`` is a torch stream, a raw
    hipStream_t address or None (the null stream)."""
    import torch
    if device_index is None:
        device_index = torch.cuda.current_device()
    key = (device_index, _stream_ptr(stream))
    h = _handles.get(key)
    if h is None:
        with torch.cuda.device(device_index):
            h = xgemm_create()
        _handles[key] = h
    return h


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return XGEMM_BF16
    if t.dtype == torch.float16:
        return XGEMM_FP16
    raise TypeError("A and B must be bfloat16 or float16 tensors, got %s" % t.dtype)


def _ld(t) -> int:
    if t.dim() != 2:
        raise ValueError("expected a 2-D tensor")
    if t.shape[1] > 1 and t.stride(1) != 1:
        raise ValueError("rows must be contiguous (stride(1) == 1)")
    if t.shape[0] <= 1:
        return max(t.shape[1], t.stride(0))
    return t.stride(0)


def bmm(A, B, out=None, stream=None):
    """out[b] = A[b] @ B[b] (fp32) for 3-D tensors through xgemm_run_strided_batched.

    A: (L, M, K), B: (L, K, N) bf16/fp16 CUDA tensors with contiguous rows (any
    batch stride, including 0 for a broadcast operand); out: optional (L, M, N)
    float32 tensor with contiguous rows.
    """
    import torch
    if A.dim() != 3 or B.dim() != 3 or A.shape[0] != B.shape[0] or A.shape[2] != B.shape[1]:
        raise ValueError("expected A (L, M, K) and B (L, K, N)")
    if A.dtype != B.dtype:
        raise TypeError("A and B must have the same dtype")
    dtype = _dtype_code(A)
    L, M, K = A.shape
    N = B.shape[2]
    if out is None:
        out = torch.empty((L, M, N), dtype=torch.float32, device=A.device)
    if out.dtype != torch.float32 or tuple(out.shape) != (L, M, N):
        raise ValueError("out must be a float32 (L, M, N) tensor")
    for t in (A, B, out):
        if t.shape[2] > 1 and t.stride(2) != 1:
            raise ValueError("rows must be contiguous")
    s = stream if stream is not None else torch.cuda.current_stream(A.device)
    h = handle(A.device.index, s)
    lda = A.stride(1) if M > 1 else max(K, 1)
    ldb = B.stride(1) if K > 1 else max(N, 1)
    ldc = out.stride(1) if M > 1 else max(N, 1)
    rc = xgemm_run_strided_batched(h, L, M, N, K, A.data_ptr() or None, lda, A.stride(0) if L > 1 else 0,
                                   B.data_ptr() or None, ldb, B.stride(0) if L > 1 else 0,
                                   out.data_ptr() or None, ldc, out.stride(0) if L > 1 else 0, dtype, s.cuda_stream)
    if rc != XGEMM_OK:
        raise XgemmError(rc, xgemm_last_error(h))
    return out


def gemm(A, B, out=None, config: xgemm_config | None = None, stream=None):
    """C = A @ B with fp32 output, through xgemm_run (or xgemm_run_config).

    A: (M, K) and B: (K, N) bfloat16/float16 CUDA tensors of one dtype with
    contiguous rows; out: optional (M, N) float32 tensor with contiguous rows.
    Enqueued on ``stream`` (default: torch's current stream).
    """
    import torch
    if A.dtype != B.dtype:
        raise TypeError("A and B must have the same dtype")
    dtype = _dtype_code(A)
    M, K = A.shape
    K2, N = B.shape
    if K2 != K:
        raise ValueError("inner dimensions differ: %d vs %d" % (K, K2))
    if not (A.is_cuda and B.is_cuda) or A.device != B.device:
        raise ValueError("A and B must be on the same GPU")
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=A.device)
    if out.dtype != torch.float32 or tuple(out.shape) != (M, N) or out.device != A.device:
        raise ValueError("out must be a float32 (M, N) tensor on A's device")
    s = stream if stream is not None else torch.cuda.current_stream(A.device)
    h = handle(A.device.index, s)
    args = (h, M, N, K, A.data_ptr() or None, _ld(A), B.data_ptr() or None, _ld(B),
            out.data_ptr() or None, _ld(out), dtype, s.cuda_stream)
    if config is None:
        rc = xgemm_run(*args)
    else:
        rc = xgemm_run_config(*args, config)
    if rc != XGEMM_OK:
        raise XgemmError(rc, xgemm_last_error(h))
    return out


def gemv(A, x, out=None, config: xgemv_config | None = None, stream=None):
    """y = A @ x for a float32 CUDA matrix A (M x K, unit column stride) and
    vector x (K, contiguous); returns y (M, float32), written into ``out`` if
    given.  Runs xgemv_run (or xgemv_run_config) on the current stream."""
    if A.dtype != torch.float32 or x.dtype != torch.float32:
        raise TypeError("gemv takes float32 A and x")
    if A.dim() != 2 or x.dim() != 1 or A.shape[1] != x.shape[0]:
        raise ValueError("shapes %s and %s do not match" % (tuple(A.shape), tuple(x.shape)))
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    M, K = A.shape
    if M > 0 and K > 1 and A.stride(1) != 1:
        raise ValueError("A must have unit stride along its rows")
    lda = A.stride(0) if M > 1 else max(K, 1)
    if out is None:
        out = torch.empty(M, dtype=torch.float32, device=A.device)
    elif out.dtype != torch.float32 or out.shape != (M,) or not out.is_contiguous():
        raise ValueError("out must be a contiguous float32 vector of %d values" % M)
    if stream is None:
        stream = torch.cuda.current_stream(A.device)
    h = handle(A.device.index, stream)
    args = (h, M, K, A.data_ptr() or None, lda, x.data_ptr() or None, out.data_ptr() or None,
            _stream_ptr(stream) or None)
    rc = xgemv_run_config(*args, config) if config is not None else xgemv_run(*args)
    if rc != XGEMM_OK:
        raise XgemmError(rc, xgemm_last_error(h))
    return out
