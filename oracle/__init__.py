"""Oracles for the dense 16-bit GEMM hot path (C = A*B) and the fp32 GEMV
(y = A*x), both evaluated in fp64.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the CPU-baseline
leg of the benchmark may import this package; the product library never does.
It shares no code with the GPU path.  Inputs are the stored 16-bit bit patterns
(numpy ``uint16`` arrays, row-major); outputs are fp64.

The arithmetic lives in ``gemm_oracle.c`` and ``gemv_oracle.c`` (plain C,
OpenMP over rows), which ``build()`` compiles with gcc into ``liboracle.so``
next to this file.  The GEMM definition is the plain one the paper's
sequential GEMM program states (Introduction; Section 2.3): C[i][j] = sum_k
A[i][k] * B[k][j], summed in ascending k, together with the tolerance scale
S[i][j] = sum_k |A[i][k]*B[k][j]|.  The GEMV is the paper's fp32
matrix-vector benchmark (Section 6): y[i] = sum_k A[i][k] * x[k] with
s[i] = sum_k |A[i][k]*x[k]|, A and x given as float32 arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = [os.path.join(_HERE, "gemm_oracle.c"), os.path.join(_HERE, "gemv_oracle.c")]
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

BF16 = 0
FP16 = 1
_DTYPES = {"bf16": BF16, "fp16": FP16, BF16: BF16, FP16: FP16}

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle sources into ``liboracle.so`` (gcc, OpenMP, no fast-math)."""
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
           "-ffp-contract=off", "-fno-fast-math"] + _SRC + ["-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    i64, p, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    lib.oracle_decode_bf16.argtypes = [ctypes.c_uint16]
    lib.oracle_decode_bf16.restype = ctypes.c_double
    lib.oracle_decode_fp16.argtypes = [ctypes.c_uint16]
    lib.oracle_decode_fp16.restype = ctypes.c_double
    lib.oracle_decode.argtypes = [p, i64, i32, p]
    lib.oracle_decode.restype = i32
    lib.oracle_gemm.argtypes = [i64, i64, i64, p, i64, p, i64, i32, p, i64, p, i64, i32]
    lib.oracle_gemm.restype = i32
    lib.oracle_gemm_rows.argtypes = [i64, i64, i64, p, i64, p, i64, i32, p, i64, p, i64, p, i64, i32]
    lib.oracle_gemm_rows.restype = i32
    lib.oracle_gemm_entries.argtypes = [i64, i64, i64, p, i64, p, i64, i32, p, p, i64, p, p, i32]
    lib.oracle_gemm_entries.restype = i32
    lib.oracle_gemv_rows.argtypes = [i64, i64, p, i64, p, p, i64, p, p, i32]
    lib.oracle_gemv_rows.restype = i32
    lib.oracle_gemv.argtypes = [i64, i64, p, i64, p, p, p, i32]
    lib.oracle_gemv.restype = i32
    lib.oracle_thread_count.argtypes = [i32]
    lib.oracle_thread_count.restype = i32
    _lib = lib
    return lib


def _dtype_code(dtype) -> int:
    try:
        return _DTYPES[dtype]
    except KeyError:
        raise ValueError("dtype must be 'bf16' or 'fp16', got %r" % (dtype,))


def _as_bits(x: np.ndarray, name: str) -> np.ndarray:
    if x.dtype != np.uint16 or x.ndim != 2:
        raise TypeError("%s must be a 2-D uint16 array of stored bit patterns" % name)
    if x.size and x.shape[1] > 1 and x.strides[1] != 2:
        raise ValueError("%s must have unit stride along its rows" % name)
    return x


def _ld(x: np.ndarray) -> int:
    """Leading dimension (row stride in elements) of a 2-D bit array."""
    if x.size == 0 or x.shape[0] == 1:
        return max(x.shape[1], x.strides[0] // 2 if x.size else 0)
    return x.strides[0] // 2


def _ptr(x: np.ndarray):
    return ctypes.c_void_p(x.ctypes.data) if x.size else None


def _check(rc: int, what: str) -> None:
    if rc == 1:
        raise ValueError("%s: invalid arguments" % what)
    if rc != 0:
        raise MemoryError("%s: allocation failed" % what)


def decode(bits: np.ndarray, dtype) -> np.ndarray:
    """Exact fp64 values of stored 16-bit patterns (any shape)."""
    lib = _load()
    src = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty(src.shape, dtype=np.float64)
    _check(lib.oracle_decode(_ptr(src), src.size, _dtype_code(dtype), _ptr(out)), "decode")
    return out


def gemm(A: np.ndarray, B: np.ndarray, dtype, nthreads: int = 0):
    """Full product. Returns (C, S), both fp64 of shape (M, N).

    ``A`` (M x K) and ``B`` (K x N) may be row-padded views; their row strides
    are passed on as the leading dimensions.
    """
    A = _as_bits(A, "A")
    B = _as_bits(B, "B")
    M, K, N = A.shape[0], B.shape[0], B.shape[1]
    lda = _ld(A)
    ldb = _ld(B)
    if A.shape[1] != K:
        raise ValueError("A has %d columns, B has %d rows" % (A.shape[1], K))
    C = np.empty((M, N), dtype=np.float64)
    S = np.empty((M, N), dtype=np.float64)
    rc = _load().oracle_gemm(M, N, K, _ptr(A), lda, _ptr(B), ldb, _dtype_code(dtype),
                             _ptr(C), N, _ptr(S), N, nthreads)
    _check(rc, "oracle_gemm")
    return C, S


def gemm_rows(A: np.ndarray, B: np.ndarray, dtype, rows, nthreads: int = 0):
    """Selected whole rows of C and S: returns (C_rows, S_rows), shape (len(rows), N)."""
    A = _as_bits(A, "A")
    B = _as_bits(B, "B")
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    M, K, N = A.shape[0], B.shape[0], B.shape[1]
    if A.shape[1] != K:
        raise ValueError("A has %d columns, B has %d rows" % (A.shape[1], K))
    C = np.empty((rows.size, N), dtype=np.float64)
    S = np.empty((rows.size, N), dtype=np.float64)
    rc = _load().oracle_gemm_rows(M, N, K, _ptr(A), _ld(A), _ptr(B), _ld(B),
                                  _dtype_code(dtype), _ptr(rows), rows.size,
                                  _ptr(C), N, _ptr(S), N, nthreads)
    _check(rc, "oracle_gemm_rows")
    return C, S


def gemm_entries(A: np.ndarray, B: np.ndarray, dtype, rows, cols, nthreads: int = 0):
    """C[rows[t], cols[t]] and S[...] for scattered entries: returns (c, s), shape (count,)."""
    A = _as_bits(A, "A")
    B = _as_bits(B, "B")
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    if rows.shape != cols.shape:
        raise ValueError("rows and cols must have the same shape")
    M, K, N = A.shape[0], B.shape[0], B.shape[1]
    if A.shape[1] != K:
        raise ValueError("A has %d columns, B has %d rows" % (A.shape[1], K))
    c = np.empty(rows.size, dtype=np.float64)
    s = np.empty(rows.size, dtype=np.float64)
    rc = _load().oracle_gemm_entries(M, N, K, _ptr(A), _ld(A), _ptr(B), _ld(B),
                                     _dtype_code(dtype), _ptr(rows), _ptr(cols), rows.size,
                                     _ptr(c), _ptr(s), nthreads)
    _check(rc, "oracle_gemm_entries")
    return c, s


def thread_count(nthreads: int = 0) -> int:
    """Threads an oracle call with this ``nthreads`` argument runs on."""
    return int(_load().oracle_thread_count(nthreads))


def _as_f32_matrix(A: np.ndarray):
    if A.dtype != np.float32 or A.ndim != 2:
        raise TypeError("A must be a 2-D float32 array")
    if A.size and A.shape[1] > 1 and A.strides[1] != 4:
        raise ValueError("A must have unit stride along its rows")
    if A.size == 0 or A.shape[0] == 1:
        lda = max(A.shape[1], A.strides[0] // 4 if A.size else 0)
    else:
        lda = A.strides[0] // 4
    return A, lda


def _as_f32_vector(x: np.ndarray, K: int) -> np.ndarray:
    if x.dtype != np.float32 or x.ndim != 1 or x.shape[0] != K:
        raise TypeError("x must be a float32 vector of %d values" % K)
    return np.ascontiguousarray(x)


def gemv(A: np.ndarray, x: np.ndarray, nthreads: int = 0):
    """y = A x for float32 A (M x K, may be a row-padded view) and x (K).
    Returns (y, s), fp64 of shape (M,)."""
    A, lda = _as_f32_matrix(A)
    M, K = A.shape
    x = _as_f32_vector(x, K)
    y = np.empty(M, dtype=np.float64)
    s = np.empty(M, dtype=np.float64)
    rc = _load().oracle_gemv(M, K, _ptr(A), lda, _ptr(x), _ptr(y), _ptr(s), nthreads)
    _check(rc, "oracle_gemv")
    return y, s


def gemv_rows(A: np.ndarray, x: np.ndarray, rows, nthreads: int = 0):
    """Selected entries of y and s: returns (y_rows, s_rows), shape (len(rows),)."""
    A, lda = _as_f32_matrix(A)
    M, K = A.shape
    x = _as_f32_vector(x, K)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    y = np.empty(rows.size, dtype=np.float64)
    s = np.empty(rows.size, dtype=np.float64)
    rc = _load().oracle_gemv_rows(M, K, _ptr(A), lda, _ptr(x), _ptr(rows), rows.size, _ptr(y), _ptr(s),
                                  nthreads)
    _check(rc, "oracle_gemv_rows")
    return y, s
