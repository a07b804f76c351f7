"""Seeded synthetic inputs: GEMM operands as stored 16-bit bit patterns, GEMV
operands as float32.

This module holds no GEMM or GEMV arithmetic.  It only draws matrices and rounds them
to the 16-bit storage formats, so that the GPU path and the CPU oracle consume
identical bits.

The paper times its kernels on hashed pseudo-random matrices (Section 6).  The
workloads here are synthetic in the same spirit, with explicit distributions
and seeds:

* one ``numpy.random.default_rng(seed)`` (PCG64) generator per problem;
* A (M x K, row-major) is drawn first, then B (K x N, row-major), in float64;
* values are cast to float32 and then rounded to the storage format with
  round-to-nearest-even (fp16 through numpy's own cast, bf16 by rounding the
  float32 bit pattern).
"""
from __future__ import annotations

import dataclasses
import hashlib

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    M: int
    N: int
    K: int
    dtype: str          # "bf16" or "fp16"
    dist: str           # "uniform" (on [lo, hi]) or "normal" (mean 0, std sigma)
    seed: int
    param: float        # uniform: half-width; normal: sigma

    @property
    def flops(self) -> int:
        return 2 * self.M * self.N * self.K

    @property
    def alg_bytes(self) -> int:
        """A and B read once (2 B/element), C written once (fp32, 4 B/element)."""
        return 2 * (self.M * self.K + self.K * self.N) + 4 * self.M * self.N


# The problem set the library is tested and measured on.
WORKLOADS = {
    "gemm256_fp16": Workload("gemm256_fp16", 256, 256, 256, "fp16", "uniform", 0, 1.0),
    "gemm4096_bf16": Workload("gemm4096_bf16", 4096, 4096, 4096, "bf16", "normal", 1, 1.0),
    "gemm8192_bf16": Workload("gemm8192_bf16", 8192, 8192, 8192, "bf16", "uniform", 2, 1.0),
    "proj16384x5120x4096_fp16": Workload("proj16384x5120x4096_fp16", 16384, 5120, 4096, "fp16",
                                         "normal", 3, 0.02),
    "proj4096x14336x4096_fp16": Workload("proj4096x14336x4096_fp16", 4096, 14336, 4096, "fp16",
                                         "normal", 3, 0.02),
    "skinny1024x1024x65536_bf16": Workload("skinny1024x1024x65536_bf16", 1024, 1024, 65536, "bf16",
                                           "uniform", 4, 1.0),
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 bit patterns, nearest-even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def to_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    """float64/float32 array -> uint16 bit patterns of the storage format."""
    x32 = np.asarray(x, dtype=np.float32)
    if dtype == "fp16":
        return x32.astype(np.float16).view(np.uint16)
    if dtype == "bf16":
        return f32_to_bf16_bits(x32)
    raise ValueError("dtype must be 'bf16' or 'fp16'")


def _draw(rng: np.random.Generator, shape, dist: str, param: float) -> np.ndarray:
    if dist == "uniform":
        return rng.uniform(-param, param, size=shape)
    if dist == "normal":
        return rng.normal(0.0, param, size=shape)
    raise ValueError("unknown distribution %r" % dist)


def make_inputs(M: int, N: int, K: int, dtype: str, dist: str, seed: int, param: float = 1.0):
    """Return (A_bits [M,K], B_bits [K,N]) as contiguous uint16 arrays."""
    rng = np.random.default_rng(seed)
    A = to_bits(_draw(rng, (M, K), dist, param), dtype)
    B = to_bits(_draw(rng, (K, N), dist, param), dtype)
    return np.ascontiguousarray(A), np.ascontiguousarray(B)


def workload_inputs(w: Workload):
    return make_inputs(w.M, w.N, w.K, w.dtype, w.dist, w.seed, w.param)


def make_int_inputs(M: int, N: int, K: int, dtype: str, seed: int, lo: int = -8, hi: int = 8):
    """Small-integer matrices (exact in bf16 and fp16), entries uniform on [lo, hi]."""
    rng = np.random.default_rng(seed)
    A = rng.integers(lo, hi + 1, size=(M, K)).astype(np.float64)
    B = rng.integers(lo, hi + 1, size=(K, N)).astype(np.float64)
    return to_bits(A, dtype), to_bits(B, dtype)


# ---------------------------------------------------------------------------
# GEMV (fp32): the paper's matrix-vector benchmark runs square problems
# (Section 6).  A (M x K, row-major) is drawn first, then x (K), in float64
# from one generator, and cast to float32.
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class GemvWorkload:
    name: str
    M: int
    K: int
    dist: str
    seed: int
    param: float
    dtype: str = "fp32"

    @property
    def flops(self) -> int:
        return 2 * self.M * self.K

    @property
    def alg_bytes(self) -> int:
        """A and x read once, y written once (4 B/element)."""
        return 4 * (self.M * self.K + self.K + self.M)


GEMV_WORKLOADS = {
    "gemv4096_fp32": GemvWorkload("gemv4096_fp32", 4096, 4096, "uniform", 5, 1.0),
    "gemv8192_fp32": GemvWorkload("gemv8192_fp32", 8192, 8192, "uniform", 6, 1.0),
    "gemv16384_fp32": GemvWorkload("gemv16384_fp32", 16384, 16384, "uniform", 7, 1.0),
    "gemv32768_fp32": GemvWorkload("gemv32768_fp32", 32768, 32768, "uniform", 8, 1.0),
}


def make_gemv_inputs(M: int, K: int, dist: str, seed: int, param: float = 1.0, rows_per_draw: int = 4096):
    """Return (A [M, K], x [K]) as contiguous float32 arrays.  A is drawn in
    blocks of rows (the same values as one draw of the whole matrix, since
    each value takes the generator's next output) to bound host memory."""
    rng = np.random.default_rng(seed)
    A = np.empty((M, K), dtype=np.float32)
    for r in range(0, M, rows_per_draw):
        n = min(rows_per_draw, M - r)
        A[r:r + n] = _draw(rng, (n, K), dist, param)
    x = _draw(rng, (K,), dist, param).astype(np.float32)
    return A, x


def gemv_workload_inputs(w: GemvWorkload):
    return make_gemv_inputs(w.M, w.K, w.dist, w.seed, w.param)


def sha256_bits(*arrays: np.ndarray) -> str:
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()
