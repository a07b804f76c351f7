"""Pins for the CPU oracle, checked against things other than itself.

Each test fixes the oracle to a value the mathematics determines independently
of its implementation: hand-worked values from the 16-bit format definitions,
exact rational arithmetic (Python ``fractions``), exact integer products, the
identity and permutation matrices, and an independent fp64 library product
(numpy/BLAS) on independently decoded inputs.  A final group plants mistakes in
a copy of the oracle's C source and checks that these pins catch each one.
"""
import ctypes
import os
import re
import shutil
import subprocess
from fractions import Fraction

import numpy as np
import pytest

from conftest import GOLDEN, ROOT
from paper_2609_16389_amd import workloads as wl


# --------------------------------------------------------------------------
# fixtures read from tests/golden
# --------------------------------------------------------------------------

def _parse_value(tok):
    if tok == "inf":
        return float("inf")
    if tok == "-inf":
        return float("-inf")
    return Fraction(tok)


def _decode_points():
    pts = []
    with open(os.path.join(GOLDEN, "decode_points.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            parts = line.split()
            pts.append((parts[0], int(parts[1], 16), _parse_value(parts[2])))
    return pts


def _worked_cases():
    cases, cur = [], None
    with open(os.path.join(GOLDEN, "worked_example.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            parts = line.split()
            if parts[0] == "case":
                cur = dict(name=parts[1], dtype=parts[2], M=int(parts[3]), N=int(parts[4]),
                           K=int(parts[5]), A=[], B=[], C=[], S=[])
                cases.append(cur)
            elif parts[0] in ("A", "B"):
                cur[parts[0]].append([int(t, 16) for t in parts[1:]])
            else:
                cur[parts[0]].append([Fraction(t) for t in parts[1:]])
    return cases


# --------------------------------------------------------------------------
# independent references (no oracle code involved)
# --------------------------------------------------------------------------

def np_decode(bits, dtype):
    """Decode through numpy's own float16 and the float32-upper-half reading of bf16."""
    bits = np.asarray(bits, dtype=np.uint16)
    if dtype == "fp16":
        return bits.view(np.float16).astype(np.float64)
    with np.errstate(invalid="ignore"):
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def frac_decode(bits, dtype):
    """Exact rational value of a finite 16-bit pattern from the field definitions."""
    if dtype == "fp16":
        s, e, f, ebits, fbits, bias = bits >> 15, (bits >> 10) & 31, bits & 1023, 5, 10, 15
    else:
        s, e, f, ebits, fbits, bias = bits >> 15, (bits >> 7) & 255, bits & 127, 8, 7, 127
    assert e != (1 << ebits) - 1, "finite patterns only"
    if e == 0:
        v = Fraction(f, 1 << fbits) * Fraction(2) ** (1 - bias)
    else:
        v = (1 + Fraction(f, 1 << fbits)) * Fraction(2) ** (e - bias)
    return -v if s else v


def int_bits(x, dtype):
    return wl.to_bits(np.asarray(x, dtype=np.float64), dtype)


# --------------------------------------------------------------------------
# decoders
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_decode_golden_points(oracle_mod, dtype):
    pts = [p for p in _decode_points() if p[0] == dtype]
    assert len(pts) >= 10
    got = oracle_mod.decode(np.array([p[1] for p in pts], dtype=np.uint16), dtype)
    for (_, bits, want), g in zip(pts, got):
        if isinstance(want, float):
            assert g == want, hex(bits)
        else:
            assert Fraction(g) == want, hex(bits)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_decode_exhaustive_against_numpy(oracle_mod, dtype):
    allbits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle_mod.decode(allbits, dtype)
    ref = np_decode(allbits, dtype)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signs of zeros too
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_decode_matches_field_definition_sampled(oracle_mod, dtype):
    rng = np.random.default_rng(7)
    bits = rng.integers(0, 65536, size=2000).astype(np.uint16)
    emax = 31 if dtype == "fp16" else 255
    shift = 10 if dtype == "fp16" else 7
    bits = bits[((bits >> shift) & emax) != emax]
    got = oracle_mod.decode(bits, dtype)
    for b, g in zip(bits.tolist(), got.tolist()):
        assert Fraction(g) == frac_decode(b, dtype)


# --------------------------------------------------------------------------
# hand-worked products
# --------------------------------------------------------------------------

@pytest.mark.parametrize("case", _worked_cases(), ids=lambda c: c["name"] + "_" + c["dtype"])
def test_worked_examples(oracle_mod, case):
    A = np.array(case["A"], dtype=np.uint16)
    B = np.array(case["B"], dtype=np.uint16)
    assert A.shape == (case["M"], case["K"]) and B.shape == (case["K"], case["N"])
    C, S = oracle_mod.gemm(A, B, case["dtype"])
    for i in range(case["M"]):
        for j in range(case["N"]):
            assert Fraction(C[i, j]) == case["C"][i][j]
            assert Fraction(S[i, j]) == case["S"][i][j]


# --------------------------------------------------------------------------
# identity, permutations, closed forms
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_identity_right_and_left(oracle_mod, dtype):
    rng = np.random.default_rng(11)
    M, K = 37, 29
    A = wl.to_bits(rng.normal(0, 3, size=(M, K)), dtype)
    I_K = int_bits(np.eye(K), dtype)
    I_M = int_bits(np.eye(M), dtype)
    C, S = oracle_mod.gemm(A, I_K, dtype)
    assert np.array_equal(C, np_decode(A, dtype))
    assert np.array_equal(S, np.abs(np_decode(A, dtype)))
    C2, _ = oracle_mod.gemm(I_M, A, dtype)
    assert np.array_equal(C2, np_decode(A, dtype))


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_identity_with_padded_leading_dims(oracle_mod, dtype):
    rng = np.random.default_rng(12)
    M, K = 20, 13
    Apad = wl.to_bits(rng.uniform(-1, 1, size=(M, K + 7)), dtype)
    A = Apad[:, :K]                       # lda = K + 7
    Ipad = int_bits(np.hstack([np.eye(K), np.full((K, 5), 9.0)]), dtype)
    I = Ipad[:, :K]                       # ldb = K + 5, padding holds 9s that must be ignored
    C, _ = oracle_mod.gemm(A, I, dtype)
    assert np.array_equal(C, np_decode(np.ascontiguousarray(A), dtype))


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_permutation_matrices(oracle_mod, dtype):
    rng = np.random.default_rng(13)
    M, K, N = 16, 24, 8
    A = wl.to_bits(rng.uniform(-1, 1, size=(M, K)), dtype)
    perm = rng.permutation(K)
    P = np.zeros((K, K))
    P[np.arange(K), perm] = 1.0
    C, _ = oracle_mod.gemm(A, int_bits(P, dtype), dtype)
    # (A P)[i][j] = A[i][k] where perm[k] == j
    inv = np.argsort(perm)
    assert np.array_equal(C, np_decode(A, dtype)[:, inv])
    del N


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_ones_give_K(oracle_mod, dtype):
    M, N, K = 5, 7, 300
    C, S = oracle_mod.gemm(int_bits(np.ones((M, K)), dtype), int_bits(np.ones((K, N)), dtype), dtype)
    assert np.all(C == K) and np.all(S == K)


def test_rank_one_powers_of_two(oracle_mod):
    # A[i][k] = 2^(i-k), B[k][j] = 2^(k+j) -> C[i][j] = K * 2^(i+j) exactly.
    M, N, K = 6, 5, 9
    A = np.array([[2.0 ** (i - k) for k in range(K)] for i in range(M)])
    B = np.array([[2.0 ** (k + j) for j in range(N)] for k in range(K)])
    C, _ = oracle_mod.gemm(int_bits(A, "bf16"), int_bits(B, "bf16"), "bf16")
    want = np.array([[K * 2.0 ** (i + j) for j in range(N)] for i in range(M)])
    assert np.array_equal(C, want)


def test_zero_K_gives_zero(oracle_mod):
    A = np.zeros((4, 0), dtype=np.uint16)
    B = np.zeros((0, 6), dtype=np.uint16)
    C, S = oracle_mod.gemm(A, B, "fp16")
    assert C.shape == (4, 6) and np.all(C == 0) and np.all(S == 0)


# --------------------------------------------------------------------------
# exact arithmetic
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("shape", [(3, 4, 5), (16, 9, 70), (64, 33, 1000)])
def test_small_integers_exact(oracle_mod, dtype, shape):
    M, N, K = shape
    A, B = wl.make_int_inputs(M, N, K, dtype, seed=M + N + K)
    Ai = np_decode(A, dtype).astype(np.int64)
    Bi = np_decode(B, dtype).astype(np.int64)
    C, S = oracle_mod.gemm(A, B, dtype)
    assert np.array_equal(C, (Ai @ Bi).astype(np.float64))
    assert np.array_equal(S, (np.abs(Ai) @ np.abs(Bi)).astype(np.float64))


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("shape", [(1, 1, 1), (2, 3, 4), (5, 3, 8), (3, 2, 64)])
def test_exact_rational_brute_force(oracle_mod, dtype, shape):
    M, N, K = shape
    rng = np.random.default_rng(100 + K)
    # spread of magnitudes so that the fp64 sum really rounds
    A = wl.to_bits(rng.normal(0, 1, size=(M, K)) * 2.0 ** rng.integers(-12, 12, size=(M, K)), dtype)
    B = wl.to_bits(rng.normal(0, 1, size=(K, N)) * 2.0 ** rng.integers(-12, 12, size=(K, N)), dtype)
    C, S = oracle_mod.gemm(A, B, dtype)
    for i in range(M):
        for j in range(N):
            terms = [frac_decode(int(A[i, k]), dtype) * frac_decode(int(B[k, j]), dtype)
                     for k in range(K)]
            exact = sum(terms, Fraction(0))
            exact_s = sum((abs(t) for t in terms), Fraction(0))
            bound = (K - 1) * Fraction(2) ** -53 * exact_s
            assert abs(Fraction(C[i, j]) - exact) <= bound
            assert abs(Fraction(S[i, j]) - exact_s) <= bound


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_against_numpy_fp64_product(oracle_mod, dtype):
    M, N, K = 96, 80, 700
    A, B = wl.make_inputs(M, N, K, dtype, "normal", seed=5)
    C, S = oracle_mod.gemm(A, B, dtype)
    Ad, Bd = np_decode(A, dtype), np_decode(B, dtype)
    ref = Ad @ Bd
    ref_s = np.abs(Ad) @ np.abs(Bd)
    assert np.all(np.abs(C - ref) <= 1e-12 * ref_s)
    assert np.all(np.abs(S - ref_s) <= 1e-12 * ref_s)


def test_linearity_and_k_block_decomposition(oracle_mod):
    M, N, K = 24, 40, 96
    A, B = wl.make_int_inputs(M, N, K, "bf16", seed=3, lo=-4, hi=4)
    C, _ = oracle_mod.gemm(A, B, "bf16")
    # sum of the products over K-slices equals the full product (exact for integers)
    parts = sum(oracle_mod.gemm(np.ascontiguousarray(A[:, k:k + 32]),
                                np.ascontiguousarray(B[k:k + 32]), "bf16")[0]
                for k in range(0, K, 32))
    assert np.array_equal(C, parts)
    # transpose identity: (A B)^T = B^T A^T
    Ct, _ = oracle_mod.gemm(np.ascontiguousarray(B.T), np.ascontiguousarray(A.T), "bf16")
    assert np.array_equal(C.T, Ct)


# --------------------------------------------------------------------------
# rows / entries agree with the full product, and argument checks
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_rows_and_entries_match_full(oracle_mod, dtype):
    M, N, K = 50, 45, 130
    A, B = wl.make_inputs(M, N, K, dtype, "uniform", seed=9)
    C, S = oracle_mod.gemm(A, B, dtype)
    rows = np.array([0, 7, 49, 7])
    Cr, Sr = oracle_mod.gemm_rows(A, B, dtype, rows)
    assert np.array_equal(Cr, C[rows]) and np.array_equal(Sr, S[rows])
    rng = np.random.default_rng(1)
    ri, ci = rng.integers(0, M, 300), rng.integers(0, N, 300)
    c, s = oracle_mod.gemm_entries(A, B, dtype, ri, ci)
    assert np.array_equal(c, C[ri, ci]) and np.array_equal(s, S[ri, ci])


def test_invalid_arguments_rejected(oracle_mod):
    A = np.zeros((4, 4), dtype=np.uint16)
    with pytest.raises(ValueError):
        oracle_mod.gemm(A, A, "fp32")
    with pytest.raises(ValueError):
        oracle_mod.gemm_rows(A, A, "bf16", [4])
    with pytest.raises(ValueError):
        oracle_mod.gemm_entries(A, A, "bf16", [0], [-1])
    with pytest.raises(TypeError):
        oracle_mod.gemm(A.astype(np.int32), A, "bf16")


def test_thread_count_positive(oracle_mod):
    assert oracle_mod.thread_count() >= 1
    assert oracle_mod.thread_count(1) == 1


# --------------------------------------------------------------------------
# sensitivity: plant mistakes in a copy of the oracle and check the pins fail
# --------------------------------------------------------------------------

MUTANTS = {
    # a dropped term: the last k is never added
    "drop_last_k": ("for (int64_t k = 0; k < K; ++k) {\n            const double a",
                    "for (int64_t k = 0; k < K - 1; ++k) {\n            const double a"),
    # a wrong index: B read transposed
    "b_transposed": ("Bd[k * N + j] = dec(B[k * ldb + j], dtype);",
                     "Bd[k * N + j] = dec(B[j * ldb + k], dtype);"),
    # a wrong leading dimension for A
    "lda_as_K": ("const double a = dec(A[i * lda + k], dtype);",
                 "const double a = dec(A[i * K + k], dtype);"),
    # a wrong exponent bias in the fp16 decoder
    "fp16_bias": ("ldexp((double)(1024 + f), e - 15 - 10)", "ldexp((double)(1024 + f), e - 16 - 10)"),
    # subnormals decoded as if normal
    "bf16_subnormal": ("v = ldexp((double)f, -126 - 7);", "v = ldexp((double)(128 + f), -126 - 7);"),
    # a sign error in the tolerance scale
    "s_signed": ("s[j] += fabs(p);", "s[j] += p;"),
}


class _MutantOracle:
    """Minimal stand-in exposing the oracle API on top of a mutated build."""

    def __init__(self, lib):
        import oracle as real
        self._lib = lib
        self._real = real

    def gemm(self, A, B, dtype):
        real = self._real
        saved = real._lib
        real._lib = self._lib
        try:
            return real.gemm(A, B, dtype)
        finally:
            real._lib = saved

    def decode(self, bits, dtype):
        real = self._real
        saved = real._lib
        real._lib = self._lib
        try:
            return real.decode(bits, dtype)
        finally:
            real._lib = saved


def _build_mutant(tmp_path, name):
    src = open(os.path.join(ROOT, "oracle", "gemm_oracle.c")).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, "mutation anchor for %s not found exactly once" % name
    path = tmp_path / ("%s.c" % name)
    path.write_text(src.replace(old, new))
    so = tmp_path / ("lib%s.so" % name)
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
                    str(path), "-o", str(so), "-lm"], check=True)
    import oracle as real
    lib = ctypes.CDLL(str(so))
    # same signatures as the real library
    for fn in ("oracle_decode", "oracle_gemm", "oracle_gemm_rows", "oracle_gemm_entries"):
        getattr(lib, fn).argtypes = getattr(real._load(), fn).argtypes
        getattr(lib, fn).restype = getattr(real._load(), fn).restype
    return _MutantOracle(lib)


def _pins_pass(orc):
    """Run a compact subset of the pins above; True if all of them hold."""
    checks = []
    for case in _worked_cases():
        A = np.array(case["A"], dtype=np.uint16)
        B = np.array(case["B"], dtype=np.uint16)
        C, S = orc.gemm(A, B, case["dtype"])
        checks.append(all(Fraction(C[i, j]) == case["C"][i][j] and Fraction(S[i, j]) == case["S"][i][j]
                          for i in range(case["M"]) for j in range(case["N"])))
    for dtype in ("bf16", "fp16"):
        allbits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
        got, ref = orc.decode(allbits, dtype), np_decode(allbits, dtype)
        ok = ~np.isnan(ref)
        checks.append(np.array_equal(got[ok], ref[ok]))
        rng = np.random.default_rng(4)
        M, K = 12, 10
        Apad = wl.to_bits(rng.normal(size=(M, K + 3)), dtype)
        A = Apad[:, :K]
        C, _ = orc.gemm(A, int_bits(np.eye(K), dtype), dtype)
        checks.append(np.array_equal(C, np_decode(np.ascontiguousarray(A), dtype)))
        A2 = wl.to_bits(rng.normal(size=(M, K)), dtype)
        B2 = wl.to_bits(rng.normal(size=(K, 7)), dtype)
        C2, _ = orc.gemm(A2, B2, dtype)
        ref2 = np_decode(A2, dtype) @ np_decode(B2, dtype)
        checks.append(np.allclose(C2, ref2, rtol=0, atol=1e-12))
    return all(checks)


def test_pins_pass_on_the_real_oracle(oracle_mod):
    assert _pins_pass(oracle_mod)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(tmp_path, oracle_mod, name):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    assert not _pins_pass(_build_mutant(tmp_path, name)), "pins did not catch mutant %s" % name
