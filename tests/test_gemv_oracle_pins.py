"""Pins of the fp32 GEMV oracle (y = A x in fp64) against what the
definition and the mathematics fix, independent of the oracle's own code:
hand-worked golden products, exact rational brute force, closed forms,
numpy's fp64 BLAS, integer arithmetic and invariants.  Planted mistakes in
a copy of the oracle must fail at least one pin."""
import ctypes
import os
import shutil
import subprocess
from fractions import Fraction

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden")


def _cases():
    cases, cur = [], None
    with open(os.path.join(GOLDEN, "gemv_worked_example.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            parts = line.split()
            if parts[0] == "case":
                cur = dict(name=parts[1], M=int(parts[2]), K=int(parts[3]), A=[], x=None, y=None, s=None)
                cases.append(cur)
            elif parts[0] == "A":
                cur["A"].append([int(t, 16) for t in parts[1:]])
            elif parts[0] == "x":
                cur["x"] = [int(t, 16) for t in parts[1:]]
            else:
                cur[parts[0]] = [Fraction(t) for t in parts[1:]]
    return cases


def f32(bits):
    return np.array(bits, dtype=np.uint32).view(np.float32)


def exact(A, x):
    """Exact y and s as Fractions (fp32 values are dyadic rationals)."""
    ys, ss = [], []
    for row in A:
        terms = [Fraction(float(a)) * Fraction(float(b)) for a, b in zip(row, x)]
        ys.append(sum(terms, Fraction(0)))
        ss.append(sum((abs(t) for t in terms), Fraction(0)))
    return ys, ss


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_worked_examples(oracle_mod, case):
    A = f32(case["A"]).reshape(case["M"], case["K"])
    x = f32(case["x"])
    y, s = oracle_mod.gemv(A, x)
    assert [Fraction(v) for v in y] == case["y"]
    assert [Fraction(v) for v in s] == case["s"]


def test_golden_values_are_the_exact_products():
    # the fixture's rationals follow from its bit patterns
    for case in _cases():
        A = f32(case["A"]).reshape(case["M"], case["K"])
        ys, ss = exact(A, f32(case["x"]))
        assert ys == case["y"] and ss == case["s"]


def test_identity_and_padding(oracle_mod):
    rng = np.random.default_rng(1)
    x = rng.normal(size=37).astype(np.float32)
    y, s = oracle_mod.gemv(np.eye(37, dtype=np.float32), x)
    assert np.array_equal(y, x.astype(np.float64)) and np.array_equal(s, np.abs(x).astype(np.float64))
    A = rng.normal(size=(9, 37 + 11)).astype(np.float32)
    y_pad, s_pad = oracle_mod.gemv(A[:, :37], x)
    y_c, s_c = oracle_mod.gemv(np.ascontiguousarray(A[:, :37]), x)
    assert np.array_equal(y_pad, y_c) and np.array_equal(s_pad, s_c)


def test_permutation_and_ones(oracle_mod):
    rng = np.random.default_rng(2)
    perm = rng.permutation(20)
    P = np.eye(20, dtype=np.float32)[perm]
    x = rng.normal(size=20).astype(np.float32)
    y, _ = oracle_mod.gemv(P, x)
    assert np.array_equal(y, x[perm].astype(np.float64))
    y, s = oracle_mod.gemv(np.ones((3, 1000), np.float32), np.ones(1000, np.float32))
    assert np.all(y == 1000) and np.all(s == 1000)


def test_rational_brute_force(oracle_mod):
    rng = np.random.default_rng(3)
    for M, K in [(1, 1), (3, 5), (4, 17), (2, 64)]:
        A = (rng.normal(size=(M, K)) * np.exp2(rng.integers(-30, 30, size=(M, K)))).astype(np.float32)
        x = (rng.normal(size=K) * np.exp2(rng.integers(-30, 30, size=K))).astype(np.float32)
        A[0, 0] = np.float32(1e-40)          # a subnormal fp32 input
        y, s = oracle_mod.gemv(A, x)
        ys, ss = exact(A, x)
        for i in range(M):
            bound = Fraction(max(K - 1, 0)) * Fraction(2) ** -53 * ss[i]
            assert abs(Fraction(y[i]) - ys[i]) <= bound
            assert abs(Fraction(s[i]) - ss[i]) <= bound


def test_numpy_fp64_blas(oracle_mod):
    rng = np.random.default_rng(4)
    A = rng.uniform(-1, 1, size=(64, 3000)).astype(np.float32)
    x = rng.uniform(-1, 1, size=3000).astype(np.float32)
    y, s = oracle_mod.gemv(A, x)
    ref = A.astype(np.float64) @ x.astype(np.float64)
    assert np.all(np.abs(y - ref) <= 1e-12 * s)
    assert np.allclose(s, np.abs(A.astype(np.float64)) @ np.abs(x.astype(np.float64)), rtol=1e-12, atol=0)


def test_small_integers_exact(oracle_mod):
    rng = np.random.default_rng(5)
    Ai = rng.integers(-100, 101, size=(30, 500))
    xi = rng.integers(-100, 101, size=500)
    y, s = oracle_mod.gemv(Ai.astype(np.float32), xi.astype(np.float32))
    assert np.array_equal(y, (Ai @ xi).astype(np.float64))
    assert np.array_equal(s, (np.abs(Ai) @ np.abs(xi)).astype(np.float64))


def test_power_of_two_scaling_is_exact(oracle_mod):
    rng = np.random.default_rng(6)
    A = rng.normal(size=(7, 300)).astype(np.float32)
    x = rng.normal(size=300).astype(np.float32)
    y1, s1 = oracle_mod.gemv(A, x)
    y2, s2 = oracle_mod.gemv(A, (x * 4).astype(np.float32))
    assert np.array_equal(y2, 4 * y1) and np.array_equal(s2, 4 * s1)


def test_empty_and_zero_k(oracle_mod):
    y, s = oracle_mod.gemv(np.zeros((5, 0), np.float32), np.zeros(0, np.float32))
    assert np.all(y == 0) and np.all(s == 0)
    y, s = oracle_mod.gemv(np.zeros((0, 4), np.float32), np.zeros(4, np.float32))
    assert y.shape == (0,)


def test_rows_match_full(oracle_mod):
    rng = np.random.default_rng(7)
    A = rng.normal(size=(40, 77)).astype(np.float32)
    x = rng.normal(size=77).astype(np.float32)
    y, s = oracle_mod.gemv(A, x)
    rows = np.array([39, 0, 17, 17])
    yr, sr = oracle_mod.gemv_rows(A, x, rows)
    assert np.array_equal(yr, y[rows]) and np.array_equal(sr, s[rows])


def test_invalid_arguments(oracle_mod):
    A = np.zeros((3, 4), np.float32)
    with pytest.raises(TypeError):
        oracle_mod.gemv(A, np.zeros(5, np.float32))
    with pytest.raises(TypeError):
        oracle_mod.gemv(A.astype(np.float64), np.zeros(4, np.float32))
    with pytest.raises(ValueError):
        oracle_mod.gemv_rows(A, np.zeros(4, np.float32), [3])


# --------------------------------------------------------------------------
# planted mistakes
# --------------------------------------------------------------------------

MUTANTS = {
    "drop_last_k": ("for (int64_t k = 0; k < K; ++k) {", "for (int64_t k = 0; k < K - 1; ++k) {"),
    "x_shifted": ("(double)a[k] * (double)x[k]", "(double)a[k] * (double)x[k > 0 ? k - 1 : 0]"),
    "lda_as_K": ("const float *a = A + rows[r] * lda;", "const float *a = A + rows[r] * K;"),
    "s_signed": ("mag += fabs(p);", "mag += p;"),
    "sum_in_fp32": ("double acc = 0.0, mag = 0.0;", "float acc = 0.0f; double mag = 0.0;"),
    "sign_flip": ("acc += p;", "acc -= p;"),
}


class _Mutant:
    def __init__(self, lib):
        import oracle as real
        self._lib, self._real = lib, real

    def gemv(self, A, x):
        saved = self._real._lib
        self._real._lib = self._lib
        try:
            return self._real.gemv(A, x)
        finally:
            self._real._lib = saved


def _build(tmp_path, name):
    src = open(os.path.join(ROOT, "oracle", "gemv_oracle.c")).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, name
    c = tmp_path / ("%s.c" % name)
    c.write_text(src.replace(old, new))
    so = tmp_path / ("lib%s.so" % name)
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", str(c),
                    "-o", str(so), "-lm"], check=True)
    import oracle as real
    lib = ctypes.CDLL(str(so))
    lib.oracle_gemv.argtypes = real._load().oracle_gemv.argtypes
    lib.oracle_gemv.restype = real._load().oracle_gemv.restype
    return _Mutant(lib)


def _pins_pass(orc):
    checks = []
    for case in _cases():
        y, s = orc.gemv(f32(case["A"]).reshape(case["M"], case["K"]), f32(case["x"]))
        checks.append([Fraction(v) for v in y] == case["y"] and [Fraction(v) for v in s] == case["s"])
    rng = np.random.default_rng(8)
    A = rng.normal(size=(6, 40 + 5)).astype(np.float32)[:, :40]
    x = rng.normal(size=40).astype(np.float32)
    y, s = orc.gemv(A, x)
    ref = A.astype(np.float64) @ x.astype(np.float64)
    checks.append(bool(np.all(np.abs(y - ref) <= 1e-12 * s)))
    checks.append(bool(np.allclose(s, np.abs(A.astype(np.float64)) @ np.abs(x.astype(np.float64)), rtol=1e-12)))
    return all(checks)


def test_pins_pass_on_the_real_oracle(oracle_mod):
    assert _pins_pass(oracle_mod)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(tmp_path, oracle_mod, name):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    assert not _pins_pass(_build(tmp_path, name)), name
