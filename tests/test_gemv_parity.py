"""GPU parity of the fp32 GEMV (xgemv_run through the C ABI) against the CPU
oracle.

Bar: |y_gpu - y_ref| <= (n 2^-24 (1 + 1e-3) + K 2^-52) s + (K + 255) 2^-150
elementwise, where s = sum_k |A[i][k] x[k]| and n = 4 ceil(K/1024) + 10.
Each operation rounds as fl(a op b) = (a op b)(1 + d) + e with |d| <= 2^-24
and |e| <= 2^-150 (e only for a subnormal result).  Every product reaches
the output through at most n operations (4 ceil(K/1024) + 1 fused
multiply-adds in its thread, 6 shuffle additions, 3 additions across
waves), which bounds the relative part; the absolute parts add up over all
K + 4 * 63 + 3 operations of the output's computation tree.  The K 2^-52
term covers the oracle's own fp64 rounding.  Bit-for-bit equality
where every partial sum is an exactly representable integer, and between
launch configurations and load widths, whose arithmetic is the same.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2609_16389_amd import workloads as wl
from paper_2609_16389_amd import xgemm as xg

pytestmark = pytest.mark.gpu

CONFIGS = [(r, u) for r in (1, 2, 4, 8) for u in (1, 2, 4)]


@pytest.fixture(scope="module", autouse=True)
def _oracle_built():
    oracle.build(force=False)


def tol(K, s, split=1):
    """The bound for a K split into `split` ranges (1: none): each range of
    at most kc values contributes 4 ceil(kc/1024) + 10 roundings, the sum
    over ranges split - 1 more."""
    kc = -(-K // split) if split > 1 else K
    n = 4 * math.ceil(kc / 1024) + 10 + (split - 1)
    return (n * 2.0 ** -24 * (1 + 1e-3) + K * 2.0 ** -52) * s + (K + 256 * split) * 2.0 ** -150


def check(y, y_ref, s, K, what, split=1):
    y = np.asarray(y, dtype=np.float64)
    assert np.all(np.isfinite(y)), what
    bad = np.abs(y - y_ref) > tol(K, s, split)
    if bad.any():
        i = int(np.argmax(bad))
        raise AssertionError("%s: %d of %d outside the bound; first row %d: gpu=%r ref=%r s=%r"
                             % (what, int(bad.sum()), bad.size, i, y[i], y_ref[i], s[i]))


def device_matrix(A, lda=None, offset=0, fill=float("nan")):
    M, K = A.shape
    lda = max(K, 1) if lda is None else lda
    buf = torch.full((offset + M * lda + 1,), fill, dtype=torch.float32)
    if M and K:
        buf[offset:offset + M * lda].view(M, lda)[:, :K] = torch.from_numpy(A)
    return buf.cuda().as_strided((M, K), (lda, 1), offset)


def device_vector(x, offset=0):
    buf = torch.full((offset + x.size + 1,), float("nan"), dtype=torch.float32)
    buf[offset:offset + x.size] = torch.from_numpy(x)
    return buf.cuda()[offset:offset + x.size]


def run(A, x, config=None, lda=None, a_offset=0, x_offset=0):
    Ad = device_matrix(A, lda, a_offset)
    xd = device_vector(x, x_offset)
    y = xg.gemv(Ad, xd, config=config)
    torch.cuda.synchronize()
    return y.cpu().numpy()


SHAPES = [(1, 1), (1, 5), (3, 4), (17, 1023), (255, 1025), (256, 4096), (1000, 3000), (4097, 777),
          (5, 100003), (3000, 8), (2, 1024 * 9 + 3), (64, 300000), (1, 262147), (200, 65536)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "%dx%d" % s)
def test_shapes_default_config(shape):
    M, K = shape
    A, x = wl.make_gemv_inputs(M, K, "uniform", M + 3 * K)
    y_ref, s = oracle.gemv(A, x)
    split = xg.xgemv_select_config(M, K, torch.cuda.get_device_properties(0).multi_processor_count).split_k
    check(run(A, x), y_ref, s, K, "gemv %dx%d" % shape, split)


@pytest.mark.parametrize("shape,split", [((64, 100003), 8), ((5, 7), 4), ((300, 5000), 3), ((1, 300000), 64),
                                         ((700, 4096), 2)], ids=lambda v: str(v))
def test_forced_k_splits(shape, split):
    """Every K split in range against the oracle; for a given split the
    result does not depend on rows, unroll or load width."""
    M, K = shape
    A, x = wl.make_gemv_inputs(M, K, "normal", 17 + split)
    y_ref, s = oracle.gemv(A, x)
    base = run(A, x, config=xg.xgemv_config(1, 4, split))
    # (when trailing ranges are empty and dropped, the bound for the
    # requested split still covers the shorter path)
    check(base, y_ref, s, K, "split %d" % split, split)
    for r, u in [(2, 1), (4, 2), (8, 4)]:
        assert np.array_equal(run(A, x, config=xg.xgemv_config(r, u, split)), base), (r, u)
    assert np.array_equal(run(A, x, config=xg.xgemv_config(1, 4, split), a_offset=1, lda=K + 3), base)


def test_every_config_is_bit_identical():
    M, K = 777, 5000
    A, x = wl.make_gemv_inputs(M, K, "normal", 9)
    y_ref, s = oracle.gemv(A, x)
    base = run(A, x)
    check(base, y_ref, s, K, "default")
    for r, u in CONFIGS:
        y = run(A, x, config=xg.xgemv_config(r, u))
        assert np.array_equal(y, base), "rows=%d unroll=%d" % (r, u)


@pytest.mark.parametrize("a_offset,lda,x_offset", [(1, None, 0), (0, 5003, 0), (0, None, 1), (2, 5001, 3)])
def test_unaligned_layouts_match_the_vector_path(a_offset, lda, x_offset):
    M, K = 300, 5000
    A, x = wl.make_gemv_inputs(M, K, "uniform", 10)
    y_ref, s = oracle.gemv(A, x)
    aligned = run(A, x)
    y = run(A, x, lda=lda, a_offset=a_offset, x_offset=x_offset)
    check(y, y_ref, s, K, "unaligned")
    assert np.array_equal(y, aligned)


def test_integer_inputs_are_exact():
    rng = np.random.default_rng(11)
    A = rng.integers(-64, 65, size=(513, 3000)).astype(np.float32)
    x = rng.integers(-64, 65, size=3000).astype(np.float32)
    y_ref, _ = oracle.gemv(A, x)
    assert np.array_equal(run(A, x).astype(np.float64), y_ref)


def test_subnormal_inputs():
    rng = np.random.default_rng(12)
    # subnormal A times 2^100: products are normal
    A = (rng.integers(1, 1 << 20, size=(64, 2000)) * rng.choice([-1, 1], size=(64, 2000))).astype(np.float64)
    A = (A * 2.0 ** -149).astype(np.float32)
    x = np.full(2000, 2.0 ** 100, dtype=np.float32)
    y_ref, s = oracle.gemv(A, x)
    check(run(A, x), y_ref, s, 2000, "subnormal A")
    # normal A times subnormal x: products and sums stay subnormal
    A2 = rng.uniform(0.5, 1.0, size=(64, 100)).astype(np.float32)
    x2 = np.full(100, 2.0 ** -140, dtype=np.float32)
    y_ref, s = oracle.gemv(A2, x2)
    y = run(A2, x2)
    assert np.all(y > 0), "subnormal products flushed to zero"
    check(y, y_ref, s, 100, "subnormal x")


def test_zero_k_and_zero_m():
    y = xg.gemv(torch.empty((7, 0), device="cuda"), torch.empty(0, device="cuda"),
                out=torch.full((7,), float("nan"), device="cuda"))
    assert torch.all(y == 0)
    y = xg.gemv(torch.empty((0, 5), device="cuda"), torch.zeros(5, device="cuda"))
    assert y.shape == (0,)


def test_output_past_m_untouched():
    A, x = wl.make_gemv_inputs(333, 700, "uniform", 13)
    y_ref, s = oracle.gemv(A, x)
    buf = torch.full((400,), float("nan"), device="cuda")
    xg.gemv(torch.from_numpy(A).cuda(), torch.from_numpy(x).cuda(), out=buf[:333])
    torch.cuda.synchronize()
    out = buf.cpu().numpy()
    check(out[:333], y_ref, s, 700, "prefix")
    assert np.all(np.isnan(out[333:]))


def test_determinism():
    A, x = wl.make_gemv_inputs(2048, 4096, "normal", 14)
    Ad, xd = torch.from_numpy(A).cuda(), torch.from_numpy(x).cuda()
    y1 = xg.gemv(Ad, xd).cpu()
    y2 = xg.gemv(Ad, xd).cpu()
    assert torch.equal(y1, y2)


def test_invalid_arguments():
    h = xg.handle()
    A = torch.zeros((4, 8), device="cuda")
    x = torch.zeros(8, device="cuda")
    y = torch.zeros(4, device="cuda")
    pa, px, py = A.data_ptr(), x.data_ptr(), y.data_ptr()
    assert xg.xgemv_run(h, 4, 8, pa, 7, px, py, None) == xg.XGEMM_ERR_INVALID_ARG      # lda < K
    assert xg.xgemv_run(h, -1, 8, pa, 8, px, py, None) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.xgemv_run(h, 4, 8, None, 8, px, py, None) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.xgemv_run(h, 4, 8, pa, 8, None, py, None) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.xgemv_run(h, 4, 8, pa, 8, px, None, None) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.xgemv_run(None, 4, 8, pa, 8, px, py, None) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.xgemv_run_config(h, 4, 8, pa, 8, px, py, None, xg.xgemv_config(3, 1)) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.xgemv_run_config(h, 4, 8, pa, 8, px, py, None, xg.xgemv_config(4, 8)) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.xgemv_run_config(h, 4, 8, pa, 8, px, py, None, None) == xg.XGEMM_ERR_INVALID_ARG


@pytest.mark.parametrize("name", ["gemv8192_fp32", "gemv16384_fp32", "gemv32768_fp32"])
def test_full_size_workloads_sampled(name):
    """The full workloads in the launch configuration the benchmark times:
    every row against the oracle is too slow for 32768^2, so edge rows and
    a seeded sample of 512 others are checked."""
    w = wl.GEMV_WORKLOADS[name]
    A, x = wl.gemv_workload_inputs(w)
    Ad, xd = torch.from_numpy(A).cuda(), torch.from_numpy(x).cuda()
    y = xg.gemv(Ad, xd).cpu().numpy()
    del Ad
    rng = np.random.default_rng(15)
    rows = np.unique(np.concatenate([[0, 1, w.M - 2, w.M - 1], rng.integers(0, w.M, size=512)]))
    y_ref, s = oracle.gemv_rows(A, x, rows)
    check(y[rows], y_ref, s, w.K, name)
    assert np.all(np.isfinite(y))
