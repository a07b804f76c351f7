"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bar: |C_gpu - C_ref| <= 1e-4 * sum_k |a_ik b_kj| elementwise, no NaN; and
bit-for-bit equality where the exact result is representable and every
partial sum is exact in fp32 (small integers, identity, permutations).
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import (CODE, check_close, check_exact, config, empty_out, run_gpu, to_device)
from paper_2609_16389_amd import workloads as wl
from paper_2609_16389_amd import xgemm as xg

pytestmark = pytest.mark.gpu

TILES = list(range(xg.XGEMM_TILE_COUNT))


@pytest.fixture(scope="module", autouse=True)
def _oracle_built():
    oracle.build(force=False)


def _case(M, N, K, dtype, seed, dist="uniform"):
    A, B = wl.make_inputs(M, N, K, dtype, dist, seed)
    C_ref, S = oracle.gemm(A, B, dtype)
    return A, B, C_ref, S


# ---------------------------------------------------------------------------
# small and ragged shapes, every tile, both dtypes
# ---------------------------------------------------------------------------

RAGGED = [(1, 1, 1), (17, 33, 65), (64, 64, 64), (255, 257, 129), (300, 520, 200),
          (513, 129, 1000), (1000, 1000, 1000)]


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("shape", RAGGED, ids=lambda s: "x".join(map(str, s)))
def test_ragged_default_config(dtype, shape):
    M, N, K = shape
    A, B, C_ref, S = _case(M, N, K, dtype, seed=M * 7 + N)
    check_close(run_gpu(A, B, dtype), C_ref, S, "default %s %s" % (dtype, shape))


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("shape", [(256, 256, 256), (255, 257, 129), (520, 300, 700)],
                         ids=lambda s: "x".join(map(str, s)))
def test_every_tile(tile, shape):
    M, N, K = shape
    for dtype in ("bf16", "fp16"):
        A, B, C_ref, S = _case(M, N, K, dtype, seed=tile + 11)
        check_close(run_gpu(A, B, dtype, config=config(tile)), C_ref, S, "tile %d %s" % (tile, dtype))


def test_workload_256_fp16_full():
    """The 256^3 fp16 workload (uniform[-1,1], seed 0), every element."""
    w = wl.WORKLOADS["gemm256_fp16"]
    A, B = wl.workload_inputs(w)
    C_ref, S = oracle.gemm(A, B, w.dtype)
    check_close(run_gpu(A, B, w.dtype), C_ref, S, w.name)


# ---------------------------------------------------------------------------
# the pipelined (direct-to-LDS) kernels: ragged M, N a multiple of 8
# ---------------------------------------------------------------------------

def _family(M, N, K, cfg):
    return xg.xgemm_kernel_family(M, N, K, 1 << 20, K, 1 << 20, N, cfg)


PIPE_SHAPES = [(256, 256, 192), (1000, 1000, 1024), (255, 264, 512), (777, 136, 4096), (64, 520, 320)]


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("shape", PIPE_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_pipelined_shapes(tile, shape):
    M, N, K = shape
    assert _family(M, N, K, config(tile)) == xg.XGEMM_KERNEL_PIPELINED
    for dtype in ("bf16", "fp16"):
        A, B, C_ref, S = _case(M, N, K, dtype, seed=M + tile)
        check_close(run_gpu(A, B, dtype, config=config(tile)), C_ref, S,
                    "pipelined tile %d %s %s" % (tile, dtype, shape))


# K a multiple of 8 but not of the K step: the pipelined kernels run the
# partial last step first and zero the LDS beyond K
PARTIAL_SHAPES = [(256, 256, 200), (1000, 1000, 1000), (300, 264, 3000), (777, 136, 4104)]


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("shape", PARTIAL_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_partial_k_step(tile, shape):
    M, N, K = shape
    assert _family(M, N, K, config(tile)) == xg.XGEMM_KERNEL_PIPELINED
    for dtype in ("bf16", "fp16"):
        A, B, C_ref, S = _case(M, N, K, dtype, seed=K + tile)
        check_close(run_gpu(A, B, dtype, config=config(tile)), C_ref, S,
                    "partial step tile %d %s %s" % (tile, dtype, shape))


# The 256 x 128 tile's two waves per block split every K step, and its K
# loop is instantiated per parity of the number of steps that issue loads
# (nk - 3): every step count from the pipeline's minimum of 3 to 9, with and
# without a partial last step, so both parities, the shortest loops and the
# loop-free case all run.
@pytest.mark.parametrize("K", [192, 256, 320, 384, 448, 512, 576, 200, 264, 328])
def test_wave_pair_step_counts(K):
    M, N = 300, 264
    assert _family(M, N, K, config(1)) == xg.XGEMM_KERNEL_PIPELINED
    for dtype in ("bf16", "fp16"):
        A, B, C_ref, S = _case(M, N, K, dtype, seed=K + 7)
        check_close(run_gpu(A, B, dtype, config=config(1)), C_ref, S, "wave pairs %s K=%d" % (dtype, K))


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_partial_k_step_never_reads_past_k(tile, dtype):
    """A's row padding past K holds NaN: any read of it would poison C."""
    M, N, K = 384, 320, 1000
    A, B, C_ref, S = _case(M, N, K, dtype, seed=31 + tile)
    nan = 0x7E00 if dtype == "fp16" else 0x7FC0
    C = run_gpu(A, B, dtype, config=config(tile), lda=K + 24, ldb=N + 8, pad=nan)
    check_close(C, C_ref, S, "NaN padding past K, tile %d" % tile)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_partial_k_step_integer_bit_exact(dtype):
    M, N, K = 520, 264, 2056
    A, B = wl.make_int_inputs(M, N, K, dtype, seed=32)
    assert _family(M, N, K, config(0)) == xg.XGEMM_KERNEL_PIPELINED
    C_ref, _ = oracle.gemm(A, B, dtype)
    check_exact(run_gpu(A, B, dtype), C_ref, "integer, partial step")


@pytest.mark.parametrize("tile,split", [(0, 3), (1, 8), (2, 4)])
def test_partial_k_step_in_last_split(tile, split):
    M, N, K = 384, 320, 8200
    assert _family(M, N, K, config(tile, split)) == xg.XGEMM_KERNEL_PIPELINED
    A, B, C_ref, S = _case(M, N, K, "bf16", seed=33 + split)
    check_close(run_gpu(A, B, "bf16", config=config(tile, split)), C_ref, S,
                "partial last split tile %d split %d" % (tile, split))


# Layouts the pipelined kernels cannot read in place:
# the library copies the operand(s) into its workspace, zero-padded
PACKED_CASES = {
    "n_odd": ((1000, 1001, 1024), {}),
    "k_odd": ((1000, 1000, 1003), {}),
    "lda_not_x8": ((1024, 1000, 1024), {"lda": 1028}),
    "ldb_not_x8": ((1000, 1024, 1024), {"ldb": 1027}),
    "misaligned_pointers": ((1000, 1000, 1024), {"offset": 1}),
    "everything_odd": ((1023, 1021, 1019), {"lda": 1022, "ldb": 1024}),
}


@pytest.mark.parametrize("name", sorted(PACKED_CASES))
@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_packed_operands(name, dtype):
    (M, N, K), kw = PACKED_CASES[name]
    lda, ldb, off = kw.get("lda", K), kw.get("ldb", N), kw.get("offset", 0)
    base = (1 << 20) + 2 * off
    assert xg.xgemm_kernel_family(M, N, K, base, lda, base, ldb, xg.xgemm_select_config(M, N, K, CODE[dtype], 256)) \
        == xg.XGEMM_KERNEL_PIPELINED
    A, B, C_ref, S = _case(M, N, K, dtype, seed=M + N + K)
    nan = 0x7E00 if dtype == "fp16" else 0x7FC0
    check_close(run_gpu(A, B, dtype, lda=lda, ldb=ldb, offset=off, pad=nan), C_ref, S,
                "packed %s %s" % (name, dtype))


@pytest.mark.parametrize("tile,split", [(0, 2), (1, 3), (2, 4)])
def test_packed_operands_split_k(tile, split):
    M, N, K = 520, 601, 1533
    A, B, C_ref, S = _case(M, N, K, "bf16", seed=41 + split)
    check_close(run_gpu(A, B, "bf16", config=config(tile, split), lda=K + 3), C_ref, S,
                "packed split tile %d split %d" % (tile, split))


def test_packed_operands_integer_bit_exact():
    M = N = K = 2047
    A, B = wl.make_int_inputs(M, N, K, "bf16", seed=42)
    C_ref, _ = oracle.gemm(A, B, "bf16")
    check_exact(run_gpu(A, B, "bf16"), C_ref, "integer, packed 2047^3")


def test_packed_then_aligned_calls_share_a_handle():
    """A packed call grows the workspace; aligned calls after it (and another
    packed call with a smaller shape) still see their own operands."""
    cases = [(1000, 1001, 1024, 1), (512, 512, 512, 2), (700, 703, 705, 3)]
    for M, N, K, seed in cases:
        A, B, C_ref, S = _case(M, N, K, "fp16", seed=seed)
        check_close(run_gpu(A, B, "fp16"), C_ref, S, "sequence %dx%dx%d" % (M, N, K))


@pytest.mark.parametrize("split", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("tile", TILES)
def test_pipelined_split_k(split, tile):
    M, N, K = 384, 320, 8192
    assert _family(M, N, K, config(tile, split)) == xg.XGEMM_KERNEL_PIPELINED
    A, B, C_ref, S = _case(M, N, K, "bf16", seed=split + 100)
    check_close(run_gpu(A, B, "bf16", config=config(tile, split)), C_ref, S,
                "pipelined tile %d split %d" % (tile, split))


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_pipelined_integer_bit_exact(dtype):
    M, N, K = 520, 264, 2048
    A, B = wl.make_int_inputs(M, N, K, dtype, seed=77)
    C_ref, _ = oracle.gemm(A, B, dtype)
    for tile in TILES:
        assert _family(M, N, K, config(tile)) == xg.XGEMM_KERNEL_PIPELINED
        check_exact(run_gpu(A, B, dtype, config=config(tile)), C_ref, "pipelined tile %d" % tile)


# ---------------------------------------------------------------------------
# split-k (the paper tries split factors 1, 2, 4, 8, 16)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("split", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("tile", TILES)
def test_split_k_factors(split, tile):
    M, N, K = 384, 320, 4100  # K not a multiple of 32: the general kernel
    A, B, C_ref, S = _case(M, N, K, "bf16", seed=split)
    check_close(run_gpu(A, B, "bf16", config=config(tile, split)), C_ref, S,
                "tile %d split %d" % (tile, split))


@pytest.mark.parametrize("split", [2, 16])
def test_split_k_integer_exact(split):
    M, N, K = 200, 136, 2048
    A, B = wl.make_int_inputs(M, N, K, "fp16", seed=split)
    C_ref, _ = oracle.gemm(A, B, "fp16")
    check_exact(run_gpu(A, B, "fp16", config=config(xg.XGEMM_TILE_128x128, split)), C_ref)


# ---------------------------------------------------------------------------
# the persistent stream-K kernel (xgemm_config.stream_k)
# ---------------------------------------------------------------------------

def _sk_cfg(grid=1):
    """The 256 x 256 tile as the persistent kernel: grid 1 = one workgroup
    per CU, n > 1 = n workgroups."""
    return config(xg.XGEMM_TILE_256x256, 1, 4, grid)


def _cu():
    return torch.cuda.get_device_properties(0).multi_processor_count


def _sk_info(M, N, K, cfg):
    return xg.xgemm_trace_plan(M, N, K, 1 << 40, K, 2 << 40, N, 3 << 40, N, cfg, _cu(), 0)


def _logical_tile(t, tiles_m, tiles_n, group_m):
    group = group_m * tiles_n
    g = t // group
    first_m = g * group_m
    gm = min(tiles_m - first_m, group_m)
    r = t - g * group
    return first_m + r % gm, r // gm


def _split_tiles(info, M, N, group_m=4):
    """(tile row, tile column) of every tile the plan splits between two
    workgroups' ranges."""
    P, kt = info.grid, info.kt
    isk = info.sk_tiles * kt
    out = []
    for lw in range(1, P):
        s0 = isk * lw // P
        if s0 % kt:
            out.append(_logical_tile(info.dp_rounds * P + s0 // kt, M // 256, N // 256, group_m))
    return out


# (M, N, K, workgroups): rounds of whole tiles, then shared ranges of
# various lengths (1 to 2 tiles, K steps per tile 3 to 16), split tiles in
# every position
SK_GRIDS = [(1024, 1280, 1024, 3), (1024, 1280, 1024, 7), (1024, 1280, 1024, 8), (1024, 1280, 1024, 13),
            (768, 768, 320, 4), (512, 768, 384, 4), (2048, 2048, 768, 24), (2048, 2048, 768, 60),
            (1536, 2560, 512, 16)]


@pytest.mark.parametrize("shape", SK_GRIDS, ids=lambda s: "%dx%dx%d_g%d" % s)
def test_persistent_kernel_small_grids(shape):
    M, N, K, grid = shape
    info = _sk_info(M, N, K, _sk_cfg(grid))
    assert info.family == xg.XGEMM_KERNEL_PERSISTENT and info.grid == grid
    for dtype in ("bf16", "fp16"):
        A, B, C_ref, S = _case(M, N, K, dtype, seed=grid + K)
        check_close(run_gpu(A, B, dtype, config=_sk_cfg(grid)), C_ref, S, "persistent %s %s" % (shape, dtype))


@pytest.mark.parametrize("shape", [(1024, 1280, 1024, 7), (2048, 2048, 768, 60)], ids=lambda s: "%dx%dx%d_g%d" % s)
def test_persistent_kernel_integer_exact_and_deterministic(shape):
    """Small-integer inputs: exact whatever the grouping; and real-valued
    inputs give the same bits on every run (a split tile is always its first
    K steps plus its last, whichever workgroup finishes it)."""
    M, N, K, grid = shape
    A, B = wl.make_int_inputs(M, N, K, "bf16", seed=grid)
    C_ref, _ = oracle.gemm(A, B, "bf16")
    check_exact(run_gpu(A, B, "bf16", config=_sk_cfg(grid)), C_ref, "persistent integer %s" % (shape,))
    A, B = wl.make_inputs(M, N, K, "fp16", "uniform", seed=grid + 1)
    runs = [run_gpu(A, B, "fp16", config=_sk_cfg(grid)) for _ in range(4)]
    for r in runs[1:]:
        assert np.array_equal(r, runs[0])


def test_persistent_kernel_counters_left_zero():
    """A split tile's finisher resets its counter: calls that follow on the
    same handle -- persistent ones, and split-k and copied-operand calls that
    use the workspace after its counters -- all stay correct."""
    h = xg.xgemm_create()
    try:
        s = torch.cuda.current_stream().cuda_stream
        cases = [(1024, 1280, 1024, _sk_cfg(7), 61), (512, 520, 4096, config(xg.XGEMM_TILE_128x128, 4), 62),
                 (1024, 1280, 1024, _sk_cfg(13), 63), (1000, 1001, 1024, None, 64), (2048, 2048, 768, _sk_cfg(60), 65)]
        for rep in range(2):
            for M, N, K, cfg, seed in cases:
                A, B, C_ref, S = _case(M, N, K, "bf16", seed=seed)
                dA, dB = to_device(A, "bf16"), to_device(B, "bf16")
                C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
                args = (h, M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, C.data_ptr(), N, xg.XGEMM_BF16, s)
                rc = xg.xgemm_run(*args) if cfg is None else xg.xgemm_run_config(*args, cfg)
                assert rc == xg.XGEMM_OK, xg.xgemm_last_error(h)
                torch.cuda.synchronize()
                check_close(C.cpu().numpy(), C_ref, S, "sequence %d %dx%dx%d" % (rep, M, N, K))
    finally:
        xg.xgemm_destroy(h)


@pytest.mark.parametrize("shape", [(1000, 1280, 1024), (1024, 1000, 1024), (1024, 1280, 1000), (1024, 1024, 65536 // 16)],
                         ids=lambda s: "x".join(map(str, s)))
def test_persistent_kernel_falls_back(shape):
    """Where the persistent kernel does not apply (M or N not whole tiles, K
    not whole steps, fewer tiles than CUs) the tile's ordinary kernel runs."""
    M, N, K = shape
    cfg = _sk_cfg(1)
    assert xg.xgemm_kernel_family(M, N, K, 1 << 20, K, 1 << 20, N, cfg) != xg.XGEMM_KERNEL_PERSISTENT
    A, B, C_ref, S = _case(M, N, K, "bf16", seed=K % 97)
    check_close(run_gpu(A, B, "bf16", config=cfg), C_ref, S, "fallback %s" % (shape,))


SK_BIG = [("gemm4096_bf16", 1), ("gemm8192_bf16", 1), ("proj16384x5120x4096_fp16", 1),
          ("proj4096x14336x4096_fp16", 1),
          # 16 tiles of K = 65536 on 12 workgroups: ranges of 1.33 tiles (1365 K steps)
          ("skinny1024x1024x65536_bf16", 12)]


@pytest.mark.parametrize("name,grid", SK_BIG, ids=lambda v: str(v))
def test_persistent_kernel_full_size_sampled(name, grid):
    """The full-size workloads through the persistent kernel on every CU (the
    skinny one, with fewer tiles than CUs, on 12 workgroups): sampled rows,
    columns and entries, plus every element of up to three split tiles
    (their two pieces meet in the hand-over) and of the first and last
    tile."""
    w = wl.WORKLOADS[name]
    cfg = _sk_cfg(grid)
    info = _sk_info(w.M, w.N, w.K, cfg)
    assert info.family == xg.XGEMM_KERNEL_PERSISTENT
    A, B = wl.workload_inputs(w)
    C = run_gpu(A, B, w.dtype, config=cfg)
    rng = np.random.default_rng(4321)
    rows = np.unique(np.concatenate([[0, w.M - 1], rng.integers(0, w.M, 4)]))
    Cr, Sr = oracle.gemm_rows(A, B, w.dtype, rows)
    check_close(C[rows], Cr, Sr, "%s rows" % name)
    ri, ci = rng.integers(0, w.M, 4096), rng.integers(0, w.N, 4096)
    c, s = oracle.gemm_entries(A, B, w.dtype, ri, ci)
    check_close(C[ri, ci][None], c[None], s[None], "%s entries" % name)
    tiles = _split_tiles(info, w.M, w.N)
    picks = [tiles[0], tiles[len(tiles) // 2], tiles[-1]] if tiles else []
    picks += [(0, 0), (w.M // 256 - 1, w.N // 256 - 1)]
    for tm, tn in picks:
        ri = np.repeat(np.arange(tm * 256, tm * 256 + 256), 256)
        ci = np.tile(np.arange(tn * 256, tn * 256 + 256), 256)
        c, s = oracle.gemm_entries(A, B, w.dtype, ri, ci)
        check_close(C[ri, ci].reshape(256, 256), c.reshape(256, 256), s.reshape(256, 256),
                    "%s tile (%d, %d)" % (name, tm, tn))
    if name == "proj4096x14336x4096_fp16":
        assert len(tiles) == 128


# ---------------------------------------------------------------------------
# exact cases
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("shape", [(128, 128, 128), (333, 260, 1111), (512, 768, 2048)],
                         ids=lambda s: "x".join(map(str, s)))
def test_small_integers_bit_exact(dtype, shape):
    M, N, K = shape
    A, B = wl.make_int_inputs(M, N, K, dtype, seed=K)
    C_ref, _ = oracle.gemm(A, B, dtype)
    for tile in TILES:
        check_exact(run_gpu(A, B, dtype, config=config(tile)), C_ref, "tile %d" % tile)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_identity_bit_exact(dtype):
    M, K = 300, 264
    A, _ = wl.make_inputs(M, 1, K, dtype, "normal", seed=3)
    I = wl.to_bits(np.eye(K), dtype)
    C_ref, _ = oracle.gemm(A, I, dtype)
    check_exact(run_gpu(A, I, dtype), C_ref, "A*I")
    I_M = wl.to_bits(np.eye(M), dtype)
    C_ref2, _ = oracle.gemm(I_M, A, dtype)
    check_exact(run_gpu(I_M, A, dtype), C_ref2, "I*A")


def test_permutation_bit_exact():
    rng = np.random.default_rng(5)
    M, K = 256, 512
    A, _ = wl.make_inputs(M, 1, K, "bf16", "uniform", seed=8)
    P = np.zeros((K, K))
    P[np.arange(K), rng.permutation(K)] = 1.0
    Pb = wl.to_bits(P, "bf16")
    C_ref, _ = oracle.gemm(A, Pb, "bf16")
    check_exact(run_gpu(A, Pb, "bf16"), C_ref, "A*P")


def test_fp16_subnormals():
    # every A entry subnormal, B powers of two: each product exact in fp32
    rng = np.random.default_rng(6)
    M, N, K = 128, 96, 256
    A = rng.integers(1, 1024, size=(M, K)).astype(np.uint16) | (rng.integers(0, 2, size=(M, K)) << 15).astype(np.uint16)
    B = wl.to_bits(2.0 ** rng.integers(-2, 8, size=(K, N)), "fp16")
    C_ref, S = oracle.gemm(A, B, "fp16")
    C = run_gpu(A, B, "fp16")
    check_close(C, C_ref, S, "subnormal")
    assert np.count_nonzero(C) > 0.9 * C.size


# ---------------------------------------------------------------------------
# layouts, alignment, degenerate sizes
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_padded_leading_dimensions(dtype):
    M, N, K = 260, 300, 200
    A, B, C_ref, S = _case(M, N, K, dtype, seed=21)
    out = empty_out(M, N, ldc=N + 12)
    C = run_gpu(A, B, dtype, lda=K + 24, ldb=N + 8, out=out)
    check_close(C, C_ref, S, "padded ld")


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_unaligned_pointers_and_odd_leading_dimensions(dtype):
    M, N, K = 131, 77, 95
    A, B, C_ref, S = _case(M, N, K, dtype, seed=22)
    out = empty_out(M, N, ldc=N + 1, offset=1)
    C = run_gpu(A, B, dtype, lda=K + 3, ldb=N + 1, offset=1, out=out)
    check_close(C, C_ref, S, "unaligned")


def test_output_padding_untouched():
    M, N, K = 64, 40, 64
    A, B, C_ref, S = _case(M, N, K, "bf16", seed=23)
    out = empty_out(M, N, ldc=N + 8, fill=123.0)
    run_gpu(A, B, "bf16", out=out)
    full = out.as_strided((M, N + 8), (N + 8, 1)).cpu().numpy()
    assert np.all(full[:, N:] == 123.0)
    check_close(full[:, :N], C_ref, S)


def test_zero_k_gives_zero():
    A = torch.empty((5, 0), dtype=torch.bfloat16, device="cuda")
    B = torch.empty((0, 7), dtype=torch.bfloat16, device="cuda")
    out = empty_out(5, 7, fill=9.0)
    xg.gemm(A, B, out=out)
    torch.cuda.synchronize()
    assert torch.all(out == 0)


def test_empty_m_or_n_is_noop():
    A = torch.ones((0, 16), dtype=torch.float16, device="cuda")
    B = torch.ones((16, 8), dtype=torch.float16, device="cuda")
    assert xg.gemm(A, B).shape == (0, 8)
    A2 = torch.ones((4, 16), dtype=torch.float16, device="cuda")
    B2 = torch.ones((16, 0), dtype=torch.float16, device="cuda")
    assert xg.gemm(A2, B2).shape == (4, 0)
    torch.cuda.synchronize()


def test_invalid_arguments_on_gpu():
    h = xg.handle()
    A = torch.zeros((4, 4), dtype=torch.bfloat16, device="cuda")
    C = torch.zeros((4, 4), dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    a, c = A.data_ptr(), C.data_ptr()
    assert xg.xgemm_run(h, 4, 4, 4, a, 3, a, 4, c, 4, 0, s) == xg.XGEMM_ERR_INVALID_ARG  # lda < K
    assert xg.xgemm_run(h, 4, 4, 4, a, 4, a, 4, c, 3, 0, s) == xg.XGEMM_ERR_INVALID_ARG  # ldc < N
    assert xg.xgemm_run(h, 4, 4, 4, a, 4, a, 4, c, 4, 5, s) == xg.XGEMM_ERR_INVALID_ARG  # dtype
    assert xg.xgemm_run(h, -1, 4, 4, a, 4, a, 4, c, 4, 0, s) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.xgemm_run(h, 4, 4, 4, None, 4, a, 4, c, 4, 0, s) == xg.XGEMM_ERR_INVALID_ARG
    bad = config(xg.XGEMM_TILE_COUNT)
    assert xg.xgemm_run_config(h, 4, 4, 4, a, 4, a, 4, c, 4, 0, s, bad) == xg.XGEMM_ERR_INVALID_ARG
    bad = config(0, split=0)
    assert xg.xgemm_run_config(h, 4, 4, 4, a, 4, a, 4, c, 4, 0, s, bad) == xg.XGEMM_ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.all(C == 0)  # nothing was enqueued


def test_workspace_allocation_failure():
    """A call whose workspace would exceed the handle's limit fails with
    XGEMM_ERR_ALLOC before anything is enqueued (C untouched), calls that
    need no workspace still run, and the handle is usable once the limit is
    lifted.  All buffers are sized for the calls made."""
    h = xg.xgemm_create()
    try:
        M, N, K = 256, 256, 1024
        Ab, Bb, C_ref, S = _case(M, N, K, "bf16", seed=90)
        Ad, Bd = to_device(Ab, "bf16"), to_device(Bb, "bf16")
        C = torch.full((M, N), 7.0, dtype=torch.float32, device="cuda")
        s = torch.cuda.current_stream().cuda_stream
        split4 = config(xg.XGEMM_TILE_128x128, 4)
        assert xg.xgemm_workspace_bytes(M, N, K, 256, split4) == 4096 + 4 * M * N * 4
        assert xg.xgemm_set_workspace_limit(h, 4096) == xg.XGEMM_OK
        assert xg.xgemm_set_workspace_limit(None, 4096) == xg.XGEMM_ERR_INVALID_ARG
        rc = xg.xgemm_run_config(h, M, N, K, Ad.data_ptr(), K, Bd.data_ptr(), N, C.data_ptr(), N, 0, s, split4)
        assert rc == xg.XGEMM_ERR_ALLOC
        assert "workspace" in xg.xgemm_last_error(h)
        torch.cuda.synchronize()
        assert torch.all(C == 7.0)
        # an unsplit aligned call needs no workspace
        assert xg.xgemm_run_config(h, M, N, K, Ad.data_ptr(), K, Bd.data_ptr(), N, C.data_ptr(), N, 0, s,
                                   config(xg.XGEMM_TILE_128x128, 1)) == xg.XGEMM_OK
        torch.cuda.synchronize()
        check_close(C.cpu().numpy(), C_ref, S, "unsplit under a workspace limit")
        # lifted: the split call runs
        C.fill_(7.0)
        assert xg.xgemm_set_workspace_limit(h, 0) == xg.XGEMM_OK
        assert xg.xgemm_run_config(h, M, N, K, Ad.data_ptr(), K, Bd.data_ptr(), N, C.data_ptr(), N, 0, s,
                                   split4) == xg.XGEMM_OK
        torch.cuda.synchronize()
        check_close(C.cpu().numpy(), C_ref, S, "after an allocation failure")
    finally:
        xg.xgemm_destroy(h)


def _two_stream_cases():
    """Two calls that both use a workspace: a forced 4-way K split (partials
    in the workspace) and a packed B (N odd: B copied into the workspace)."""
    split = (512, 512, 4096, config(xg.XGEMM_TILE_128x128, 4), 71)
    packed = (1000, 1001, 1024, None, 72)
    out = []
    for M, N, K, cfg, seed in (split, packed):
        A, B, C_ref, S = _case(M, N, K, "bf16", seed=seed)
        out.append((M, N, K, cfg, to_device(A, "bf16"), to_device(B, "bf16"), C_ref, S))
    return out


def test_two_streams_own_handles_concurrent():
    """Split-k and packed-operand calls through gemm() on two torch streams
    at once, several rounds without synchronisation in between: the binding
    keys its handles on (device, stream), so each stream writes its own
    workspace.  Every result matches the oracle elementwise."""
    cases = _two_stream_cases()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [[torch.full((M, N), float("nan"), device="cuda") for (M, N, *_ ) in cases] for _ in streams]
    torch.cuda.synchronize()
    assert xg.handle(0, streams[0]) != xg.handle(0, streams[1])
    for _ in range(4):
        for si, st in enumerate(streams):
            with torch.cuda.stream(st):
                for ci, (M, N, K, cfg, dA, dB, _, _) in enumerate(cases):
                    xg.gemm(dA, dB, out=outs[si][ci], config=cfg, stream=st)
    torch.cuda.synchronize()
    for si in range(2):
        for ci, (M, N, K, cfg, dA, dB, C_ref, S) in enumerate(cases):
            check_close(outs[si][ci].cpu().numpy(), C_ref, S, "stream %d case %d" % (si, ci))


def test_two_streams_share_one_handle():
    """The same calls through one C handle on two streams, enqueued without
    synchronisation: the handle makes each workspace user wait for the last
    one on the other stream, so the shared workspace is never written by two
    calls at once.  Every result matches the oracle elementwise."""
    cases = _two_stream_cases()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    h = xg.xgemm_create()
    try:
        outs = [[torch.full((M, N), float("nan"), device="cuda") for (M, N, *_ ) in cases] for _ in streams]
        torch.cuda.synchronize()
        for _ in range(4):
            for ci, (M, N, K, cfg, dA, dB, _, _) in enumerate(cases):
                for si, st in enumerate(streams):
                    args = (h, M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, outs[si][ci].data_ptr(), N,
                            xg.XGEMM_BF16, st.cuda_stream)
                    rc = xg.xgemm_run(*args) if cfg is None else xg.xgemm_run_config(*args, cfg)
                    assert rc == xg.XGEMM_OK, xg.xgemm_last_error(h)
        torch.cuda.synchronize()
        for si in range(2):
            for ci, (M, N, K, cfg, dA, dB, C_ref, S) in enumerate(cases):
                check_close(outs[si][ci].cpu().numpy(), C_ref, S, "shared handle, stream %d case %d" % (si, ci))
    finally:
        torch.cuda.synchronize()
        xg.xgemm_destroy(h)


def test_own_handle_lifecycle_and_stream():
    h = xg.xgemm_create()
    try:
        M, N, K = 200, 300, 400
        A, B, C_ref, S = _case(M, N, K, "fp16", seed=31)
        dA, dB = to_device(A, "fp16"), to_device(B, "fp16")
        C = torch.empty((M, N), dtype=torch.float32, device="cuda")
        st = torch.cuda.Stream()
        with torch.cuda.stream(st):
            rc = xg.xgemm_run_config(h, M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, C.data_ptr(), N,
                                     xg.XGEMM_FP16, st.cuda_stream, config(xg.XGEMM_TILE_256x256, 4))
            assert rc == xg.XGEMM_OK, xg.xgemm_last_error(h)
        st.synchronize()
        check_close(C.cpu().numpy(), C_ref, S, "own handle")
    finally:
        assert xg.xgemm_destroy(h) == xg.XGEMM_OK


def test_run_to_run_deterministic():
    M, N, K = 512, 512, 8192
    A, B = wl.make_inputs(M, N, K, "bf16", "normal", seed=41)
    for cfg in (None, config(xg.XGEMM_TILE_128x128, 8)):
        c1 = run_gpu(A, B, "bf16", config=cfg)
        c2 = run_gpu(A, B, "bf16", config=cfg)
        assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32))


def test_transpose_identity():
    M, N, K = 320, 192, 640
    A, B, C_ref, S = _case(M, N, K, "bf16", seed=51)
    Ct = run_gpu(np.ascontiguousarray(B.T), np.ascontiguousarray(A.T), "bf16")
    check_close(Ct.T, C_ref, S, "(B^T A^T)^T")


# ---------------------------------------------------------------------------
# full-size workloads in the configuration the benchmark times; outputs
# sampled (whole rows, whole columns, scattered entries) and checked one by
# one against the oracle
# ---------------------------------------------------------------------------

BIG = ["gemm4096_bf16", "gemm8192_bf16", "proj16384x5120x4096_fp16", "proj4096x14336x4096_fp16",
       "skinny1024x1024x65536_bf16"]


@pytest.mark.parametrize("name", BIG)
def test_full_size_workload_sampled(name):
    w = wl.WORKLOADS[name]
    A, B = wl.workload_inputs(w)
    C = run_gpu(A, B, w.dtype)
    rng = np.random.default_rng(1234)
    rows = np.unique(np.concatenate([[0, w.M - 1], rng.integers(0, w.M, 6)]))
    Cr, Sr = oracle.gemm_rows(A, B, w.dtype, rows)
    check_close(C[rows], Cr, Sr, "%s rows" % name)
    cols = np.unique(np.concatenate([[0, w.N - 1], rng.integers(0, w.N, 6)]))
    ri = np.repeat(np.arange(w.M), cols.size)
    ci = np.tile(cols, w.M)
    c, s = oracle.gemm_entries(A, B, w.dtype, ri, ci)
    check_close(C[ri, ci].reshape(w.M, cols.size), c.reshape(w.M, cols.size), s.reshape(w.M, cols.size),
                "%s cols" % name)
    ri = rng.integers(0, w.M, 4096)
    ci = rng.integers(0, w.N, 4096)
    c, s = oracle.gemm_entries(A, B, w.dtype, ri, ci)
    check_close(C[ri, ci][None], c[None], s[None], "%s entries" % name)


def test_full_size_8192_every_element():
    """The 8192^3 bf16 benchmark workload (uniform[-1,1], seed 2) in the
    benchmark's plan: every one of the 67M outputs against the oracle's full
    product (about 30 s of host time on 16 cores)."""
    w = wl.WORKLOADS["gemm8192_bf16"]
    A, B = wl.workload_inputs(w)
    C = run_gpu(A, B, w.dtype)
    C_ref, S = oracle.gemm(A, B, w.dtype)
    check_close(C, C_ref, S, "8192^3 every element")


def test_full_size_8192_integer_every_element():
    """8192^3 with integer entries in [-8, 8], every output bit-exact against
    the oracle's full product."""
    M = N = K = 8192
    A, B = wl.make_int_inputs(M, N, K, "bf16", seed=2)
    C = run_gpu(A, B, "bf16")
    C_ref, _ = oracle.gemm(A, B, "bf16")
    check_exact(C, C_ref, "8192^3 integer every element")


def test_full_size_8192_integer_exact_sampled():
    """8192^3 with integer entries in [-8, 8]: every partial sum is an integer
    below 2^24, so the fp32 result must equal the oracle exactly."""
    M = N = K = 8192
    A, B = wl.make_int_inputs(M, N, K, "bf16", seed=2)
    C = run_gpu(A, B, "bf16")
    rng = np.random.default_rng(99)
    rows = rng.integers(0, M, 4)
    Cr, _ = oracle.gemm_rows(A, B, "bf16", rows)
    check_exact(C[rows], Cr, "int rows")
    ri, ci = rng.integers(0, M, 4096), rng.integers(0, N, 4096)
    c, _ = oracle.gemm_entries(A, B, "bf16", ri, ci)
    check_exact(C[ri, ci][None], c[None], "int entries")


# ---------------------------------------------------------------------------
# body + band plans: xgemm_run cutting C in two launches
# ---------------------------------------------------------------------------

# (M, N, K, dtype): bands of columns, of rows, and one with both operands
# copied (N and M odd)
BANDED = [(2560, 6656, 1000, "bf16"), (3072, 5632, 1024, "fp16"), (9472, 2048, 1000, "bf16"),
          (2047, 10239, 1000, "fp16"), (4096, 6144, 1000, "bf16")]   # the last: a band of 256 x 128 wave-pair tiles


def _band_or_skip(M, N, K, dtype):
    cu = torch.cuda.get_device_properties(0).multi_processor_count
    b = xg.xgemm_select_band(M, N, K, CODE[dtype], cu)
    if b.axis == xg.XGEMM_BAND_NONE:
        pytest.skip("the selector takes no band for this shape on a %d-CU device" % cu)
    return b


def _cut_samples(b, M, N, rng):
    """Rows and columns to check: the edges of C, both sides of the cut and
    a few random ones."""
    rows = [0, M - 1] + list(rng.integers(0, M, 4))
    cols = [0, N - 1] + list(rng.integers(0, N, 4))
    if b.axis == xg.XGEMM_BAND_ROWS:
        rows += [b.extent - 1, b.extent]
    else:
        cols += [b.extent - 1, b.extent]
    return np.unique(rows), np.unique(cols)


@pytest.mark.parametrize("shape", BANDED, ids=lambda s: "%dx%dx%d_%s" % s)
def test_band_plan_sampled(shape):
    M, N, K, dtype = shape
    b = _band_or_skip(M, N, K, dtype)
    A, B = wl.make_inputs(M, N, K, dtype, "uniform", seed=M + N)
    C = run_gpu(A, B, dtype)
    rng = np.random.default_rng(M * 7 + N)
    rows, cols = _cut_samples(b, M, N, rng)
    Cr, Sr = oracle.gemm_rows(A, B, dtype, rows)
    check_close(C[rows], Cr, Sr, "band rows")
    ri = np.repeat(np.arange(M), cols.size)
    ci = np.tile(cols, M)
    c, s = oracle.gemm_entries(A, B, dtype, ri, ci)
    check_close(C[ri, ci].reshape(M, cols.size), c.reshape(M, cols.size), s.reshape(M, cols.size), "band cols")
    ri, ci = rng.integers(0, M, 4096), rng.integers(0, N, 4096)
    c, s = oracle.gemm_entries(A, B, dtype, ri, ci)
    check_close(C[ri, ci][None], c[None], s[None], "band entries")


def test_band_plan_integer_exact():
    M, N, K = 2560, 6656, 1000
    b = _band_or_skip(M, N, K, "bf16")
    A, B = wl.make_int_inputs(M, N, K, "bf16", seed=17)
    C = run_gpu(A, B, "bf16")
    rng = np.random.default_rng(3)
    rows, cols = _cut_samples(b, M, N, rng)
    Cr, _ = oracle.gemm_rows(A, B, "bf16", rows)
    check_exact(C[rows], Cr, "int band rows")
    ri = np.repeat(np.arange(M), cols.size)
    ci = np.tile(cols, M)
    c, _ = oracle.gemm_entries(A, B, "bf16", ri, ci)
    check_exact(C[ri, ci].reshape(M, cols.size), c.reshape(M, cols.size), "int band cols")


@pytest.mark.parametrize("shape", [BANDED[0], BANDED[2]], ids=lambda s: "%dx%dx%d_%s" % s)
def test_band_plan_padded_leading_dimensions(shape):
    """The band's sub-matrices start ext rows (A, C) or ext columns (B, C)
    into the caller's arrays: with padded lda, ldb and ldc the cut must still
    land on the right elements, and C's padding must stay untouched."""
    M, N, K, dtype = shape
    b = _band_or_skip(M, N, K, dtype)
    A, B = wl.make_inputs(M, N, K, dtype, "uniform", seed=M + 3 * N)
    lda, ldb, ldc = K + 24, N + 8, N + 12
    out = empty_out(M, N, ldc=ldc, fill=-7.0)
    C = run_gpu(A, B, dtype, out=out, lda=lda, ldb=ldb)
    flat = out.as_strided((M * ldc,), (1,), out.storage_offset()).cpu().numpy().reshape(M, ldc)
    assert np.all(flat[:, N:] == -7.0), "C padding written"
    rng = np.random.default_rng(11)
    rows, cols = _cut_samples(b, M, N, rng)
    Cr, Sr = oracle.gemm_rows(A, B, dtype, rows)
    check_close(C[rows], Cr, Sr, "padded band rows")
    ri = np.repeat(np.arange(M), cols.size)
    ci = np.tile(cols, M)
    c, s = oracle.gemm_entries(A, B, dtype, ri, ci)
    check_close(C[ri, ci].reshape(M, cols.size), c.reshape(M, cols.size), s.reshape(M, cols.size),
                "padded band cols")


@pytest.mark.parametrize("shape", [BANDED[0], BANDED[2], BANDED[3]], ids=lambda s: "%dx%dx%d_%s" % s)
def test_band_plan_equals_one_launch(shape):
    """With no K split in either part, a banded call sums every element in
    the same order as one launch of the whole call: the results agree bit for
    bit."""
    M, N, K, dtype = shape
    b = _band_or_skip(M, N, K, dtype)
    cu = torch.cuda.get_device_properties(0).multi_processor_count
    whole = xg.xgemm_select_config(M, N, K, CODE[dtype], cu)
    if b.band.split_k != 1 or whole.split_k != 1:
        pytest.skip("a K split regroups the sums")
    A, B = wl.make_inputs(M, N, K, dtype, "uniform", seed=M + 2 * N)
    C1 = run_gpu(A, B, dtype)
    C2 = run_gpu(A, B, dtype, config=whole)
    assert np.array_equal(C1, C2)


# ---------------------------------------------------------------------------
# strided batched products
# ---------------------------------------------------------------------------

def _batched_case(L, M, N, K, dtype, seed, shared_a=False):
    As, Bs = [], []
    for b in range(L):
        A, B = wl.make_inputs(M, N, K, dtype, "uniform", seed=seed * 100 + b)
        As.append(A)
        Bs.append(B)
    if shared_a:
        As = [As[0]] * L
    return As, Bs


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("shape", [(3, 512, 264, 1024), (4, 300, 200, 100), (5, 64, 520, 320)],
                         ids=lambda s: "x".join(map(str, s)))
def test_strided_batched(dtype, shape):
    L, M, N, K = shape
    As, Bs = _batched_case(L, M, N, K, dtype, seed=L + M)
    A = torch.stack([to_device(a, dtype) for a in As])
    B = torch.stack([to_device(b, dtype) for b in Bs])
    C = xg.bmm(A, B)
    torch.cuda.synchronize()
    C = C.cpu().numpy()
    for b in range(L):
        C_ref, S = oracle.gemm(As[b], Bs[b], dtype)
        check_close(C[b], C_ref, S, "batch %d of %s" % (b, shape))


@pytest.mark.parametrize("K", [1000, 100], ids=["copied", "general"])
def test_strided_batched_unaligned(K):
    """Odd N and a padded, odd lda: at K = 1000 every problem's operands are
    copied into the workspace and the pipelined kernel runs; at K = 100 (two
    K steps) the general kernel reads them in place."""
    L, M, N = 3, 300, 201
    As, Bs, refs = [], [], []
    for b in range(L):
        A, B, C_ref, S = _case(M, N, K, "bf16", seed=60 + b)
        As.append(A); Bs.append(B); refs.append((C_ref, S))
    lda = K + 3
    abuf = np.full((L, M, lda), 0x7FC0, dtype=np.uint16)   # NaN row padding, never read
    for b in range(L):
        abuf[b, :, :K] = As[b]
    Ad = torch.from_numpy(abuf.view(np.int16)).cuda().view(torch.bfloat16)[:, :, :K]
    Bd = torch.from_numpy(np.stack(Bs).view(np.int16)).cuda().view(torch.bfloat16)
    assert Ad.stride(1) == lda and Bd.stride(1) == N
    C = xg.bmm(Ad, Bd)
    torch.cuda.synchronize()
    for b in range(L):
        check_close(C[b].cpu().numpy(), *refs[b], "batched unaligned K=%d problem %d" % (K, b))


def test_strided_batched_unaligned_shared_b():
    """A shared B (stride 0) with odd N is copied once; A per problem."""
    L, M, N, K = 4, 256, 129, 512
    As, refs = [], []
    _, B, _, _ = _case(M, N, K, "fp16", seed=70)
    for b in range(L):
        A, _, _, _ = _case(M, N, K, "fp16", seed=71 + b)
        C_ref, S = oracle.gemm(A, B, "fp16")
        As.append(A); refs.append((C_ref, S))
    Ad = torch.from_numpy(np.stack(As).view(np.int16)).cuda().view(torch.float16)
    Bd = torch.from_numpy(B.view(np.int16)).cuda().view(torch.float16).unsqueeze(0).expand(L, K, N)
    C = xg.bmm(Ad, Bd)
    torch.cuda.synchronize()
    for b in range(L):
        check_close(C[b].cpu().numpy(), *refs[b], "batched shared B problem %d" % b)


def test_strided_batched_shared_a_and_padding():
    L, M, N, K = 3, 260, 136, 448
    As, Bs = _batched_case(L, M, N, K, "bf16", seed=7, shared_a=True)
    h = xg.handle()
    dA = to_device(As[0], "bf16")                         # stride_a = 0: one A for all
    sb = K * N + 64                                       # padded batch stride for B
    Bbuf = torch.zeros(L * sb, dtype=torch.bfloat16, device="cuda")
    for b in range(L):
        Bbuf[b * sb:b * sb + K * N] = to_device(Bs[b], "bf16").reshape(-1)
    ldc, sc = N + 8, (M + 2) * (N + 8)                    # padded rows and batch stride for C
    Cbuf = torch.full((L * sc,), 777.0, dtype=torch.float32, device="cuda")
    rc = xg.xgemm_run_strided_batched(h, L, M, N, K, dA.data_ptr(), K, 0, Bbuf.data_ptr(), N, sb,
                                      Cbuf.data_ptr(), ldc, sc, xg.XGEMM_BF16,
                                      torch.cuda.current_stream().cuda_stream)
    assert rc == xg.XGEMM_OK, xg.xgemm_last_error(h)
    torch.cuda.synchronize()
    Ch = Cbuf.cpu().numpy()
    for b in range(L):
        C_ref, S = oracle.gemm(As[0], Bs[b], "bf16")
        blk = Ch[b * sc:b * sc + M * ldc].reshape(M, ldc)
        check_close(blk[:, :N], C_ref, S, "shared-A batch %d" % b)
        assert np.all(blk[:, N:] == 777.0)                # row padding untouched
        assert np.all(Ch[b * sc + M * ldc:(b + 1) * sc] == 777.0)


@pytest.mark.parametrize("L", [64, 56], ids=["4rounds", "3.5rounds"])
def test_strided_batched_persistent(L):
    """Enough 256 x 256 tiles over the problems for the persistent kernel:
    64 problems of 1024 x 1024 (16 tiles each) are four whole rounds on 256
    CUs; 56 are three and a half, with tiles shared between workgroups (one
    problem's tile may be split between two of them) and their partial sums
    in the workspace.  C has padded rows and a padded batch stride, which
    stay untouched; every problem is checked against the oracle."""
    M = N = 1024
    K = 512
    cu = torch.cuda.get_device_properties(0).multi_processor_count
    if cu != 256:
        pytest.skip("the case is sized for 256 CUs")
    As, Bs = _batched_case(L, M, N, K, "bf16", seed=L)
    A = torch.stack([to_device(a, "bf16") for a in As])
    B = torch.stack([to_device(b, "bf16") for b in Bs])
    ldc, sc = N + 4, (M + 1) * (N + 4)
    Cbuf = torch.full((L * sc,), 777.0, dtype=torch.float32, device="cuda")
    h = xg.handle()
    rc = xg.xgemm_run_strided_batched(h, L, M, N, K, A.data_ptr(), K, M * K, B.data_ptr(), N, K * N,
                                      Cbuf.data_ptr(), ldc, sc, xg.XGEMM_BF16,
                                      torch.cuda.current_stream().cuda_stream)
    assert rc == xg.XGEMM_OK, xg.xgemm_last_error(h)
    torch.cuda.synchronize()
    Ch = Cbuf.cpu().numpy()
    for b in range(L):
        C_ref, S = oracle.gemm(As[b], Bs[b], "bf16")
        blk = Ch[b * sc:b * sc + M * ldc].reshape(M, ldc)
        check_close(blk[:, :N], C_ref, S, "persistent batch %d of %d" % (b, L))
        assert np.all(blk[:, N:] == 777.0)
        assert np.all(Ch[b * sc + M * ldc:(b + 1) * sc] == 777.0)
    # the same call again gives the same bits (the counters were left zero)
    Cbuf2 = torch.full((L * sc,), 777.0, dtype=torch.float32, device="cuda")
    assert xg.xgemm_run_strided_batched(h, L, M, N, K, A.data_ptr(), K, M * K, B.data_ptr(), N, K * N,
                                        Cbuf2.data_ptr(), ldc, sc, xg.XGEMM_BF16,
                                        torch.cuda.current_stream().cuda_stream) == xg.XGEMM_OK
    torch.cuda.synchronize()
    assert np.array_equal(Cbuf2.cpu().numpy(), Ch)


def test_persistent_switch():
    """xgemm_set_persistent(h, 0): the handle's selected plans leave out the
    persistent kernel (8192 x 8192 x 2048 bf16 is four whole rounds of 256 x
    256 tiles; with the switch off it runs one workgroup per tile, the same
    sums in the same order for whole tiles, so the same bits); other values
    are rejected; forced configurations are unaffected."""
    M, N, K = 8192, 8192, 2048
    cu = torch.cuda.get_device_properties(0).multi_processor_count
    if cu != 256:
        pytest.skip("the case is sized for 256 CUs")
    assert xg.xgemm_select_band(M, N, K, xg.XGEMM_BF16, cu).body.stream_k == 1
    A, B = wl.make_inputs(M, N, K, "bf16", "uniform", seed=91)
    dA, dB = to_device(A, "bf16"), to_device(B, "bf16")
    s = torch.cuda.current_stream().cuda_stream
    h = xg.xgemm_create()
    try:
        outs = []
        for enable in (1, 0):
            assert xg.xgemm_set_persistent(h, enable) == xg.XGEMM_OK
            C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
            assert xg.xgemm_run(h, M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, C.data_ptr(), N,
                                xg.XGEMM_BF16, s) == xg.XGEMM_OK, xg.xgemm_last_error(h)
            torch.cuda.synchronize()
            outs.append(C.cpu().numpy())
        assert np.array_equal(outs[0], outs[1])
        rows = np.array([0, 1, 255, 256, 4097, 8191])
        C_ref, S = oracle.gemm_rows(A, B, "bf16", rows)
        check_close(outs[1][rows], C_ref, S, "persistent switch off")
        assert xg.xgemm_set_persistent(h, 2) == xg.XGEMM_ERR_INVALID_ARG
        # a forced persistent configuration still runs it
        assert xg.xgemm_set_persistent(h, 0) == xg.XGEMM_OK
        C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        cfg = xg.xgemm_config(tile=0, split_k=1, group_m=4, stream_k=1)
        assert xg.xgemm_run_config(h, M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, C.data_ptr(), N,
                                   xg.XGEMM_BF16, s, cfg) == xg.XGEMM_OK
        torch.cuda.synchronize()
        assert np.array_equal(C.cpu().numpy(), outs[0])
    finally:
        torch.cuda.synchronize()
        xg.xgemm_destroy(h)


def test_strided_batched_integer_exact_and_single():
    L, M, N, K = 2, 256, 256, 512
    As, Bs = [], []
    for b in range(L):
        A, B = wl.make_int_inputs(M, N, K, "fp16", seed=b)
        As.append(A)
        Bs.append(B)
    A = torch.stack([to_device(a, "fp16") for a in As])
    B = torch.stack([to_device(b, "fp16") for b in Bs])
    C = xg.bmm(A, B).cpu().numpy()
    for b in range(L):
        check_exact(C[b], oracle.gemm(As[b], Bs[b], "fp16")[0], "int batch %d" % b)
    # batch of one equals the plain call
    C1 = xg.bmm(A[:1], B[:1]).cpu().numpy()
    check_exact(C1[0], oracle.gemm(As[0], Bs[0], "fp16")[0], "batch 1")


def test_strided_batched_arguments():
    h = xg.handle()
    s = torch.cuda.current_stream().cuda_stream
    A = torch.zeros((2, 64, 64), dtype=torch.bfloat16, device="cuda")
    C = torch.zeros((2, 64, 64), dtype=torch.float32, device="cuda")
    a, c = A.data_ptr(), C.data_ptr()
    ok = xg.xgemm_run_strided_batched(h, 0, 64, 64, 64, a, 64, 4096, a, 64, 4096, c, 64, 4096, 0, s)
    assert ok == xg.XGEMM_OK                                   # batch 0: no-op
    bad = xg.xgemm_run_strided_batched(h, 2, 64, 64, 64, a, 64, 4096, a, 64, 4096, c, 64, 100, 0, s)
    assert bad == xg.XGEMM_ERR_INVALID_ARG                     # overlapping outputs
    bad = xg.xgemm_run_strided_batched(h, 2, 64, 64, 64, a, 64, -1, a, 64, 4096, c, 64, 4096, 0, s)
    assert bad == xg.XGEMM_ERR_INVALID_ARG                     # negative stride
    bad = xg.xgemm_run_strided_batched(h, -1, 64, 64, 64, a, 64, 4096, a, 64, 4096, c, 64, 4096, 0, s)
    assert bad == xg.XGEMM_ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.all(C == 0)


# ---------------------------------------------------------------------------
# seeded random layouts: shapes, padding, offsets and forced configurations
# ---------------------------------------------------------------------------

def _random_cases(n, seed):
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        big = rng.random() < 0.4   # a share of larger shapes
        hi = 900 if big else 300
        M, N, K = (int(v) for v in rng.integers(1, hi, size=3))
        lda = K + int(rng.choice([0, 0, 1, 3, 8]))
        ldb = N + int(rng.choice([0, 0, 1, 5, 8]))
        ldc = N + int(rng.choice([0, 0, 1, 4]))
        off = int(rng.choice([0, 0, 0, 1]))
        cfg = None if rng.random() < 0.5 else config(int(rng.integers(0, 3)), int(rng.choice([1, 1, 2, 4])))
        cases.append((M, N, K, lda, ldb, ldc, off, cfg, str(rng.choice(["bf16", "fp16"]))))
    return cases


@pytest.mark.parametrize("case", _random_cases(40, 2024), ids=lambda c: "%dx%dx%d" % c[:3])
def test_random_layouts(case):
    M, N, K, lda, ldb, ldc, off, cfg, dtype = case
    A, B, C_ref, S = _case(M, N, K, dtype, seed=M * 7 + N * 3 + K)
    out = empty_out(M, N, ldc=ldc, offset=off)
    C = run_gpu(A, B, dtype, config=cfg, out=out, lda=lda, ldb=ldb, offset=off, pad=0x7FC0 if dtype == "bf16"
                else 0x7E00)
    check_close(C, C_ref, S, "random %s" % (case,))
