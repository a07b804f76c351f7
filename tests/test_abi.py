"""The C-ABI library: it loads, exports what the header declares, and its
host-only entry points (configuration selection, tile info, argument checks)
behave as documented.  No GPU work is launched here."""
import ctypes
import math

import pytest

from paper_2609_16389_amd import workloads as wl
from paper_2609_16389_amd import xgemm as xg


def test_every_header_function_is_exported():
    names = xg.header_functions()
    assert "xgemm_create" in names and "xgemm_run" in names and "xgemm_destroy" in names
    for n in names:
        assert hasattr(xg.lib, n), "libxgemm.so does not export %s" % n


def test_strerror_codes():
    for code in range(5):
        assert xg.xgemm_strerror(code) not in ("", "unknown status")
    assert xg.xgemm_strerror(99) == "unknown status"


def test_null_handle_is_invalid_argument():
    assert xg.xgemm_run(None, 1, 1, 1, None, 1, None, 1, None, 1, xg.XGEMM_BF16, None) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.xgemm_destroy(None) == xg.XGEMM_OK
    assert xg.xgemm_last_error(None) == "no handle"
    assert xg.lib.xgemm_create(None) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.xgemm_set_persistent(None, 0) == xg.XGEMM_ERR_INVALID_ARG


def test_tile_info():
    seen = set()
    for t in range(xg.XGEMM_TILE_COUNT):
        bm, bn, bk, threads = xg.xgemm_tile_info(t)
        assert bm % 32 == 0 and bn % 32 == 0 and bk % 16 == 0 and threads % 64 == 0
        # two LDS stages fit in 160 KiB
        assert 2 * (bm + bn) * bk * 2 <= 160 * 1024
        seen.add((bm, bn))
    assert len(seen) == xg.XGEMM_TILE_COUNT
    with pytest.raises(xg.XgemmError):
        xg.xgemm_tile_info(xg.XGEMM_TILE_COUNT)


@pytest.mark.parametrize("name", sorted(wl.WORKLOADS))
def test_selector_on_workloads(name):
    w = wl.WORKLOADS[name]
    dt = xg.XGEMM_BF16 if w.dtype == "bf16" else xg.XGEMM_FP16
    cfg = xg.xgemm_select_config(w.M, w.N, w.K, dt, 256)
    assert 0 <= cfg.tile < xg.XGEMM_TILE_COUNT and 1 <= cfg.split_k <= 16 and cfg.group_m >= 1
    bm, bn, bk, _ = xg.xgemm_tile_info(cfg.tile)
    tiles = math.ceil(w.M / bm) * math.ceil(w.N / bn)
    # every split has a non-empty K range
    chunk = math.ceil(math.ceil(w.K / cfg.split_k) / bk) * bk
    assert chunk * (cfg.split_k - 1) < w.K
    if name == "skinny1024x1024x65536_bf16":
        # 1024 x 1024 has too few output tiles to fill 256 CUs without splitting K
        assert cfg.split_k > 1 and tiles * cfg.split_k >= 128
    if name == "gemm8192_bf16":
        assert cfg.split_k == 1 and (bm, bn) == (256, 256)


def test_selector_rejects_bad_arguments():
    cfg = xg.xgemm_config()
    assert xg.lib.xgemm_select_config(-1, 1, 1, 0, 256, ctypes.byref(cfg)) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.lib.xgemm_select_config(1, 1, 1, 7, 256, ctypes.byref(cfg)) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.lib.xgemm_select_config(1, 1, 1, 0, 0, ctypes.byref(cfg)) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.lib.xgemm_select_config(1, 1, 1, 0, 256, None) == xg.XGEMM_ERR_INVALID_ARG


PREFIX = 4096   # the workspace's counter prefix


def test_workspace_bytes():
    cfg = xg.xgemm_config(tile=0, split_k=1, group_m=4, stream_k=0)
    assert xg.xgemm_workspace_bytes(1024, 1024, 4096, 256, cfg) == 0
    cfg.split_k = 16
    assert xg.xgemm_workspace_bytes(1024, 1024, 65536, 256, cfg) == PREFIX + 16 * 1024 * 1024 * 4
    # rows of partials padded to 4 floats; N = 5 also copies B (65536 x 8, after the partials)
    assert xg.xgemm_workspace_bytes(10, 5, 65536, 256, cfg) == PREFIX + 16 * 10 * 8 * 4 + 65536 * 8 * 2
    cfg.stream_k = 1                        # the persistent kernel needs split_k == 1
    assert xg.xgemm_workspace_bytes(10, 5, 65536, 256, cfg) == 0
    cfg.stream_k, cfg.tile = 0, 99
    assert xg.xgemm_workspace_bytes(10, 5, 65536, 256, cfg) == 0
    cfg.tile, cfg.split_k, cfg.stream_k = 0, 1, 1024   # at most 1023 workgroups
    assert xg.xgemm_workspace_bytes(4096, 4096, 4096, 256, cfg) == 0


def _sk_info(M, N, K, stream_k=1, cu=256, tile=0, ldc=None, c=3 << 40):
    cfg = xg.xgemm_config(tile=tile, split_k=1, group_m=4, stream_k=stream_k)
    return xg.xgemm_trace_plan(M, N, K, 1 << 40, K, 2 << 40, N, c, N if ldc is None else ldc, cfg, cu, 0)


def test_persistent_plan():
    """The persistent stream-K plan: whole rounds of tiles, then the rest as
    K-step ranges of at least one tile each; partial sums in the workspace
    only when tiles are split."""
    # 4096 x 14336 with 256 x 256 tiles: 896 tiles = 3 rounds of 256 + 128
    w = wl.WORKLOADS["proj4096x14336x4096_fp16"]
    info = _sk_info(w.M, w.N, w.K)
    assert info.family == xg.XGEMM_KERNEL_PERSISTENT and info.grid == 256 and info.threads == 512
    assert (info.dp_rounds, info.sk_tiles, info.kt) == (2, 384, 64)
    assert info.workspace_bytes == PREFIX + 2 * 256 * 256 * 256 * 4 and info.data_offset == PREFIX
    assert info.lds_bytes == 2 * 65536 + 256
    # whole rounds (8192^3: 1024 tiles on 256 CUs): no split, no workspace
    info = _sk_info(8192, 8192, 8192)
    assert (info.dp_rounds, info.sk_tiles, info.kt) == (4, 0, 128)
    assert info.workspace_bytes == 0
    # an explicit grid: 20 tiles on 8 workgroups = 1 round, then 12 tiles shared
    info = _sk_info(1024, 1280, 1024, stream_k=8)
    assert (info.grid, info.dp_rounds, info.sk_tiles) == (8, 1, 12)
    # the ordinary kernel where the persistent one does not apply
    family = lambda *a, **k: _sk_info(*a, **k).family
    assert family(1024, 1024, 65536) == xg.XGEMM_KERNEL_PIPELINED       # 16 tiles < 256 CUs
    assert family(4096, 4096 + 8, 4096) == xg.XGEMM_KERNEL_PIPELINED    # N not whole tiles
    assert family(4096, 4096, 4096 + 8) == xg.XGEMM_KERNEL_PIPELINED    # K not whole steps
    assert family(4096, 4096, 4096, tile=1) == xg.XGEMM_KERNEL_PIPELINED
    assert family(4096, 4096, 4096, c=(3 << 40) + 4) == xg.XGEMM_KERNEL_PIPELINED   # C misaligned
    assert family(4096, 4096, 4096, ldc=(1 << 22)) == xg.XGEMM_KERNEL_PIPELINED     # 256 rows > 4 GiB
    assert family(4096, 4096, 4096) == xg.XGEMM_KERNEL_PERSISTENT
    # not chosen by the selector unless it wins (see the selector tests)
    assert xg.xgemm_select_config(8192, 8192, 8192, xg.XGEMM_BF16, 256).stream_k in (0, 1)


def test_persistent_ranges_cover_every_step_once():
    """Host replica of the kernel's work split (one workgroup's logical id,
    rounds of whole tiles, then equal K-step ranges of the rest): every
    (tile, K step) is computed exactly once, every range holds at least one
    tile's steps, and a tile is split between at most two neighbouring
    ranges -- its first steps ending range lw, its last starting lw + 1."""
    for T, P, kt in [(896, 256, 64), (300, 256, 7), (257, 256, 3), (20, 8, 16), (9, 8, 2), (1024, 256, 128),
                     (511, 256, 64), (13, 13, 5)]:
        rounds, rem = divmod(T, P)
        dp = rounds if rem == 0 else rounds - 1
        sk = 0 if rem == 0 else rem + P
        seen = {}
        owners = {}
        for lw in range(P):
            s0, s1 = sk * kt * lw // P, sk * kt * (lw + 1) // P
            if sk:
                assert s1 - s0 >= kt
            steps = [(lw + r * P, k) for r in range(dp) for k in range(kt)]
            steps += [(dp * P + i // kt, i % kt) for i in range(s0, s1)]
            for t, k in steps:
                seen[(t, k)] = seen.get((t, k), 0) + 1
                owners.setdefault(t, {}).setdefault(lw, []).append(k)
        assert len(seen) == T * kt and set(seen.values()) == {1}, (T, P, kt)
        for t, by in owners.items():
            assert len(by) <= 2, (T, P, kt, t)
            if len(by) == 2:
                a, b = sorted(by)
                assert b == a + 1 and min(by[a]) == 0 and max(by[b]) == kt - 1 and max(by[a]) + 1 == min(by[b])


def test_single_hip_runtime_in_process():
    """libxgemm.so must bind to the HIP runtime torch loaded, not a second copy,
    whatever the import order (torch's device pointers and streams belong to
    its runtime)."""
    import subprocess
    import sys
    code = ("import ctypes, sys; sys.path.insert(0, %r)\n"
            "import paper_2609_16389_amd.xgemm\n"
            "import torch\n"
            "maps = open('/proc/self/maps').read().split('\\n')\n"
            "libs = sorted({l.split()[-1] for l in maps if 'libamdhip64' in l})\n"
            "print(len(libs), libs)\n") % xg._PKG.rsplit("/", 1)[0]
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, check=True).stdout
    assert out.startswith("1 "), out


def test_kernel_family_rules():
    cfg = xg.xgemm_config(tile=0, split_k=1, group_m=4, stream_k=0)
    al = 1 << 20  # a 16-byte aligned stand-in address (only alignment is inspected)
    fam = lambda M, N, K, a=al, lda=None, b=al, ldb=None, c=cfg: xg.xgemm_kernel_family(
        M, N, K, a, K if lda is None else lda, b, N if ldb is None else ldb, c)
    P, G = xg.XGEMM_KERNEL_PIPELINED, xg.XGEMM_KERNEL_GENERAL
    assert fam(8192, 8192, 8192) == P
    assert fam(1000, 1000, 1024) == P          # ragged M and N, N % 8 == 0
    assert fam(1000, 1000, 1000) == P          # K % 64 != 0 but K % 8 == 0: a partial last step
    assert fam(1000, 1000, 1056) == P          # the same
    assert fam(1000, 1000, 128) == G           # fewer than 3 K steps of 64
    assert fam(1000, 1000, 136) == P           # 2 full steps and a partial one
    assert fam(1000, 1000, 120) == G           # 1 full step and a partial one
    # operands the pipelined kernels cannot read in place are copied into
    # the workspace when that makes the pipelined kernel eligible; with too
    # few K steps the general kernel reads them in place
    short = 120   # one full K step and a partial one
    assert fam(300, 301, 304) == P and fam(300, 301, short) == G                  # N % 8 != 0
    assert fam(300, 304, 301, lda=304) == P and fam(300, 304, 117, lda=120) == G  # K % 8 != 0
    assert fam(300, 304, 304, a=al + 2) == P and fam(300, 304, short, a=al + 2) == G  # misaligned A
    assert fam(300, 304, 304, lda=308) == P and fam(300, 304, short, lda=124) == G  # lda % 8 != 0
    assert fam(300, 304, 304, ldb=308) == P and fam(300, 304, short, ldb=308) == G  # ldb % 8 != 0
    cfg16 = xg.xgemm_config(tile=0, split_k=16, group_m=4, stream_k=0)
    assert fam(1024, 1024, 65536, c=cfg16) == P
    assert fam(1024, 1024, 1024, c=cfg16) == G   # 64-element splits are too short
    assert fam(0, 8, 32) == -1
    bad = xg.xgemm_config(tile=7, split_k=1, group_m=4, stream_k=0)
    assert fam(8, 8, 32, c=bad) == -1


def test_batched_null_handle():
    assert xg.xgemm_run_strided_batched(None, 1, 1, 1, 1, None, 1, 0, None, 1, 0, None, 1, 0, 0, None) \
        == xg.XGEMM_ERR_INVALID_ARG


def test_gemv_selector():
    c = xg.xgemv_select_config(16384, 16384, 256)
    assert (c.rows, c.unroll, c.split_k) == (2, 4, 1)
    assert xg.xgemv_select_config(256, 262144, 256).rows == 1
    assert xg.xgemv_select_config(2048, 10, 256).rows == 2
    assert xg.xgemv_select_config(2047, 10, 256).rows == 1
    # few rows: K is split until there are about two workgroups per CU, each
    # range keeping at least 65536 values, at most 256 ranges
    assert xg.xgemv_select_config(64, 1000000, 256).split_k == 8
    assert xg.xgemv_select_config(1, 4194304, 256).split_k == 64
    assert xg.xgemv_select_config(1, 300000, 256).split_k == 4
    assert xg.xgemv_select_config(1, 100000, 256).split_k == 1
    assert xg.xgemv_select_config(1, 2 ** 30, 256).split_k == 256
    assert xg.xgemv_select_config(64, 3000, 256).split_k == 1
    assert xg.xgemv_select_config(512, 10 ** 6, 256).split_k == 1
    with pytest.raises(xg.XgemmError):
        xg.xgemv_select_config(-1, 5, 256)
    with pytest.raises(xg.XgemmError):
        xg.xgemv_select_config(5, 5, 0)


def test_gemv_null_handle_and_trace_arguments():
    assert xg.xgemv_run(None, 4, 4, 16, 4, 16, 16, None) == xg.XGEMM_ERR_INVALID_ARG
    import ctypes
    counts = (ctypes.c_int64 * 256)()
    cfg = xg.xgemv_config(2, 4)
    tr = xg.lib.xgemv_trace_workgroup
    # block out of range, unsupported configs, K == 0
    assert tr(4, 4, 16, 4, 16, 16, 32, ctypes.byref(cfg), 2, None, 0, counts) == xg.XGEMM_ERR_INVALID_ARG
    for bad in (xg.xgemv_config(3, 4), xg.xgemv_config(2, 4, 0), xg.xgemv_config(2, 4, 257)):
        assert tr(4, 4, 16, 4, 16, 16, 32, ctypes.byref(bad), 0, None, 0, counts) == xg.XGEMM_ERR_INVALID_ARG
    assert tr(4, 0, 16, 4, 16, 16, 32, ctypes.byref(cfg), 0, None, 0, counts) == xg.XGEMM_ERR_INVALID_ARG
    assert tr(4, 4, 16, 4, 16, 16, 32, ctypes.byref(cfg), 0, None, 0, counts) == xg.XGEMM_OK
    # a K split needs the partials' address and has split x row-block workgroups
    split = xg.xgemv_config(2, 4, 2)
    assert tr(4, 4096, 16, 4096, 16, 16, None, ctypes.byref(split), 0, None, 0, counts) == xg.XGEMM_ERR_INVALID_ARG
    assert tr(4, 4096, 16, 4096, 16, 16, 32, ctypes.byref(split), 3, None, 0, counts) == xg.XGEMM_OK
    assert tr(4, 4096, 16, 4096, 16, 16, 32, ctypes.byref(split), 4, None, 0, counts) == xg.XGEMM_ERR_INVALID_ARG


def test_sweep_candidates_host_logic():
    """The selector sweep (bench.py --sweep, a GPU measurement) enumerates
    configurations on the host: the selector's choice is always timed, splits
    shorter than 3 K steps and launches above the workgroup cap are left out."""
    import bench
    c = bench.sweep_candidates(1024, 1024, 65536, (1, 8), xg)
    assert (1, 8) in c and (0, 1) in c and (2, 16) in c and len(c) == len(set(c))
    small = bench.sweep_candidates(256, 256, 256, (2, 1), xg)
    assert all(s == 1 for _, s in small)          # K = 256: every split would be under 3 steps
    big = bench.sweep_candidates(16384, 16384, 4096, (0, 1), xg)
    for t, s in big:
        bm, bn, _, _ = xg.xgemm_tile_info(t)
        assert (16384 // bm) * (16384 // bn) * s <= bench.SWEEP_MAX_WORKGROUPS or (t, s) == (0, 1)


def test_packed_plan_layout():
    """Packed operands sit after the split partials in the workspace, 256-byte
    aligned, with K and N rounded up to 8 and the kernel reading them with
    those leading dimensions."""
    cfg = xg.xgemm_config(tile=0, split_k=2, group_m=4, stream_k=0)
    M, N, K = 1000, 1001, 2003
    info = xg.xgemm_trace_plan(M, N, K, 1 << 20, K, 1 << 21, N, 1 << 22, N, cfg, 256, 0)
    assert info.family == xg.XGEMM_KERNEL_PIPELINED and info.packed == 3   # K % 8 != 0: both
    assert info.k == 2008 and info.lda == 2008 and info.ldb == 1008
    split_bytes = 2 * M * 1004 * 4                     # two partials of M x ceil4(N) floats
    assert info.a_offset == PREFIX + (split_bytes + 255) // 256 * 256
    assert info.b_offset == (info.a_offset + M * 2008 * 2 + 255) // 256 * 256
    assert info.workspace_bytes == info.b_offset + 2008 * 1008 * 2
    assert xg.xgemm_workspace_bytes(M, N, K, 256, cfg) == info.workspace_bytes
    # only B misses the layout: A is read in place
    info = xg.xgemm_trace_plan(M, N, 2000, 1 << 20, 2000, 1 << 21, N, 1 << 22, N,
                               xg.xgemm_config(tile=0, split_k=1, group_m=4, stream_k=0), 256, 0)
    assert info.packed == 2 and info.a_offset == -1 and info.lda == 2000 and info.ldb == 1008
    # aligned operands: nothing packed
    info = xg.xgemm_trace_plan(1024, 1024, 1024, 1 << 20, 1024, 1 << 21, 1024, 1 << 22, 1024,
                               xg.xgemm_config(tile=0, split_k=1, group_m=4, stream_k=0), 256, 0)
    assert info.packed == 0 and info.a_offset == -1 and info.b_offset == -1 and info.workspace_bytes == 0


# ---------------------------------------------------------------------------
# body + band plans (host-only selection)
# ---------------------------------------------------------------------------

def _band(M, N, K, dtype=xg.XGEMM_BF16, cu=256):
    return xg.xgemm_select_band(M, N, K, dtype, cu)


def test_band_selection_on_workloads():
    # 6144^3: 576 tiles of 256 x 256 are 2.25 rounds on 256 CUs; the body
    # takes 21 tile columns (504 tiles) and a 128 x 128 band the last 768
    # columns
    b = _band(6144, 6144, 6144)
    assert (b.axis, b.extent, b.body.tile, b.body.split_k, b.body.stream_k) == (xg.XGEMM_BAND_COLUMNS, 5376, 0, 1, 0)
    assert (b.band.tile, b.band.split_k, b.band.stream_k) == (2, 1, 0)
    # the persistent kernel: four or more whole rounds of 256 x 256 tiles
    # (8192^3: 4, 16384 x 5120: 5), or three and a half (4096 x 14336: 896
    # tiles); not banded
    for shape, sk in [((8192, 8192, 8192), 1), ((16384, 5120, 4096), 1), ((4096, 14336, 4096), 1),
                      ((6144, 8192, 4096), 0), ((4096, 8192, 4096), 0), ((4096, 4096, 4096), 0),
                      ((5120, 5120, 5120), 0), ((1024, 1024, 65536), 0), ((256, 256, 256), 0),
                      ((2048, 5120, 4096), 0), ((3072, 3072, 4096), 0)]:
        b = _band(*shape)
        assert b.axis == xg.XGEMM_BAND_NONE and b.extent == 0, shape
        whole = xg.xgemm_select_config(*shape, xg.XGEMM_BF16, 256)
        assert (b.body.tile, b.body.split_k, b.body.group_m) == (whole.tile, whole.split_k, whole.group_m)
        assert b.body.stream_k == sk, shape
        assert (b.band.tile, b.band.split_k, b.band.group_m, b.band.stream_k) == (0, 0, 0, 0)
    # the rule is in whole rounds of the device's CUs: 8192^3 on 304 CUs is
    # 3.37 rounds
    assert _band(8192, 8192, 8192, xg.XGEMM_BF16, 304).body.stream_k == 0
    # without the persistent kernel: the one-launch plan, or the band plan
    b = xg.xgemm_select_plan(8192, 8192, 8192, xg.XGEMM_BF16, 256, 0)
    assert (b.axis, b.body.tile, b.body.split_k, b.body.stream_k) == (xg.XGEMM_BAND_NONE, 0, 1, 0)
    b = xg.xgemm_select_plan(4096, 14336, 4096, xg.XGEMM_FP16, 256, 0)
    assert (b.axis, b.extent, b.body.tile, b.body.stream_k) == (xg.XGEMM_BAND_COLUMNS, 12288, 0, 0)
    assert (b.band.tile, b.band.split_k) == (1, 1)
    for shape in [(4096, 14336, 4096), (6144, 6144, 6144), (1024, 1024, 65536)]:
        a, b = _band(*shape), xg.xgemm_select_plan(*shape, xg.XGEMM_BF16, 256, 1)
        assert (a.axis, a.extent, a.body.tile, a.body.split_k, a.body.stream_k) == \
               (b.axis, b.extent, b.body.tile, b.body.split_k, b.body.stream_k)
    with pytest.raises(xg.XgemmError):
        xg.xgemm_select_plan(64, 64, 64, xg.XGEMM_BF16, 256, 2)
    # a band of rows
    b = _band(9472, 2048, 1000)
    assert (b.axis, b.extent) == (xg.XGEMM_BAND_ROWS, 8192)


@pytest.mark.parametrize("cu", [256, 304, 80])
def test_band_plan_invariants(cu):
    """Every banded plan cuts C at a whole number of the body's tiles, leaves
    a non-empty band, runs the body without split-k, and names valid
    configurations, the band's being the selector's for its shape."""
    seen = 0
    for M in (1000, 2048, 3000, 5120, 7168, 9472):
        for N in (1000, 2048, 3584, 6656, 10240, 14336):
            for K in (256, 1000, 4096):
                b = _band(M, N, K, xg.XGEMM_BF16, cu)
                assert b.axis in (xg.XGEMM_BAND_NONE, xg.XGEMM_BAND_COLUMNS, xg.XGEMM_BAND_ROWS)
                if b.axis == xg.XGEMM_BAND_NONE:
                    continue
                seen += 1
                bm, bn, _, _ = xg.xgemm_tile_info(b.body.tile)
                along, step = (N, bn) if b.axis == xg.XGEMM_BAND_COLUMNS else (M, bm)
                assert 0 < b.extent < along and b.extent % step == 0
                assert b.body.split_k == 1 and b.body.stream_k == 0 and b.body.group_m >= 1
                assert 0 <= b.band.tile < xg.XGEMM_TILE_COUNT and 1 <= b.band.split_k <= 16
                assert b.band.stream_k == 0 and b.band.group_m >= 1
                # the band's configuration is the selector's for the band's shape
                rm, rn = (M, N - b.extent) if b.axis == xg.XGEMM_BAND_COLUMNS else (M - b.extent, N)
                whole = xg.xgemm_select_config(rm, rn, K, xg.XGEMM_BF16, cu)
                assert (b.band.tile, b.band.split_k) == (whole.tile, whole.split_k)
    assert seen > 0


def test_band_selection_rejects_bad_arguments():
    out = xg.xgemm_band()
    assert xg.lib.xgemm_select_band(-1, 1, 1, 0, 256, ctypes.byref(out)) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.lib.xgemm_select_band(1, 1, 1, 5, 256, ctypes.byref(out)) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.lib.xgemm_select_band(1, 1, 1, 0, 0, ctypes.byref(out)) == xg.XGEMM_ERR_INVALID_ARG
    assert xg.lib.xgemm_select_band(1, 1, 1, 0, 256, None) == xg.XGEMM_ERR_INVALID_ARG
    # empty problems: no band
    assert xg.lib.xgemm_select_band(0, 4096, 4096, 0, 256, ctypes.byref(out)) == xg.XGEMM_OK
    assert out.axis == xg.XGEMM_BAND_NONE


def test_kernels_use_no_scratch(tmp_path):
    """No kernel of libxgemm.so has a private (scratch) segment.  A kernel
    that spills registers gets one, and the runtime then allocates scratch
    memory at its first launch: xgemm_run_noalloc would allocate after all.
    Reads the gfx950 code object's metadata (objcopy, the offload bundler and
    llvm-readelf of this image)."""
    import os
    import re
    import shutil
    import subprocess
    bundler = "/opt/rocm/llvm/bin/clang-offload-bundler"
    readelf = "/opt/rocm/llvm/bin/llvm-readelf"
    if not (shutil.which("objcopy") and os.path.exists(bundler) and os.path.exists(readelf)):
        pytest.skip("objcopy / clang-offload-bundler / llvm-readelf not available")
    fat, co = tmp_path / "fat.bin", tmp_path / "gfx950.co"
    subprocess.run(["objcopy", "-O", "binary", "--only-section=.hip_fatbin", xg._LIB_PATH, str(fat)], check=True)
    subprocess.run([bundler, "--unbundle", "--type=o", "--input=" + str(fat),
                    "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", "--output=" + str(co)], check=True)
    notes = subprocess.run([readelf, "--notes", str(co)], check=True, capture_output=True, text=True).stdout
    symbols = re.findall(r"\.symbol:\s+(\S+)\.kd", notes)
    sizes = [int(v) for v in re.findall(r"\.private_segment_fixed_size:\s+(\d+)", notes)]
    assert len(sizes) == len(symbols) >= 20, (len(sizes), len(symbols))
    assert all(v == 0 for v in sizes), [(n, v) for n, v in zip(symbols, sizes) if v]
