"""Synchronisation checker (the abstract machine over the kernels' own
traces, Section 5 of the paper): the pipelined GEMM kernel and the GEMV.

1. The machine is pinned on hand-built wave programs whose verdicts follow
   from the hardware's ordering rules (a wait retires the issuing wave's
   operations; a barrier orders what each wave had retired before arriving).
2. The kernel's traces pass at concrete sizes: every tile, pipeline depths
   from the minimum up, ragged edges, padded leading dimensions, split-k and
   the tail split.
3. Planted mistakes in a real trace (a wait too weak, a missing LDS wait, a
   missing or unmatched barrier, a read hoisted above its barrier, output
   written twice, a load outside A and B) are all caught.
CPU only: the traces come from the library's host-side replay of the kernel
body, no GPU is touched."""
import dataclasses

import numpy as np
import pytest

import paper_2609_16389_amd.xgemm as xg
from paper_2609_16389_amd import syncheck as sc

LANE = np.arange(64, dtype=np.int64)
LDS = 4096


def prog(*ops):
    """A wave program: ('load', base) a 16-byte direct load per lane to
    base + 16*lane; ('read', base) a 16-byte read per lane at base +
    16*lane; ('read8', addrs) an 8-byte read at per-lane addrs; ('wvm', n),
    ('wlgkm', n); ('bar',)."""
    op, arg, lds = [], [], []
    for o in ops:
        k = o[0]
        if k == "load":
            op.append(sc.LDS_LOAD); arg.append(16); lds.append(np.full(64, o[1]))
        elif k == "read":
            op.append(sc.LDS_READ); arg.append(16); lds.append(o[1] + 16 * LANE)
        elif k == "read8":
            op.append(sc.LDS_READ); arg.append(8); lds.append(np.asarray(o[1], dtype=np.int64))
        elif k == "wvm":
            op.append(sc.WAIT_VM); arg.append(o[1]); lds.append(np.zeros(64))
        elif k == "wlgkm":
            op.append(sc.WAIT_LGKM); arg.append(o[1]); lds.append(np.zeros(64))
        elif k == "bar":
            op.append(sc.BARRIER); arg.append(0); lds.append(np.zeros(64))
        elif k == "vmem":
            op.append(sc.VMEM); arg.append(o[1]); lds.append(np.zeros(64))
        else:
            raise ValueError(k)
    n = len(op)
    return sc.WaveStream(op=np.array(op, dtype=np.int32), arg=np.array(arg, dtype=np.int32),
                         lds=np.array(lds, dtype=np.int64).reshape(n, 64), addr=np.zeros((n, 64), np.int64))


def verdict(*waves, lds=LDS):
    return {v.kind for v in sc.check_workgroup_lds(list(waves), lds)}


# ---------------------------------------------------------------------------
# 1. the machine on programs with known verdicts
# ---------------------------------------------------------------------------

def test_load_wait_barrier_read_is_ordered():
    assert verdict(prog(("load", 0), ("wvm", 0), ("bar",)),
                   prog(("bar",), ("read", 0))) == set()


def test_missing_wait_is_a_read_after_write_race():
    assert verdict(prog(("load", 0), ("bar",)),
                   prog(("bar",), ("read", 0))) == {"raw", "inflight_exit"}


def test_wait_after_the_barrier_does_not_order_other_waves():
    assert verdict(prog(("load", 0), ("bar",), ("wvm", 0)),
                   prog(("bar",), ("read", 0))) == {"raw"}


def test_missing_barrier_is_a_race_even_with_the_wait():
    assert verdict(prog(("load", 0), ("wvm", 0)),
                   prog(("read", 0))) == {"raw"}


def test_race_found_whichever_wave_is_visited_first():
    w_load = prog(("load", 0), ("wvm", 0))
    w_read = prog(("read", 0))
    assert "raw" in verdict(w_load, w_read)
    # reader visited first: it sees no write (uninit), then the write finds
    # an unordered read of its location
    assert {"uninit", "war"} <= verdict(w_read, w_load)


def test_own_load_needs_only_the_wait():
    assert verdict(prog(("load", 0), ("wvm", 0), ("read", 0))) == set()
    assert verdict(prog(("load", 0), ("read", 0), ("wvm", 0))) == {"raw"}


def test_vmcnt_retires_all_but_the_most_recent():
    # two loads, vmcnt(1): the first has landed, the second may not have
    assert verdict(prog(("load", 0), ("load", 1024), ("wvm", 1), ("read", 0), ("wvm", 0))) == set()
    assert verdict(prog(("load", 0), ("load", 1024), ("wvm", 1), ("read", 1024), ("wvm", 0))) == {"raw"}


def test_overwrite_after_reads_needs_their_completion_and_a_barrier():
    setup = (("load", 0), ("wvm", 0), ("bar",))
    ok = verdict(prog(*setup, ("bar",), ("load", 0), ("wvm", 0)),
                 prog(("bar",), ("read", 0), ("wlgkm", 0), ("bar",)))
    assert ok == set()
    no_lgkm = verdict(prog(*setup, ("bar",), ("load", 0), ("wvm", 0)),
                      prog(("bar",), ("read", 0), ("bar",)))
    assert no_lgkm == {"war"}
    no_barrier = verdict(prog(*setup, ("load", 0), ("wvm", 0), ("bar",)),
                         prog(("bar",), ("read", 0), ("wlgkm", 0), ("bar",)))
    assert "war" in no_barrier or "raw" in no_barrier


def test_two_unordered_loads_to_one_location():
    assert verdict(prog(("load", 0), ("wvm", 0)), prog(("load", 0), ("wvm", 0))) == {"waw"}
    assert verdict(prog(("load", 0), ("wvm", 0), ("bar",)),
                   prog(("bar",), ("load", 0), ("wvm", 0))) == set()


def test_read_of_unwritten_lds():
    assert verdict(prog(("read", 0))) == {"uninit"}
    # partial coverage: the load covers bytes 0..1023, the read 1024..2047
    assert verdict(prog(("load", 0), ("wvm", 0), ("read", 1024))) == {"uninit"}


def test_unmatched_barriers():
    assert "barrier_count" in verdict(prog(("bar",)), prog())


def test_load_in_flight_at_exit():
    assert verdict(prog(("load", 0))) == {"inflight_exit"}


def test_lds_bounds():
    assert "lds_bounds" in verdict(prog(("load", LDS - 16), ("wvm", 0)))
    assert "lds_bounds" in verdict(prog(("load", 0), ("wvm", 0), ("read8", np.full(64, -8))))


def test_global_stores_count_in_the_vector_memory_counter():
    # a direct load, then 3 global stores: vmcnt(3) retires the load, vmcnt(4) does not
    assert verdict(prog(("load", 0), ("vmem", 3), ("wvm", 3), ("read", 0), ("wvm", 0))) == set()
    assert verdict(prog(("load", 0), ("vmem", 3), ("wvm", 4), ("read", 0), ("wvm", 0))) == {"raw"}


def test_masked_global_runs_count_their_minimum_over_lanes():
    """Lane 0 issues 2 stores, the other lanes 3, between a direct load and a
    wait: the wave stream counts 2, so vmcnt(2) retires the load in the model
    (as on the hardware, which issued at least 2) but vmcnt(3) does not."""
    def trace(wait):
        ev = np.zeros((64, 8), dtype=xg.TRACE_EVENT_DTYPE)
        counts = np.zeros(64, dtype=np.int64)
        for lane in range(64):
            row = [(sc.LDS_LOAD, 16, 0, 0)] + [(sc.STORE, 4, 0, 1 << 40)] * (2 if lane == 0 else 3) + \
                  [(sc.WAIT_VM, wait, 0, 0), (sc.LDS_READ, 16, 16 * lane, 0), (sc.WAIT_VM, 0, 0, 0)]
            counts[lane] = len(row)
            for i, r in enumerate(row):
                ev[lane, i] = r
        return sc.wave_streams(ev, counts)
    waves = trace(2)
    assert list(waves[0].op[:3]) == [sc.LDS_LOAD, sc.VMEM, sc.WAIT_VM] and waves[0].arg[1] == 2
    assert sc.check_workgroup_lds(waves, LDS) == []
    assert {v.kind for v in sc.check_workgroup_lds(trace(3), LDS)} == {"raw"}


def test_per_lane_read_granules():
    # 8-byte reads touch one granule each: reading only the first half of
    # what was loaded is fine, one byte past it is not
    assert verdict(prog(("load", 0), ("wvm", 0), ("read8", 8 * LANE))) == set()
    assert verdict(prog(("load", 0), ("wvm", 0), ("read8", 1024 + 0 * LANE))) == {"uninit"}


# ---------------------------------------------------------------------------
# 2. the kernel's own traces
# ---------------------------------------------------------------------------

def cfg(tile, split=1, group_m=4, stream_k=0):
    return xg.xgemm_config(tile, split, group_m, stream_k)


def stages(tile):
    info = xg.xgemm_trace_plan(512, 512, 64 * 8, sc.BASE_A, 512, sc.BASE_B, 512, sc.BASE_C, 512, cfg(tile),
                               256, 0)
    bm, bn, bk, _ = xg.xgemm_tile_info(tile)
    return info.lds_bytes // (2 * bk * (bm + bn))


@pytest.mark.parametrize("tile", [0, 1, 2])
def test_kernel_trace_structure(tile):
    """Per wave: one barrier after the prologue and one per K step (one more
    where two waves along K add their sums through LDS), and the direct
    loads of every K step exactly once."""
    bm, bn, bk, threads = xg.xgemm_tile_info(tile)
    nk = stages(tile) + 3
    K = nk * bk
    ev, counts = sc.trace_workgroup(bm, bn, K, K, bn, bn, cfg(tile), 256, 0, 0, threads)
    waves = sc.wave_streams(ev, counts)
    loads_per_step = (bm + bn) * bk * 2 // 1024 // len(waves)
    # the 256 x 128 tile: eight waves, two on each 128 x 64 block of C
    exchange = 1 if tile == 1 and threads == 512 else 0
    for ws in waves:
        assert (ws.op == sc.BARRIER).sum() == nk + 1 + exchange
        assert (ws.op == sc.LDS_LOAD).sum() == nk * loads_per_step
    # every byte of every stage is loaded once per step that uses it
    base = np.concatenate([ws.lds[ws.op == sc.LDS_LOAD, 0] for ws in waves])
    per_stage = np.bincount(base // 1024, minlength=stages(tile) * (bm + bn) * bk * 2 // 1024)
    assert per_stage.sum() == nk * loads_per_step * len(waves)


@pytest.mark.parametrize("tile", [0, 1, 2])
@pytest.mark.parametrize("extra", [0, 1, 2, 5])
def test_kernel_pipeline_depths_are_race_free(tile, extra):
    bm, bn, bk, _ = xg.xgemm_tile_info(tile)
    nk = max(stages(tile), 3) + extra
    rep = sc.check_launch(bm, bn, nk * bk, cfg(tile))
    assert rep.ok, [str(v) for v in rep.violations]


@pytest.mark.parametrize("shape,tile", [((255, 264, 512), 2), ((1000, 1000, 1024), 1), ((264, 520, 320), 0),
                                        ((130, 136, 192), 0)])
def test_kernel_ragged_edges(shape, tile):
    rep = sc.check_launch(*shape, cfg(tile))
    assert rep.ok, [str(v) for v in rep.violations]


def test_kernel_padded_leading_dimensions():
    rep = sc.check_launch(300, 264, 448, cfg(2), lda=448 + 72, ldb=264 + 8, ldc=264 + 12)
    assert rep.ok, [str(v) for v in rep.violations]


@pytest.mark.parametrize("tile,split", [(2, 4), (1, 2), (0, 3)])
def test_kernel_split_k_partials(tile, split):
    bm, bn, bk, _ = xg.xgemm_tile_info(tile)
    rep = sc.check_launch(bm + 40, bn * 2, split * 3 * bk, cfg(tile, split))
    assert rep.ok, [str(v) for v in rep.violations]


# the persistent stream-K kernel on small grids: (M, N, K, workgroups)
SK_CASES = [
    (512, 768, 64 * 6, 4),     # 6 tiles on 4: all shared (1.5 tiles each)
    (768, 768, 64 * 5, 4),     # 9 tiles on 4: one round, then 5 shared, kt = 5
    (1024, 1280, 64 * 4, 8),   # 20 tiles on 8: one round, then 12 shared (6 steps of 4 each)
    (512, 512, 64 * 3, 3),     # 4 tiles on 3: 4 tiles shared, ranges of 4 steps over kt = 3
    (1024, 512, 64 * 3, 8),    # 8 tiles on 8: one whole round, nothing split
    (512, 256, 64 * 4, 2),     # 2 tiles on 2: one whole round
]


@pytest.mark.parametrize("M,N,K,grid", SK_CASES, ids=lambda v: str(v))
def test_persistent_kernel_is_race_free(M, N, K, grid):
    """Every workgroup of the persistent kernel, under both orders in which
    the pieces of a split tile count in: LDS ordering across the tiles of a
    range (the next tile's loads in flight during the last steps, the
    previous tile's stores under the next one's first rows), loads inside A,
    B and the workspace, C stored exactly once, partial sums written once and
    read only where written."""
    c = cfg(0, 1, 4, grid)
    info = xg.xgemm_trace_plan(M, N, K, sc.BASE_A, K, sc.BASE_B, N, sc.BASE_C, N, c, 256, 0)
    assert info.family == xg.XGEMM_KERNEL_PERSISTENT and info.grid == grid
    rep = sc.check_launch(M, N, K, c)
    assert rep.ok, [str(v) for v in rep.violations]


def test_persistent_kernel_trace_structure():
    """Ranges of 1.5 tiles (6 tiles of 256 x 256 on 4 workgroups, K = 384, all
    shared out):
    one barrier after the prologue and one per K step, plus the hand-over's
    barriers; direct loads in the prologue (two steps) and in every step
    (the last two steps repeat the range's last step); the split tile's pieces
    publish (schedule 0: the last steps, at the start of their range) or add
    (the first steps, at the end of theirs) as expected."""
    M, N, K, grid = 512, 768, 64 * 6, 4
    c = cfg(0, 1, 4, grid)
    info = xg.xgemm_trace_plan(M, N, K, sc.BASE_A, K, sc.BASE_B, N, sc.BASE_C, N, c, 256, 0)
    assert (info.dp_rounds, info.sk_tiles, info.kt) == (0, 6, 6)
    for block in range(grid):
        lw = (block % 8) * (grid // 8) + block // 8 if block < (grid // 8) * 8 else block
        s0, s1 = 6 * 6 * lw // grid, 6 * 6 * (lw + 1) // grid
        G = s1 - s0
        ev, counts = sc.trace_workgroup(M, N, K, K, N, N, c, 256, 0, block, info.threads)
        waves = sc.wave_streams(ev, counts)
        tail, head = s0 % 6 != 0, s1 % 6 != 0
        # prologue + per step, publish (release + count) and hand-over words
        extra = (2 if tail else 0) + (1 if head else 0)
        for ws in waves:
            assert (ws.op == sc.LDS_LOAD).sum() == (G + 2) * 8
            assert (ws.op == sc.BARRIER).sum() == 1 + G + extra, (block, lw, G, tail, head)
        # thread 0's partial-sum loads (16 bytes each): only the head adds them
        t0 = ev[0][:counts[0]]
        part_loads = ((t0["op"] == sc.LOAD) & (t0["arg"] == 16)).sum()
        assert part_loads == (32 if head else 0)


def test_persistent_kernel_planted_mistake_is_caught():
    """The checker is not blind to the persistent kernel: the same traces with
    the wait before one K step's barrier removed (a planted mistake, in the
    trace only) fail with a read-after-write race."""
    M, N, K, grid = 512, 768, 64 * 6, 4
    c = cfg(0, 1, 4, grid)
    info = xg.xgemm_trace_plan(M, N, K, sc.BASE_A, K, sc.BASE_B, N, sc.BASE_C, N, c, 256, 0)
    ev, counts = sc.trace_workgroup(M, N, K, K, N, N, c, 256, 0, 1, info.threads)
    waves = sc.wave_streams(ev, counts)
    assert not sc.check_workgroup_lds(waves, info.lds_bytes)
    # drop every wave's second vector-memory wait (the first K step's, for
    # the second step's loads): that stage is then read right after the
    # barrier before its direct loads are known to have landed
    for ws in waves:
        idx = np.nonzero(ws.op == sc.WAIT_VM)[0][1]
        keep = np.ones(len(ws.op), bool)
        keep[idx] = False
        ws.op, ws.arg, ws.lds, ws.addr = ws.op[keep], ws.arg[keep], ws.lds[keep], ws.addr[keep]
    kinds = {v.kind for v in sc.check_workgroup_lds(waves, info.lds_bytes)}
    assert "raw" in kinds


@pytest.mark.parametrize("shape,c,lds", [
    ((100, 100, 100), cfg(2), {}),                    # K not a multiple of 64
    ((300, 260, 120), cfg(0), {}),                    # N not a multiple of 8, K too short to copy for
    ((256, 256, 128), cfg(1), {}),                    # 2 K steps: too few for the pipeline
    ((129, 136, 320), cfg(2, 2), {"lda": 323}),       # lda not a multiple of 8
    ((200, 130, 400), cfg(1, 4), {"ldb": 131}),       # split-k over the general kernel (2 steps per split)
])
def test_general_kernel_traces_are_race_free(shape, c, lds):
    info = xg.xgemm_trace_plan(*shape[:3], sc.BASE_A, lds.get("lda", shape[2]), sc.BASE_B, lds.get("ldb", shape[1]),
                               sc.BASE_C, shape[1], c, 256, 0)
    assert info.family == xg.XGEMM_KERNEL_GENERAL
    rep = sc.check_launch(*shape, c, **lds)
    assert rep.ok, [str(v) for v in rep.violations]


def test_general_kernel_trace_structure():
    """General kernel, n K steps: one barrier after the first tile store and
    one per K step; each K step's tiles written to LDS once."""
    # lda = 2^23: a tile's byte offsets exceed 32 bits, so the general kernel
    # runs (the layout is aligned, so no copy is made); K = 328: 6 K steps
    K, lda = 5 * 64 + 8, 1 << 23
    info = xg.xgemm_trace_plan(256, 256, K, sc.BASE_A, lda, sc.BASE_B, 256, sc.BASE_C, 256, cfg(0), 256, 0)
    assert info.family == xg.XGEMM_KERNEL_GENERAL and info.packed == 0
    ev, counts = sc.trace_workgroup(256, 256, K, lda, 256, 256, cfg(0), 256, 0, 0, info.threads)
    waves = sc.wave_streams(ev, counts)
    nk = 6
    for ws in waves:
        assert (ws.op == sc.BARRIER).sum() == nk + 1
        # per thread and K step: 8 of the 2048 16-byte A chunks, and one of
        # the 256 8 x 8 B blocks written as 8 transposed columns
        assert (ws.op == sc.LDS_WRITE).sum() == nk * (8 + 8)


@pytest.mark.parametrize("name,keep", [
    ("no barrier", lambda op: op != sc.BARRIER),
    ("no LDS wait", lambda op: op != sc.WAIT_LGKM),
])
def test_general_kernel_planted_mistakes(name, keep):
    # lda = 2^23 keeps the general kernel (32-bit tile offsets overflow)
    K, lda = 5 * 64 + 8, 1 << 23
    info = xg.xgemm_trace_plan(256, 256, K, sc.BASE_A, lda, sc.BASE_B, 256, sc.BASE_C, 256, cfg(0), 256, 0)
    assert info.family == xg.XGEMM_KERNEL_GENERAL
    ev, counts = sc.trace_workgroup(256, 256, K, lda, 256, 256, cfg(0), 256, 0, 0, info.threads)
    waves = sc.wave_streams(ev, counts)
    lds = info.lds_bytes
    assert sc.check_workgroup_lds(waves, lds) == []
    mutated = [edit(ws, keep=keep) for ws in waves]
    assert sc.check_workgroup_lds(mutated, lds), name


# ---------------------------------------------------------------------------
# 3. planted mistakes in a real trace
# ---------------------------------------------------------------------------

def real_waves(tile, extra=3):
    bm, bn, bk, threads = xg.xgemm_tile_info(tile)
    nk = max(stages(tile), 3) + extra
    ev, counts = sc.trace_workgroup(bm, bn, nk * bk, nk * bk, bn, bn, cfg(tile), 256, 0, 0, threads)
    info = xg.xgemm_trace_plan(bm, bn, nk * bk, sc.BASE_A, nk * bk, sc.BASE_B, bn, sc.BASE_C, bn, cfg(tile), 256, 0)
    return sc.wave_streams(ev, counts), info.lds_bytes


def edit(ws, keep=None, arg=None):
    op, a, lds, addr = ws.op.copy(), ws.arg.copy(), ws.lds.copy(), ws.addr.copy()
    if arg is not None:
        a = arg(op, a)
    if keep is not None:
        k = keep(op)
        op, a, lds, addr = op[k], a[k], lds[k], addr[k]
    return sc.WaveStream(op=op, arg=a, lds=lds, addr=addr)


def nth(op, kind, n):
    return np.nonzero(op == kind)[0][n]


MUTANTS = {
    "vmcnt one too weak": lambda w, ws: edit(ws, arg=lambda op, a: np.where(op == sc.WAIT_VM, a + 1, a)),
    "no LDS waits": lambda w, ws: edit(ws, keep=lambda op: op != sc.WAIT_LGKM),
    "no vector-memory waits": lambda w, ws: edit(ws, keep=lambda op: op != sc.WAIT_VM),
    "third barrier dropped": lambda w, ws: edit(ws, keep=lambda op: np.arange(len(op)) != nth(op, sc.BARRIER, 2)),
    "one wave skips a barrier": lambda w, ws: ws if w else edit(
        ws, keep=lambda op: np.arange(len(op)) != nth(op, sc.BARRIER, 3)),
}


@pytest.mark.parametrize("tile", [0, 1])
def test_unmutated_trace_passes(tile):
    waves, lds = real_waves(tile)
    assert sc.check_workgroup_lds(waves, lds) == []


@pytest.mark.parametrize("tile", [0, 1])
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_schedule_mistakes_are_caught(tile, name):
    waves, lds = real_waves(tile)
    mutated = [MUTANTS[name](w, ws) for w, ws in enumerate(waves)]
    found = {v.kind for v in sc.check_workgroup_lds(mutated, lds)}
    assert found, name


@pytest.mark.parametrize("tile", [0, 1])
def test_read_hoisted_above_its_barrier_is_caught(tile):
    waves, lds = real_waves(tile)
    out = []
    for ws in waves:
        b = nth(ws.op, sc.BARRIER, 3)
        r = b + 1 + int(np.argmax(ws.op[b + 1:] == sc.LDS_READ))
        order = np.arange(len(ws.op))
        order[b], order[r] = r, b          # the first read after the barrier moves before it
        out.append(sc.WaveStream(op=ws.op[order], arg=ws.arg[order], lds=ws.lds[order], addr=ws.addr[order]))
    assert {v.kind for v in sc.check_workgroup_lds(out, lds)} & {"raw", "war"}


# ---------------------------------------------------------------------------
# a partial last K step (K a multiple of 8, not of the K step)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("tile", [0, 1, 2])
@pytest.mark.parametrize("shape", [(256, 256, 3 * 64 + 8), (300, 264, 4 * 64 + 56), (520, 136, 2 * 64 + 32)],
                         ids=lambda s: "x".join(map(str, s)))
def test_partial_k_step_traces_are_race_free(tile, shape):
    """The partial step runs first; its clamped loads stay inside A and B,
    the zero fill of the LDS beyond K is ordered before every fragment read,
    and the output is still covered once."""
    M, N, K = shape
    assert xg.xgemm_kernel_family(M, N, K, 1 << 20, K, 1 << 20, N, cfg(tile)) == xg.XGEMM_KERNEL_PIPELINED
    rep = sc.check_launch(M, N, K, cfg(tile))
    assert rep.ok, [str(v) for v in rep.violations]


@pytest.mark.parametrize("tile", [0, 1])
def test_partial_k_step_with_split_k(tile):
    # K = 1224 in 3 splits: 448, 448 and a last one of 328 (5 full steps and 8)
    rep = sc.check_launch(384, 256, 1224, cfg(tile, 3))
    assert rep.ok, [str(v) for v in rep.violations]


def partial_waves(tile):
    bm, bn, bk, _ = xg.xgemm_tile_info(tile)
    K = 4 * bk + 24
    info = xg.xgemm_trace_plan(bm, bn, K, sc.BASE_A, K, sc.BASE_B, bn, sc.BASE_C, bn, cfg(tile), 256, 0)
    ev, counts = sc.trace_workgroup(bm, bn, K, K, bn, bn, cfg(tile), 256, 0, 0, info.threads)
    return sc.wave_streams(ev, counts), info.lds_bytes


@pytest.mark.parametrize("tile", [0, 1])
def test_partial_k_step_zero_fill_is_traced(tile):
    waves, lds = partial_waves(tile)
    assert sc.check_workgroup_lds(waves, lds) == []
    # the 256 x 128 tile's wave pairs write half their sums to LDS after the
    # second-to-last barrier (16 blocks of 16 x 16 each)
    pair = tile == 1 and len(waves) == 8
    for ws in waves:
        # the zero fill: LDS writes between the first barrier and the second
        b0, b1 = nth(ws.op, sc.BARRIER, 0), nth(ws.op, sc.BARRIER, 1)
        assert (ws.op[b0:b1] == sc.LDS_WRITE).sum() > 0
        nbar = int((ws.op == sc.BARRIER).sum())
        end = nth(ws.op, sc.BARRIER, nbar - 2) if pair else len(ws.op)
        assert (ws.op[b1:end] == sc.LDS_WRITE).sum() == 0
        assert (ws.op[end:] == sc.LDS_WRITE).sum() == (16 if pair else 0)


@pytest.mark.parametrize("tile", [0, 1])
def test_partial_k_step_missing_barrier_is_caught(tile):
    """Without the barrier after the zero fill, a wave could read fragments
    before another wave has zeroed them."""
    waves, lds = partial_waves(tile)
    mutated = [edit(ws, keep=lambda op: np.arange(len(op)) != nth(op, sc.BARRIER, 1)) for ws in waves]
    assert {v.kind for v in sc.check_workgroup_lds(mutated, lds)} & {"raw", "war", "waw"}


@pytest.mark.parametrize("which", [-2, -1])
def test_pair_exchange_barriers_are_needed(which):
    """The 256 x 128 tile's wave pairs add their sums through LDS: without
    the last K step's barrier, a wave's writes overwrite a stage that
    another wave may still read; without the one between the writes and the
    reads, a wave reads its partner's half before it is written."""
    bm, bn, bk, threads = xg.xgemm_tile_info(1)
    assert threads == 512
    K = 6 * bk
    ev, counts = sc.trace_workgroup(bm, bn, K, K, bn, bn, cfg(1), 256, 0, 0, threads)
    waves = sc.wave_streams(ev, counts)
    lds = xg.xgemm_trace_plan(bm, bn, K, sc.BASE_A, K, sc.BASE_B, bn, sc.BASE_C, bn, cfg(1), 256, 0).lds_bytes
    assert sc.check_workgroup_lds(waves, lds) == []

    def drop(ws):
        n = int((ws.op == sc.BARRIER).sum())
        return edit(ws, keep=lambda op: np.arange(len(op)) != nth(op, sc.BARRIER, n + which))
    kinds = {v.kind for v in sc.check_workgroup_lds([drop(ws) for ws in waves], lds)}
    assert kinds & ({"war", "waw"} if which == -2 else {"raw"})


# ---------------------------------------------------------------------------
# operands packed into the workspace (layouts the kernels cannot read in place)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("shape,lds,tile,split", [
    ((1000, 1001, 1024), {}, 0, 1),                      # N % 8 != 0: B packed
    ((1000, 1000, 1003), {"lda": 1003, "ldb": 1000}, 0, 1),   # K % 8 != 0: both packed
    ((520, 600, 1536), {"lda": 1540}, 1, 2),             # lda % 8 != 0 with split-k: A packed
    ((1030, 512, 1290), {"ldb": 516}, 2, 1),             # ldb % 8 != 0, partial K step: B packed
], ids=["n_odd", "k_odd", "lda_split", "ldb_partial"])
def test_packed_operand_traces(shape, lds, tile, split):
    """The pipelined kernel reads the packed copies (inside the workspace)
    and never the caller's arrays; the checker takes their bounds from the
    plan.  Large shapes: the first workgroups of each launch are traced."""
    M, N, K = shape
    c = cfg(tile, split)
    info = xg.xgemm_trace_plan(M, N, K, sc.BASE_A, lds.get("lda", K), sc.BASE_B, lds.get("ldb", N), sc.BASE_C, N,
                               c, 256, 0)
    assert info.family == xg.XGEMM_KERNEL_PIPELINED and info.packed != 0
    rep = sc.check_launch(M, N, K, c, max_blocks=3, **lds)
    assert rep.ok, [str(v) for v in rep.violations]


def test_packed_operand_bounds_are_enforced(monkeypatch):
    """A load of the caller's B where the plan reads a packed copy is flagged."""
    real = sc.trace_workgroup

    def to_caller_b(*args, **kw):
        ev, counts = real(*args, **kw)
        ev = ev.copy()
        moved = (ev["op"] == sc.LDS_LOAD) & (ev["addr"] >= sc.BASE_W)
        ev["addr"] = np.where(moved, sc.BASE_B, ev["addr"])
        return ev, counts
    monkeypatch.setattr(sc, "trace_workgroup", to_caller_b)
    # B is packed (N % 8 != 0) and A read in place, so the caller's B is not
    # an operand of the kernel at all
    info = xg.xgemm_trace_plan(1000, 1001, 1024, sc.BASE_A, 1024, sc.BASE_B, 1001, sc.BASE_C, 1001, cfg(0), 256, 0)
    assert info.packed == 2
    rep = sc.check_launch(1000, 1001, 1024, cfg(0), max_blocks=1)
    assert "global_bounds" in {v.kind for v in rep.violations}


def test_duplicate_workgroup_output_is_caught(monkeypatch):
    real = sc.trace_workgroup
    monkeypatch.setattr(sc, "trace_workgroup",
                        lambda M, N, K, lda, ldb, ldc, c, cu, seg, block, threads, capacity=None, schedule=0:
                        real(M, N, K, lda, ldb, ldc, c, cu, seg, 0, threads, capacity, schedule))
    rep = sc.check_launch(512, 512, 256, cfg(0))
    assert "coverage" in {v.kind for v in rep.violations}
    # the persistent kernel's workgroups: one range traced for all
    rep = sc.check_launch(512, 768, 64 * 6, cfg(0, 1, 4, 4))
    assert "coverage" in {v.kind for v in rep.violations}


def test_persistent_partial_sum_races_are_caught(monkeypatch):
    """Under a schedule where both pieces of every split tile find the other
    already counted in (not a real order: one of them must count in first),
    both would add the other's partial and store C: the coverage check
    reports the double stores."""
    real = sc.trace_workgroup

    def both(*args, **kw):
        ev0, c0 = real(*args, **dict(kw, schedule=0))
        ev1, c1 = real(*args, **dict(kw, schedule=1))
        # the head's events come from schedule 0 (it adds), the tail's from 1
        # (it adds too): keep whichever trace stores more of C per thread
        n0 = ((ev0["op"] == sc.STORE) & (ev0["arg"] == 16)).sum()
        n1 = ((ev1["op"] == sc.STORE) & (ev1["arg"] == 16)).sum()
        return (ev0, c0) if n0 >= n1 else (ev1, c1)
    monkeypatch.setattr(sc, "trace_workgroup", both)
    rep = sc.check_launch(512, 768, 64 * 6, cfg(0, 1, 4, 4), schedules=(0,))
    assert "coverage" in {v.kind for v in rep.violations}


def test_load_outside_a_and_b_is_caught(monkeypatch):
    real = sc.trace_workgroup

    def shifted(*args, **kw):
        ev, counts = real(*args, **kw)
        ev = ev.copy()
        ev["addr"] = np.where(ev["op"] == sc.LDS_LOAD, ev["addr"] + 2 * 256 * 256, ev["addr"])
        return ev, counts
    monkeypatch.setattr(sc, "trace_workgroup", shifted)
    rep = sc.check_launch(256, 256, 256, cfg(0))
    assert "global_bounds" in {v.kind for v in rep.violations}


@pytest.mark.parametrize("shape", [(2560, 6656, 1000), (9472, 2048, 1000), (2047, 10239, 1000)],
                         ids=["columns", "rows", "columns_packed"])
def test_band_plan_parts_are_race_free(shape):
    """xgemm_run's body and band launches, each checked on its sub-matrix of
    the full operands (the first workgroups of each launch)."""
    M, N, K = shape
    reps = sc.check_call(M, N, K, max_blocks=2)
    assert len(reps) == 2
    for rep in reps:
        assert rep.ok, [str(v) for v in rep.violations]


def test_band_plan_cli(capsys):
    assert sc.main(["2560", "6656", "1000", "--max-blocks", "1"]) == 0
    out = capsys.readouterr().out
    assert out.count("OK") == 2


def test_cli_reports_ok(capsys):
    assert sc.main(["256", "512", "448", "--tile", "0", "--split", "1"]) == 0
    assert "OK" in capsys.readouterr().out


# ---------------------------------------------------------------------------
# the GEMV kernel: LDS writes from registers, lane-masked accesses
# ---------------------------------------------------------------------------

def prog_w(*ops):
    """As prog, plus ('write', base) a 4-byte LDS write by lane 0 only."""
    plain = [o for o in ops]
    out = prog(*[("wvm", 0) if o[0] == "write" else o for o in plain])
    for i, o in enumerate(plain):
        if o[0] == "write":
            out.op[i] = sc.LDS_WRITE
            out.arg[i] = 4
            out.lds[i] = sc.INACTIVE
            out.lds[i, 0] = o[1]
    return out


def test_lds_write_needs_lgkm_wait_and_barrier():
    reader = prog(("bar",), ("read8", np.where(LANE == 0, 0, sc.INACTIVE)))
    assert verdict(prog_w(("write", 0), ("write", 4), ("wlgkm", 0), ("bar",)), reader) == set()
    assert verdict(prog_w(("write", 0), ("write", 4), ("bar",)), reader) == {"raw"}
    # a vector-memory wait does not retire LDS writes
    assert verdict(prog_w(("write", 0), ("write", 4), ("wvm", 0), ("bar",)), reader) == {"raw"}


def test_neighbouring_4_byte_writes_of_two_waves_do_not_conflict():
    assert verdict(prog_w(("write", 0), ("wlgkm", 0)), prog_w(("write", 4), ("wlgkm", 0))) == set()
    assert verdict(prog_w(("write", 0), ("wlgkm", 0)), prog_w(("write", 0), ("wlgkm", 0))) == {"waw"}


@pytest.mark.parametrize("shape", [(1, 1), (5, 7), (300, 5000), (4097, 777), (64, 100003)])
@pytest.mark.parametrize("rows,unroll", [(1, 1), (2, 4), (4, 2), (8, 4)])
def test_gemv_launch_is_race_free(shape, rows, unroll):
    rep = sc.check_gemv_launch(*shape, xg.xgemv_config(rows, unroll))
    assert rep.ok, [str(v) for v in rep.violations]


@pytest.mark.parametrize("shape,split", [((64, 100003), 8), ((5, 7), 4), ((300, 5000), 3), ((1, 300000), 64)])
def test_gemv_k_split_is_race_free(shape, split):
    rep = sc.check_gemv_launch(*shape, xg.xgemv_config(1, 4, split))
    assert rep.ok, [str(v) for v in rep.violations]
    assert rep.workgroups == shape[0] * sc.gemv_split(shape[1], split)[0]


def test_gemv_padded_rows():
    rep = sc.check_gemv_launch(77, 1001, xg.xgemv_config(4, 2), lda=1007)
    assert rep.ok, [str(v) for v in rep.violations]


def gemv_waves(rows=4):
    ev, counts = sc.trace_gemv_workgroup(64, 4096, 4096, xg.xgemv_config(rows, 2), 0)
    return sc.wave_streams(ev, counts), 16 * rows


@pytest.mark.parametrize("name,keep,expect", [
    # without the barrier, wave 0 (checked first) reads slots the others have
    # not written yet, and their writes then find its unordered reads
    ("no barrier", lambda op: op != sc.BARRIER, {"uninit", "war"}),
    ("no LDS wait", lambda op: op != sc.WAIT_LGKM, {"raw"}),
])
def test_gemv_planted_mistakes(name, keep, expect):
    waves, lds = gemv_waves()
    assert sc.check_workgroup_lds(waves, lds) == []
    mutated = [edit(ws, keep=keep) for ws in waves]
    assert {v.kind for v in sc.check_workgroup_lds(mutated, lds)} == expect, name


def test_gemv_partials_written_to_one_slot_race():
    waves, lds = gemv_waves()
    out = []
    for w, ws in enumerate(waves):
        ws = edit(ws)
        wr = ws.op == sc.LDS_WRITE
        ws.lds[wr] = np.where(ws.lds[wr] == sc.INACTIVE, sc.INACTIVE, ws.lds[wr] % 16)  # every wave: wave 0's slots
        out.append(ws)
    assert "waw" in {v.kind for v in sc.check_workgroup_lds(out, lds)}


def test_gemv_duplicate_rows_are_caught(monkeypatch):
    real = sc.trace_gemv_workgroup
    monkeypatch.setattr(sc, "trace_gemv_workgroup", lambda M, K, lda, cfg, block, capacity=None:
                        real(M, K, lda, cfg, 0, capacity))
    rep = sc.check_gemv_launch(64, 256, xg.xgemv_config(4, 2))
    assert "coverage" in {v.kind for v in rep.violations}


def test_random_small_plans_are_race_free():
    """Seeded random shapes, leading dimensions and configurations, every
    workgroup of every launch traced."""
    rng = np.random.default_rng(7)
    for _ in range(12):
        M, N = (int(v) for v in rng.integers(1, 400, size=2))
        K = int(rng.integers(1, 600))
        lda, ldb = K + int(rng.choice([0, 3, 8])), N + int(rng.choice([0, 5, 8]))
        c = cfg(int(rng.integers(0, 3)), int(rng.choice([1, 2, 4])))
        rep = sc.check_launch(M, N, K, c, lda=lda, ldb=ldb)
        assert rep.ok, ((M, N, K, lda, ldb, c.tile, c.split_k), [str(v) for v in rep.violations][:3])
