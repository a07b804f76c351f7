"""Synchronisation checker for the GEMM and GEMV kernels: an abstract machine
run over the kernels' own operation traces at concrete sizes.

The paper makes every kernel's synchronisation checkable by interpreting an
abstract machine over the program for concrete problem sizes (Section 5,
Abstract Machine): each access to shared memory leaves a read or mutate
record with a visibility level per thread, fences, barrier arrivals and
waits raise those levels, and an access fails its check when an earlier
conflicting record is not yet visible to the accessing thread.  Its
evaluation times that interpreter over square GEMM sizes (Section 6).

Here the same idea is applied to what gfx950 actually synchronises:

* The traces cover both GEMM kernel families (the pipelined kernel with
  direct global-to-LDS loads and explicit waits, the general kernel with
  loads through registers, LDS writes and ``__syncthreads``) and the GEMV.
* Records live on granules of the workgroup's LDS allocation: the largest
  power of two (up to 16 bytes) that divides every access's offset and
  size in the trace, so no granule is shared by accesses that do not
  overlap.  A direct global-to-LDS load or an LDS write leaves a mutate
  record, an LDS read a read record; each record remembers the wave that issued it and its position
  in that wave's counter (vector memory for direct loads and stores, LDS
  for LDS reads), because on this hardware an access completes
  asynchronously and only ``s_waitcnt`` makes its completion known.
* Visibility levels, lowest first: *in flight* (issued, not known to have
  completed); *issuer-ordered* (the issuing wave's ``s_waitcnt`` retired
  it, so it is ordered before that wave's later operations: the paper's
  temporally ordered level for a single thread); *workgroup-ordered* (it
  was issuer-ordered when its wave arrived at an ``s_barrier``, so it is
  ordered before every wave's operations after that barrier: the paper's
  fully ordered level).  ``s_waitcnt`` plays the role of the paper's Fence
  and ``s_barrier`` of Arrive plus Await.
* Checks (the paper's CheckReads / CheckMutates / CheckBarrier): a read
  needs the location's mutate record visible to the reader (no
  read-after-write race) and the location written at all; a direct load
  needs every earlier read and mutate record of its locations visible to
  its wave (no write-after-read or write-after-write race); every wave
  must execute the same number of barriers; no direct load may still be in
  flight when the wave exits (its LDS would be handed to the next
  workgroup); every LDS access stays inside the allocation.

Counters retire in issue order: ``s_waitcnt vmcnt(n)`` means all but the n
most recent vector-memory operations of the wave have completed, and
likewise for ``lgkmcnt``.  A record that the model cannot prove ordered is
reported; the model never assumes an ordering the hardware does not
guarantee (for example it ignores waits the compiler adds for register
dependences, which can only make real executions safer).

Barrier epochs are interpreted in lock step: all waves' operations between
barrier e-1 and barrier e are checked before any after barrier e.  Two
conflicting accesses in the same epoch from different waves are never
ordered, and whichever is checked second fails, so the order in which
waves are visited inside an epoch does not change the verdict.

Beyond the LDS, ``check_launch`` checks each launch's global accesses: every
direct load reads inside A or B, and the stores of all workgroups together
write each element of the launch's output (C, or the split-k partials)
exactly once and nothing else -- two workgroups of one launch are never
ordered, so any overlap is a race.  Partials are summed by a later launch
on the same stream, which the kernel boundary orders after all of them.
"""
from __future__ import annotations

import dataclasses
import hashlib
import time

import numpy as np

from . import xgemm as xg

LANES = 64           # wavefront width

LDS_LOAD = xg.XGEMM_TRACE_LDS_LOAD
LDS_READ = xg.XGEMM_TRACE_LDS_READ
WAIT_VM = xg.XGEMM_TRACE_WAIT_VM
WAIT_LGKM = xg.XGEMM_TRACE_WAIT_LGKM
BARRIER = xg.XGEMM_TRACE_BARRIER
STORE = xg.XGEMM_TRACE_STORE
LDS_WRITE = xg.XGEMM_TRACE_LDS_WRITE
LOAD = xg.XGEMM_TRACE_LOAD
INACTIVE = -1        # LDS offset of a lane that sits out a lane-masked access
VMEM = 100           # wave-stream entry: `arg` global loads or stores (vector-memory counter)


@dataclasses.dataclass
class Violation:
    kind: str        # raw, war, waw, uninit, lds_bounds, barrier_count, inflight_exit, divergent,
                     # global_bounds, coverage
    wave: int        # -1 when not tied to one wave
    event: int       # index in the wave's event stream (-1 if none)
    detail: str

    def __str__(self):
        return "%s (wave %d, event %d): %s" % (self.kind, self.wave, self.event, self.detail)


@dataclasses.dataclass
class WaveStream:
    """One wave's operations in program order; per-lane fields are [n, 64]."""
    op: np.ndarray     # [n] int32
    arg: np.ndarray    # [n] int32
    lds: np.ndarray    # [n, 64] int64
    addr: np.ndarray   # [n, 64] int64


def _collapse_global(events, counts):
    """Per-thread traces with their global loads and stores into registers
    taken out, and for every remaining event the number of such
    vector-memory operations the thread issued since the previous remaining
    event (``before``, one more column for those after the last).

    Lane-masked global accesses (edge tiles, K tails) make lanes of a wave
    issue different numbers of them, so they cannot stand in the wave's
    stream one by one.  They matter to the synchronisation only through the
    vector-memory counter, which they advance; the wave stream gets, before
    each event, the smallest such count over the wave's lanes.  Counting
    fewer operations than were issued makes every ``s_waitcnt vmcnt``
    retire fewer direct loads in the model than on the hardware, so the
    approximation can only report more, never fewer, hazards."""
    threads, cap = events.shape
    valid = np.arange(cap)[None, :] < counts[:, None]
    glob = valid & ((events["op"] == STORE) | (events["op"] == LOAD))
    if not glob.any():
        return events, counts, np.zeros((threads, cap + 1), dtype=np.int64)
    keep = valid & ~glob
    new_counts = keep.sum(axis=1)
    n = max(int(new_counts.max()), 1)
    out = np.zeros((threads, n), dtype=events.dtype)
    before = np.zeros((threads, n + 1), dtype=np.int64)
    for t in range(threads):
        k = np.nonzero(keep[t])[0]
        out[t, :len(k)] = events[t][k]
        g = np.concatenate([[0], np.cumsum(glob[t])])      # g[i]: global ops at positions < i
        at = g[k]
        before[t, :len(k)] = np.diff(np.concatenate([[0], at]))
        before[t, len(k)] = g[counts[t]] - (at[-1] if len(k) else 0)
    return out, new_counts, before


def wave_streams(events: np.ndarray, counts: np.ndarray, violations: list | None = None):
    """Group a workgroup trace (threads x capacity records, per-thread
    counts) into per-wave streams of its direct LDS loads, LDS reads and
    writes, waits and barriers, with VMEM entries standing for the global
    loads and stores between them (see _collapse_global).  Lanes of one
    wave must issue the same operations with the same wave-uniform
    operands; a lane that does not is reported as a divergence and the
    wave's stream is cut there."""
    threads = events.shape[0]
    assert threads % LANES == 0
    events, counts, before = _collapse_global(events, counts)
    out = []
    for w in range(threads // LANES):
        lanes = slice(w * LANES, (w + 1) * LANES)
        cnt = counts[lanes]
        n = int(cnt.min())
        if int(cnt.max()) != n and violations is not None:
            violations.append(Violation("divergent", w, n, "lanes issue %d to %d operations" %
                                        (n, int(cnt.max()))))
        ev = events[lanes, :n]
        op = ev["op"][0].copy()
        arg = ev["arg"][0].copy()
        same = (ev["op"] == op).all(axis=0) & (ev["arg"] == arg).all(axis=0)
        uniform_lds = (op == LDS_LOAD)
        same &= ~uniform_lds | (ev["lds"] == ev["lds"][0]).all(axis=0)
        if not same.all():
            cut = int(np.argmin(same))
            if violations is not None:
                violations.append(Violation("divergent", w, cut, "lanes disagree on the operation"))
            n = cut
            op, arg, ev = op[:n], arg[:n], ev[:, :n]
        vm = before[lanes, :n + 1].min(axis=0)
        lds = ev["lds"].T
        addr = ev["addr"].T
        if vm.any():
            # insert a VMEM entry before every event (and after the last) that
            # follows global operations in every lane
            pos = np.nonzero(vm[:n])[0]
            op = np.insert(op, pos, VMEM)
            arg = np.insert(arg, pos, vm[pos].astype(arg.dtype))
            lds = np.insert(lds, pos, 0, axis=0)
            addr = np.insert(addr, pos, 0, axis=0)
            if vm[n]:
                op = np.append(op, np.int32(VMEM))
                arg = np.append(arg, np.int32(vm[n]))
                lds = np.vstack([lds, np.zeros((1, LANES), lds.dtype)])
                addr = np.vstack([addr, np.zeros((1, LANES), addr.dtype)])
        out.append(WaveStream(op=op.astype(np.int32), arg=arg.astype(np.int32), lds=np.ascontiguousarray(lds),
                              addr=np.ascontiguousarray(addr)))
    return out


class LdsMachine:
    """Abstract machine over one workgroup's LDS (see the module docstring)."""

    def __init__(self, lds_bytes: int, nwaves: int, granule: int = 8, max_reports: int = 20):
        self.lds_bytes = lds_bytes
        self.nw = nwaves
        self.granule = granule
        g = (lds_bytes + granule - 1) // granule
        self.mut_w = np.full(g, -1, dtype=np.int64)     # wave of the live mutate record
        self.mut_s = np.full(g, -1, dtype=np.int64)     # its position in that wave's counter
        self.mut_c = np.zeros(g, dtype=np.int8)         # the counter: 0 vector memory, 1 LDS
        self.rd_s = np.full((g, nwaves), -1, dtype=np.int64)  # latest read per wave since then
        self.issued = {"vm": np.zeros(nwaves, np.int64), "lgkm": np.zeros(nwaves, np.int64)}
        self.done = {"vm": np.zeros(nwaves, np.int64), "lgkm": np.zeros(nwaves, np.int64)}
        self.seen = {"vm": np.zeros(nwaves, np.int64), "lgkm": np.zeros(nwaves, np.int64)}
        self.last_load = np.full(nwaves, -1, dtype=np.int64)  # counter position of the last direct load
        self.violations: list[Violation] = []
        self.max_reports = max_reports
        self.n_reported = {}

    # -- helpers -------------------------------------------------------------
    def _report(self, kind, wave, event, detail):
        k = self.n_reported.get(kind, 0)
        self.n_reported[kind] = k + 1
        if k < self.max_reports:
            self.violations.append(Violation(kind, wave, event, detail))

    def _visible(self, counter, owner, pos, x):
        """Records (owner wave, counter position) visible to wave x."""
        return (pos < self.seen[counter][owner]) | ((owner == x) & (pos < self.done[counter][x]))

    def _mut_visible(self, g, x):
        """Live mutate records of granules g (all present) visible to wave x."""
        w, pos, c = self.mut_w[g], self.mut_s[g], self.mut_c[g]
        return np.where(c == 0, self._visible("vm", w, pos, x), self._visible("lgkm", w, pos, x))

    def _granules(self, wave, i, start, nbytes):
        """Granules covered by per-lane accesses [start, start + nbytes)."""
        if (start < 0).any() or (start + nbytes > self.lds_bytes).any():
            bad = start[(start < 0) | (start + nbytes > self.lds_bytes)]
            self._report("lds_bounds", wave, i, "LDS bytes [%d, %d) outside the %d-byte allocation" %
                         (int(bad[0]), int(bad[0]) + nbytes, self.lds_bytes))
            start = start[(start >= 0) & (start + nbytes <= self.lds_bytes)]
        first = start // self.granule
        last = (start + nbytes - 1) // self.granule
        span = int((last - first).max()) + 1 if len(first) else 0
        g = (first[:, None] + np.arange(span)[None, :])
        g = g[g <= last[:, None]]
        return np.unique(g)

    # -- operations ----------------------------------------------------------
    def lds_load(self, w, i, base, nbytes):
        """Direct load: lane l writes nbytes at base + nbytes * l."""
        g = self._granules(w, i, base + nbytes * np.arange(LANES, dtype=np.int64), nbytes)
        self._mutate(w, i, g, "vm", "direct load")
        self.last_load[w] = self.issued["vm"][w] - 1

    def lds_write(self, w, i, addrs, nbytes):
        """LDS write from registers by the active lanes."""
        g = self._granules(w, i, addrs[addrs != INACTIVE], nbytes)
        self._mutate(w, i, g, "lgkm", "LDS write")

    def _mutate(self, w, i, g, counter, what):
        mw = self.mut_w[g]
        has = mw >= 0
        if has.any():
            ok = self._mut_visible(g[has], w)
            if not ok.all():
                bad = g[has][~ok][0]
                self._report("waw", w, i, "LDS byte %d: earlier write by wave %d not ordered before this %s"
                             % (bad * self.granule, int(self.mut_w[bad]), what))
        rs = self.rd_s[g]                                     # [len(g), nw]
        has = rs >= 0
        if has.any():
            owners = np.broadcast_to(np.arange(self.nw), rs.shape)[has]
            ok = self._visible("lgkm", owners, rs[has], w)
            if not ok.all():
                rows, cols = np.nonzero(has)
                k = int(np.argmin(ok))
                self._report("war", w, i, "LDS byte %d: read by wave %d not complete and ordered before "
                             "this %s overwrites it" % (g[rows[k]] * self.granule, int(cols[k]), what))
        self.mut_w[g] = w
        self.mut_s[g] = self.issued[counter][w]
        self.mut_c[g] = 0 if counter == "vm" else 1
        self.rd_s[g] = -1
        self.issued[counter][w] += 1

    def lds_read(self, w, i, addrs, nbytes):
        g = self._granules(w, i, addrs[addrs != INACTIVE], nbytes)
        mw = self.mut_w[g]
        if (mw < 0).any():
            bad = g[mw < 0][0]
            self._report("uninit", w, i, "LDS byte %d read but never written" % (bad * self.granule))
        has = mw >= 0
        if has.any():
            ok = self._mut_visible(g[has], w)
            if not ok.all():
                bad = g[has][~ok][0]
                self._report("raw", w, i, "LDS byte %d: write by wave %d not complete and ordered "
                             "before this read" % (bad * self.granule, int(self.mut_w[bad])))
        self.rd_s[g, w] = self.issued["lgkm"][w]
        self.issued["lgkm"][w] += 1

    def wait(self, w, counter, n):
        self.done[counter][w] = max(self.done[counter][w], self.issued[counter][w] - n)

    def barrier(self):
        for c in ("vm", "lgkm"):
            self.seen[c] = self.done[c].copy()

    # -- driver --------------------------------------------------------------
    def run(self, waves: list[WaveStream]):
        """Interpret every wave's stream; returns the violations found."""
        assert len(waves) == self.nw
        cuts = []
        for ws in waves:
            b = np.nonzero(ws.op == BARRIER)[0]
            cuts.append(np.concatenate([[-1], b, [len(ws.op)]]))
        nb = [len(c) - 2 for c in cuts]
        if len(set(nb)) != 1:
            self._report("barrier_count", -1, -1, "waves execute %s barriers (a workgroup barrier "
                         "needs every wave)" % nb)
        epochs = min(nb) + 1
        for e in range(epochs):
            for w, ws in enumerate(waves):
                lo, hi = cuts[w][e] + 1, cuts[w][e + 1]
                for i in range(lo, hi):
                    op = ws.op[i]
                    if op == LDS_LOAD:
                        self.lds_load(w, i, int(ws.lds[i, 0]), int(ws.arg[i]))
                    elif op == LDS_READ:
                        self.lds_read(w, i, ws.lds[i], int(ws.arg[i]))
                    elif op == LDS_WRITE:
                        self.lds_write(w, i, ws.lds[i], int(ws.arg[i]))
                    elif op == VMEM:
                        self.issued["vm"][w] += int(ws.arg[i])
                    elif op == WAIT_VM:
                        self.wait(w, "vm", int(ws.arg[i]))
                    elif op == WAIT_LGKM:
                        self.wait(w, "lgkm", int(ws.arg[i]))
            if e + 1 < epochs:
                self.barrier()
        for w in range(self.nw):
            if self.last_load[w] >= self.done["vm"][w]:
                self._report("inflight_exit", w, len(waves[w].op),
                             "direct loads into LDS still in flight when the wave exits")
        return self.violations


def granule_for(waves: list[WaveStream]) -> int:
    """Largest power of two up to 16 dividing every LDS access's offset and
    size in these streams."""
    g = 16
    for ws in waves:
        acc = np.isin(ws.op, (LDS_LOAD, LDS_READ, LDS_WRITE))
        if not acc.any():
            continue
        vals = [ws.arg[acc].astype(np.int64)]
        lds = ws.lds[acc]
        vals.append(lds[lds != INACTIVE])
        for v in vals:   # (lane l of a direct load lands at base + arg * l)
            while g > 1 and (v % g).any():
                g //= 2
    return g


def check_workgroup_lds(waves: list[WaveStream], lds_bytes: int) -> list[Violation]:
    return LdsMachine(lds_bytes, len(waves), granule_for(waves)).run(waves)


# ---------------------------------------------------------------------------
# whole launches
# ---------------------------------------------------------------------------

# Stand-in addresses for traced calls: 16-byte aligned, far apart, never
# dereferenced.
BASE_A = 1 << 40
BASE_B = 2 << 40
BASE_C = 3 << 40
BASE_W = 4 << 40


@dataclasses.dataclass
class LaunchReport:
    shape: tuple
    config: str
    segments: int
    workgroups: int
    lds_classes: int         # distinct LDS operation streams interpreted
    events: int              # operations traced (all threads)
    seconds: float
    violations: list

    @property
    def ok(self):
        return not self.violations


def trace_workgroup(M, N, K, lda, ldb, ldc, cfg, cu_count, seg, block, threads, capacity=None, schedule=0):
    """(events [threads, capacity], counts [threads]) of one workgroup.
    `threads` must be the launch's thread count (xgemm_trace_plan's
    info.threads): the library writes that many counts.  `schedule` is the
    order in which the two pieces of a persistent kernel's split tile count
    in (0: its last K steps first)."""
    import ctypes
    info = xg.xgemm_trace_plan(M, N, K, BASE_A, lda, BASE_B, ldb, BASE_C, ldc, cfg, cu_count, seg)
    if threads != info.threads:
        raise ValueError("trace_workgroup: the launch has %d threads per workgroup, not %d" % (info.threads, threads))
    counts = np.zeros(threads, dtype=np.int64)
    cptr = counts.ctypes.data_as(ctypes.c_void_p)
    args = (M, N, K, BASE_A, lda, BASE_B, ldb, BASE_C, ldc, BASE_W, ctypes.byref(cfg), cu_count, seg, block,
            schedule)
    if capacity is None:
        rc = xg.lib.xgemm_trace_workgroup(*args, None, 0, cptr)
        if rc != xg.XGEMM_OK:
            raise xg.XgemmError(rc)
        capacity = max(int(counts.max()), 1)
    ev = np.zeros((threads, capacity), dtype=xg.TRACE_EVENT_DTYPE)
    rc = xg.lib.xgemm_trace_workgroup(*args, ev.ctypes.data_as(ctypes.c_void_p), capacity, cptr)
    if rc != xg.XGEMM_OK:
        raise xg.XgemmError(rc)
    if int(counts.max()) > capacity:
        return trace_workgroup(M, N, K, lda, ldb, ldc, cfg, cu_count, seg, block, threads, int(counts.max()),
                               schedule)
    return ev, counts


class _Coverage:
    """Counts how often each element of a launch's outputs is stored: C, the
    full-matrix split partials, or (the persistent kernel) C and its
    partial sums, two per slot of BM x BN floats; the persistent kernel's
    4-byte counter stores are only checked to hit the counter prefix."""

    def __init__(self, info, M, N, ldc, bm, bn):
        self.reduce = info.reduce
        self.sk = info.family == xg.XGEMM_KERNEL_PERSISTENT
        self.M, self.N, self.ldc, self.bm, self.bn = M, N, ldc, bm, bn
        self.split = info.split
        self.count = np.zeros((M, N), dtype=np.uint8) if info.reduce == 0 else None
        self.ldw = (N + 3) // 4 * 4
        if info.reduce == 1:
            self.pbase = BASE_W + info.data_offset
            self.part = np.zeros((info.split, M, N), dtype=np.uint8)
        elif self.sk:
            self.pbase = BASE_W + info.data_offset
            self.part = np.zeros(2 * info.grid * bm * bn, dtype=np.uint8)
        else:
            self.part = None

    def _c(self, off):
        e = off // 4
        i, j = e // self.ldc, e % self.ldc
        ok = (e >= 0) & (i < self.M) & (j < self.N)
        return ok, (i[ok], j[ok])

    def _p(self, off):
        e = off // 4
        if self.reduce == 1:
            per = self.M * self.ldw
            p, r = e // per, e % per
            i, j = r // self.ldw, r % self.ldw
            ok = (e >= 0) & (p < self.split) & (j < self.N)
            return ok, (p[ok], i[ok], j[ok])
        ok = (e >= 0) & (e < len(self.part))
        return ok, (e[ok],)

    def add(self, addr, nbytes):
        """Record stores of nbytes at each address; returns a list of problems."""
        bad = []
        if self.sk and nbytes == 4:
            # counter resets
            off = addr - BASE_W
            if ((off < 0) | (off >= PREFIX_BYTES) | (off % 4 != 0)).any():
                bad.append("4-byte store outside the counter prefix")
            return bad
        in_c = (addr >= BASE_C) & (addr < BASE_W) if self.count is not None else np.zeros(len(addr), bool)
        for sel, base, region in ((in_c, BASE_C, "C"), (~in_c, getattr(self, "pbase", BASE_W), "partials")):
            a = addr[sel]
            if not len(a):
                continue
            off = a - base
            if (off % 4).any():
                bad.append("store not aligned to a float")
            for k in range(nbytes // 4):
                ok, idx = self._c(off + 4 * k) if region == "C" else (self._p(off + 4 * k) if self.part is not None
                                                                       else (np.zeros(len(off), bool), None))
                if not ok.all():
                    bad.append("store outside the output at byte offset %d" % int(off[~ok][0] + 4 * k))
                if idx is not None:
                    np.add.at(self.count if region == "C" else self.part, idx, 1)
        return bad

    def written(self, addr, nbytes):
        """Whether the partial elements that loads of nbytes at addr read were
        all stored by some workgroup of the launch."""
        off = addr - self.pbase
        ok = np.ones(len(addr), bool)
        for k in range(nbytes // 4):
            inside, idx = self._p(off + 4 * k)
            ok &= inside
            ok[inside] &= self.part[idx] == 1
        return ok

    def result(self):
        arr = self.count if self.reduce == 0 else self.part
        zero = int((arr == 0).sum())
        many = int((arr > 1).sum())
        return zero, many

    def partial_many(self):
        return int((self.part > 1).sum()) if self.part is not None else 0


PREFIX_BYTES = 4096   # the workspace's counter prefix


def check_launch(M, N, K, cfg, cu_count=256, lda=None, ldb=None, ldc=None, max_blocks=None, schedules=None):
    """Trace every workgroup of every launch of the plan for this call and
    run the checks; returns a LaunchReport.  max_blocks limits the
    workgroups traced per launch (for quick checks of large shapes; the
    coverage check is then skipped).  A persistent launch that splits tiles
    is checked under both orders of its split tiles' pieces (schedules 0
    and 1) unless `schedules` names them."""
    lda = K if lda is None else lda
    ldb = N if ldb is None else ldb
    ldc = N if ldc is None else ldc
    t0 = time.perf_counter()
    violations: list[Violation] = []
    lds_seen = set()
    n_events = 0
    n_blocks = 0
    bm, bn, _, _ = xg.xgemm_tile_info(cfg.tile)
    info0 = xg.xgemm_trace_plan(M, N, K, BASE_A, lda, BASE_B, ldb, BASE_C, ldc, cfg, cu_count, 0)
    # the operands as the kernels read them: the caller's A and B, or their
    # zero-padded copies in the workspace (M x k and k x ldb)
    if info0.packed & 1:
        a_lo = BASE_W + info0.a_offset
        a_hi = a_lo + 2 * ((M - 1) * info0.lda + info0.k)
    else:
        a_lo, a_hi = BASE_A, BASE_A + 2 * ((M - 1) * lda + K)
    if info0.packed & 2:
        b_lo = BASE_W + info0.b_offset
        b_hi = b_lo + 2 * info0.k * info0.ldb
    else:
        b_lo, b_hi = BASE_B, BASE_B + 2 * ((K - 1) * ldb + N)
    for seg in range(info0.segments):
        info = xg.xgemm_trace_plan(M, N, K, BASE_A, lda, BASE_B, ldb, BASE_C, ldc, cfg, cu_count, seg)
        sk = info.family == xg.XGEMM_KERNEL_PERSISTENT
        scheds = schedules if schedules is not None else ((0, 1) if sk and info.sk_tiles > 0 else (0,))
        nblk = info.grid if max_blocks is None else min(info.grid, max_blocks)
        for schedule in scheds:
            cov = _Coverage(info, M, N, ldc, bm, bn)
            part_loads = []
            for block in range(nblk):
                ev, counts = trace_workgroup(M, N, K, lda, ldb, ldc, cfg, cu_count, seg, block, info.threads,
                                             schedule=schedule)
                n_blocks += 1
                n_events += int(counts.sum())
                valid = np.arange(ev.shape[1])[None, :] < counts[:, None]
                # global reads: direct (to LDS) and register loads; the
                # persistent kernel also reads its counters and partial sums
                ld = valid & ((ev["op"] == LDS_LOAD) | (ev["op"] == LOAD))
                ga = ev["addr"][ld]
                nb = ev["arg"][ld]
                inside = ((ga >= a_lo) & (ga + nb <= a_hi)) | ((ga >= b_lo) & (ga + nb <= b_hi))
                if sk:
                    ctr = (ga >= BASE_W) & (ga + nb <= BASE_W + PREFIX_BYTES) & (nb == 4)
                    part = (ga >= BASE_W + info.data_offset) & (ga + nb <= BASE_W + info.workspace_bytes) & (nb == 16)
                    inside |= ctr | part
                    part_loads.append(ga[part])
                if not inside.all():
                    violations.append(Violation("global_bounds", -1, -1, "launch %d workgroup %d: load "
                                                "reads outside A and B at address %#x" %
                                                (seg, block, int(ga[~inside][0]))))
                # global stores
                st = valid & (ev["op"] == STORE)
                for nbytes in np.unique(ev["arg"][st]):
                    sel = st & (ev["arg"] == nbytes)
                    for msg in cov.add(ev["addr"][sel], int(nbytes)):
                        violations.append(Violation("global_bounds", -1, -1, "launch %d workgroup %d: %s" %
                                                    (seg, block, msg)))
                # LDS: one interpretation per distinct operation stream
                key = hashlib.sha1()
                for f in ("op", "arg", "lds"):
                    key.update(np.where(valid, ev[f], 0).tobytes())
                key.update(counts.tobytes())
                key = key.digest()
                if key not in lds_seen:
                    lds_seen.add(key)
                    pre = []
                    waves = wave_streams(ev, counts, pre)
                    violations.extend(pre)
                    for v in check_workgroup_lds(waves, info.lds_bytes):
                        v.detail = "launch %d workgroup %d: %s" % (seg, block, v.detail)
                        violations.append(v)
            if max_blocks is not None:
                continue
            zero, many = cov.result()
            tag = "launch %d%s" % (seg, " (schedule %d)" % schedule if sk else "")
            if many:
                violations.append(Violation("coverage", -1, -1, "%s: %d output elements stored by more than one "
                                            "store (unordered workgroups race)" % (tag, many)))
            if zero and info.reduce == 1:
                violations.append(Violation("coverage", -1, -1, "%s: %d partial elements never written" %
                                            (tag, zero)))
            if info.reduce == 0 and zero:
                violations.append(Violation("coverage", -1, -1, "%s: %d elements of C never written" % (tag, zero)))
            if sk:
                if cov.partial_many():
                    violations.append(Violation("coverage", -1, -1, "%s: %d partial-sum elements stored twice" %
                                                (tag, cov.partial_many())))
                pl = np.concatenate(part_loads) if part_loads else np.zeros(0, np.int64)
                if len(pl) and not cov.written(pl, 16).all():
                    violations.append(Violation("coverage", -1, -1, "%s: a partial sum read that no workgroup "
                                                "stores" % tag))
    return LaunchReport(shape=(M, N, K), config=repr(cfg), segments=info0.segments, workgroups=n_blocks,
                        lds_classes=len(lds_seen), events=n_events, seconds=time.perf_counter() - t0,
                        violations=violations)


def trace_gemv_workgroup(M, K, lda, cfg, block, capacity=None):
    """(events [256, capacity], counts [256]) of one GEMV workgroup, with A
    at BASE_A, x at BASE_B and y at BASE_C."""
    import ctypes
    threads = 256
    counts = np.zeros(threads, dtype=np.int64)
    cptr = counts.ctypes.data_as(ctypes.c_void_p)
    args = (M, K, BASE_A, lda, BASE_B, BASE_C, BASE_W, ctypes.byref(cfg), block)
    if capacity is None:
        rc = xg.lib.xgemv_trace_workgroup(*args, None, 0, cptr)
        if rc != xg.XGEMM_OK:
            raise xg.XgemmError(rc)
        capacity = max(int(counts.max()), 1)
    ev = np.zeros((threads, capacity), dtype=xg.TRACE_EVENT_DTYPE)
    rc = xg.lib.xgemv_trace_workgroup(*args, ev.ctypes.data_as(ctypes.c_void_p), capacity, cptr)
    if rc != xg.XGEMM_OK:
        raise xg.XgemmError(rc)
    if int(counts.max()) > capacity:
        return trace_gemv_workgroup(M, K, lda, cfg, block, int(counts.max()))
    return ev, counts


def gemv_split(K, split):
    """The K split a GEMV launch runs after empty trailing ranges are
    dropped, and the K values per range (the library's rule)."""
    def chunk(s):
        return -(-(-(-K // s)) // 4) * 4
    kc = chunk(split)
    while split > 1 and kc * (split - 1) >= K:
        split -= 1
        kc = chunk(split)
    return split, kc


def check_gemv_launch(M, K, cfg, lda=None):
    """Trace every workgroup of the GEMV launch and run the checks: the LDS
    machine on each distinct workgroup stream, global loads inside A and x,
    and every y[i] (or, with a K split, every partial sum) stored exactly
    once.  The partial sums are added by a later launch on the same stream."""
    import ctypes
    lda = K if lda is None else lda
    t0 = time.perf_counter()
    violations: list[Violation] = []
    lds_seen = set()
    n_events = 0
    split, _ = gemv_split(K, cfg.split_k)
    grid = -(-M // cfg.rows) * split
    counts = np.zeros(256, dtype=np.int64)
    beyond = xg.lib.xgemv_trace_workgroup(M, K, BASE_A, lda, BASE_B, BASE_C, BASE_W, ctypes.byref(cfg), grid, None,
                                          0, counts.ctypes.data_as(ctypes.c_void_p))
    if beyond != xg.XGEMM_ERR_INVALID_ARG:
        violations.append(Violation("coverage", -1, -1, "the library runs more than %d workgroups" % grid))
    lds_bytes = 4 * 4 * cfg.rows
    a_lo, a_hi = BASE_A, BASE_A + 4 * ((M - 1) * lda + K)
    x_lo, x_hi = BASE_B, BASE_B + 4 * K
    out_base = BASE_C if split == 1 else BASE_W
    cov = np.zeros(M * split, dtype=np.int64)
    for block in range(grid):
        ev, counts = trace_gemv_workgroup(M, K, lda, cfg, block)
        n_events += int(counts.sum())
        valid = np.arange(ev.shape[1])[None, :] < counts[:, None]
        ld = valid & (ev["op"] == LOAD)
        ga, nb = ev["addr"][ld], ev["arg"][ld]
        inside = ((ga >= a_lo) & (ga + nb <= a_hi)) | ((ga >= x_lo) & (ga + nb <= x_hi))
        if not inside.all():
            violations.append(Violation("global_bounds", -1, -1, "workgroup %d: load outside A and x at %#x"
                                        % (block, int(ga[~inside][0]))))
        st = valid & (ev["op"] == STORE)
        off = ev["addr"][st] - out_base
        ok = (off >= 0) & (off % 4 == 0) & (off // 4 < M * split) & (ev["arg"][st] == 4)
        if not ok.all():
            violations.append(Violation("global_bounds", -1, -1, "workgroup %d: store outside %s" %
                                        (block, "y" if split == 1 else "the partial sums")))
        np.add.at(cov, off[ok] // 4, 1)
        key = hashlib.sha1()
        for f in ("op", "arg", "lds"):
            key.update(np.where(valid & (ev["op"] != LOAD) & (ev["op"] != STORE), ev[f], 0).tobytes())
        key = key.digest()
        if key not in lds_seen:
            lds_seen.add(key)
            pre = []
            waves = wave_streams(ev, counts, pre)
            violations.extend(pre)
            for v in check_workgroup_lds(waves, lds_bytes):
                v.detail = "workgroup %d: %s" % (block, v.detail)
                violations.append(v)
    if (cov != 1).any():
        violations.append(Violation("coverage", -1, -1, "%d entries of %s not stored exactly once"
                                    % (int((cov != 1).sum()), "y" if split == 1 else "the partial sums")))
    return LaunchReport(shape=(M, K), config=repr(cfg), segments=1, workgroups=grid, lds_classes=len(lds_seen),
                        events=n_events, seconds=time.perf_counter() - t0, violations=violations)


def check_call(M, N, K, dtype=0, cu_count=256, max_blocks=None):
    """Check the launches xgemm_run makes for a call with 16-byte aligned A,
    B and C at lda = K, ldb = ldc = N: one plan, or a body and a band of C
    (xgemm_select_band), each checked as its own call on the sub-matrix.
    Returns one LaunchReport per part."""
    band = xg.xgemm_select_band(M, N, K, dtype, cu_count)
    if band.axis == xg.XGEMM_BAND_NONE:
        return [check_launch(M, N, K, band.body, cu_count, max_blocks=max_blocks)]
    e = band.extent
    if band.axis == xg.XGEMM_BAND_COLUMNS:
        parts = [((M, e), band.body), ((M, N - e), band.band)]
    else:
        parts = [((e, N), band.body), ((M - e, N), band.band)]
    return [check_launch(m, n, K, c, cu_count, lda=K, ldb=N, ldc=N, max_blocks=max_blocks)
            for (m, n), c in parts]


def main(argv=None):
    import argparse
    ap = argparse.ArgumentParser(description="synchronisation check of the GEMM kernels for one call")
    ap.add_argument("M", type=int)
    ap.add_argument("N", type=int)
    ap.add_argument("K", type=int)
    ap.add_argument("--tile", type=int, default=None)
    ap.add_argument("--split", type=int, default=None)
    ap.add_argument("--stream-k", type=int, default=0,
                    help="the persistent stream-K kernel: 1 on every CU, n > 1 on n workgroups")
    ap.add_argument("--group-m", type=int, default=None)
    ap.add_argument("--cu-count", type=int, default=256)
    ap.add_argument("--max-blocks", type=int, default=None)
    args = ap.parse_args(argv)
    if all(v is None for v in (args.tile, args.split, args.group_m)) and args.stream_k == 0:
        # the selector's plan, as xgemm_run makes it (possibly a body and a band)
        reps = check_call(args.M, args.N, args.K, xg.XGEMM_BF16, args.cu_count, args.max_blocks)
        for rep in reps:
            print("%s %s: %d launch(es), %d workgroups, %d LDS streams, %d events, %.2f s: %s" % (
                rep.shape, rep.config, rep.segments, rep.workgroups, rep.lds_classes, rep.events, rep.seconds,
                "OK" if rep.ok else "%d violation(s)" % len(rep.violations)))
            for v in rep.violations[:20]:
                print("  ", v)
        return 0 if all(r.ok for r in reps) else 1
    cfg = xg.xgemm_select_config(args.M, args.N, args.K, xg.XGEMM_BF16, args.cu_count)
    if args.tile is not None:
        cfg.tile = args.tile
    if args.split is not None:
        cfg.split_k = args.split
    if args.group_m is not None:
        cfg.group_m = args.group_m
    cfg.stream_k = args.stream_k
    try:
        rep = check_launch(args.M, args.N, args.K, cfg, args.cu_count, max_blocks=args.max_blocks)
    except xg.XgemmError as e:
        print("%s %r: not checked: %s" % ((args.M, args.N, args.K), cfg, e))
        return 2
    print("%s %s: %d launch(es), %d workgroups, %d LDS streams, %d events, %.2f s: %s" % (
        rep.shape, rep.config, rep.segments, rep.workgroups, rep.lds_classes, rep.events, rep.seconds,
        "OK" if rep.ok else "%d violation(s)" % len(rep.violations)))
    for v in rep.violations[:20]:
        print("  ", v)
    return 0 if rep.ok else 1


if __name__ == "__main__":
    raise SystemExit(main())
