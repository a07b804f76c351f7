// Persistent stream-K GEMM kernel for gfx950 (the 256 x 256 tile, eight
// waves of 128 x 64, as gemm_kernel_dma).
//
// The paper's kernels are persistent: a fixed grid walks a task generator
// over the output tiles (Section 4.2, code generation), and it attributes
// the variation it sees on small and very long-K problems to wave
// quantisation (Section 6).  Here one workgroup runs per CU and walks a
// fixed list of K steps:
//   * dp_rounds rounds of whole tiles (tile lw + r * grid in round r, lw the
//     workgroup's logical id), then
//   * a contiguous range of K steps of the remaining tiles (stream-K): the
//     steps of those sk_tiles tiles, tile after tile, are cut into `grid`
//     ranges of equal length.  Every range holds at least one tile's worth
//     of steps, so a tile is split between at most two neighbouring ranges:
//     the first steps (from k = 0) at the end of range lw, the rest at the
//     start of range lw + 1.
// The tiles may belong to the problems of a strided batch (tile t is tile
// t % tiles_per of problem t / tiles_per).
// The LDS pipeline runs across tile boundaries: during a tile's last K
// steps the loads of the next tile's first steps are already in flight, and
// a finished tile's C stores (streaming stores) are issued at the start of
// the next tile's first step, whose MFMAs start from zero, so no second set
// of accumulators is needed.  That step waits while the memory side takes
// the stores (all workgroups of a round store at once); no tile after a
// workgroup's first has a prologue of its own.
//
// A tile split between ranges lw and lw + 1 (its slot is lw + 1) is
// finished by whichever of its two pieces completes second, without any
// wait.  The piece of the last steps (at the start of range lw + 1) writes
// its partial sum to its half of the slot with device-scope stores, waits
// for them to complete and counts in with an atomic add.  The piece of the
// first steps (at the end of range lw) reads the counter: if the other
// piece has counted in, it adds that partial (device-scope loads) and
// stores C; otherwise it publishes its own partial the same way.  Whichever
// piece's add returns 1 forms the sum and resets the counter, so every call
// leaves all counters zero.  The sum is always the tile's first steps plus
// its last steps (fp32 addition is commutative, so the bits do not depend on
// which piece finishes it).  In the usual order the last steps are done long
// before the first steps, so one partial is written and read per split
// tile.  Device-scope accesses make the partials visible across XCDs
// without writing back or invalidating whole L2 caches.
#pragma once

#include "gemm_kernel.hpp"

namespace xgemm_dev {

struct SkParams {
    const uint16_t *A;
    const uint16_t *B;
    float *C;
    float *part;      // partial sums of slot s: 2 * BM * BN floats at part + s * 2 * BM * BN
                      // (the tile's first steps, then its last steps)
    int *flags;       // counter of slot s: flags[s] (pieces counted in; zero between calls)
    int64_t lda, ldb, ldc;
    int M, N, K;      // M and N multiples of the tile, K of the K step
    int tiles_m, tiles_n, group_m;
    int tiles_per;    // tiles of one problem (tiles_m * tiles_n); tile t is tile t % tiles_per of
                      // problem t / tiles_per, whose A, B and C start stride_a, stride_b,
                      // stride_c elements (times the problem index) after A, B and C
    int64_t stride_a, stride_b, stride_c;
    int kt;           // K steps per tile (K is a multiple of the K step)
    int grid;         // workgroups of the launch (one per CU)
    int dp_rounds;    // rounds of whole tiles before the shared ones
    int sk_tiles;     // tiles after those rounds, shared out as K-step ranges
};

// LDS bytes of the persistent kernel: two stages and the words through
// which thread 0 tells the workgroup what a split tile's counter said.
template <int BM, int BN, int BK>
constexpr int sk_lds_bytes()
{
    return 2 * (BM * BK * 2 + BK * BN * 2) + 256;
}

// Logical workgroup id: the hardware hands workgroup ids to the XCDs
// round-robin; consecutive logical ids are gathered onto one XCD, so that
// the tiles an XCD works on at one time are neighbours (as map_tile).
__host__ __device__ __forceinline__ int sk_logical(int block, int grid)
{
    const int per = grid / kNumXcd;
    return block < per * kNumXcd ? (block % kNumXcd) * per + block / kNumXcd : block;
}

// A tile of the launch: problem b, tile (m, n) of that problem's C.
struct SkTile {
    int b, m, n;
};

__host__ __device__ __forceinline__ SkTile sk_tile_of(const SkParams &p, int t)
{
    SkTile r;
    r.b = t / p.tiles_per;
    logical_tile(t - r.b * p.tiles_per, p.tiles_m, p.tiles_n, p.group_m, r.m, r.n);
    return r;
}

// The K-step range of logical workgroup lw: steps [0, gdp) are its whole
// tiles, [gdp, G) its share [s0, s1) of the stream-K steps.
struct SkRange {
    int gdp, G, s0, s1;
};

__host__ __device__ __forceinline__ SkRange sk_range(const SkParams &p, int lw)
{
    SkRange r;
    const int64_t isk = (int64_t)p.sk_tiles * p.kt;
    r.s0 = (int)(isk * lw / p.grid);
    r.s1 = (int)(isk * (lw + 1) / p.grid);
    r.gdp = p.dp_rounds * p.kt;
    r.G = r.gdp + (r.s1 - r.s0);
    return r;
}

// Step g of logical workgroup lw's range -> (logical tile t, K step k).
__host__ __device__ __forceinline__ void sk_locate(const SkParams &p, const SkRange &r, int lw, int g, int &t,
                                                   int &k)
{
    if (g < r.gdp) {
        const int q = g / p.kt;
        t = lw + q * p.grid;
        k = g - q * p.kt;
    } else {
        const int i = r.s0 + (g - r.gdp);
        const int q = i / p.kt;
        t = p.dp_rounds * p.grid + q;
        k = i - q * p.kt;
    }
}

// One workgroup (id `block`) of the persistent kernel, as seen by thread
// `tid`; every memory access, MFMA, wait, barrier and flag operation goes
// through `ops`.
template <int BM, int BN, int BK, int WGM, int WGN, int DT, class Ops>
__host__ __device__ __forceinline__ void sk_tile(const Ops &ops, const SkParams &p, int block, int tid)
{
    constexpr int MI = 16;
    constexpr int NW = WGM * WGN;
    constexpr int TM = BM / WGM, TN = BN / WGN;
    constexpr int FM = TM / MI, FN = TN / MI;   // 16 x 16 MFMA blocks per wave
    constexpr int KI = 32;                       // k per MFMA
    constexpr int NG = 64 / MI;                  // lane groups along k
    constexpr int A_ROWB = BK * 2;
    constexpr int B_ROWB = BN * 2;
    constexpr int A_BYTES = BM * A_ROWB;
    constexpr int B_BYTES = BK * B_ROWB;
    constexpr int STAGE = A_BYTES + B_BYTES;
    constexpr int A_LD = A_BYTES / 1024 / NW;    // direct loads per wave per K step
    constexpr int B_LD = B_BYTES / 1024 / NW;
    constexpr int LD = A_LD + B_LD;
    constexpr int A_ROWS_PER_LD = 1024 / A_ROWB;
    constexpr int B_ROWS_PER_LD = 1024 / B_ROWB;
    constexpr int NSTORE = FM * FN;              // 16-byte stores of one wave's accumulators
    constexpr int R = 1;                         // rows of sub-step 1 issued before the barrier
    constexpr int LSTEP = ((FM - R) * FN) / LD > 0 ? ((FM - R) * FN) / LD : 1;
    static_assert(NW == 8 && BK == 64 && BK / KI == 2 && FN <= FM - R, "the eight-wave 16 x 16 x 32 schedule");
    static_assert(A_LD * NW * 1024 == A_BYTES && B_LD * NW * 1024 == B_BYTES, "load split");
    static_assert(LSTEP * (LD - 1) < (FM - R) * FN, "load spacing");
    static_assert(NSTORE < 64 && LD < 64, "vmcnt range");
    typedef float accT __attribute__((ext_vector_type(4)));

    const int lw = sk_logical(block, p.grid);
    const SkRange rg = sk_range(p, lw);
    const int lane = tid & 63;
    const int wave = ops.uniform(tid >> 6);
    const int wm = wave % WGM, wn = wave / WGM;
    const int64_t lda = p.lda, ldb = p.ldb;
    char *const smem = ops.lds();
    char *const bcast = smem + 2 * STAGE;        // counter words (two, 64 bytes apart)

    auto bswz = [](int k) { return ((k & 3) << 1) | ((k >> 3) & 1); };

    // --- per-lane direct-load offsets (every tile is whole) ---
    uint32_t a_goff[A_LD], b_goff[B_LD];
#pragma unroll
    for (int j = 0; j < A_LD; ++j) {
        const int r = (wave * A_LD + j) * A_ROWS_PER_LD + lane / (A_ROWB / 16);
        const int c = (lane % (A_ROWB / 16)) ^ aswz<A_ROWB>(r);
        a_goff[j] = (uint32_t)((r * lda + c * 8) * 2);
    }
#pragma unroll
    for (int j = 0; j < B_LD; ++j) {
        const int k = (wave * B_LD + j) * B_ROWS_PER_LD + lane / (B_ROWB / 16);
        const int q = lane % (B_ROWB / 16);
        const int c = (q >> 1) ^ bswz(k);
        b_goff[j] = (uint32_t)((k * ldb + c * 16 + (q & 1) * 8) * 2);
    }
    // where the loads of one K step read from
    struct Src {
        const uint16_t *a, *b;
    };
    // direct load j (0 .. LD-1) of the step described by s into `stage`
    auto load_j = [&](const Src &s, int stage, int j) {
        const uint32_t sA = ops.lds_addr(smem) + stage * STAGE;
        if (j < A_LD)
            ops.load16(s.a, a_goff[j], sA + (wave * A_LD + j) * 1024);
        else
            ops.load16(s.b, b_goff[j - A_LD], sA + A_BYTES + (wave * B_LD + (j - A_LD)) * 1024);
    };

    // --- fragments (as dma_tile's eight-wave schedule) ---
    const int lr = lane % MI;
    const int kg = lane / MI;
    const int a_x = kg ^ aswz<A_ROWB>(lr);
    const int a_lane = (wm * TM + lr) * A_ROWB;
    const int s16 = lane & 15;
    const int c16 = lr >> 4;
    const int t4 = s16 >> 2;
    const int b_lane = (8 * kg + t4) * B_ROWB + 8 * (s16 & 3);
    const int b_c0 = wn * (TN / 16) + c16;
    const int b_sw = bswz(8 * kg + t4);
    auto frag_A = [&](int stage, int kk, int i) {
        const char *sA = smem + stage * STAGE + a_lane + ((((KI / 8) * kk) ^ a_x) << 4);
        return ops.read16(sA + i * MI * A_ROWB);
    };
    auto frag_B = [&](int stage, int kk, int j) {
        const char *pb = smem + stage * STAGE + A_BYTES + kk * KI * B_ROWB + b_lane +
                         (((b_c0 + j * (MI / 16)) ^ b_sw) << 5);
        const v4i16 lo = ops.read_tr8(pb);
        const v4i16 hi = ops.read_tr8(pb + 4 * B_ROWB);
        u32x4 v;
        v.x = __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 0, 1));
        v.y = __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 2, 3));
        v.z = __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 0, 1));
        v.w = __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 2, 3));
        return v;
    };

    accT acc[FM][FN];
    const accT zero = {0.0f, 0.0f, 0.0f, 0.0f};
    auto clear_acc = [&]() {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
                acc[i][j] = zero;
    };
    clear_acc();
    u32x4 ga[2][FM], gb[2][FN];

    // --- stores ---
    // Buffer accesses: a descriptor of a uniform base, a 32-bit per-lane
    // byte offset and a uniform byte offset (the host keeps 256 rows of C
    // within 4 GiB and C 16-byte aligned).  Lane l's accumulators hold row
    // lr, columns 4 kg .. 4 kg + 3 of each 16 x 16 block.
    // this wave's block of C in tile u
    auto c_base = [&](const SkTile &u) {
        return p.C + u.b * p.stride_c + (int64_t)(u.m * BM + wm * TM) * p.ldc + u.n * BN + wn * TN;
    };
    // C of tile u, block row i (FN 16-byte stores per lane): streaming
    // stores, whose lines an XCD's L2 does not keep, so that they take no L2
    // space from the operands of the tiles that follow.  Pairs of blocks are
    // first rearranged into whole 128-byte rows (line_pair: lane l then
    // writes row l % 8, or 8 + l % 8, at column 16 ((l % 16) / 8) + 4 (l / 16)
    // of the pair).  Measured 712 against 748 us at 8192^3 (3-9% on the
    // persistent kernel's shapes) over storing the blocks as they are.
    const uint32_t c_line = (uint32_t)(((lr & 7) * p.ldc + (lr >> 3) * 16 + kg * 4) * 4);
    static_assert(FN % 2 == 0, "pairs of block columns");
    auto store_pair = [&](typename Ops::Rsrc r, uint32_t soff, int j, accT &b0, accT &b1) {
        ops.line_pair(b0, b1);
        ops.buf_store4_nt(r, c_line + j * MI * 4, soff, b0);
        ops.buf_store4_nt(r, c_line + j * MI * 4, soff + (uint32_t)(8 * p.ldc * 4), b1);
    };
    auto store_c_row = [&](const SkTile &u, int i) {
        const auto r = ops.rsrc(c_base(u));
        const uint32_t soff = (uint32_t)(i * MI * p.ldc * 4);
#pragma unroll
        for (int j = 0; j < FN; j += 2)
            store_pair(r, soff, j, acc[i][j], acc[i][j + 1]);
    };
    // partial sums of slot s, piece 0 (first steps) or 1 (last steps): block
    // (i, j) of wave w is 64 lanes x 16 bytes, contiguous, in the
    // accumulators' own layout
    const uint32_t p_lane = (uint32_t)lane * 16;
    auto part_rsrc = [&](int s, int piece) {
        return ops.rsrc(p.part + ((int64_t)s * 2 + piece) * (BM * BN) + wave * (FM * FN * 256));
    };

    // A cursor walks the range step by step, without divisions except where
    // it enters a new tile.
    struct Cursor {
        int g, t, k;
        SkTile u;
    };
    const SkRange &L = rg;
    auto set_tile = [&](Cursor &c) { c.u = sk_tile_of(p, c.t); };
    auto start = [&](Cursor &c, int g) {
        c.g = g;
        sk_locate(p, rg, lw, g, c.t, c.k);
        set_tile(c);
    };
    auto advance = [&](Cursor &c) {
        ++c.g;
        ++c.k;
        if (c.g >= L.G)
            return;   // past the range's last step: nothing to locate
        if (c.g == rg.gdp) {
            // from the whole tiles to the stream-K range
            sk_locate(p, rg, lw, c.g, c.t, c.k);
            set_tile(c);
        } else if (c.k == p.kt) {
            c.k = 0;
            c.t += c.g < rg.gdp ? p.grid : 1;
            set_tile(c);
        }
    };
    auto src_of = [&](const Cursor &c) {
        Src s;
        const int m0 = c.u.m * BM, n0 = c.u.n * BN;
        s.a = p.A + c.u.b * p.stride_a + (int64_t)m0 * lda + c.k * BK;
        s.b = p.B + c.u.b * p.stride_b + (int64_t)c.k * BK * ldb + n0;
        return s;
    };

    // --- one K step g of the range ---
    // With `flush` (once per tile) the step first stores the previous tile's
    // accumulators (tile f) and clears them; the stores drain under
    // the step's MFMAs.  Sub-step 0 works from ga[0] / gb[0] and reads
    // sub-step 1 of the same stage.  Then R
    // rows of sub-step 1, the waits, the barrier, and the other rows of
    // sub-step 1 with the direct loads of step g + 2 (from s) into the stage
    // just freed and the reads of step g + 1's sub-step 0.  Every step is the
    // same: past the range's end the loads repeat its last step (into a
    // stage no later step reads) and the reads take what those loads
    // brought, so no branch interrupts the MFMAs; the range waits for its
    // last loads before it ends.
    auto kstep = [&](int g, bool flush, const SkTile &f, const Src &s) {
        const int stage = g & 1, next = stage ^ 1;
        if (__builtin_expect(flush, 0)) {
#pragma unroll
            for (int i = 0; i < FM; ++i)
                store_c_row(f, i);
            clear_acc();
        }
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int j = 0; j < FN; ++j)
                acc[i][j] = ops.template mfma<DT>(gb[0][j], ga[0][i], acc[i][j]);
            ga[1][i] = frag_A(stage, 1, i);
            if (i < FN)
                gb[1][i] = frag_B(stage, 1, i);
            ops.fence();
        }
#pragma unroll
        for (int i = 0; i < R; ++i) {
#pragma unroll
            for (int j = 0; j < FN; ++j)
                acc[i][j] = ops.template mfma<DT>(gb[1][j], ga[1][i], acc[i][j]);
            ops.fence();
        }
        // stage g fully read by this wave; step g + 1 landed for this wave
        // (the flushed stores, issued after its loads, may still be in flight)
        ops.wait_lgkm0();
        if (__builtin_expect(flush, 0))
            ops.template wait_vm<NSTORE>();
        else
            ops.template wait_vm<0>();
        ops.barrier();
        ops.fence();
        ops.template priority<1>();
#pragma unroll
        for (int i = 0; i < R; ++i)
            ga[0][i] = frag_A(next, 0, i);
#pragma unroll
        for (int i = R; i < FM; ++i) {
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                acc[i][j] = ops.template mfma<DT>(gb[1][j], ga[1][i], acc[i][j]);
                const int q = (i - R) * FN + j;
                if (q % LSTEP == 0 && q / LSTEP < LD)
                    load_j(s, stage, q / LSTEP);
            }
            ga[0][i] = frag_A(next, 0, i);
            if (i - R < FN)
                gb[0][i - R] = frag_B(next, 0, i - R);
            ops.fence();
        }
        ops.template priority<0>();
    };

    // Tell the workgroup the value thread 0 got (an LDS word, a barrier).
    auto broadcast = [&](char *word, int v) {
        ops.lds_write4(word, v, tid == 0);
        ops.wait_lgkm0();
        ops.barrier();
        return ops.lds_read4(word);
    };
    // Publish this piece's partial sum (piece 0: the first steps, 1: the
    // last steps of slot s) and count in; returns the counter's value before.
    auto publish = [&](int s, int piece) {
        const auto r = part_rsrc(s, piece);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
                ops.buf_store4_dev(r, p_lane + j * 1024, i * FN * 1024, acc[i][j]);
        // every wave's partial complete (visible to every XCD), then count in
        ops.stores_done();
        ops.barrier();
        int old = 0;
        if (tid == 0)
            old = ops.flag_add(p.flags + s, 1);
        return broadcast(bcast + 64, old);
    };
    // The first steps of tile u (slot s) are in acc (the end of
    // the range): add the last steps' partial once published, row by row,
    // and store C; or publish the first steps when the last are not done.
    auto finish_head = [&](int s, const SkTile &u) {
        int v = 0;
        if (tid == 0)
            v = ops.flag_load(p.flags + s);
        if (broadcast(bcast, v) != 1 && publish(s, 0) != 1)
            return;
        const auto r = part_rsrc(s, 1);
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int j = 0; j < FN; ++j)
                acc[i][j] = acc[i][j] + ops.buf_load4_dev(r, p_lane + j * 1024, i * FN * 1024);
            store_c_row(u, i);
            ops.fence();
        }
        if (tid == 0)
            ops.flag_store(p.flags + s, 0);
    };
    // Both partials of slot s are published (this workgroup's last steps
    // counted in second): C of tile u is their sum, read back
    // (the same sum as finish_head's: fp32 addition commutes).
    auto combine = [&](int s, const SkTile &u) {
        const auto r0 = part_rsrc(s, 0), r1 = part_rsrc(s, 1);
        const auto rc = ops.rsrc(c_base(u));
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int j = 0; j < FN; j += 2) {
                accT x0 = ops.buf_load4_dev(r0, p_lane + j * 1024, i * FN * 1024) +
                          ops.buf_load4_dev(r1, p_lane + j * 1024, i * FN * 1024);
                accT x1 = ops.buf_load4_dev(r0, p_lane + (j + 1) * 1024, i * FN * 1024) +
                          ops.buf_load4_dev(r1, p_lane + (j + 1) * 1024, i * FN * 1024);
                store_pair(rc, (uint32_t)(i * MI * p.ldc * 4), j, x0, x1);
            }
            ops.fence();
        }
        if (tid == 0)
            ops.flag_store(p.flags + s, 0);
    };

    if (L.G == 0)
        return;      // the host gives every workgroup at least one tile's steps
    Cursor cc, lc;   // the step computed, and the step loaded two ahead
    start(cc, 0);
    // prologue: the first two steps in flight, the first landed
    {
        const Src s0 = src_of(cc);
#pragma unroll
        for (int j = 0; j < LD; ++j)
            load_j(s0, 0, j);
        lc = cc;
        if (lc.g + 1 < L.G)
            advance(lc);
        const Src s1 = src_of(lc);
#pragma unroll
        for (int j = 0; j < LD; ++j)
            load_j(s1, 1, j);
        ops.template wait_vm<LD>();
        ops.barrier();
#pragma unroll
        for (int i = 0; i < FM; ++i)
            ga[0][i] = frag_A(0, 0, i);
#pragma unroll
        for (int j = 0; j < FN; ++j)
            gb[0][j] = frag_B(0, 0, j);
    }

    // A range's stream-K part starting inside a tile begins with that
    // tile's last steps (split with range lw - 1, slot lw): they end at
    // step tail_end - 1.
    const int k_sk = rg.s0 % p.kt;
    const int tail_end = (rg.s1 > rg.s0 && k_sk > 0) ? rg.gdp + (p.kt - k_sk) : 0;

    // Steps 0 .. G - 1, lc the step loaded two ahead.  Most steps are plain:
    // the step computed and the one loaded lie in one tile and nothing ends;
    // they run in an inner loop that only moves the load pointers along K.
    // The steps around a tile boundary take the general path: the first
    // step of a tile stores the previous whole tile under its MFMAs
    // (flush), and the last step of a range stores its whole tile.  The
    // range's tail (if any) and its head are handed over between passes and
    // after the last.
    bool flush = false;   // the tile f is stored under the next step
    SkTile f{0, 0, 0};
    int kfirst = cc.k;    // K step the current unit started at
    bool tail_combine = false;
    SkTile tt{0, 0, 0};   // the tail's tile
    // two passes: up to the end of the tail (if any), then the rest
#pragma nounroll
    for (int pass = tail_end > 0 ? 0 : 1; pass < 2; ++pass) {
        const int g_end = pass == 0 ? tail_end : L.G;
        while (cc.g < g_end) {
            if (cc.k == 0 || cc.g == rg.gdp)
                kfirst = cc.k;
            // plain steps: lc advances within its tile, cc stays two behind it
            int n = (!flush && cc.t == lc.t) ? min(p.kt - 1 - lc.k, L.G - 1 - lc.g) : 0;
            if (n > 0) {
                Src s = src_of(lc);
                for (; n > 0; --n) {
                    s.a += BK;
                    s.b += (int64_t)BK * ldb;
                    kstep(cc.g, false, f, s);
                    ++cc.g;
                    ++cc.k;
                }
                lc.g = cc.g + 1;
                lc.k = cc.k + 1;
            }
            // one general step
            if (cc.k == 0 || cc.g == rg.gdp)
                kfirst = cc.k;
            const bool fl = flush;
            flush = false;
            if (lc.g + 1 < L.G)
                advance(lc);   // step g + 2, or the last step again
            kstep(cc.g, fl, f, src_of(lc));
            if (kfirst == 0 && cc.k == p.kt - 1) {
                if (cc.g + 1 < L.G) {
                    flush = true;
                    f = cc.u;
                } else {
#pragma unroll
                    for (int i = 0; i < FM; ++i)
                        store_c_row(cc.u, i);
                    clear_acc();
                }
            }
            advance(cc);
        }
        if (pass == 0) {
            // the tail's last steps: publish them; if the first steps are
            // already published, the sum is formed after the range
            tail_combine = publish(lw, 1) == 1;
            int t, k;
            sk_locate(p, rg, lw, tail_end - 1, t, k);
            tt = sk_tile_of(p, t);
            clear_acc();
        }
    }
    ops.template wait_vm<0>();   // the repeated last loads landed: no LDS write in flight at exit
    // A range ending inside a tile ends with that tile's first steps (split
    // with range lw + 1, slot lw + 1).
    if (L.G > 0 && (rg.s1 > rg.s0) && rg.s1 % p.kt != 0) {
        int t, k;
        sk_locate(p, rg, lw, L.G - 1, t, k);
        finish_head(lw + 1, sk_tile_of(p, t));
    }
    if (tail_combine)
        combine(lw, tt);
}

template <int BM, int BN, int BK, int WGM, int WGN, int DT>
__global__ void __launch_bounds__(WGM * WGN * 64, 1)
gemm_kernel_sk(SkParams p)
{
    __shared__ __attribute__((aligned(1024))) char smem[sk_lds_bytes<BM, BN, BK>()];
    const DeviceOps ops{smem};
    sk_tile<BM, BN, BK, WGM, WGN, DT>(ops, p, blockIdx.x, threadIdx.x);
}

}  // namespace xgemm_dev
