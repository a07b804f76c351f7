// Device code for C = A * B (16-bit inputs, fp32 accumulate, fp32 out) on
// gfx950.
//
// One workgroup computes a BM x BN tile of C (or, with split-k, the partial
// sum of that tile over one K range).  Per K step of BK:
//   global -> registers  16-byte loads of the A tile (BM x BK, k contiguous)
//                        and of the B tile (BK x BN, n contiguous); each B
//                        unit is an 8 x 8 block that the thread transposes
//                        in registers so that k becomes contiguous;
//   registers -> LDS     both tiles stored k-contiguous, 16-byte chunks
//                        XOR-swizzled per row so that the fragment reads of
//                        consecutive rows fall in different banks;
//   LDS -> MFMA          v_mfma_f32_32x32x16_{bf16,f16}, each wave owning a
//                        (BM/WGM) x (BN/WGN) block of fp32 accumulators.
// Two LDS stages: while the waves multiply stage s, the loads for the next K
// step are in flight and land in stage s^1; one barrier per K step.
//
// The paper's kernels overlap bulk copies with tensor-core work through
// split barriers (Section 2.1, explicit synchronization); here the same
// overlap comes from double-buffered LDS with s_waitcnt ordering on the
// loads and a single workgroup barrier per K step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

namespace xgemm_dev {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

constexpr int kNumXcd = 8;  // MI355X: 8 accelerator complex dies, each with its own L2

struct GemmParams {
    const uint16_t *A;
    const uint16_t *B;
    float *C;               // C, or the split-k workspace
    int64_t lda, ldb, ldc;  // ldc: leading dimension of the array written
    int64_t split_stride;   // elements between split partials (0 when split == 1)
    int M, N, K;
    int k_chunk;            // K elements per split, a multiple of BK
    int split;
    int tiles_m, tiles_n;
    int group_m;
    int vec_ab;             // A, B 16-byte aligned, lda and ldb multiples of 8
    int vec_c;              // output 16-byte aligned, ldc a multiple of 4
    int tile_base;          // this launch covers logical tiles [tile_base, tile_base + tile_count)
    int tile_count;
    int batch;              // independent problems; problem b uses A + b*stride_a, B + b*stride_b,
    int64_t stride_a;       //   C + b*stride_c (elements); batched launches have split == 1
    int64_t stride_b;
    int64_t stride_c;
    int grid;               // workgroups of the launch; a 2-D grid may hold more, which exit
};

// Linear workgroup id of a launch whose grid may be 2-D (x fastest, as the
// hardware dispatches them): launches with more than 2^32 threads need the
// second dimension.
__device__ __forceinline__ int linear_block() { return (int)(blockIdx.y * gridDim.x + blockIdx.x); }

template <int DT>
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c);

template <>
__device__ __forceinline__ f32x16 mfma32<0>(u32x4 a, u32x4 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

template <>
__device__ __forceinline__ f32x16 mfma32<1>(u32x4 a, u32x4 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

template <int DT>
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c);

template <>
__device__ __forceinline__ f32x4 mfma16<0>(u32x4 a, u32x4 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

template <>
__device__ __forceinline__ f32x4 mfma16<1>(u32x4 a, u32x4 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// 16-byte chunk slot of logical chunk c in tile row r.  Rows r and r^j for
// j < 16 never share a slot among 8 consecutive rows, nor a (row parity,
// slot) pair among 16 consecutive rows.
__host__ __device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Logical tile id -> (tile_m, tile_n): tiles are walked in groups of
// group_m tile rows, column by column within a group, so that consecutive
// ids share rows of A and columns of B.  Shared by the GEMM kernels and the
// tile reduction, which must agree on it.
__host__ __device__ __forceinline__ void logical_tile(int t, int tiles_m, int tiles_n, int group_m, int &tm,
                                                      int &tn)
{
    const int group = group_m * tiles_n;
    const int g = t / group;
    const int first_m = g * group_m;
    const int gm = min(tiles_m - first_m, group_m);
    const int r = t - g * group;
    tm = first_m + r % gm;
    tn = r / gm;
}

// Workgroup -> (tile_m, tile_n, split, local tile index).  The hardware
// hands workgroup ids to the XCDs round-robin; consecutive logical ids are
// first gathered onto one XCD, so that the workgroups an XCD runs at the
// same time are neighbours in the grouped tile order and share rows of A
// and columns of B in its L2.  The split index is outermost: workgroups of
// one K range run together.  (The paper's persistent kernels hand out tasks
// in lexicographic order and leave other orders to future work, Section
// 4.2.)
// The batch index is outermost of all: the problems of a batch run one
// after another across the grid.  w is the workgroup id and total the grid
// size.  Returns the workgroup's parameters with A, B and C moved to its
// problem.
__host__ __device__ __forceinline__ GemmParams map_tile(const GemmParams &p_in, int w, int total, int &tm, int &tn,
                                                       int &ks, int &local)
{
    const int per = total / kNumXcd;
    int lid = (w < per * kNumXcd) ? (w % kNumXcd) * per + w / kNumXcd : w;
    const int per_batch = p_in.tile_count * p_in.split;
    const int b = lid / per_batch;
    lid -= b * per_batch;
    ks = lid / p_in.tile_count;
    local = lid - ks * p_in.tile_count;
    logical_tile(p_in.tile_base + local, p_in.tiles_m, p_in.tiles_n, p_in.group_m, tm, tn);
    GemmParams p = p_in;
    p.A += b * p_in.stride_a;
    p.B += b * p_in.stride_b;
    p.C += b * p_in.stride_c;
    return p;
}

// Output placement: row-major C, or split ks's full-matrix partial, at
// base + row * ld + col.
struct OutView {
    float *base;
    int64_t ld;
    int r0, c0;
};

template <int BM, int BN>
__host__ __device__ __forceinline__ OutView out_view(const GemmParams &p, int ks, int, int, int)
{
    OutView o;
    o.base = p.C + (int64_t)ks * p.split_stride;
    o.ld = p.ldc;
    o.r0 = 0;
    o.c0 = 0;
    return o;
}

// Eight 16-bit values starting at base[off], the first `cnt` of them read
// from memory (through ops) and the rest zero.
template <class Ops>
__host__ __device__ __forceinline__ u32x4 load8_masked(const Ops &ops, const uint16_t *base, int64_t off, int cnt)
{
    uint32_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
        h[e] = (e < cnt) ? (uint32_t)ops.gload2(base + off + e) : 0u;
    u32x4 v;
    v.x = h[0] | (h[1] << 16);
    v.y = h[2] | (h[3] << 16);
    v.z = h[4] | (h[5] << 16);
    v.w = h[6] | (h[7] << 16);
    return v;
}

// Column c (0..7) of an 8 x 8 block of 16-bit values held as 8 rows of 4
// dwords: returns the 8 values of that column, row 0 in the low half of
// dword 0.
__host__ __device__ __forceinline__ u32x4 column8(const u32x4 (&v)[8], int c)
{
    u32x4 w;
    const int d = c >> 1;
    if ((c & 1) == 0) {
        w.x = (v[0][d] & 0xFFFFu) | (v[1][d] << 16);
        w.y = (v[2][d] & 0xFFFFu) | (v[3][d] << 16);
        w.z = (v[4][d] & 0xFFFFu) | (v[5][d] << 16);
        w.w = (v[6][d] & 0xFFFFu) | (v[7][d] << 16);
    } else {
        w.x = (v[0][d] >> 16) | (v[1][d] & 0xFFFF0000u);
        w.y = (v[2][d] >> 16) | (v[3][d] & 0xFFFF0000u);
        w.z = (v[4][d] >> 16) | (v[5][d] & 0xFFFF0000u);
        w.w = (v[6][d] >> 16) | (v[7][d] & 0xFFFF0000u);
    }
    return w;
}

// LDS bytes the general kernel allocates.
template <int BM, int BN, int BK>
constexpr int general_lds_bytes()
{
    return 2 * (BM + BN) * BK * 2;
}

// One workgroup (id `block` of `nblocks`) of the general kernel, as seen by
// thread `tid`; every memory access, MFMA and barrier goes through `ops`
// (see DeviceOps).
template <int BM, int BN, int BK, int WGM, int WGN, int DT, class Ops>
__host__ __device__ __forceinline__ void general_tile(const Ops &ops, const GemmParams &p_in, int block, int nblocks,
                                                      int tid)
{
    constexpr int NT = WGM * WGN * 64;
    constexpr int TM = BM / WGM, TN = BN / WGN;   // wave tile
    constexpr int FM = TM / 32, FN = TN / 32;     // 32x32 MFMA blocks per wave
    constexpr int KC = BK / 8;                    // 16-byte chunks per tile row
    constexpr int KS = BK / 16;                   // MFMA k steps per K step
    constexpr int ROWB = BK * 2;                  // bytes per LDS tile row
    constexpr int A_UNITS = BM * KC;              // 16-byte chunks of the A tile
    constexpr int A_IT = (A_UNITS + NT - 1) / NT;
    constexpr int B_UNITS = KC * (BN / 8);        // 8 x 8 blocks of the B tile
    constexpr int B_IT = (B_UNITS + NT - 1) / NT;
    constexpr int A_BYTES = BM * ROWB, B_BYTES = BN * ROWB;
    constexpr int STAGE = A_BYTES + B_BYTES;
    static_assert(TM % 32 == 0 && TN % 32 == 0 && BK % 16 == 0 && KC <= 16, "tile shape");
    static_assert(2 * STAGE <= 160 * 1024 && 2 * STAGE == general_lds_bytes<BM, BN, BK>(), "LDS budget");

    char *const smem = ops.lds();

    int tm, tn, ks, local;
    const GemmParams p = map_tile(p_in, block, nblocks, tm, tn, ks, local);
    const int m0 = tm * BM, n0 = tn * BN;
    const int kbeg = ks * p.k_chunk;
    const int kend = min(p.K, kbeg + p.k_chunk);
    const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;

    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WGM, wn = wave / WGM;
    const bool interior = (m0 + BM <= p.M) && (n0 + BN <= p.N);

    const int64_t lda = p.lda, ldb = p.ldb;

    // Per-thread load assignments (fixed for the whole K loop).
    int a_row[A_IT], a_c[A_IT];
    int64_t a_off[A_IT];
#pragma unroll
    for (int it = 0; it < A_IT; ++it) {
        const int u = tid + it * NT;
        a_row[it] = u / KC;
        a_c[it] = u % KC;
        a_off[it] = (int64_t)a_row[it] * lda + a_c[it] * 8;
    }
    int b_kg[B_IT], b_ng[B_IT];
    int64_t b_off[B_IT];
#pragma unroll
    for (int it = 0; it < B_IT; ++it) {
        const int u = tid + it * NT;
        b_kg[it] = u % KC;
        b_ng[it] = u / KC;
        b_off[it] = (int64_t)(b_kg[it] * 8) * ldb + b_ng[it] * 8;
    }

    u32x4 ra[A_IT];
    u32x4 rb[B_IT][8];

    auto load_tiles = [&](int k0) {
        const uint16_t *Ab = p.A + (int64_t)m0 * lda + k0;
        const uint16_t *Bb = p.B + (int64_t)k0 * ldb + n0;
        const bool full = p.vec_ab && interior && (k0 + BK <= kend);
        if (full) {
#pragma unroll
            for (int it = 0; it < A_IT; ++it)
                if (A_UNITS % NT == 0 || tid + it * NT < A_UNITS)
                    ra[it] = ops.gload16(Ab + a_off[it]);
#pragma unroll
            for (int it = 0; it < B_IT; ++it)
                if (B_UNITS % NT == 0 || tid + it * NT < B_UNITS)
#pragma unroll
                    for (int r = 0; r < 8; ++r)
                        rb[it][r] = ops.gload16(Bb + b_off[it] + r * ldb);
        } else {
#pragma unroll
            for (int it = 0; it < A_IT; ++it)
                if (A_UNITS % NT == 0 || tid + it * NT < A_UNITS) {
                    const int gm = m0 + a_row[it];
                    const int gk = k0 + a_c[it] * 8;
                    const int cnt = (gm < p.M) ? max(0, min(8, kend - gk)) : 0;
                    ra[it] = load8_masked(ops, Ab, a_off[it], cnt);
                }
#pragma unroll
            for (int it = 0; it < B_IT; ++it)
                if (B_UNITS % NT == 0 || tid + it * NT < B_UNITS) {
                    const int gn = n0 + b_ng[it] * 8;
                    const int ncnt = max(0, min(8, p.N - gn));
#pragma unroll
                    for (int r = 0; r < 8; ++r) {
                        const int gk = k0 + b_kg[it] * 8 + r;
                        rb[it][r] = load8_masked(ops, Bb, b_off[it] + r * ldb, gk < kend ? ncnt : 0);
                    }
                }
        }
    };

    auto store_tiles = [&](int stage) {
        char *sA = smem + stage * STAGE;
        char *sB = sA + A_BYTES;
#pragma unroll
        for (int it = 0; it < A_IT; ++it)
            if (A_UNITS % NT == 0 || tid + it * NT < A_UNITS) {
                const int r = a_row[it];
                ops.lds_write16(sA + r * ROWB + ((a_c[it] ^ swz(r)) << 4), ra[it]);
            }
#pragma unroll
        for (int it = 0; it < B_IT; ++it)
            if (B_UNITS % NT == 0 || tid + it * NT < B_UNITS) {
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    const int n = b_ng[it] * 8 + c;
                    ops.lds_write16(sB + n * ROWB + ((b_kg[it] ^ swz(n)) << 4), column8(rb[it], c));
                }
            }
    };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                acc[i][j][e] = 0.0f;

    // Fragment addressing: lane l reads row (l % 32) of each 32-row block at
    // chunk 2*kk + l/32.  Rows of a block start at a multiple of 32, so the
    // swizzle depends on the lane only.
    const int l32 = lane & 31;
    const int xk = (lane >> 5) ^ swz(l32);
    const int frag_lane = l32 * ROWB;

    auto compute = [&](int stage) {
        const char *sA = smem + stage * STAGE + (wm * TM) * ROWB + frag_lane;
        const char *sB = smem + stage * STAGE + A_BYTES + (wn * TN) * ROWB + frag_lane;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            const int co = ((2 * kk) ^ xk) << 4;
            u32x4 fa[FM], fb[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                fa[i] = ops.read16(sA + i * 32 * ROWB + co);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                fb[j] = ops.read16(sB + j * 32 * ROWB + co);
            // B fragment as the first operand: the result lands with lanes
            // along rows of C and 4 consecutive columns per register quad.
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = ops.template mfma<DT>(fb[j], fa[i], acc[i][j]);
        }
    };

    if (nk > 0) {
        load_tiles(kbeg);
        store_tiles(0);
        ops.sync();
        for (int kt = 0; kt < nk; ++kt) {
            const int cur = kt & 1;
            if (kt + 1 < nk)
                load_tiles(kbeg + (kt + 1) * BK);
            compute(cur);
            if (kt + 1 < nk)
                store_tiles(cur ^ 1);
            ops.sync();
        }
    }

    // Epilogue: lane l holds rows (l % 32) of each 32 x 32 block and, in
    // register quad q, columns 8q + 4(l / 32) .. +3.
    const OutView ov = out_view<BM, BN>(p, ks, local, m0, n0);
    float *Cb = ov.base;
    const int64_t ldc = ov.ld;
    const bool vec_store = p.vec_c && interior;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int row = m0 + wm * TM + i * 32 + l32;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int col = n0 + wn * TN + j * 32 + q * 8 + (lane >> 5) * 4;
                f32x4 v;
                v.x = acc[i][j][4 * q + 0];
                v.y = acc[i][j][4 * q + 1];
                v.z = acc[i][j][4 * q + 2];
                v.w = acc[i][j][4 * q + 3];
                if (vec_store) {
                    ops.store4(Cb + (int64_t)(row - ov.r0) * ldc + (col - ov.c0), v);
                } else if (row < p.M) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (col + e < p.N)
                            ops.store1(Cb + (int64_t)(row - ov.r0) * ldc + (col - ov.c0) + e, v[e]);
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Pipelined kernel for 16-byte aligned operands with K a multiple of BK.
//
// Global -> LDS without registers: each wave issues 16-byte direct-to-LDS
// loads (a lane's 16 bytes land at LDS base + 16 * lane), so the LDS layout
// is chosen by which global chunk each lane fetches.  STAGES K steps are in
// flight at once.  Fragments:
//   A  (BM x BK, k contiguous, rows of BK*2 bytes): ds_read_b128 of 8
//      consecutive k of one row; 16-byte chunk c of row r is stored at slot
//      c ^ aswz(r) (see aswz), so 16 consecutive rows read at one logical
//      chunk cover all 16 slots of a 256-byte bank window;
//   B  (BK x BN, n contiguous as in memory, rows of BN*2 bytes):
//      ds_read_b64_tr_b16 -- within each group of 16 lanes, lane i receives
//      element (i % 4) of the 8 bytes addressed by lane 4e + i / 4 as its
//      element e, which turns a 4 (k) x 16 (n) block into the k-packed
//      MFMA operand; 32-byte chunk c of row k is stored at chunk
//      c ^ bswz(k) so the rows one read instruction touches fall in
//      different banks.
// M and N edges: rows and columns beyond the matrix are clamped to the last
// valid one (they only feed outputs that are never stored).
//
// Schedule of K step t with one wave per SIMD (fragment buffers alternate
// between K sub-steps):
//   read fragments of the last sub-step of t         (LDS stage t)
//   MFMAs of the other sub-steps of t
//   wait: own fragment reads done, own loads of stage t+1 landed; barrier
//   issue direct loads of step t+STAGES into stage t (now free)
//   read fragments of sub-step 0 of t+1               (LDS stage t+1)
//   MFMAs of the last sub-step of t
// With eight waves (two per SIMD) the same order holds, with each row's
// fragment reads issued right after that row's MFMAs (see kstep_pair below).
// ---------------------------------------------------------------------------

typedef short v4i16 __attribute__((ext_vector_type(4)));

// 16 bytes per lane from global (scalar base + per-lane byte offset) to LDS
// at lds_addr + 16 * lane.  Issued as inline assembly so that the compiler's
// wait insertion does not treat it as a pending LDS write (it would otherwise
// wait for every such load before each LDS read); the kernels place their
// own vmcnt waits.
__device__ __forceinline__ void lds_load16(const void *gbase, uint32_t voff, uint32_t lds_addr)
{
    asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(gbase), "{m0}"(lds_addr) : "memory");
}

__device__ __forceinline__ uint32_t lds_address(const void *p)
{
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char *)p;
}

__device__ __forceinline__ v4i16 ds_read_tr16(const char *p)
{
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16 *)p);
}

// s_waitcnt with only vmcnt constrained (gfx9 encoding: vmcnt bits 3:0 and
// 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ void wait_lgkmcnt0()
{
    __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));
}

// Workgroup barrier that the compiler may not move memory accesses across;
// it adds no waits of its own (they are explicit at each use).
__device__ __forceinline__ void barrier_only()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Fence for the compiler's instruction scheduler: nothing moves across it,
// so the code order between fences is the issue order.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// Cache-policy bits of the buffer load/store builtins on gfx950: nt
// (streaming) and sc1 (device scope).
constexpr int kCpolNt = 2;
constexpr int kCpolSc1 = 16;

// Chunk swizzle of the A tile for rows of ROWB bytes (4 or 8 chunks): with
// 64-byte rows, four rows share a 256-byte bank window and rows r, r+4,
// r+8, r+12 get distinct slots; with 128-byte rows, two rows share a window
// and rows of one parity within 16 get distinct slots.
template <int ROWB>
__host__ __device__ __forceinline__ int aswz(int r)
{
    static_assert(ROWB == 64 || ROWB == 128, "A row size");
    return ROWB == 64 ? ((r >> 2) & 3) : ((r >> 1) & 7);
}

// Operations of the pipelined kernel as the device executes them.  The
// kernel body (dma_tile) issues every direct load, LDS read, MFMA, wait,
// barrier and global store through such an object, so that the same body
// can be run on the host with an object that records these operations
// instead (the synchronisation checker replays the record).
struct DeviceOps {
    char *smem;
    __device__ __forceinline__ char *lds() const { return smem; }
    // LDS address of a pointer into the workgroup's LDS
    __device__ __forceinline__ uint32_t lds_addr(const char *q) const { return lds_address(q); }
    __device__ __forceinline__ int uniform(int x) const { return __builtin_amdgcn_readfirstlane(x); }
    // 16 bytes per lane from gbase + goff to LDS address lds + 16 * lane
    __device__ __forceinline__ void load16(const void *gbase, uint32_t goff, uint32_t lds) const
    {
        lds_load16(gbase, goff, lds);
    }
    __device__ __forceinline__ u32x4 read16(const char *q) const { return *(const u32x4 *)q; }
    __device__ __forceinline__ v4i16 read_tr8(const char *q) const { return ds_read_tr16(q); }
    template <int DT>
    __device__ __forceinline__ f32x16 mfma(u32x4 a, u32x4 b, f32x16 c) const
    {
        return mfma32<DT>(a, b, c);
    }
    template <int DT>
    __device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) const
    {
        return mfma16<DT>(a, b, c);
    }
    template <int N>
    __device__ __forceinline__ void wait_vm() const
    {
        wait_vmcnt<N>();
    }
    __device__ __forceinline__ void wait_lgkm0() const { wait_lgkmcnt0(); }
    __device__ __forceinline__ void barrier() const { barrier_only(); }
    __device__ __forceinline__ void fence() const { sched_fence(); }
    // issue priority of this wave among the waves of its SIMD (0 .. 3)
    template <int P>
    __device__ __forceinline__ void priority() const
    {
        __builtin_amdgcn_s_setprio(P);
    }
    __device__ __forceinline__ void store4(float *q, f32x4 v) const { *(f32x4 *)q = v; }
    __device__ __forceinline__ void store1(float *q, float v) const { *q = v; }
    // general kernel: loads into registers, LDS writes, a full barrier
    __device__ __forceinline__ u32x4 gload16(const uint16_t *q) const { return *(const u32x4 *)q; }
    __device__ __forceinline__ uint16_t gload2(const uint16_t *q) const { return *q; }
    __device__ __forceinline__ void lds_write16(char *q, u32x4 v) const { *(u32x4 *)q = v; }
    // lane-masked: only lanes with `on` write
    __device__ __forceinline__ void lds_write16(char *q, u32x4 v, bool on) const
    {
        if (on)
            *(u32x4 *)q = v;
    }
    __device__ __forceinline__ void sync() const { __syncthreads(); }
    // persistent kernel: buffer accesses (a descriptor of a base address in
    // SGPRs, a 32-bit per-lane byte offset, a uniform byte offset), flags and
    // the LDS words of the split-tile hand-over
    typedef __amdgpu_buffer_rsrc_t Rsrc;
    // raw buffer over `base` (no stride, no range limit; gfx9 descriptor
    // word 3: 32-bit data format)
    __device__ __forceinline__ Rsrc rsrc(const void *base) const
    {
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)0xffffffff, 0x00020000);
    }
    __device__ __forceinline__ void buf_store4(Rsrc r, uint32_t voff, uint32_t soff, f32x4 v) const
    {
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, voff, soff, 0);
    }
    // Two 16 x 16 accumulator blocks of one block row (block columns 2p and
    // 2p + 1; lane l holds row l % 16, columns 4 (l / 16) .. +3 of each),
    // rearranged so that each holds 8 whole rows of their 32 columns: b0
    // rows 0-7, b1 rows 8-15, lane l holding row l % 8 (+ 8 in b1), columns
    // 16 ((l % 16) / 8) + 4 (l / 16) .. +3.  One 16-byte store per lane then
    // writes 8 rows of 128 bytes, whole lines, where the plain layout writes
    // 16 half lines (the memory side counted 1.2-1.37x the bytes of C for
    // half-line streaming stores).  Lanes 8-15 of each row of 16 trade with
    // lanes 0-7 (DPP row rotation by 8, bank masks select the halves).  The
    // elements are copied out before the bit casts (a bit cast of a vector
    // element in place read element 0 for every element).
    __device__ __forceinline__ void line_pair(f32x4 &b0, f32x4 &b1) const
    {
        f32x4 r0, r1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float a = b0[e], b = b1[e];
            const int ia = __builtin_bit_cast(int, a), ib = __builtin_bit_cast(int, b);
            const int t = __builtin_amdgcn_mov_dpp(ia, 0x128, 0xF, 0xF, false);   // row_ror:8
            r0[e] = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(ia, ib, 0x128, 0xF, 0xC, false));
            r1[e] = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(ib, t, 0xE4, 0xF, 0x3, false));
        }
        b0 = r0;
        b1 = r1;
    }
    // streaming store (nt): the XCD's L2 does not keep the line for reuse
    __device__ __forceinline__ void buf_store4_nt(Rsrc r, uint32_t voff, uint32_t soff, f32x4 v) const
    {
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, voff, soff, kCpolNt);
    }
    // partial sums: device-scope (sc1) stores and loads.  A device-scope
    // store, once complete, is visible to loads of that scope from every
    // XCD, and such loads do not return stale copies from a CU's L1 or an
    // XCD's L2; so the hand-over needs neither a write-back of the whole L2
    // (buffer_wbl2) nor an invalidation (buffer_inv).
    __device__ __forceinline__ void buf_store4_dev(Rsrc r, uint32_t voff, uint32_t soff, f32x4 v) const
    {
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, voff, soff, kCpolSc1);
    }
    __device__ __forceinline__ f32x4 buf_load4_dev(Rsrc r, uint32_t voff, uint32_t soff) const
    {
        return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kCpolSc1));
    }
    // every store of this wave complete (s_waitcnt vmcnt(0)): for the
    // device-scope partial sums, visible to every XCD
    __device__ __forceinline__ void stores_done() const { wait_vmcnt<0>(); }
    // the counters: device-scope atomics (relaxed: the partial sums they
    // publish are device-scope accesses themselves, ordered by stores_done
    // before the count and by the count's value before the loads)
    __device__ __forceinline__ int flag_load(int *f) const
    {
        return __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __device__ __forceinline__ void flag_store(int *f, int v) const
    {
        __hip_atomic_store(f, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // atomic add; returns the value before it
    __device__ __forceinline__ int flag_add(int *f, int v) const
    {
        return __hip_atomic_fetch_add(f, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __device__ __forceinline__ void lds_write4(char *q, int v, bool on) const
    {
        if (on)
            *(int *)q = v;
    }
    __device__ __forceinline__ int lds_read4(const char *q) const { return *(const int *)q; }
};

template <int BM, int BN, int BK, int WGM, int WGN, int DT>
__global__ void __launch_bounds__(WGM * WGN * 64)
gemm_kernel(GemmParams p_in)
{
    __shared__ __attribute__((aligned(16))) char smem[general_lds_bytes<BM, BN, BK>()];
    const int w = linear_block();
    if (w >= p_in.grid)
        return;
    const DeviceOps ops{smem};
    general_tile<BM, BN, BK, WGM, WGN, DT>(ops, p_in, w, p_in.grid, threadIdx.x);
}

// LDS bytes the pipelined kernel allocates.
template <int BM, int BN, int BK, int STAGES>
constexpr int dma_lds_bytes()
{
    return STAGES * (BM * BK * 2 + BK * BN * 2);
}

// One workgroup (id `block` of `nblocks`) of the pipelined kernel, as seen
// by thread `tid`.  The host launches it only when every split has at least
// STAGES K steps.
//
// MI is the MFMA block: 32 (v_mfma_f32_32x32x16, 16 k per instruction) or
// 16 (v_mfma_f32_16x16x32, 32 k per instruction).  Both do the same work per
// K step from the same LDS bytes.  On random data the GPU is power-capped;
// there the 16 x 16 shape sustains more flops (MFMA-only, about 2100
// against 1840 TFLOP/s, with the accumulators in VGPRs or AGPRs alike).
//
// KW is the number of waves along K: with 2, two waves own each (BM/WGM) x
// (BN/WGN) block of C, each multiplying one of the two MFMA sub-steps of
// every K step, and their sums are added at the end.
template <int BM, int BN, int BK, int STAGES, int WGM, int WGN, int DT, int MI, int KW, class Ops>
__host__ __device__ __forceinline__ void dma_tile(const Ops &ops, const GemmParams &p_in, int block, int nblocks,
                                                  int tid)
{
    static_assert(MI == 16 || MI == 32, "MFMA block");
    static_assert(KW == 1 || KW == 2, "waves along K");
    constexpr int NMN = WGM * WGN;               // waves along M and N
    constexpr int NW = NMN * KW;
    constexpr int TM = BM / WGM, TN = BN / WGN;
    constexpr int FM = TM / MI, FN = TN / MI;   // MFMA blocks per wave
    constexpr int KI = 512 / MI;                 // k per MFMA
    constexpr int KS = BK / KI;                  // MFMA k sub-steps per K step
    constexpr int NG = 64 / MI;                  // lane groups along k, 8 values each
    constexpr int AE = MI * MI / 64;             // accumulators per lane and block
    constexpr bool TWO_PER_SIMD = NW == 8 && KW == 1;   // the two-waves-per-SIMD schedule below
    typedef float accT __attribute__((ext_vector_type(AE)));
    constexpr int A_ROWB = BK * 2;
    constexpr int B_ROWB = BN * 2;
    constexpr int A_BYTES = BM * A_ROWB;
    constexpr int B_BYTES = BK * B_ROWB;
    constexpr int STAGE = A_BYTES + B_BYTES;
    constexpr int A_LD = A_BYTES / 1024 / NW;    // direct loads per wave per K step
    constexpr int B_LD = B_BYTES / 1024 / NW;
    constexpr int LD = A_LD + B_LD;
    constexpr int A_ROWS_PER_LD = 1024 / A_ROWB; // tile rows one load instruction fills
    constexpr int B_ROWS_PER_LD = 1024 / B_ROWB;
    static_assert(BK == 32 || BK == 64, "A rows of 64 or 128 bytes");
    static_assert(BN % 32 == 0 && B_ROWB >= 256 && B_ROWB <= 1024 && 1024 % B_ROWB == 0, "B layout");
    static_assert(A_LD * NW * 1024 == A_BYTES && B_LD * NW * 1024 == B_BYTES, "load split");
    static_assert(KS >= 2 && STAGES >= 2 && STAGES * STAGE <= 160 * 1024, "pipeline shape");
    static_assert((STAGES - 1) * LD < 64, "vmcnt range");

    int tm, tn, ks, local;
    const GemmParams p = map_tile(p_in, block, nblocks, tm, tn, ks, local);
    const int m0 = tm * BM, n0 = tn * BN;
    const int kbeg = ks * p.k_chunk;
    const int kend = min(p.K, kbeg + p.k_chunk);
    // A K range that is not a whole number of steps (K a multiple of 8, so
    // every 16-byte chunk is wholly inside or outside it) ends in a partial
    // step of tk values.  It runs first, as step 0: its loads read clamped,
    // valid addresses, and the prologue zeroes the LDS chunks of A and rows
    // of B beyond K before any fragment read.  Full steps follow from kbeg.
    const int klen = kend > kbeg ? kend - kbeg : 0;
    const int tk = klen % BK;
    const int nk = klen / BK + (tk > 0 ? 1 : 0);
    auto step_k0 = [&](int u) { return tk > 0 ? (u == 0 ? kend - tk : kbeg + (u - 1) * BK) : kbeg + u * BK; };

    const int lane = tid & 63;
    const int wave = ops.uniform(tid >> 6);
    const int wmn = wave % NMN, wk = wave / NMN;
    const int wm = wmn % WGM, wn = wmn / WGM;
    const int64_t lda = p.lda, ldb = p.ldb;
    char *const smem = ops.lds();

    // B rows keep n contiguous; the 32-byte chunks of row k are permuted by
    // XOR with bswz(k), so that the transpose reads of one instruction (4
    // consecutive rows per 16 lanes; with MI 16, rows 8 apart in the other
    // 16 lanes of a half-wave) fall in distinct banks.
    auto bswz = [](int k) { return MI == 32 ? (k & 3) << 1 : ((k & 3) << 1) | ((k >> 3) & 1); };

    // --- per-lane byte offsets of the direct loads (relative to the tile) ---
    uint32_t a_goff[A_LD], b_goff[B_LD];
    const int mmax = p.M - 1 - m0;               // last valid tile row
    const int nmax = ((p.N - 1) / 8) * 8 - n0;   // last valid 8-column chunk
#pragma unroll
    for (int j = 0; j < A_LD; ++j) {
        const int r = (wave * A_LD + j) * A_ROWS_PER_LD + lane / (A_ROWB / 16);
        const int c = (lane % (A_ROWB / 16)) ^ aswz<A_ROWB>(r);
        a_goff[j] = (uint32_t)((min(r, mmax) * lda + c * 8) * 2);
    }
#pragma unroll
    for (int j = 0; j < B_LD; ++j) {
        const int k = (wave * B_LD + j) * B_ROWS_PER_LD + lane / (B_ROWB / 16);
        const int q = lane % (B_ROWB / 16);          // physical 16-byte chunk in the row
        const int c = (q >> 1) ^ bswz(k);            // logical 32-byte chunk
        const int n = c * 16 + (q & 1) * 8;
        b_goff[j] = (uint32_t)((k * ldb + min(n, nmax)) * 2);
    }

    auto issue_loads = [&](int kstep, int stage) {
        const int k0 = step_k0(kstep);
        const uint16_t *Ab = p.A + (int64_t)m0 * lda + k0;
        const uint16_t *Bb = p.B + (int64_t)k0 * ldb + n0;
        const uint32_t sA = ops.lds_addr(smem) + stage * STAGE;
        const uint32_t sB = sA + A_BYTES;
        const bool partial = tk > 0 && kstep == 0;
#pragma unroll
        for (int j = 0; j < A_LD; ++j) {
            // a chunk beyond K reads the row's first chunk instead
            const int r = (wave * A_LD + j) * A_ROWS_PER_LD + lane / (A_ROWB / 16);
            const int c = (lane % (A_ROWB / 16)) ^ aswz<A_ROWB>(r);
            const uint32_t off = partial && c * 8 >= tk ? a_goff[j] - (uint32_t)(c * 16) : a_goff[j];
            ops.load16(Ab, off, sA + (wave * A_LD + j) * 1024);
        }
#pragma unroll
        for (int j = 0; j < B_LD; ++j) {
            // a row beyond K reads row tk - 1 instead
            const int k = (wave * B_LD + j) * B_ROWS_PER_LD + lane / (B_ROWB / 16);
            const uint32_t off =
                partial && k >= tk ? b_goff[j] - (uint32_t)((int64_t)(k - tk + 1) * ldb * 2) : b_goff[j];
            ops.load16(Bb, off, sB + (wave * B_LD + j) * 1024);
        }
    };
    // After the partial step has landed in stage 0 (and a barrier): zero the
    // A chunks and B rows beyond K, then a barrier before the fragment reads.
    auto zero_partial = [&]() {
        if (tk > 0) {
            constexpr int NT = NW * 64;
            const u32x4 z = {0u, 0u, 0u, 0u};
            static_assert((BM * (BK / 8)) % NT == 0 && (BK * (B_ROWB / 16)) % NT == 0, "whole passes");
            for (int idx = tid; idx < BM * (BK / 8); idx += NT) {
                const int r = idx / (BK / 8), c = idx % (BK / 8);
                ops.lds_write16(smem + r * A_ROWB + ((c ^ aswz<A_ROWB>(r)) << 4), z, c * 8 >= tk);
            }
            for (int idx = tid; idx < BK * (B_ROWB / 16); idx += NT)
                ops.lds_write16(smem + A_BYTES + idx * 16, z, idx / (B_ROWB / 16) >= tk);
            ops.wait_lgkm0();
            ops.barrier();
        }
    };

    // --- fragment addressing ---
    const int lr = lane % MI;                     // A row / B column within an MFMA block
    const int kg = lane / MI;                     // k group of the MFMA operand (8 values)
    // A: row wm*TM + i*MI + lr, logical chunk (KI/8)*kk + kg
    const int a_x = kg ^ aswz<A_ROWB>(lr);
    const int a_lane = (wm * TM + lr) * A_ROWB;
    // B: rows kk*KI + 8*kg + t4 (and 4 more), columns wn*TN + j*MI + 16*c16 + 4*(s16%4)
    const int s16 = lane & 15;
    const int c16 = lr >> 4;                      // 16-column half of a 32-column block
    const int t4 = s16 >> 2;                      // equals row & 3
    const int b_lane = (8 * kg + t4) * B_ROWB + 8 * (s16 & 3);
    const int b_c0 = wn * (TN / 16) + c16;        // logical 32-byte chunk of block 0
    const int b_sw = bswz(8 * kg + t4);           // the same for every kk and the 4 rows below

    accT acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int e = 0; e < AE; ++e)
                acc[i][j][e] = 0.0f;

    u32x4 fa[2][FM], fb[2][FN];

    // A fragment of MFMA block row i and B fragment of block column j for
    // sub-step kk of the K step held in LDS stage `stage`
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
    auto read_A = [&](int stage, int kk, int buf, int i) {
        const char *sA = smem + stage * STAGE + a_lane + ((((KI / 8) * kk) ^ a_x) << 4);
        fa[buf][i] = ops.read16(sA + i * MI * A_ROWB);
    };
    auto read_B = [&](int stage, int kk, int buf, int j) {
        const char *pb = smem + stage * STAGE + A_BYTES + kk * KI * B_ROWB + b_lane +
                         (((b_c0 + j * (MI / 16)) ^ b_sw) << 5);
        const v4i16 lo = ops.read_tr8(pb);
        const v4i16 hi = ops.read_tr8(pb + 4 * B_ROWB);
        u32x4 v;
        v.x = __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 0, 1));
        v.y = __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 2, 3));
        v.z = __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 0, 1));
        v.w = __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 2, 3));
        fb[buf][j] = v;
    };
    // The fragment reads of one sub-step as FM + FN units in the order the
    // MFMAs below first need them: A0, B0 .. B(FN-1), A1 .. A(FM-1).  Unit u
    // is issued after MFMA u * SP of the sub-step before, so that the reads
    // spread over the first half of its MFMAs (with 16 x 16 blocks, 16 units
    // among 64 MFMAs: one every second MFMA).
    constexpr int NU = FM + FN;
    constexpr int SP = (FM * FN / 2) / NU > 0 ? (FM * FN / 2) / NU : 1;
    auto read_unit = [&](int stage, int kk, int buf, int u) {
        if (u == 0)
            read_A(stage, kk, buf, 0);
        else if (u <= FN)
            read_B(stage, kk, buf, u - 1);
        else
            read_A(stage, kk, buf, u - FN);
    };
    auto read_frags = [&](int stage, int kk, int buf) {
#pragma unroll
        for (int u = 0; u < NU; ++u)
            read_unit(stage, kk, buf, u);
    };
    // MFMA n of a sub-step, row-major over the (i, j) blocks.
    auto mfma_n = [&](int buf, int n) {
        const int i = n / FN, j = n % FN;
        acc[i][j] = ops.template mfma<DT>(fb[buf][j], fa[buf][i], acc[i][j]);
    };

    // Direct load j (0 .. LD-1) of K step u into LDS stage `stage`.
    auto load_j = [&](int u, int stage, int j) {
        const int k0 = step_k0(u);
        const uint32_t sA = ops.lds_addr(smem) + stage * STAGE;
        if (j < A_LD) {
            const uint16_t *Ab = p.A + (int64_t)m0 * lda + k0;
            ops.load16(Ab, a_goff[j], sA + (wave * A_LD + j) * 1024);
        } else {
            const uint16_t *Bb = p.B + (int64_t)k0 * ldb + n0;
            ops.load16(Bb, b_goff[j - A_LD], sA + A_BYTES + (wave * B_LD + (j - A_LD)) * 1024);
        }
    };
    // With three or more stages the loads of one K step are issued in two
    // halves: the first after the barrier that frees their stage, the
    // second during the next step's sub-steps before its barrier.  This
    // spaces the direct loads one per few MFMAs (a burst of them fills the
    // vector-memory queue and blocks the wave's MFMA issue) while each load
    // still has about STAGES-2 K steps to land.  With two stages every load
    // must be issued right after the barrier.
    constexpr bool SPLIT = STAGES >= 3;
    constexpr int H1 = SPLIT ? (LD + 1) / 2 : LD;   // loads issued after the barrier
    constexpr int H2 = LD - H1;                      // loads issued before the next barrier
    constexpr int STEP1 = H1 > 0 ? (FM * FN) / H1 > 0 ? (FM * FN) / H1 : 1 : 1;
    constexpr int H2D = H2 > 0 ? H2 : 1;
    constexpr int STEP2 = ((KS - 1) * FM * FN) / H2D > 0 ? ((KS - 1) * FM * FN) / H2D : 1;

    // One K step t.  LOAD1: issue the first half of step t+STAGES's loads
    // (into stage t, freed by this step's barrier).  LOAD2: issue the second
    // half of step t-1+STAGES's loads (into stage t-1).  WAIT: number of this
    // wave's load groups allowed in flight once step t+1 has landed (-1: t
    // is the last step).
    auto kstep = [&]<bool LOAD1, bool LOAD2, int WAIT>(int t) {
        const int stage = t % STAGES;
        const int prev = (t + STAGES - 1) % STAGES;
        // sub-steps 0 .. KS-2: MFMAs of kk, with the read units of kk+1 (and,
        // spread out, the second-half loads) between them, in this order
#pragma unroll
        for (int kk = 0; kk < KS - 1; ++kk) {
#pragma unroll
            for (int n = 0; n < FM * FN; ++n) {
                mfma_n(kk & 1, n);
                if (n % SP == 0 && n / SP < NU)
                    read_unit(stage, kk + 1, (kk + 1) & 1, n / SP);
                if constexpr (LOAD2) {
                    const int gi = kk * FM * FN + n;
                    if (gi % STEP2 == 0 && gi / STEP2 < H2)
                        load_j(t - 1 + STAGES, prev, H1 + gi / STEP2);
                }
                ops.fence();
            }
        }
        // stage t fully read by this wave; stage t+1 landed for this wave
        ops.wait_lgkm0();
        if constexpr (WAIT >= 0)
            ops.template wait_vm<WAIT * LD>();
        ops.barrier();
        ops.fence();
        // last sub-step: its MFMAs, with the first-half loads of step
        // t+STAGES into the freed stage and the reads of step t+1's first
        // sub-step
        const int next = (t + 1) % STAGES;
#pragma unroll
        for (int n = 0; n < FM * FN; ++n) {
            mfma_n((KS - 1) & 1, n);
            if constexpr (WAIT >= 0) {
                if (n % SP == 0 && n / SP < NU)
                    read_unit(next, 0, 0, n / SP);
            }
            if constexpr (LOAD1) {
#pragma unroll
                for (int q = 0; q < (H1 + FM * FN - 1) / (FM * FN); ++q) {
                    const int j = (H1 <= FM * FN) ? (n % STEP1 == 0 ? n / STEP1 : H1) : n * ((H1 + FM * FN - 1) / (FM * FN)) + q;
                    if (j < H1)
                        load_j(t + STAGES, stage, j);
                }
            }
            ops.fence();
        }
    };

    if constexpr (TWO_PER_SIMD) {
        // Two waves per SIMD, 16 x 16 x 32 MFMAs, BK 64 (two sub-steps), two
        // LDS stages; each wave owns 128 accumulator registers, and the two
        // waves of a SIMD cover each other's waits (measured 1-4.5% faster
        // than one wave per SIMD owning a 128 x 128 block, although the
        // waves read 1.5 times the LDS bytes).  A and B fragments are
        // double-buffered between the sub-steps (252 registers): block row
        // i of the next sub-step is read as soon as row i of the current
        // one has issued its MFMAs.  (Reading A into the registers row i
        // has just used, which saves 32 registers, measured 6-8% slower.)
        // One row of sub-step 1 runs before the barrier: 0 rows exposed the
        // last A read's latency (4.5% slower), 2 or more left fewer MFMAs
        // to space the direct loads over (1-3% slower).
        constexpr int R = 1;                      // rows of sub-step 1 issued before the barrier
        static_assert(MI == 16 && STAGES == 2 && KS == 2 && FN <= FM - R, "two-per-SIMD schedule shape");
        constexpr int LSTEP = ((FM - R) * FN) / LD > 0 ? ((FM - R) * FN) / LD : 1;
        static_assert(LSTEP * (LD - 1) < (FM - R) * FN, "load spacing");
        u32x4 ga[2][FM], gb[2][FN];
        auto row = [&](int b, int i) {
#pragma unroll
            for (int j = 0; j < FN; ++j)
                acc[i][j] = ops.template mfma<DT>(gb[b][j], ga[b][i], acc[i][j]);
        };
        // One K step t.  Sub-step 0 works from ga[0] / gb[0] and reads sub-step
        // 1 of the same stage (ga[1], gb[1]).  Before the barrier:
        // the first R rows of sub-step 1 (registers only, which gives the
        // last A read time to land), then the waits.  After it: the rest of
        // sub-step 1 with the reads of step t+1's sub-step 0 (ga[0], gb[0])
        // and, if LOAD, the direct loads of step t+2 into the stage
        // just freed.  WAIT < 0: t is the last step.
        auto kstep_pair = [&]<bool LOAD, int WAIT>(int t) {
            const int stage = t & 1, next = stage ^ 1;
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                row(0, i);
                ga[1][i] = frag_A(stage, 1, i);
                if (i < FN)
                    gb[1][i] = frag_B(stage, 1, i);
                ops.fence();
            }
#pragma unroll
            for (int i = 0; i < R; ++i) {
                row(1, i);
                ops.fence();
            }
            // stage t fully read by this wave; stage t+1 landed for this wave
            ops.wait_lgkm0();
            if constexpr (WAIT >= 0)
                ops.template wait_vm<0>();
            ops.barrier();
            ops.fence();
            // the rows that issue the direct loads run at a raised priority
            // against the other wave of the SIMD (measured 0.6-0.8% faster)
            ops.template priority<1>();
            if constexpr (WAIT >= 0) {
#pragma unroll
                for (int i = 0; i < R; ++i)
                    ga[0][i] = frag_A(next, 0, i);
            }
#pragma unroll
            for (int i = R; i < FM; ++i) {
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    acc[i][j] = ops.template mfma<DT>(gb[1][j], ga[1][i], acc[i][j]);
                    const int g = (i - R) * FN + j;
                    if constexpr (LOAD) {
                        if (g % LSTEP == 0 && g / LSTEP < LD)
                            load_j(t + 2, stage, g / LSTEP);
                    }
                }
                if constexpr (WAIT >= 0) {
                    ga[0][i] = frag_A(next, 0, i);
                    if (i - R < FN)
                        gb[0][i - R] = frag_B(next, 0, i - R);
                }
                ops.fence();
            }
            ops.template priority<0>();
        };
        if (nk >= 2) {
            issue_loads(0, 0);
            issue_loads(1, 1);
            ops.template wait_vm<LD>();
            ops.barrier();
            zero_partial();
#pragma unroll
            for (int i = 0; i < FM; ++i)
                ga[0][i] = frag_A(0, 0, i);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                gb[0][j] = frag_B(0, 0, j);
            for (int t = 0; t < nk - 2; ++t)
                kstep_pair.template operator()<true, 0>(t);
            kstep_pair.template operator()<false, 0>(nk - 2);
            kstep_pair.template operator()<false, -1>(nk - 1);
        }
    } else if constexpr (KW == 2) {
        // Two waves per SIMD on a tile too narrow for two 128 x 64 blocks
        // per SIMD: the waves of a pair own the same 128 x 64 block and
        // split every K step, wave wk multiplying sub-step wk (32 of the 64
        // k).  Each wave thus reads the LDS bytes per flop of a 128 x 64
        // block, and the other wave of its SIMD covers its barrier and load
        // waits.  Three stages: the loads of step t+3 go into the stage that
        // step t's barrier frees (its fragments were read during step t-1)
        // and have two steps to land.  A wave's fragments of step t+1 are
        // read during step t into the other register buffer, so the buffer
        // alternates with the step's parity (a template argument: register
        // arrays are not indexed at run time).
        constexpr int R = 1;                      // rows of a step issued before its barrier
        static_assert(MI == 16 && STAGES == 3 && KS == 2 && FN <= FM - R && FM % 2 == 0, "K-pair schedule shape");
        constexpr int LSTEP = ((FM - R) * FN) / LD > 0 ? ((FM - R) * FN) / LD : 1;
        static_assert(LSTEP * (LD - 1) < (FM - R) * FN, "load spacing");
        u32x4 ga[2][FM], gb[2][FN];
        // One K step t in buffer BUF (t's parity).  LOAD: issue the loads of
        // step t+3 into stage t % 3.  WAIT: this wave's load groups allowed
        // in flight once step t+1 has landed (-1: t is the last step).
        auto kstep_k = [&]<int BUF, bool LOAD, int WAIT>(int t) {
            const int stage = t % 3;
            const int next = stage == 2 ? 0 : stage + 1;
#pragma unroll
            for (int i = 0; i < R; ++i) {
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = ops.template mfma<DT>(gb[BUF][j], ga[BUF][i], acc[i][j]);
                ops.fence();
            }
            // stage t fully read by every wave; step t+1 landed for this wave
            ops.wait_lgkm0();
            if constexpr (WAIT >= 0)
                ops.template wait_vm<WAIT * LD>();
            ops.barrier();
            ops.fence();
            ops.template priority<1>();
            if constexpr (WAIT >= 0) {
#pragma unroll
                for (int i = 0; i < R; ++i)
                    ga[BUF ^ 1][i] = frag_A(next, wk, i);
            }
#pragma unroll
            for (int i = R; i < FM; ++i) {
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    acc[i][j] = ops.template mfma<DT>(gb[BUF][j], ga[BUF][i], acc[i][j]);
                    const int g = (i - R) * FN + j;
                    if constexpr (LOAD) {
                        if (g % LSTEP == 0 && g / LSTEP < LD)
                            load_j(t + 3, stage, g / LSTEP);
                    }
                }
                if constexpr (WAIT >= 0) {
                    ga[BUF ^ 1][i] = frag_A(next, wk, i);
                    if (i - R < FN)
                        gb[BUF ^ 1][i - R] = frag_B(next, wk, i - R);
                }
                ops.fence();
            }
            ops.template priority<0>();
        };
        // the last three steps: no more loads, then exact waits
        auto last3 = [&]<int BUF>(int t) {
            kstep_k.template operator()<BUF, false, 1>(t);
            kstep_k.template operator()<BUF ^ 1, false, 0>(t + 1);
            kstep_k.template operator()<BUF, false, -1>(t + 2);
        };
        // Add the pair's sums through LDS (every stage is free once every
        // wave is past the last step's barrier, which follows its last
        // fragment reads): wave WK keeps block rows
        // [WK FM/2, WK FM/2 + FM/2), hands the other half to its partner and
        // moves the kept rows to acc[0 .. FM/2).  Sub-step 0's sum is the
        // first operand of every addition.  WK is the wave's wk as a template
        // argument, so that the halves are chosen at compile time (a run-time
        // choice keeps both live).
        constexpr int FH = FM / 2;
        static_assert(NW * FH * FN * 1024 <= STAGES * STAGE, "exchange fits the stages");
        char *const give = smem + (wmn * KW + wk) * FH * FN * 1024 + lane * 16;
        const char *const take = smem + (wmn * KW + (wk ^ 1)) * FH * FN * 1024 + lane * 16;
        auto exchange = [&]<int WK>() {
            constexpr int GIVE = WK ? 0 : FH, KEEP = WK ? FH : 0;
#pragma unroll
            for (int h = 0; h < FH; ++h)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    ops.lds_write16(give + (h * FN + j) * 1024, __builtin_bit_cast(u32x4, acc[GIVE + h][j]));
            ops.wait_lgkm0();
            ops.barrier();
#pragma unroll
            for (int h = 0; h < FH; ++h)
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    const accT other = __builtin_bit_cast(accT, ops.read16(take + (h * FN + j) * 1024));
                    acc[h][j] = WK ? other + acc[KEEP + h][j] : acc[KEEP + h][j] + other;
                }
        };
        // Steps 0 .. nk-4 issue loads (nl of them).  The K loop is
        // instantiated per parity of nl: the fragment buffers alternate with
        // the step, and with an odd nl step 0 runs from buffer 1, so that the
        // loop of two steps and the last three always start from buffer 0.
        // The loop body runs at least once (nk = 3 and 4 are straight-line
        // code of their own): a path that skipped it kept the first
        // fragments live across it and spilled.  After the last step only the
        // accumulators are live, and the exchange is instantiated per wk.
        // (buffer 1 is read B first: the branches then begin differently, so
        // the compiler does not hoist the common reads above them, where
        // they would stay live across the loop)
        auto first_frags = [&]<int P>() {
            if constexpr (P == 1) {
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    gb[P][j] = frag_B(0, wk, j);
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
                ga[P][i] = frag_A(0, wk, i);
            if constexpr (P == 0) {
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    gb[P][j] = frag_B(0, wk, j);
            }
        };
        auto k_loop = [&]<int P>() {
            const int nl = nk - 3;
            first_frags.template operator()<P>();
            int t = 0;
            if constexpr (P == 1) {
                kstep_k.template operator()<1, true, 1>(0);
                t = 1;
            }
            do {
                kstep_k.template operator()<0, true, 1>(t);
                kstep_k.template operator()<1, true, 1>(t + 1);
                t += 2;
            } while (t + 2 <= nl);
            last3.template operator()<0>(t);
        };
        if (nk >= 3) {
            issue_loads(0, 0);
            issue_loads(1, 1);
            issue_loads(2, 2);
            ops.template wait_vm<2 * LD>();
            ops.barrier();
            zero_partial();
            if (nk == 3) {
                first_frags.template operator()<0>();
                last3.template operator()<0>(0);
            } else if (nk == 4) {
                first_frags.template operator()<1>();
                kstep_k.template operator()<1, true, 1>(0);
                last3.template operator()<0>(1);
            } else if ((nk - 3) & 1) {
                k_loop.template operator()<1>();
            } else {
                k_loop.template operator()<0>();
            }
            if (wk)
                exchange.template operator()<1>();
            else
                exchange.template operator()<0>();
        }
    } else if (nk >= STAGES) {
        // prologue: fill every stage, wait for stage 0
#pragma unroll
        for (int t = 0; t < STAGES; ++t)
            issue_loads(t, t);
        ops.template wait_vm<(STAGES - 1) * LD>();
        ops.barrier();
        zero_partial();
        read_frags(0, 0, 0);
        if (nk > STAGES) {
            // step 0: the prologue issued all of step STAGES-1's loads
            kstep.template operator()<true, false, STAGES - 2>(0);
            // steady state
            for (int t = 1; t < nk - STAGES; ++t)
                kstep.template operator()<true, SPLIT, STAGES - 2>(t);
            // the last STAGES steps: no more first halves, exact waits
            kstep.template operator()<false, SPLIT, STAGES - 2>(nk - STAGES);
            [&]<int... I>(std::integer_sequence<int, I...>) {
                (kstep.template operator()<false, false, (I + 2 < STAGES ? STAGES - 3 - I : -1)>(nk - STAGES + 1 + I),
                 ...);
            }(std::make_integer_sequence<int, STAGES - 1>{});
        } else {
            [&]<int... I>(std::integer_sequence<int, I...>) {
                (kstep.template operator()<false, false, (I + 1 < STAGES ? STAGES - 2 - I : -1)>(I), ...);
            }(std::make_integer_sequence<int, STAGES>{});
        }
    }

    // epilogue: B is the MFMA's first operand, so lane l holds, for block
    // (i, j), row lr and groups of 4 consecutive columns 4*kg + 4*NG*q
    const OutView ov = out_view<BM, BN>(p, ks, local, m0, n0);
    float *Cb = ov.base;
    const int64_t ldc = ov.ld;
    const bool vec_store = p.vec_c && (m0 + BM <= p.M) && (n0 + BN <= p.N);
    // with two waves along K, each stores its FM / 2 kept block rows
    constexpr int FO = FM / KW;
#pragma unroll
    for (int i = 0; i < FO; ++i) {
        const int row = m0 + wm * TM + (wk * FO + i) * MI + lr;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
#pragma unroll
            for (int q = 0; q < AE / 4; ++q) {
                const int col = n0 + wn * TN + j * MI + q * 4 * NG + kg * 4;
                f32x4 v;
                v.x = acc[i][j][4 * q + 0];
                v.y = acc[i][j][4 * q + 1];
                v.z = acc[i][j][4 * q + 2];
                v.w = acc[i][j][4 * q + 3];
                if (vec_store) {
                    ops.store4(Cb + (int64_t)(row - ov.r0) * ldc + (col - ov.c0), v);
                } else if (row < p.M) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (col + e < p.N)
                            ops.store1(Cb + (int64_t)(row - ov.r0) * ldc + (col - ov.c0) + e, v[e]);
                }
            }
        }
    }
}

template <int BM, int BN, int BK, int STAGES, int WGM, int WGN, int DT, int MI, int KW>
__global__ void __launch_bounds__(WGM * WGN * KW * 64, 1)
gemm_kernel_dma(GemmParams p_in)
{
    __shared__ __attribute__((aligned(1024))) char smem[dma_lds_bytes<BM, BN, BK, STAGES>()];
    const int w = linear_block();
    if (w >= p_in.grid)
        return;
    const DeviceOps ops{smem};
    dma_tile<BM, BN, BK, STAGES, WGM, WGN, DT, MI, KW>(ops, p_in, w, p_in.grid, threadIdx.x);
}

// C[i][j] = sum over p of W[p][i][j], p ascending (a fixed order, so the
// result does not depend on scheduling).  The paper's split-k kernels reduce
// partials into global memory with bulk reduce-add copies (Section 6).
__global__ void __launch_bounds__(256)
splitk_reduce(const float *W, int64_t split_stride, int64_t ldw, int split,
              float *C, int64_t ldc, int M, int N, int vec_c)
{
    const int64_t nvec = (int64_t)M * ((N + 3) / 4);
    const int64_t cols4 = (N + 3) / 4;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < nvec;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int i = (int)(t / cols4);
        const int j = (int)(t - (int64_t)i * cols4) * 4;
        const float *w = W + (int64_t)i * ldw + j;
        f32x4 s = *(const f32x4 *)w;
        for (int q = 1; q < split; ++q) {
            const f32x4 x = *(const f32x4 *)(w + q * split_stride);
            s += x;
        }
        float *c = C + (int64_t)i * ldc + j;
        if (vec_c && j + 4 <= N) {
            *(f32x4 *)c = s;
        } else {
            for (int e = 0; e < 4; ++e)
                if (j + e < N)
                    c[e] = s[e];
        }
    }
}

// C[0:M, 0:N] = 0 (the K == 0 product).
__global__ void __launch_bounds__(256)
fill_zero(float *C, int64_t ldc, int M, int N)
{
    const int64_t n = (int64_t)M * N;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int i = (int)(t / N);
        const int j = (int)(t - (int64_t)i * N);
        C[(int64_t)i * ldc + j] = 0.0f;
    }
}

}  // namespace xgemm_dev
