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
};

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

// 16-byte chunk slot of logical chunk c in tile row r.  Rows r and r^j for
// j < 16 never share a slot among 8 consecutive rows, nor a (row parity,
// slot) pair among 16 consecutive rows.
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Workgroup -> (tile_m, tile_n, split).  The hardware hands workgroup ids to
// the XCDs round-robin; consecutive logical ids are first gathered onto one
// XCD, then walked in groups of group_m tile rows so that the workgroups an
// XCD runs at the same time share rows of A and columns of B in its L2.  The
// split index is outermost: workgroups of one K range run together.
// (The paper's persistent kernels hand out tasks in lexicographic order and
// leave other orders to future work, Section 4.2.)
__device__ __forceinline__ void map_tile(const GemmParams &p, int &tm, int &tn, int &ks)
{
    const int total = gridDim.x;
    const int w = blockIdx.x;
    const int per = total / kNumXcd;
    const int lid = (w < per * kNumXcd) ? (w % kNumXcd) * per + w / kNumXcd : w;
    const int tiles = p.tiles_m * p.tiles_n;
    ks = lid / tiles;
    const int t = lid - ks * tiles;
    const int group = p.group_m * p.tiles_n;
    const int g = t / group;
    const int first_m = g * p.group_m;
    const int gm = min(p.tiles_m - first_m, p.group_m);
    const int r = t - g * group;
    tm = first_m + r % gm;
    tn = r / gm;
}

// Eight 16-bit values starting at base[off], the first `cnt` of them read
// from memory and the rest zero.
__device__ __forceinline__ u32x4 load8_masked(const uint16_t *base, int64_t off, int cnt)
{
    uint32_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
        h[e] = (e < cnt) ? (uint32_t)base[off + e] : 0u;
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
__device__ __forceinline__ u32x4 column8(const u32x4 (&v)[8], int c)
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

template <int BM, int BN, int BK, int WGM, int WGN, int DT>
__global__ void __launch_bounds__(WGM * WGN * 64)
gemm_kernel(GemmParams p)
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
    static_assert(2 * STAGE <= 160 * 1024, "LDS budget");

    __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

    int tm, tn, ks;
    map_tile(p, tm, tn, ks);
    const int m0 = tm * BM, n0 = tn * BN;
    const int kbeg = ks * p.k_chunk;
    const int kend = min(p.K, kbeg + p.k_chunk);
    const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;

    const int tid = threadIdx.x;
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
                    ra[it] = *(const u32x4 *)(Ab + a_off[it]);
#pragma unroll
            for (int it = 0; it < B_IT; ++it)
                if (B_UNITS % NT == 0 || tid + it * NT < B_UNITS)
#pragma unroll
                    for (int r = 0; r < 8; ++r)
                        rb[it][r] = *(const u32x4 *)(Bb + b_off[it] + r * ldb);
        } else {
#pragma unroll
            for (int it = 0; it < A_IT; ++it)
                if (A_UNITS % NT == 0 || tid + it * NT < A_UNITS) {
                    const int gm = m0 + a_row[it];
                    const int gk = k0 + a_c[it] * 8;
                    const int cnt = (gm < p.M) ? max(0, min(8, kend - gk)) : 0;
                    ra[it] = load8_masked(Ab, a_off[it], cnt);
                }
#pragma unroll
            for (int it = 0; it < B_IT; ++it)
                if (B_UNITS % NT == 0 || tid + it * NT < B_UNITS) {
                    const int gn = n0 + b_ng[it] * 8;
                    const int ncnt = max(0, min(8, p.N - gn));
#pragma unroll
                    for (int r = 0; r < 8; ++r) {
                        const int gk = k0 + b_kg[it] * 8 + r;
                        rb[it][r] = load8_masked(Bb, b_off[it] + r * ldb, gk < kend ? ncnt : 0);
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
                *(u32x4 *)(sA + r * ROWB + ((a_c[it] ^ swz(r)) << 4)) = ra[it];
            }
#pragma unroll
        for (int it = 0; it < B_IT; ++it)
            if (B_UNITS % NT == 0 || tid + it * NT < B_UNITS) {
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    const int n = b_ng[it] * 8 + c;
                    *(u32x4 *)(sB + n * ROWB + ((b_kg[it] ^ swz(n)) << 4)) = column8(rb[it], c);
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
                fa[i] = *(const u32x4 *)(sA + i * 32 * ROWB + co);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                fb[j] = *(const u32x4 *)(sB + j * 32 * ROWB + co);
            // B fragment as the first operand: the result lands with lanes
            // along rows of C and 4 consecutive columns per register quad.
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = mfma32<DT>(fb[j], fa[i], acc[i][j]);
        }
    };

    if (nk > 0) {
        load_tiles(kbeg);
        store_tiles(0);
        __syncthreads();
        for (int kt = 0; kt < nk; ++kt) {
            const int cur = kt & 1;
            if (kt + 1 < nk)
                load_tiles(kbeg + (kt + 1) * BK);
            compute(cur);
            if (kt + 1 < nk)
                store_tiles(cur ^ 1);
            __syncthreads();
        }
    }

    // Epilogue: lane l holds rows (l % 32) of each 32 x 32 block and, in
    // register quad q, columns 8q + 4(l / 32) .. +3.
    float *Cb = p.C + (int64_t)ks * p.split_stride;
    const int64_t ldc = p.ldc;
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
                    *(f32x4 *)(Cb + (int64_t)row * ldc + col) = v;
                } else if (row < p.M) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (col + e < p.N)
                            Cb[(int64_t)row * ldc + col + e] = v[e];
                }
            }
        }
    }
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
