// Device code for y = A * x in fp32 (A row-major M x K, x and y vectors).
//
// The paper's second benchmark is a full-precision fp32 GEMV that uses no
// matrix instructions (Section 6); its bound is memory bandwidth: every
// element of A is read once for one multiply-add, so the ideal time is the
// time to stream A from HBM.
//
// Workgroup: 256 threads (4 waves) own R consecutive rows (and, when the
// rows alone give too few workgroups to fill the GPU, one of `split` K
// ranges of them; a second kernel then adds the ranges' partial sums).  The K range is
// cut into 16-byte chunks of 4 values; thread t takes chunks t, t + 256,
// t + 512, ... of every one of its R rows, so that each load instruction of
// a wave reads 1 KiB of one row contiguously.  Per iteration a thread
// issues U chunks of x and R x U chunks of A before using any of them (the
// loads are in flight together); a chunk of x is reused for the R rows from
// registers.  Each thread keeps one fp32 accumulator per row, updated with
// fused multiply-adds in ascending k.  Reduction: across the 64 lanes of a
// wave with butterfly shuffles, then across the 4 waves through LDS (one
// barrier), summing the wave partials in ascending wave order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xgemv_dev {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

struct GemvParams {
    const float *A;
    const float *x;
    float *y;
    float *part;  // split > 1: partial sums, part[q * M + i] for K range q
    int64_t lda;
    int M, K;
    int k_chunk;  // K values per split, a multiple of 4 (K when split == 1)
    int split;
    int vec;      // A and x 16-byte aligned and lda a multiple of 4: 16-byte loads
    int blocks;   // workgroups of the launch, ceil(M / R) * split; a 2-D grid may hold more, which exit
};

// Operations of the GEMV kernel on the device (the body below is also run on
// the host with a recording stand-in, for the synchronisation checker).
struct DeviceOps {
    float *red;  // kWaves * R floats of LDS
    __device__ __forceinline__ float *lds() const { return red; }
    __device__ __forceinline__ f32x4 load4(const float *q) const { return *(const f32x4 *)q; }
    __device__ __forceinline__ float load1(const float *q) const { return *q; }
    __device__ __forceinline__ float wave_sum(float v) const
    {
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1)
            v += __shfl_xor(v, off, 64);
        return v;
    }
    // LDS accesses of the lanes with `on` set (the others do nothing)
    __device__ __forceinline__ void lds_write1(float *q, float v, bool on) const
    {
        if (on)
            *q = v;
    }
    __device__ __forceinline__ float lds_read1(const float *q, bool on) const { return on ? *q : 0.0f; }
    // LDS writes of this wave complete, then a workgroup barrier that the
    // compiler may not move memory accesses across
    __device__ __forceinline__ void sync() const
    {
        __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));  // lgkmcnt(0)
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    }
    __device__ __forceinline__ void store1(float *q, float v) const { *q = v; }
};

__host__ __device__ __forceinline__ float fma4(f32x4 a, f32x4 b, float acc)
{
    acc = fmaf(a.x, b.x, acc);
    acc = fmaf(a.y, b.y, acc);
    acc = fmaf(a.z, b.z, acc);
    acc = fmaf(a.w, b.w, acc);
    return acc;
}

// Workgroup `block` is K range q = block / ceil(M / R) (the range's splits
// outermost, so that the workgroups reading one slice of x run together)
// and rows [rb * R, rb * R + R) with rb = block % ceil(M / R); thread tid's
// part of it.  Without a split (q = 0, the whole K range) the rows' sums go
// to y, otherwise to the partials.
template <int R, int U, class Ops>
__host__ __device__ __forceinline__ void gemv_block(const Ops &ops, const GemvParams &p, int block, int tid)
{
    const int row_blocks = (p.M + R - 1) / R;
    const int q = block / row_blocks;
    const int row0 = (block - q * row_blocks) * R;
    const int kb = q * p.k_chunk;
    const int kn = min(p.K, kb + p.k_chunk) - kb;   // K values of this range
    const float *xq = p.x + kb;
    const int lane = tid & 63, wave = tid >> 6;
    // rows past M read the last row (their sums are never stored)
    const float *arow[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        arow[r] = p.A + (int64_t)min(row0 + r, p.M - 1) * p.lda + kb;
    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        acc[r] = 0.0f;

    const int K4 = kn / 4;  // whole chunks of 4 values
    int c = tid;
    if (p.vec) {
        for (; c + (U - 1) * kThreads < K4; c += U * kThreads) {
            f32x4 xv[U], av[R][U];
#pragma unroll
            for (int u = 0; u < U; ++u)
                xv[u] = ops.load4(xq + 4 * (c + u * kThreads));
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < U; ++u)
                    av[r][u] = ops.load4(arow[r] + 4 * (c + u * kThreads));
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int r = 0; r < R; ++r)
                    acc[r] = fma4(av[r][u], xv[u], acc[r]);
        }
        for (; c < K4; c += kThreads) {
            const f32x4 xv = ops.load4(xq + 4 * c);
#pragma unroll
            for (int r = 0; r < R; ++r)
                acc[r] = fma4(ops.load4(arow[r] + 4 * c), xv, acc[r]);
        }
    } else {
        for (; c < K4; c += kThreads) {
            f32x4 xv;
            xv.x = ops.load1(xq + 4 * c);
            xv.y = ops.load1(xq + 4 * c + 1);
            xv.z = ops.load1(xq + 4 * c + 2);
            xv.w = ops.load1(xq + 4 * c + 3);
#pragma unroll
            for (int r = 0; r < R; ++r) {
                f32x4 av;
                av.x = ops.load1(arow[r] + 4 * c);
                av.y = ops.load1(arow[r] + 4 * c + 1);
                av.z = ops.load1(arow[r] + 4 * c + 2);
                av.w = ops.load1(arow[r] + 4 * c + 3);
                acc[r] = fma4(av, xv, acc[r]);
            }
        }
    }
    // the range's last kn % 4 values, one per thread
    const int kt = 4 * K4 + tid;
    if (kt < kn) {
        const float xs = ops.load1(xq + kt);
#pragma unroll
        for (int r = 0; r < R; ++r)
            acc[r] = fmaf(ops.load1(arow[r] + kt), xs, acc[r]);
    }

    float *red = ops.lds();
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const float s = ops.wave_sum(acc[r]);
        ops.lds_write1(red + wave * R + r, s, lane == 0);
    }
    ops.sync();
    // thread r < R sums row r's wave partials
    const bool own = tid < R && row0 + tid < p.M;
    const int r = own ? tid : 0;
    float s = ops.lds_read1(red + r, own);
#pragma unroll
    for (int w = 1; w < kWaves; ++w)
        s += ops.lds_read1(red + w * R + r, own);
    if (own)
        ops.store1(p.split == 1 ? p.y + row0 + tid : p.part + (int64_t)q * p.M + row0 + tid, s);
}

// y[i] = sum over q of part[q * M + i], q ascending (a fixed order).
__global__ void __launch_bounds__(256)
gemv_reduce(const float *part, int split, int M, float *y)
{
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < M; i += gridDim.x * blockDim.x) {
        float s = part[i];
        for (int q = 1; q < split; ++q)
            s += part[(int64_t)q * M + i];
        y[i] = s;
    }
}

template <int R, int U>
__global__ void __launch_bounds__(kThreads)
gemv_kernel(GemvParams p)
{
    __shared__ float red[kWaves * R];
    const int block = (int)(blockIdx.y * gridDim.x + blockIdx.x);
    if (block >= p.blocks)
        return;
    const DeviceOps ops{red};
    gemv_block<R, U>(ops, p, block, threadIdx.x);
}

}  // namespace xgemv_dev
