// Copies of 16-bit GEMM operands into the library's workspace.
//
// The pipelined GEMM kernels load whole 16-byte chunks of A and B rows
// straight into LDS, so they need 16-byte aligned rows, K a multiple of 8
// and B rows readable to a multiple of 8 columns.  An operand that is not
// laid out that way is copied once per call into a dense, zero-padded
// buffer that is: rows x cols with cols the logical width rounded up to a
// multiple of 8.  The padding is zero, so padded K positions contribute
// exactly zero to every product; padded columns of B only feed outputs that
// are never stored.  The copy is bound by HBM bandwidth.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xgemm_dev {

typedef uint32_t pack_u32x4 __attribute__((ext_vector_type(4)));

// destination columns per workgroup iteration: 256 threads x 4 chunks of 8,
// which keeps 16 KiB per workgroup in flight before each barrier
constexpr int kPackSeg = 8192;

// dst[b * dst_stride + r * ldd + c] = src[b * src_stride + r * lds + c] for
// r < src_rows and c < src_cols, and 0 elsewhere in each of the `batch`
// rows x (8 * cols8) destinations.  dst and dst_stride keep every destination
// 16-byte aligned, ldd is a multiple of 8; src is 2-byte aligned with any
// leading dimension and batch stride.
//
// A workgroup copies one segment of kPackSeg destination columns of one row
// per iteration of a grid-stride loop.  Its source elements are staged in
// LDS through 16-byte aligned loads (the 16-byte chunks that lie wholly
// inside the segment's source span; the first and last chunk, which may
// reach outside it, are read element by element), so every global load
// stays inside the source row; then the threads write the destination row's
// 16-byte chunks from LDS, shifted by the source's misalignment.
__global__ void __launch_bounds__(256) pack16(const uint16_t *__restrict__ src, int64_t lds, int64_t src_stride,
                                              int src_rows, int src_cols, uint16_t *__restrict__ dst, int64_t ldd,
                                              int64_t dst_stride, int rows, int cols8, int batch)
{
    __shared__ __attribute__((aligned(16))) uint16_t span[kPackSeg + 16];
    const int tid = threadIdx.x;
    const int cols = cols8 * 8;
    const int segs = (cols + kPackSeg - 1) / kPackSeg;
    const int64_t per = (int64_t)rows * segs;
    const int64_t items = per * batch;
    for (int64_t w = blockIdx.x; w < items; w += gridDim.x) {
        const int64_t b = w / per;
        const int r = (int)((w - b * per) / segs);
        const int c_begin = (int)((w - b * per) % segs) * kPackSeg;
        const int c_end = min(c_begin + kPackSeg, cols);
        // valid source columns of this segment: [c_begin, v_end)
        const int v_end = r < src_rows ? min(c_end, src_cols) : c_begin;
        int shift = 0;  // elements of the first aligned chunk before c_begin
        if (v_end > c_begin) {
            const uint16_t *s0 = src + b * src_stride + (int64_t)r * lds + c_begin;
            const uintptr_t a0 = (uintptr_t)s0, a_end = (uintptr_t)(s0 + (v_end - c_begin));
            const uintptr_t a_lo = a0 & ~(uintptr_t)15;
            shift = (int)(a0 - a_lo) / 2;
            const int nchunks = (int)((a_end - a_lo + 15) / 16);
            for (int q = tid; q < nchunks; q += 256) {
                const uintptr_t a = a_lo + (uintptr_t)q * 16;
                if (a >= a0 && a + 16 <= a_end) {
                    *(pack_u32x4 *)(span + 8 * q) = *(const pack_u32x4 *)a;
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const uintptr_t ae = a + 2 * e;
                        span[8 * q + e] = (ae >= a0 && ae < a_end) ? *(const uint16_t *)ae : (uint16_t)0;
                    }
                }
            }
        }
        __syncthreads();
        for (int c = c_begin + 8 * tid; c < c_end; c += 8 * 256) {
            uint32_t v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int c2 = c + 2 * e;
                const uint32_t lo = c2 < v_end ? span[shift + c2 - c_begin] : 0u;
                const uint32_t hi = c2 + 1 < v_end ? span[shift + c2 + 1 - c_begin] : 0u;
                v[e] = lo | (hi << 16);
            }
            pack_u32x4 out = {v[0], v[1], v[2], v[3]};
            *(pack_u32x4 *)(dst + b * dst_stride + (int64_t)r * ldd + c) = out;
        }
        __syncthreads();
    }
}

}  // namespace xgemm_dev
