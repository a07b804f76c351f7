// MFMA-only microbenchmark for MI355X (gfx950): the issue rate of the GEMM's
// matrix instructions and the throughput the GPU sustains when nothing but
// MFMAs run, on random and on all-zero operands.  No memory traffic inside
// the timed loop, so the result bounds every GEMM kernel on the same data.
//
//   mfma_ceiling            prints one markdown table row per configuration
//
// Each wave keeps NACC independent accumulators and 8 + 8 distinct operand
// registers (loaded once from a buffer of 16-bit values: random, drawn like
// a workload's inputs, or all zero) and issues NACC MFMAs per loop
// iteration, so consecutive MFMAs never depend on each other and every
// instruction sees new operand bits.
// Configurations:
//   shape     16x16x32 or 32x32x16 bf16 -> fp32, 16x16x32 fp16 -> fp32
//   place     where the accumulators live: "vgpr" / "agpr" place them by an
//             inline-asm register constraint (operands in VGPRs); "builtin"
//             uses the compiler builtin with twice the accumulators, so that
//             more than 256 registers are live and the compiler puts the
//             accumulators in AGPRs itself (the situation of a 4-wave GEMM
//             tile whose waves each own a 128 x 128 block)
//   waves     waves per SIMD (1 or 2)
// A second table runs the 16 x 16 x 32 instruction of each GEMM workload's
// type on operands drawn like that workload's inputs (two waves per SIMD,
// accumulators in VGPRs, as in the 256 x 256 GEMM tile).
// The clock comes from s_memtime cycles over s_memrealtime (100 MHz) ticks
// around the loop of the first wave; TFLOP/s from HIP events over the last of
// 20 back-to-back launches of a few milliseconds each (the power limit
// settles within the first launches); cycles per MFMA per SIMD from the
// event time at that clock, divided by the MFMAs one SIMD issues.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <type_traits>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kBufQuads = 4096;  // operand source: 4096 x 16 bytes
constexpr int kCUs = 256;        // one workgroup per CU

enum { SHAPE16 = 0, SHAPE32 = 1, SHAPE16H = 2 };  // bf16, bf16, fp16
enum { PLACE_VGPR = 0, PLACE_AGPR = 1, PLACE_BUILTIN = 2 };

template <int SHAPE, int PLACE>
constexpr int nacc()
{
    // asm placements: 128 accumulator registers per wave (fits two waves
    // per SIMD); builtin: 256, so that they cannot share the 256 VGPRs with
    // the operands
    return SHAPE != SHAPE32 ? (PLACE == PLACE_BUILTIN ? 64 : 32) : (PLACE == PLACE_BUILTIN ? 16 : 8);
}

template <int SHAPE, int PLACE, int WPS>
__global__ void __launch_bounds__(256 * WPS, 1)
mfma_loop(const u32x4 *__restrict__ src, float *__restrict__ out, int iters, long long *__restrict__ clk)
{
    constexpr int N = nacc<SHAPE, PLACE>();
    typedef typename std::conditional<SHAPE != SHAPE32, f32x4, f32x16>::type acc_t;
    static_assert(SHAPE != SHAPE16H || PLACE == PLACE_VGPR, "fp16: VGPR placement only");
    const int tid = threadIdx.x;
    u32x4 a[8], b[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = src[(i * 512 + tid) % kBufQuads];
        b[i] = src[(i * 512 + 256 + tid) % kBufQuads];
    }
    acc_t acc[N];
#pragma unroll
    for (int n = 0; n < N; ++n)
        acc[n] = acc_t{};
    // the zeroing above is ordinary VALU code; give it time to retire
    // before the first MFMA reads the registers
    asm volatile("s_nop 7\n\ts_nop 7" ::: "memory");
    const long long t0 = __builtin_readcyclecounter();
    const long long w0 = __builtin_amdgcn_s_memrealtime();
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int n = 0; n < N; ++n) {
            const u32x4 x = b[n % 8], y = a[(n / 8) % 8];
            if constexpr (PLACE == PLACE_BUILTIN) {
                if constexpr (SHAPE == SHAPE16)
                    acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, x),
                                                                     __builtin_bit_cast(bf16x8, y), acc[n], 0, 0, 0);
                else
                    acc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, x),
                                                                     __builtin_bit_cast(bf16x8, y), acc[n], 0, 0, 0);
            } else if constexpr (SHAPE == SHAPE16H) {
                asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+v"(acc[n]) : "v"(x), "v"(y));
            } else if constexpr (SHAPE == SHAPE16) {
                if constexpr (PLACE == PLACE_VGPR)
                    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(acc[n]) : "v"(x), "v"(y));
                else
                    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc[n]) : "v"(x), "v"(y));
            } else {
                if constexpr (PLACE == PLACE_VGPR)
                    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc[n]) : "v"(x), "v"(y));
                else
                    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc[n]) : "v"(x), "v"(y));
            }
        }
    }
    // the last MFMAs must finish before ordinary code reads their results
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
    const long long t1 = __builtin_readcyclecounter();
    const long long w1 = __builtin_amdgcn_s_memrealtime();
    float s = 0.0f;
#pragma unroll
    for (int n = 0; n < N; ++n)
#pragma unroll
        for (int e = 0; e < (SHAPE != SHAPE32 ? 4 : 16); ++e)
            s += acc[n][e];
    out[blockIdx.x * blockDim.x + tid] = s;
    if (tid == 0 && blockIdx.x == 0) {
        clk[0] = t1 - t0;
        clk[1] = w1 - w0;
    }
}

uint16_t bf16_rne(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

bool check(hipError_t e, const char *what)
{
    if (e != hipSuccess) {
        fprintf(stderr, "mfma_ceiling: %s: %s\n", what, hipGetErrorString(e));
        return false;
    }
    return true;
}

enum { DATA_ZERO, DATA_UNIFORM_BF16, DATA_NORMAL1_BF16, DATA_UNIFORM_FP16, DATA_NORMAL002_FP16 };

// kBufQuads x 8 16-bit operands: zeros, or values drawn from splitmix64
// uniforms (normals by Box-Muller), rounded to nearest even in bf16 or fp16.
void fill(uint16_t *h, int data)
{
    uint64_t x = 0x9e3779b97f4a7c15ull;
    auto uni = [&x]() {
        x += 0x9e3779b97f4a7c15ull;
        uint64_t z = x;
        z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
        z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
        z ^= z >> 31;
        return (double)(z >> 11) * (1.0 / 9007199254740992.0);  // [0, 1)
    };
    for (int i = 0; i < kBufQuads * 8; ++i) {
        double v = 0.0;
        if (data == DATA_UNIFORM_BF16 || data == DATA_UNIFORM_FP16) {
            v = 2.0 * uni() - 1.0;
        } else if (data != DATA_ZERO) {
            const double u1 = 1.0 - uni(), u2 = uni();
            v = sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2) * (data == DATA_NORMAL1_BF16 ? 1.0 : 0.02);
        }
        if (data == DATA_UNIFORM_FP16 || data == DATA_NORMAL002_FP16) {
            const _Float16 f = (_Float16)(float)v;
            memcpy(&h[i], &f, 2);
        } else {
            h[i] = bf16_rne((float)v);
        }
    }
}

template <int SHAPE, int PLACE, int WPS>
bool run(const u32x4 *src, float *out, long long *clk, const char *data)
{
    constexpr int N = nacc<SHAPE, PLACE>();
    constexpr double kFlopsPerMfma = 16384.0 * (SHAPE != SHAPE32 ? 1 : 2);
    // about 4 ms per launch at 2 GHz
    const int iters = (int)(8.0e6 / (N * WPS * 16.0 * (SHAPE != SHAPE32 ? 1 : 2)));
    const dim3 grid(kCUs), block(256 * WPS);
    hipEvent_t e0, e1;
    if (!check(hipEventCreate(&e0), "event") || !check(hipEventCreate(&e1), "event"))
        return false;
    float ms = 0.0f;
    for (int r = 0; r < 20; ++r) {
        (void)hipEventRecord(e0);
        hipLaunchKernelGGL((mfma_loop<SHAPE, PLACE, WPS>), grid, block, 0, 0, src, out, iters, clk);
        (void)hipEventRecord(e1);
        if (!check(hipGetLastError(), "launch") || !check(hipEventSynchronize(e1), "sync"))
            return false;
        (void)hipEventElapsedTime(&ms, e0, e1);
    }
    long long h[2] = {0, 0};
    if (!check(hipMemcpy(h, clk, sizeof(h), hipMemcpyDeviceToHost), "copy"))
        return false;
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    const double mfmas = (double)kCUs * 4 * WPS * iters * N;  // per launch
    const double ghz = (double)h[0] / ((double)h[1] / 100e6) / 1e9;
    const double cyc = ms * 1e-3 * ghz * 1e9 / ((double)iters * N * WPS);  // per MFMA per SIMD
    printf("| %s | %s | %s | %d | %.2f | %.3f | %.1f |\n",
           SHAPE == SHAPE16 ? "16x16x32 bf16" : SHAPE == SHAPE32 ? "32x32x16 bf16" : "16x16x32 fp16",
           PLACE == PLACE_VGPR ? "vgpr (asm)" : PLACE == PLACE_AGPR ? "agpr (asm)" : "builtin, >256 live", data, WPS,
           cyc, ghz, mfmas * kFlopsPerMfma / (ms * 1e-3) / 1e12);
    fflush(stdout);
    return true;
}

}  // namespace

int main()
{
    hipDeviceProp_t prop;
    if (!check(hipGetDeviceProperties(&prop, 0), "device"))
        return 1;
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) {
        fprintf(stderr, "mfma_ceiling: needs gfx950, found %s\n", prop.gcnArchName);
        return 1;
    }
    u32x4 *src = nullptr;
    float *out = nullptr;
    long long *clk = nullptr;
    if (!check(hipMalloc(&src, kBufQuads * sizeof(u32x4)), "malloc") ||
        !check(hipMalloc(&out, (size_t)kCUs * 512 * sizeof(float)), "malloc") ||
        !check(hipMalloc(&clk, 2 * sizeof(long long)), "malloc"))
        return 1;
    uint16_t *h = (uint16_t *)malloc(kBufQuads * sizeof(u32x4));
    printf("| MFMA | accumulators | operands | waves per SIMD | cycles per MFMA per SIMD | clock (GHz) | TFLOP/s |\n");
    printf("|---|---|---|---|---|---|---|\n");
    for (int pass = 0; pass < 2; ++pass) {
        fill(h, pass == 0 ? DATA_UNIFORM_BF16 : DATA_ZERO);
        if (!check(hipMemcpy(src, h, kBufQuads * sizeof(u32x4), hipMemcpyHostToDevice), "copy"))
            return 1;
        const char *d = pass == 0 ? "uniform[-1,1]" : "zeros";
        bool ok = run<SHAPE16, PLACE_VGPR, 1>(src, out, clk, d) && run<SHAPE16, PLACE_AGPR, 1>(src, out, clk, d) &&
                  run<SHAPE16, PLACE_BUILTIN, 1>(src, out, clk, d) && run<SHAPE16, PLACE_VGPR, 2>(src, out, clk, d) &&
                  run<SHAPE16, PLACE_AGPR, 2>(src, out, clk, d) && run<SHAPE32, PLACE_VGPR, 1>(src, out, clk, d) &&
                  run<SHAPE32, PLACE_AGPR, 1>(src, out, clk, d) && run<SHAPE32, PLACE_BUILTIN, 1>(src, out, clk, d);
        if (!ok)
            return 1;
    }
    // the operand distributions of the GEMM workloads
    printf("\n| MFMA | accumulators | operands | waves per SIMD | cycles per MFMA per SIMD | clock (GHz) | TFLOP/s |\n");
    printf("|---|---|---|---|---|---|---|\n");
    const struct {
        int data;
        const char *name;
    } wl[] = {{DATA_UNIFORM_BF16, "uniform[-1,1] bf16"},
              {DATA_NORMAL1_BF16, "normal(0,1) bf16"},
              {DATA_UNIFORM_FP16, "uniform[-1,1] fp16"},
              {DATA_NORMAL002_FP16, "normal(0,0.02) fp16"}};
    for (const auto &w : wl) {
        fill(h, w.data);
        if (!check(hipMemcpy(src, h, kBufQuads * sizeof(u32x4), hipMemcpyHostToDevice), "copy"))
            return 1;
        const bool ok = (w.data == DATA_UNIFORM_FP16 || w.data == DATA_NORMAL002_FP16)
                            ? run<SHAPE16H, PLACE_VGPR, 2>(src, out, clk, w.name)
                            : run<SHAPE16, PLACE_VGPR, 2>(src, out, clk, w.name);
        if (!ok)
            return 1;
    }
    free(h);
    (void)hipFree(src);
    (void)hipFree(out);
    (void)hipFree(clk);
    return 0;
}
