// Host side of libxgemm: argument checks, configuration selection, the
// split-k workspace and kernel launches.  The C ABI is declared in
// include/xgemm.h.
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <new>

#include "xgemm.h"
#include "gemm_kernel.hpp"

using xgemm_dev::GemmParams;

struct xgemm_ctx {
    int device;
    int cu_count;
    void *workspace;
    size_t ws_bytes;
    char last_error[256];
};

namespace {

struct TileShape {
    int bm, bn, bk, threads, wg_per_cu;
};

// Workgroups per CU follow from LDS use: two stages of (bm + bn) x bk
// 16-bit values out of 160 KiB.
constexpr TileShape kTiles[XGEMM_TILE_COUNT] = {
    {256, 256, 64, 256, 1},  // XGEMM_TILE_256x256: 4 waves of 128 x 128, 128 KiB LDS
    {256, 128, 64, 256, 1},  // XGEMM_TILE_256x128: 4 waves of 128 x 64,   96 KiB LDS
    {128, 128, 64, 256, 2},  // XGEMM_TILE_128x128: 4 waves of 64 x 64,    64 KiB LDS
};

constexpr int64_t kMaxDim = (int64_t)1 << 31;

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

void set_error(xgemm_ctx *h, const char *what, hipError_t e)
{
    if (h)
        snprintf(h->last_error, sizeof(h->last_error), "%s: %s", what, hipGetErrorString(e));
}

bool valid_config(const xgemm_config *c)
{
    return c && c->tile >= 0 && c->tile < XGEMM_TILE_COUNT && c->split_k >= 1 && c->split_k <= 64 &&
           c->group_m >= 1 && c->group_m <= 64 && c->reserved == 0;
}

// K elements each split covers: K / split rounded up to the K step, so that
// every split but the last starts on a K-step boundary.
int64_t split_chunk(int64_t K, int split, int bk)
{
    return cdiv(cdiv(K, split), bk) * bk;
}

// Modelled cost of a configuration in units of MFMA-peak cycles of one CU:
// the number of full waves of workgroups times the cycles one workgroup
// needs at the tile's sustained rate, plus the split-k traffic through HBM.
double model_cost(int64_t M, int64_t N, int64_t K, int cu_count, int tile, int split)
{
    const TileShape &t = kTiles[tile];
    static const double kTileEff[XGEMM_TILE_COUNT] = {1.0, 0.9, 0.75};
    const int64_t tiles = cdiv(M, t.bm) * cdiv(N, t.bn);
    const int64_t kc = split_chunk(K, split, t.bk);
    const int64_t slots = (int64_t)cu_count * t.wg_per_cu;
    const int64_t waves = cdiv(tiles * split, slots);
    // one CU retires 4096 flops per cycle at peak; a workgroup shares its CU
    const double wg_cycles = 2.0 * t.bm * t.bn * (double)kc * t.wg_per_cu / 4096.0 / kTileEff[tile];
    double cost = (double)waves * wg_cycles;
    if (split > 1) {
        // partials written once and read once, C written once; ~3.3 KB per
        // cycle of HBM bandwidth (8 TB/s at 2.4 GHz), plus a launch
        const double bytes = (2.0 * split + 1.0) * 4.0 * (double)M * (double)N;
        cost += bytes / 3333.0 + 4000.0;
    }
    return cost;
}

void select_config(int64_t M, int64_t N, int64_t K, int cu_count, xgemm_config *out)
{
    double best = 0.0;
    int best_tile = XGEMM_TILE_256x256, best_split = 1;
    for (int tile = 0; tile < XGEMM_TILE_COUNT; ++tile) {
        for (int split = 1; split <= 16; split *= 2) {
            if (split > 1 && split_chunk(K, split, kTiles[tile].bk) * (split - 1) >= K)
                break;  // the last split would be empty
            const double c = model_cost(M, N, K, cu_count, tile, split);
            if (best == 0.0 || c < best * 0.98) {
                best = c;
                best_tile = tile;
                best_split = split;
            }
        }
    }
    out->tile = best_tile;
    out->split_k = best_split;
    out->group_m = 4;
    out->reserved = 0;
}

size_t workspace_bytes(int64_t M, int64_t N, int split)
{
    if (split <= 1)
        return 0;
    const int64_t ldw = cdiv(N, 4) * 4;
    return (size_t)split * (size_t)M * (size_t)ldw * sizeof(float);
}

template <int BM, int BN, int BK, int WGM, int WGN>
hipError_t launch_gemm(int dtype, const GemmParams &p, int grid, hipStream_t s)
{
    if (dtype == XGEMM_BF16)
        hipLaunchKernelGGL((xgemm_dev::gemm_kernel<BM, BN, BK, WGM, WGN, 0>), dim3(grid),
                           dim3(WGM * WGN * 64), 0, s, p);
    else
        hipLaunchKernelGGL((xgemm_dev::gemm_kernel<BM, BN, BK, WGM, WGN, 1>), dim3(grid),
                           dim3(WGM * WGN * 64), 0, s, p);
    return hipGetLastError();
}

template <int BM, int BN, int BK, int STAGES, int WGM, int WGN>
hipError_t launch_dma(int dtype, const GemmParams &p, int grid, hipStream_t s)
{
    if (dtype == XGEMM_BF16)
        hipLaunchKernelGGL((xgemm_dev::gemm_kernel_dma<BM, BN, BK, STAGES, WGM, WGN, 0>), dim3(grid),
                           dim3(WGM * WGN * 64), 0, s, p);
    else
        hipLaunchKernelGGL((xgemm_dev::gemm_kernel_dma<BM, BN, BK, STAGES, WGM, WGN, 1>), dim3(grid),
                           dim3(WGM * WGN * 64), 0, s, p);
    return hipGetLastError();
}

// K step of the pipelined (direct-to-LDS) kernels; LDS stages per tile.
constexpr int kDmaBK = 64;
constexpr int kDmaStages256x256 = 2;  // 2 x 64 KiB
constexpr int kDmaStages256x128 = 3;  // 3 x 48 KiB
constexpr int kDmaStages128x128 = 2;  // 2 x 32 KiB, two workgroups per CU
constexpr int kDmaMinStages = 3;

// The pipelined kernels need 16-byte aligned A and B with lda, ldb multiples
// of 8, N a multiple of 8 (whole 16-byte chunks of B rows), K a multiple of
// their K step, at least as many K steps in every split as the deepest
// pipeline has stages, and per-tile byte offsets that fit in 32 bits.
bool dma_eligible(const GemmParams &p, int bm)
{
    const int64_t last = (int64_t)p.K - (int64_t)(p.split - 1) * p.k_chunk;
    const int64_t min_steps = (p.k_chunk < last ? p.k_chunk : last) / kDmaBK;
    return p.vec_ab && p.N % 8 == 0 && p.K % kDmaBK == 0 && min_steps >= kDmaMinStages &&
           (int64_t)bm * p.lda * 2 < ((int64_t)1 << 32) && (int64_t)kDmaBK * p.ldb * 2 < ((int64_t)1 << 32);
}

hipError_t launch_tile(int tile, bool dma, int dtype, const GemmParams &p, int grid, hipStream_t s)
{
    switch (tile) {
    case XGEMM_TILE_256x256:
        return dma ? launch_dma<256, 256, kDmaBK, kDmaStages256x256, 2, 2>(dtype, p, grid, s)
                   : launch_gemm<256, 256, 64, 2, 2>(dtype, p, grid, s);
    case XGEMM_TILE_256x128:
        return dma ? launch_dma<256, 128, kDmaBK, kDmaStages256x128, 2, 2>(dtype, p, grid, s)
                   : launch_gemm<256, 128, 64, 2, 2>(dtype, p, grid, s);
    case XGEMM_TILE_128x128:
        return dma ? launch_dma<128, 128, kDmaBK, kDmaStages128x128, 2, 2>(dtype, p, grid, s)
                   : launch_gemm<128, 128, 64, 2, 2>(dtype, p, grid, s);
    default: return hipErrorInvalidValue;
    }
}

int check_args(xgemm_ctx *h, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
               const void *B, int64_t ldb, const float *C, int64_t ldc, int dtype)
{
    if (!h)
        return XGEMM_ERR_INVALID_ARG;
    if (M < 0 || N < 0 || K < 0 || M >= kMaxDim || N >= kMaxDim || K >= kMaxDim)
        return XGEMM_ERR_INVALID_ARG;
    if (lda < K || ldb < N || ldc < N || lda < 0 || ldb < 0 || ldc < 0)
        return XGEMM_ERR_INVALID_ARG;
    if (dtype != XGEMM_BF16 && dtype != XGEMM_FP16)
        return XGEMM_ERR_INVALID_ARG;
    if ((M > 0 && K > 0 && !A) || (K > 0 && N > 0 && !B) || (M > 0 && N > 0 && !C))
        return XGEMM_ERR_INVALID_ARG;
    // every element offset must fit in 63 bits
    const double span_a = (double)M * (double)lda, span_b = (double)K * (double)ldb,
                 span_c = (double)M * (double)ldc;
    if (span_a > 9.0e18 || span_b > 9.0e18 || span_c > 9.0e18)
        return XGEMM_ERR_INVALID_ARG;
    return XGEMM_OK;
}

// Everything about a launch that follows from the arguments on the host.
struct Plan {
    GemmParams p;
    int tile;
    int split;
    int64_t grid;
    bool dma;       // pipelined direct-to-LDS kernel (else the general one)
    size_t ws;      // split-k workspace bytes
    int64_t ldw;    // workspace row stride (floats)
};

// Plan a launch for K > 0 and M, N > 0 with configuration cfg.  Device
// pointers are only inspected for their alignment.
int make_plan(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb,
              const float *C, int64_t ldc, const xgemm_config &cfg, Plan *out)
{
    const TileShape &t = kTiles[cfg.tile];
    // drop trailing splits that would have no K range
    int split = cfg.split_k;
    int64_t kc = split_chunk(K, split, t.bk);
    while (split > 1 && kc * (split - 1) >= K) {
        --split;
        kc = split_chunk(K, split, t.bk);
    }
    const int64_t tiles_m = cdiv(M, t.bm), tiles_n = cdiv(N, t.bn);
    const int64_t grid = tiles_m * tiles_n * split;
    if (grid > 0x7fffffff)
        return XGEMM_ERR_INVALID_ARG;

    GemmParams &p = out->p;
    p.A = (const uint16_t *)A;
    p.B = (const uint16_t *)B;
    p.lda = lda;
    p.ldb = ldb;
    p.M = (int)M;
    p.N = (int)N;
    p.K = (int)K;
    p.k_chunk = (int)kc;
    p.split = split;
    p.tiles_m = (int)tiles_m;
    p.tiles_n = (int)tiles_n;
    p.group_m = cfg.group_m;
    p.vec_ab = ((uintptr_t)A % 16 == 0) && ((uintptr_t)B % 16 == 0) && (lda % 8 == 0) && (ldb % 8 == 0);
    out->ldw = cdiv(N, 4) * 4;
    if (split == 1) {
        p.C = (float *)C;
        p.ldc = ldc;
        p.split_stride = 0;
        p.vec_c = ((uintptr_t)C % 16 == 0) && (ldc % 4 == 0);
    } else {
        p.C = nullptr;  // the workspace, filled in at launch
        p.ldc = out->ldw;
        p.split_stride = M * out->ldw;
        p.vec_c = 1;
    }
    out->tile = cfg.tile;
    out->split = split;
    out->grid = grid;
    out->dma = dma_eligible(p, t.bm);
    out->ws = workspace_bytes(M, N, split);
    return XGEMM_OK;
}

int run(xgemm_ctx *h, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B,
        int64_t ldb, float *C, int64_t ldc, int dtype, void *stream, const xgemm_config *forced)
{
    int rc = check_args(h, M, N, K, A, lda, B, ldb, C, ldc, dtype);
    if (rc != XGEMM_OK)
        return rc;
    if (forced && !valid_config(forced))
        return XGEMM_ERR_INVALID_ARG;
    h->last_error[0] = '\0';
    hipStream_t s = (hipStream_t)stream;
    if (M == 0 || N == 0)
        return XGEMM_OK;
    hipError_t e;
    if (K == 0) {
        const int64_t n = M * N;
        const int grid = (int)(cdiv(n, 256) < 4096 ? cdiv(n, 256) : 4096);
        hipLaunchKernelGGL(xgemm_dev::fill_zero, dim3(grid), dim3(256), 0, s, C, ldc, (int)M, (int)N);
        e = hipGetLastError();
        if (e != hipSuccess) {
            set_error(h, "fill_zero launch", e);
            return XGEMM_ERR_HIP;
        }
        return XGEMM_OK;
    }

    xgemm_config cfg;
    if (forced)
        cfg = *forced;
    else
        select_config(M, N, K, h->cu_count, &cfg);
    Plan plan;
    rc = make_plan(M, N, K, A, lda, B, ldb, C, ldc, cfg, &plan);
    if (rc != XGEMM_OK)
        return rc;

    if (plan.ws > h->ws_bytes) {
        // the old workspace may still be in use by work on this stream
        if (h->workspace) {
            e = hipStreamSynchronize(s);
            if (e != hipSuccess) {
                set_error(h, "hipStreamSynchronize", e);
                return XGEMM_ERR_HIP;
            }
            (void)hipFree(h->workspace);
            h->workspace = nullptr;
            h->ws_bytes = 0;
        }
        e = hipMalloc(&h->workspace, plan.ws);
        if (e != hipSuccess) {
            h->workspace = nullptr;
            (void)hipGetLastError();
            set_error(h, "hipMalloc workspace", e);
            return XGEMM_ERR_ALLOC;
        }
        h->ws_bytes = plan.ws;
    }
    if (plan.split > 1)
        plan.p.C = (float *)h->workspace;

    e = launch_tile(plan.tile, plan.dma, dtype, plan.p, (int)plan.grid, s);
    if (e != hipSuccess) {
        set_error(h, "gemm launch", e);
        return XGEMM_ERR_HIP;
    }
    if (plan.split > 1) {
        const int64_t nvec = M * cdiv(N, 4);
        const int grid = (int)(cdiv(nvec, 256) < 8192 ? cdiv(nvec, 256) : 8192);
        const int vec_c = ((uintptr_t)C % 16 == 0) && (ldc % 4 == 0);
        hipLaunchKernelGGL(xgemm_dev::splitk_reduce, dim3(grid), dim3(256), 0, s,
                           (const float *)h->workspace, (int64_t)(M * plan.ldw), plan.ldw, plan.split, C,
                           ldc, (int)M, (int)N, vec_c);
        e = hipGetLastError();
        if (e != hipSuccess) {
            set_error(h, "split-k reduce launch", e);
            return XGEMM_ERR_HIP;
        }
    }
    return XGEMM_OK;
}

}  // namespace

extern "C" {

int xgemm_create(xgemm_handle_t *out)
{
    if (!out)
        return XGEMM_ERR_INVALID_ARG;
    *out = nullptr;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return XGEMM_ERR_HIP;
    }
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
        (void)hipGetLastError();
        return XGEMM_ERR_HIP;
    }
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return XGEMM_ERR_UNSUPPORTED;
    xgemm_ctx *h = new (std::nothrow) xgemm_ctx;
    if (!h)
        return XGEMM_ERR_ALLOC;
    h->device = dev;
    h->cu_count = prop.multiProcessorCount;
    h->workspace = nullptr;
    h->ws_bytes = 0;
    h->last_error[0] = '\0';
    *out = h;
    return XGEMM_OK;
}

int xgemm_destroy(xgemm_handle_t h)
{
    if (!h)
        return XGEMM_OK;
    int rc = XGEMM_OK;
    if (h->workspace && hipFree(h->workspace) != hipSuccess) {
        (void)hipGetLastError();
        rc = XGEMM_ERR_HIP;
    }
    delete h;
    return rc;
}

int xgemm_run(xgemm_handle_t h, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
              const void *B, int64_t ldb, float *C, int64_t ldc, int dtype, void *stream)
{
    return run(h, M, N, K, A, lda, B, ldb, C, ldc, dtype, stream, nullptr);
}

int xgemm_run_config(xgemm_handle_t h, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                     const void *B, int64_t ldb, float *C, int64_t ldc, int dtype, void *stream,
                     const xgemm_config *cfg)
{
    if (!cfg)
        return XGEMM_ERR_INVALID_ARG;
    return run(h, M, N, K, A, lda, B, ldb, C, ldc, dtype, stream, cfg);
}

int xgemm_select_config(int64_t M, int64_t N, int64_t K, int dtype, int cu_count, xgemm_config *out)
{
    if (!out || M < 0 || N < 0 || K < 0 || cu_count < 1 || (dtype != XGEMM_BF16 && dtype != XGEMM_FP16))
        return XGEMM_ERR_INVALID_ARG;
    select_config(M, N, K, cu_count, out);
    return XGEMM_OK;
}

int xgemm_tile_info(int tile, int *bm, int *bn, int *bk, int *threads)
{
    if (tile < 0 || tile >= XGEMM_TILE_COUNT || !bm || !bn || !bk || !threads)
        return XGEMM_ERR_INVALID_ARG;
    *bm = kTiles[tile].bm;
    *bn = kTiles[tile].bn;
    *bk = kTiles[tile].bk;
    *threads = kTiles[tile].threads;
    return XGEMM_OK;
}

int xgemm_kernel_family(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B,
                        int64_t ldb, const xgemm_config *cfg)
{
    if (!valid_config(cfg) || M <= 0 || N <= 0 || K <= 0 || M >= kMaxDim || N >= kMaxDim || K >= kMaxDim ||
        lda < K || ldb < N)
        return -1;
    Plan plan;
    // C's alignment does not affect the choice
    if (make_plan(M, N, K, A, lda, B, ldb, nullptr, N, *cfg, &plan) != XGEMM_OK)
        return -1;
    return plan.dma ? XGEMM_KERNEL_PIPELINED : XGEMM_KERNEL_GENERAL;
}

size_t xgemm_workspace_bytes(int64_t M, int64_t N, const xgemm_config *cfg)
{
    if (!valid_config(cfg) || M < 0 || N < 0)
        return 0;
    return workspace_bytes(M, N, cfg->split_k);
}

const char *xgemm_strerror(int status)
{
    switch (status) {
    case XGEMM_OK: return "success";
    case XGEMM_ERR_INVALID_ARG: return "invalid argument";
    case XGEMM_ERR_UNSUPPORTED: return "unsupported device (gfx950 required)";
    case XGEMM_ERR_ALLOC: return "workspace allocation failed";
    case XGEMM_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
    }
}

const char *xgemm_last_error(xgemm_handle_t h)
{
    if (!h)
        return "no handle";
    return h->last_error;
}

}  // extern "C"
