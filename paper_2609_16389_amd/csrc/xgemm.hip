// Host side of libxgemm: argument checks, configuration selection, the
// split-k workspace and kernel launches.  The C ABI is declared in
// include/xgemm.h.
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <type_traits>
#include <vector>

#include "xgemm.h"
#include "gemm_kernel.hpp"
#include "gemv_kernel.hpp"
#include "pack_kernel.hpp"
#include "sk_kernel.hpp"

using xgemm_dev::GemmParams;

// Scratch of xgemm_run_noalloc: split-k partials and operand copies of the
// calls that may not allocate.  One array per GPU, held by the code object
// until the process ends; every such call on a GPU uses the same one.  Host
// code never passes this name to a kernel or a copy: the device address of
// each GPU's array comes from hipGetSymbolAddress (see xgemm_create).
constexpr size_t kScratchBytes = XGEMM_NOALLOC_SCRATCH_BYTES;
static __device__ __attribute__((aligned(256))) char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each device (null until looked up)
}  // namespace

struct xgemm_ctx {
    int device;
    int cu_count;
    void *workspace;
    size_t ws_bytes;
    // Calls that share the workspace never overlap, whichever streams they
    // are enqueued on.  While a handle's calls all come on one stream, the
    // stream's order is enough and nothing is recorded (an event record
    // between two GEMMs leaves the GPU idle for about 10 us).  The first
    // call on another stream waits for the device to drain (the previous
    // stream may no longer exist), and from then on every call records
    // ws_event on its stream after its last launch, and a call on another
    // stream makes its stream wait for that event.  The workspace is only
    // freed (to grow it) once its last user has completed.
    hipEvent_t ws_event;
    hipStream_t ws_stream;  // stream of the last call that used the workspace
    bool ws_used;           // ws_stream is set
    bool ws_recorded;       // ws_event follows the last use on ws_stream
    bool ws_multi;          // calls have come on more than one stream
    size_t ws_limit;        // largest workspace the handle may allocate (0: no limit)
    bool persistent;        // the selected plans may use the persistent kernel
    void *scratch;          // this device's `scratch` array (xgemm_run_noalloc)
    char last_error[256];
};

namespace {

struct TileShape {
    int bm, bn, bk, wg_per_cu;
};

// Workgroups per CU follow from LDS use: two stages of (bm + bn) x bk
// 16-bit values out of 160 KiB.  (Waves per workgroup are in the kernel
// tables below: DmaTile, GeneralTile.)
constexpr TileShape kTiles[XGEMM_TILE_COUNT] = {
    {256, 256, 64, 1},  // XGEMM_TILE_256x256: 128 KiB LDS
    {256, 128, 64, 1},  // XGEMM_TILE_256x128:  96 KiB LDS
    {128, 128, 64, 2},  // XGEMM_TILE_128x128:  64 KiB LDS
};

constexpr int64_t kMaxDim = (int64_t)1 << 31;

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

void set_error(xgemm_ctx *h, const char *what, hipError_t e)
{
    if (h)
        snprintf(h->last_error, sizeof(h->last_error), "%s: %s", what, hipGetErrorString(e));
}

// Counter words of the persistent kernel's split tiles: the first bytes of
// every workspace, zero when the workspace is allocated and zero again after
// every call that uses them; the other workspace users start after them.
constexpr size_t kWsPrefix = 4096;
constexpr int kMaxSkGrid = (int)(kWsPrefix / sizeof(int));

bool valid_config(const xgemm_config *c)
{
    return c && c->tile >= 0 && c->tile < XGEMM_TILE_COUNT && c->split_k >= 1 && c->split_k <= 64 &&
           c->group_m >= 1 && c->group_m <= 64 && c->stream_k >= 0 && c->stream_k < kMaxSkGrid &&
           (c->stream_k == 0 || c->split_k == 1);
}

// K elements each split covers: K / split rounded up to the K step, so that
// every split but the last starts on a K-step boundary.
int64_t split_chunk(int64_t K, int split, int bk)
{
    return cdiv(cdiv(K, split), bk) * bk;
}

// Modelled time of a configuration in microseconds on MI355X: the rounds
// of workgroups (waves), each a fixed cost (prologue, epilogue stores) plus
// its K steps at the tile's measured rate, plus, for split-k, the reduction
// kernel and the partials' traffic (written once, read once, with C written
// once).  A 128 x 128 workgroup shares its CU with a second one in a round
// that fills every CU twice, which makes each step slower; a last round
// with at most one workgroup per CU runs at the unshared rate (this per-
// round charge picks a configuration within 3.4% of the fastest measured,
// geometric mean over 60 shapes, against 5.7% when every round of a launch
// was charged as shared).  The constants
// were fitted (least squares on log time) to 180 measured (tile, split)
// timings over 21 shapes from 256^3 to 8192^3 and 1024 x 1024 x 65536; the
// fit picks a configuration within 7% of the fastest measured one on every
// shape, and the fastest on the five benchmark workloads.  Re-checked after
// the 256 x 128 tile moved to eight waves: the fastest on 20 of 25 shapes,
// within 4.6% on the others (refitting that tile alone made the large
// shapes pick it, 10-20% slower).
struct TileCost {
    double fixed_us, step_us, step_shared_us;
};
constexpr TileCost kTileCost[XGEMM_TILE_COUNT] = {
    {9.78, 1.487, 1.487},  // 256 x 256: 8 waves, one workgroup per CU
    {6.29, 0.852, 0.852},  // 256 x 128: 8 waves (pairs split K), one workgroup per CU
    {3.22, 0.585, 1.050},  // 128 x 128: 4 waves, one or two workgroups per CU
};

double model_cost(int64_t M, int64_t N, int64_t K, int cu_count, int tile, int split)
{
    const TileShape &t = kTiles[tile];
    const TileCost &c = kTileCost[tile];
    const int64_t tiles = cdiv(M, t.bm) * cdiv(N, t.bn);
    const int64_t kc = split_chunk(K, split, t.bk);
    const int64_t slots = (int64_t)cu_count * t.wg_per_cu;
    const int64_t n = tiles * split;
    const double steps = (double)cdiv(std::min(kc, K), t.bk);
    // whole rounds fill every slot (two workgroups per CU share it where the
    // tile allows); a last partial round shares CUs only past one workgroup
    // per CU, its step rate taken between the two in proportion to the CUs
    // that hold two
    const int64_t full = n / slots, last = n % slots;
    double cost = (double)full * (c.fixed_us + steps * (t.wg_per_cu > 1 ? c.step_shared_us : c.step_us));
    if (last > 0) {
        const double twice = last > cu_count ? (double)(last - cu_count) / cu_count : 0.0;
        cost += c.fixed_us + steps * (c.step_us + (c.step_shared_us - c.step_us) * twice);
    }
    if (split > 1)
        cost += 3.70 + 0.411 * split + (2.0 * split + 1.0) * 4.0 * (double)M * (double)N / 8.494e6;
    return cost;
}

// Tile rows per group in the launch order.  Each XCD runs a contiguous
// share of the logical tile ids; when eight whole tile rows fit in one
// share, groups of eight keep an XCD's concurrent tiles square-ish across
// the whole share, otherwise groups of four.
int choose_group_m(int64_t tiles_m, int64_t tiles_n, int split)
{
    const int64_t share = tiles_m * tiles_n * split / xgemm_dev::kNumXcd;
    return (tiles_n * 8 <= share && tiles_m >= 8) ? 8 : 4;
}

void select_config_batched(int64_t batch, int64_t M, int64_t N, int64_t K, int cu_count, xgemm_config *out);

void select_config(int64_t M, int64_t N, int64_t K, int cu_count, xgemm_config *out)
{
    select_config_batched(1, M, N, K, cu_count, out);
}

// The configuration for `batch` independent problems of one shape: the
// batch multiplies the workgroups of a wave, and batched launches do not
// split K.
void select_config_batched(int64_t batch, int64_t M, int64_t N, int64_t K, int cu_count, xgemm_config *out)
{
    double best = 0.0;
    int best_tile = XGEMM_TILE_256x256, best_split = 1;
    for (int tile = 0; tile < XGEMM_TILE_COUNT; ++tile) {
        for (int split = 1; split <= (batch > 1 ? 1 : 16); split *= 2) {
            if (split > 1 && split_chunk(K, split, kTiles[tile].bk) * (split - 1) >= K)
                break;  // the last split would be empty
            const double c = model_cost(M * batch, N, K, cu_count, tile, split);
            // a faster configuration wins; within 0.5%, the one with fewer
            // K splits (less workspace, fewer partials).  (A 2% window cost
            // 14% at 2048 x 2048 x 16384, where 256 x 256 split 4 beats the
            // 256 x 128 split 2 it kept, and 0.6% over the validation set.)
            if (best == 0.0 || c < best * 0.995 || (c < best * 1.005 && split < best_split)) {
                best = c;
                best_tile = tile;
                best_split = split;
            }
        }
    }
    const TileShape &t = kTiles[best_tile];
    out->tile = best_tile;
    out->split_k = best_split;
    out->group_m = choose_group_m(cdiv(M, t.bm), cdiv(N, t.bn), best_split * (int)(batch < 64 ? batch : 64));
    out->stream_k = 0;
}

// Body + band plans.  When the output tiles of the chosen configuration end
// in a partial round of workgroups, C may instead be cut into a body of
// whole rounds of one tile shape and a band (the columns on the right, or
// the rows at the bottom) that the band's own configuration covers in fewer
// rounds; the two are launched one after the other, each an ordinary call on
// a sub-matrix.  Measured: 4096 x 14336 x 4096 (3.5 rounds of 256 x 256
// tiles) 379 against 396 us with a 2048-column band of 256 x 128 tiles;
// 6144^3 365 against 438 us; 3-28% on 23 shapes of 2 to 5 rounds.  The
// time model charges each plan its rounds, plus the second launch; a banded
// plan must come out kBandMargin cheaper, since the model does not see that
// a partial round runs at a higher clock.  Of 16 shapes the model put 0-8%
// ahead when cut, the 14 a 4% margin cuts gained 1-13%; cutting the other
// two gained nothing and lost 4%.
constexpr double kBandMargin = 0.04;
constexpr double kBandLaunchUs = 3.0;

struct BandPlan {
    int axis = XGEMM_BAND_NONE;
    int64_t extent = 0;  // columns (XGEMM_BAND_COLUMNS) or rows (XGEMM_BAND_ROWS) of C in the body
    xgemm_config body{}, band{};
};

// The persistent kernel (one workgroup per CU walking its tiles, each
// tile's C stores draining under the next tile's MFMAs) in place of one
// workgroup per 256 x 256 tile, where it measured faster: four or more whole
// rounds (8192^3 742 against 762 us, 8192 x 14336 x 4096 679 against 701,
// 12288 x 12288 x 4096 fp16 917 against 988; 8192 x 8192 x 2048 even), or
// three or more and a half (4096 x 14336 x 4096 fp16 390 against 398 with
// the band plan).  With two or three whole rounds it measured 3-6% slower.
// Other partial rounds stay with the band plans: there the shared ranges
// start at many different K offsets, so the tiles an XCD runs at one time
// share no operand rows in its L2 (6144^3: 404 against 357 us).
bool use_persistent(int64_t M, int64_t N, int64_t K, int cu_count, const xgemm_config &whole, int64_t batch = 1)
{
    const TileShape &t = kTiles[XGEMM_TILE_256x256];
    if (whole.tile != XGEMM_TILE_256x256 || whole.split_k != 1 || M % t.bm || N % t.bn || K % t.bk ||
        cu_count < 1 || cu_count >= kMaxSkGrid)
        return false;
    const int64_t tiles = (M / t.bm) * (N / t.bn) * batch, rounds = tiles / cu_count, rem = tiles % cu_count;
    return rem == 0 ? rounds >= 4 : (2 * rem == cu_count && rounds >= 3);
}

BandPlan select_band(int64_t M, int64_t N, int64_t K, int cu_count, bool persistent = true)
{
    BandPlan out;
    xgemm_config whole;
    select_config(M, N, K, cu_count, &whole);
    out.body = whole;
    if (whole.split_k > 1)
        return out;  // a K split already spreads the problem over the GPU
    if (persistent && use_persistent(M, N, K, cu_count, whole)) {
        out.body.stream_k = 1;
        return out;
    }
    {
        // one round or less: the call already takes one tile time, and a
        // partial round runs at a higher clock than the model charges
        // (measured: 2048 x 5120 x 4096, 160 tiles, 83 us in one launch
        // against 92 us as a body and a band)
        const TileShape &t = kTiles[whole.tile];
        if (cdiv(M, t.bm) * cdiv(N, t.bn) <= (int64_t)cu_count * t.wg_per_cu)
            return out;
    }
    const double unbanded = model_cost(M, N, K, cu_count, whole.tile, 1);
    double best = unbanded * (1.0 - kBandMargin);
    for (int axis = XGEMM_BAND_COLUMNS; axis <= XGEMM_BAND_ROWS; ++axis) {
        const int64_t along = axis == XGEMM_BAND_COLUMNS ? N : M;   // the dimension the band cuts
        const int64_t across = axis == XGEMM_BAND_COLUMNS ? M : N;
        for (int tb = 0; tb < XGEMM_TILE_COUNT; ++tb) {
            const TileShape &t = kTiles[tb];
            const int64_t step = axis == XGEMM_BAND_COLUMNS ? t.bn : t.bm;
            const int64_t tiles_across = cdiv(across, axis == XGEMM_BAND_COLUMNS ? t.bm : t.bn);
            const int64_t slots = (int64_t)cu_count * t.wg_per_cu;
            // bodies of the most whole rounds that fit (R) or one fewer: as
            // many whole tile columns or rows as r rounds hold.  (An
            // exhaustive search over r picked R on all 177 banded shapes of
            // a 1024..16384 grid.)
            const int64_t R = (along / step) * tiles_across / slots;
            for (int64_t r = R > 1 ? R - 1 : 1; r <= R; ++r) {
                const int64_t j = r * slots / tiles_across;
                const int64_t ext = j * step;
                if (j < 1 || ext >= along)
                    continue;
                const int64_t bm = axis == XGEMM_BAND_COLUMNS ? M : ext, bn = axis == XGEMM_BAND_COLUMNS ? ext : N;
                const int64_t rm = axis == XGEMM_BAND_COLUMNS ? M : M - ext, rn = axis == XGEMM_BAND_COLUMNS ? N - ext : N;
                xgemm_config bandcfg;
                select_config(rm, rn, K, cu_count, &bandcfg);
                const double c = model_cost(bm, bn, K, cu_count, tb, 1) +
                                 model_cost(rm, rn, K, cu_count, bandcfg.tile, bandcfg.split_k) + kBandLaunchUs;
                if (c < best) {
                    best = c;
                    out.axis = axis;
                    out.extent = ext;
                    out.body.tile = tb;
                    out.body.split_k = 1;
                    out.body.group_m = choose_group_m(cdiv(bm, t.bm), cdiv(bn, t.bn), 1);
                    out.body.stream_k = 0;
                    out.band = bandcfg;
                }
            }
        }
    }
    return out;
}

size_t workspace_bytes(int64_t M, int64_t N, int split)
{
    if (split <= 1)
        return 0;
    const int64_t ldw = cdiv(N, 4) * 4;
    return (size_t)split * (size_t)M * (size_t)ldw * sizeof(float);
}

// Grid of `blocks` workgroups (blocks < 2^31): one dimension while the
// launch has fewer than 2^32 threads at 1024 threads per workgroup, else
// rows of 65536 workgroups (the kernels take the linear id and let the
// workgroups past `blocks` exit).
dim3 grid_of(int64_t blocks)
{
    constexpr int64_t kRow = 65536;
    if (blocks < ((int64_t)1 << 22))
        return dim3((unsigned)blocks);
    return dim3((unsigned)kRow, (unsigned)cdiv(blocks, kRow));
}

template <int BM, int BN, int BK, int WGM, int WGN>
hipError_t launch_gemm(int dtype, GemmParams p, int grid, hipStream_t s)
{
    p.grid = grid;
    if (dtype == XGEMM_BF16)
        hipLaunchKernelGGL((xgemm_dev::gemm_kernel<BM, BN, BK, WGM, WGN, 0>), grid_of(grid),
                           dim3(WGM * WGN * 64), 0, s, p);
    else
        hipLaunchKernelGGL((xgemm_dev::gemm_kernel<BM, BN, BK, WGM, WGN, 1>), grid_of(grid),
                           dim3(WGM * WGN * 64), 0, s, p);
    return hipGetLastError();
}

template <int BM, int BN, int BK, int STAGES, int WGM, int WGN, int MI, int KW>
hipError_t launch_dma(int dtype, GemmParams p, int grid, hipStream_t s)
{
    p.grid = grid;
    if (dtype == XGEMM_BF16)
        hipLaunchKernelGGL((xgemm_dev::gemm_kernel_dma<BM, BN, BK, STAGES, WGM, WGN, 0, MI, KW>), grid_of(grid),
                           dim3(WGM * WGN * KW * 64), 0, s, p);
    else
        hipLaunchKernelGGL((xgemm_dev::gemm_kernel_dma<BM, BN, BK, STAGES, WGM, WGN, 1, MI, KW>), grid_of(grid),
                           dim3(WGM * WGN * KW * 64), 0, s, p);
    return hipGetLastError();
}

// K step of the pipelined (direct-to-LDS) kernels; LDS stages per tile.
constexpr int kDmaBK = 64;
constexpr int kDmaStages256x256 = 2;  // 2 x 64 KiB
constexpr int kDmaStages256x128 = 3;  // 3 x 48 KiB
constexpr int kDmaStages128x128 = 2;  // 2 x 32 KiB, two workgroups per CU
constexpr int kDmaMinStages = 3;
// MFMA block of the pipelined kernels (32: 32x32x16, 16: 16x16x32)
#ifndef XGEMM_MI_256x256
#define XGEMM_MI_256x256 16
#endif
#ifndef XGEMM_MI_256x128
#define XGEMM_MI_256x128 16
#endif
#ifndef XGEMM_MI_128x128
#define XGEMM_MI_128x128 16
#endif
// Waves along M and N of the 256 x 256 pipelined tile: 8 waves (two per
// SIMD) of 128 x 64, measured 1-4.5% faster on the large shapes than 4
// waves of 128 x 128 (2 x 2).
#ifndef XGEMM_WGM_256x256
#define XGEMM_WGM_256x256 2
#define XGEMM_WGN_256x256 4
#endif
// Waves along K of the 256 x 128 pipelined tile: 2 (eight waves, two per
// SIMD, each pair splitting the K steps of one 128 x 64 block) or 1 (four
// waves, one per SIMD).
#ifndef XGEMM_KW_256x128
#define XGEMM_KW_256x128 2
#endif

// The pipelined kernels need 16-byte aligned A and B with lda, ldb multiples
// of 8, N and K multiples of 8 (whole 16-byte chunks of B rows and of A rows
// within K; a last partial K step is zero-filled; N may be ragged when B's
// rows are padded to a multiple of 8 columns, as packed copies are), at
// least as many K steps (counting a partial one) in every split as the
// deepest pipeline has stages, and per-tile byte offsets that fit in 32 bits.
bool dma_eligible(const GemmParams &p, int bm, bool b_padded = false)
{
    const int64_t last = (int64_t)p.K - (int64_t)(p.split - 1) * p.k_chunk;
    const int64_t min_steps = cdiv(p.k_chunk < last ? p.k_chunk : last, kDmaBK);
    return p.vec_ab && (p.N % 8 == 0 || b_padded) && p.K % 8 == 0 && min_steps >= kDmaMinStages &&
           (int64_t)bm * p.lda * 2 < ((int64_t)1 << 32) && (int64_t)kDmaBK * p.ldb * 2 < ((int64_t)1 << 32);
}

// Template arguments of the pipelined kernel per tile (tile rows and
// columns, K step, LDS stages, waves along M and N, MFMA block).  Launches
// and host traces both take them from here, so a trace follows the kernel
// that runs.
template <int BM_, int BN_, int STAGES_, int MI_, int WGM_ = 2, int WGN_ = 2, int KW_ = 1>
struct DmaTile {
    static constexpr int BM = BM_, BN = BN_, BK = kDmaBK, STAGES = STAGES_, WGM = WGM_, WGN = WGN_, MI = MI_,
                         KW = KW_;
};

template <class F>
auto with_dma_tile(int tile, F &&f)
{
    switch (tile) {
    case XGEMM_TILE_256x256: return f(DmaTile<256, 256, kDmaStages256x256, XGEMM_MI_256x256, XGEMM_WGM_256x256, XGEMM_WGN_256x256>{});
    case XGEMM_TILE_256x128: return f(DmaTile<256, 128, kDmaStages256x128, XGEMM_MI_256x128, 2, 2, XGEMM_KW_256x128>{});
    default: return f(DmaTile<128, 128, kDmaStages128x128, XGEMM_MI_128x128>{});
    }
}

// Template arguments of the general kernel per tile, shared by launches and
// traces like DmaTile.
template <int BM_, int BN_>
struct GeneralTile {
    static constexpr int BM = BM_, BN = BN_, BK = 64, WGM = 2, WGN = 2;
};

template <class F>
auto with_general_tile(int tile, F &&f)
{
    switch (tile) {
    case XGEMM_TILE_256x256: return f(GeneralTile<256, 256>{});
    case XGEMM_TILE_256x128: return f(GeneralTile<256, 128>{});
    default: return f(GeneralTile<128, 128>{});
    }
}

// Threads per workgroup of a tile's pipelined (dma) or general kernel.
int tile_threads(int tile, bool dma)
{
    if (dma)
        return with_dma_tile(tile, [](auto t) { return decltype(t)::WGM * decltype(t)::WGN * decltype(t)::KW * 64; });
    return with_general_tile(tile, [](auto t) { return decltype(t)::WGM * decltype(t)::WGN * 64; });
}

hipError_t launch_tile(int tile, bool dma, int dtype, const GemmParams &p, int grid, hipStream_t s)
{
    if (tile < 0 || tile >= XGEMM_TILE_COUNT)
        return hipErrorInvalidValue;
    if (dma)
        return with_dma_tile(tile, [&](auto t) {
            using T = decltype(t);
            return launch_dma<T::BM, T::BN, T::BK, T::STAGES, T::WGM, T::WGN, T::MI, T::KW>(dtype, p, grid, s);
        });
    return with_general_tile(tile, [&](auto t) {
        using T = decltype(t);
        return launch_gemm<T::BM, T::BN, T::BK, T::WGM, T::WGN>(dtype, p, grid, s);
    });
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

// One kernel launch of a plan: a range of logical tiles, its split-k
// factor and where its output goes.
struct Segment {
    GemmParams p;
    int64_t grid;
    bool dma;    // pipelined direct-to-LDS kernel (else the general one)
    bool sk;     // the persistent stream-K kernel (the 256 x 256 tile; dma is set too)
    int reduce;  // 0: writes C; 1: full-matrix partials + splitk_reduce
    int dp_rounds, sk_tiles, kt;  // persistent kernel: rounds of whole tiles, shared tiles, K steps per tile
};

// Operands copied into the workspace (pack16) so that the pipelined kernels
// can run: A as M x k8 (leading dimension k8), B as k8 x n8 (leading
// dimension n8), with k8 and n8 the K and N rounded up to multiples of 8 and
// zero padding.  Offsets are bytes from the workspace base.
struct Pack {
    bool a = false, b = false;
    int64_t k8 = 0, n8 = 0;
    size_t a_off = 0, b_off = 0;
};

// Everything about a call that follows from the arguments on the host.
struct Plan {
    int tile;
    Segment seg[2];
    int nseg;
    size_t ws;      // workspace bytes (split partials, then packed operands)
    int64_t ldw;    // full-matrix workspace row stride (floats)
    Pack pack;
};

// K range per split with trailing empty splits dropped; returns the split.
int trim_split(int64_t K, int split, int bk, int64_t *kc)
{
    *kc = split_chunk(K, split, bk);
    while (split > 1 && *kc * (split - 1) >= K) {
        --split;
        *kc = split_chunk(K, split, bk);
    }
    return split;
}

// The persistent kernel's schedule of `tiles` tiles of kt K steps over
// `grid` workgroups (one per CU): whole rounds, then the K steps of the last
// partial round and one more round shared out as equal ranges (each at least
// a tile's steps, so a tile is split between at most two ranges).  Returns
// false, leaving g unchanged, where the schedule does not apply; the
// workspace it needs (two partial sums per slot, none without shared tiles)
// is sk_workspace(g).
bool sk_schedule(Segment &g, int64_t tiles, int64_t kt, int grid)
{
    if (kt < 1 || grid < 1 || grid >= kMaxSkGrid || tiles < grid || tiles * kt >= 0x7fffffff)
        return false;
    const int64_t rounds = tiles / grid, rem = tiles % grid;
    g.sk = true;
    g.grid = grid;
    g.kt = (int)kt;
    g.dp_rounds = (int)(rem == 0 ? rounds : rounds - 1);
    g.sk_tiles = (int)(rem == 0 ? 0 : rem + grid);
    return true;
}

size_t sk_workspace(const Segment &g)
{
    return g.sk && g.sk_tiles > 0 ? (size_t)2 * g.grid * kTiles[XGEMM_TILE_256x256].bm *
                                        kTiles[XGEMM_TILE_256x256].bn * sizeof(float)
                                  : 0;
}

// Plan a call for K > 0 and M, N > 0 with configuration cfg on a device
// with cu_count CUs.  Device pointers are only inspected for alignment.
int make_plan_with(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb,
                   const float *C, int64_t ldc, const xgemm_config &cfg, int cu_count, Pack pk, Plan *out);

// With allow_pack, operands the pipelined kernels cannot read in place are
// copied into the workspace when the copies make the pipelined kernel
// eligible (the packed operands' addresses in the plan are then byte offsets
// from the workspace base, rebased at launch).  Measured from 127 x 129 x 131
// (14 against 24 us) to 8191^3 (990 against 7454 us), copying and running the
// pipelined kernel beats the general kernel reading the operands in place.
int make_plan(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb,
              const float *C, int64_t ldc, const xgemm_config &cfg, int cu_count, Plan *out, bool allow_pack)
{
    const int rc = make_plan_with(M, N, K, A, lda, B, ldb, C, ldc, cfg, cu_count, Pack{}, out);
    if (rc != XGEMM_OK || !allow_pack || out->seg[0].dma)
        return rc;
    Pack pk;
    pk.k8 = cdiv(K, 8) * 8;
    pk.n8 = cdiv(N, 8) * 8;
    const bool k_ok = K % 8 == 0;
    pk.a = !(k_ok && (uintptr_t)A % 16 == 0 && lda % 8 == 0);
    pk.b = !(k_ok && (uintptr_t)B % 16 == 0 && ldb % 8 == 0 && N % 8 == 0);
    if (!pk.a && !pk.b)
        return rc;  // aligned operands: the general kernel runs for another reason
    Plan packed;
    const int rc2 = make_plan_with(M, N, K, A, lda, B, ldb, C, ldc, cfg, cu_count, pk, &packed);
    if (rc2 == XGEMM_OK && packed.seg[0].dma)
        *out = packed;
    return XGEMM_OK;
}

int make_plan_with(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb,
                   const float *C, int64_t ldc, const xgemm_config &cfg, int cu_count, Pack pk, Plan *out)
{
    const TileShape &t = kTiles[cfg.tile];
    const int64_t tiles_m = cdiv(M, t.bm), tiles_n = cdiv(N, t.bn);
    const int64_t tiles = tiles_m * tiles_n;
    if (pk.a || pk.b)
        K = pk.k8;  // zero-padded K (both operands are packed when K % 8 != 0)
    int64_t kc;
    const int split = trim_split(K, cfg.split_k, t.bk, &kc);
    if (tiles * split > 0x7fffffff || tiles * 8 > 0x7fffffff)
        return XGEMM_ERR_INVALID_ARG;

    GemmParams base;
    // a packed operand's address is its byte offset in the (256-byte aligned)
    // workspace, set below once the split partials' bytes are known
    base.A = pk.a ? nullptr : (const uint16_t *)A;
    base.B = pk.b ? nullptr : (const uint16_t *)B;
    base.lda = pk.a ? pk.k8 : lda;
    base.ldb = pk.b ? pk.n8 : ldb;
    base.M = (int)M;
    base.N = (int)N;
    base.K = (int)K;
    base.tiles_m = (int)tiles_m;
    base.tiles_n = (int)tiles_n;
    base.group_m = cfg.group_m;
    base.vec_ab = ((uintptr_t)base.A % 16 == 0) && ((uintptr_t)base.B % 16 == 0) && (base.lda % 8 == 0) &&
                  (base.ldb % 8 == 0);
    base.tile_base = 0;
    base.batch = 1;
    base.stride_a = base.stride_b = base.stride_c = 0;
    out->tile = cfg.tile;
    out->ldw = cdiv(N, 4) * 4;
    out->ws = 0;
    out->nseg = 0;
    out->pack = pk;

    auto add = [&](int64_t first, int64_t count, int sp, int64_t kchunk, int reduce) {
        Segment &g = out->seg[out->nseg++];
        g.p = base;
        g.p.tile_base = (int)first;
        g.p.tile_count = (int)count;
        g.p.split = sp;
        g.p.k_chunk = (int)kchunk;
        g.reduce = reduce;
        if (reduce == 0) {
            g.p.C = (float *)C;
            g.p.ldc = ldc;
            g.p.split_stride = 0;
            g.p.vec_c = ((uintptr_t)C % 16 == 0) && (ldc % 4 == 0);
        } else {
            g.p.C = nullptr;  // the workspace, filled in at launch
            g.p.ldc = out->ldw;
            g.p.split_stride = M * out->ldw;
            g.p.vec_c = 1;
        }
        g.grid = count * sp;
        g.dma = dma_eligible(g.p, t.bm, pk.b);
        g.sk = false;
        g.dp_rounds = g.sk_tiles = g.kt = 0;
    };

    // packed operands follow the split partials in the workspace
    auto finish = [&]() {
        if (pk.a || pk.b) {
            pk.a_off = (out->ws + 255) / 256 * 256;
            const size_t a_bytes = pk.a ? (size_t)M * (size_t)pk.k8 * 2 : 0;
            pk.b_off = (pk.a_off + a_bytes + 255) / 256 * 256;
            out->ws = pk.b ? pk.b_off + (size_t)pk.k8 * (size_t)pk.n8 * 2 : pk.a_off + a_bytes;
            for (int i = 0; i < out->nseg; ++i) {
                if (pk.a)
                    out->seg[i].p.A = (const uint16_t *)(uintptr_t)pk.a_off;
                if (pk.b)
                    out->seg[i].p.B = (const uint16_t *)(uintptr_t)pk.b_off;
            }
            out->pack = pk;
        }
        return (int)XGEMM_OK;
    };
    if (split > 1) {
        add(0, tiles, split, kc, 1);
        out->ws = workspace_bytes(M, N, split);
        return finish();
    }
    add(0, tiles, 1, kc, 0);
    // the persistent stream-K kernel: the 256 x 256 tile on whole tiles of C
    // and whole K steps, at least as many tiles as workgroups (so that each
    // workgroup's range holds a tile's worth of steps), C 16-byte aligned
    // with 256 of its rows within 4 GiB
    if (cfg.stream_k > 0 && cfg.tile == XGEMM_TILE_256x256 && !pk.a && !pk.b) {
        Segment &g = out->seg[0];
        if (g.dma && M % t.bm == 0 && N % t.bn == 0 && K % t.bk == 0 && g.p.vec_c &&
            (int64_t)t.bm * ldc * 4 < ((int64_t)1 << 32))
            if (sk_schedule(g, tiles, K / t.bk, cfg.stream_k == 1 ? cu_count : cfg.stream_k))
                out->ws = sk_workspace(g);
    }
    return finish();
}

// Make the handle's workspace usable by work enqueued next on stream s with
// at least `bytes` after its counter prefix (it never shrinks).  Work of
// earlier calls on other streams that used the workspace is ordered before
// s's next work (a wait on the handle's event); a buffer being replaced is
// freed only after that work has completed, and a new one gets its counter
// prefix zeroed on s.  Every caller enqueues its workspace users and then
// calls release_workspace on the same stream.
int acquire_workspace(xgemm_ctx *h, size_t bytes, hipStream_t s)
{
    hipError_t e;
    bytes += kWsPrefix;
    if (h->ws_limit > 0 && bytes > h->ws_limit) {
        snprintf(h->last_error, sizeof(h->last_error), "workspace of %zu bytes exceeds the handle's limit of %zu",
                 bytes, h->ws_limit);
        return XGEMM_ERR_ALLOC;
    }
    if (h->ws_used && h->ws_stream != s) {
        // the last user is on another stream: wait for its event, or (the
        // first switch of streams, nothing recorded) for the whole device
        e = h->ws_recorded ? hipStreamWaitEvent(s, h->ws_event, 0) : hipDeviceSynchronize();
        if (e != hipSuccess) {
            set_error(h, h->ws_recorded ? "hipStreamWaitEvent" : "hipDeviceSynchronize", e);
            return XGEMM_ERR_HIP;
        }
        h->ws_multi = true;
    }
    if (bytes <= h->ws_bytes)
        return XGEMM_OK;
    if (h->workspace) {
        // the last user completes before the buffer goes: its event, or this
        // stream (the last user was on it, or the device has drained)
        e = h->ws_recorded ? hipEventSynchronize(h->ws_event) : hipStreamSynchronize(s);
        if (e != hipSuccess) {
            set_error(h, "workspace drain", e);
            return XGEMM_ERR_HIP;
        }
        (void)hipFree(h->workspace);
        h->workspace = nullptr;
        h->ws_bytes = 0;
    }
    e = hipMalloc(&h->workspace, bytes);
    if (e != hipSuccess) {
        h->workspace = nullptr;
        (void)hipGetLastError();
        set_error(h, "hipMalloc workspace", e);
        return XGEMM_ERR_ALLOC;
    }
    h->ws_bytes = bytes;
    hipLaunchKernelGGL(xgemm_dev::fill_zero, dim3(1), dim3(256), 0, s, (float *)h->workspace, (int64_t)0, 1,
                       (int)(kWsPrefix / sizeof(float)));
    e = hipGetLastError();
    if (e != hipSuccess) {
        set_error(h, "workspace prefix clear", e);
        return XGEMM_ERR_HIP;
    }
    return XGEMM_OK;
}

// The workspace's data after its counter prefix.
char *ws_data(void *ws) { return (char *)ws + kWsPrefix; }

// Mark the end of the workspace users just enqueued on stream s.
int release_workspace(xgemm_ctx *h, hipStream_t s)
{
    h->ws_stream = s;
    h->ws_used = true;
    h->ws_recorded = false;
    if (!h->ws_multi)
        return XGEMM_OK;
    const hipError_t e = hipEventRecord(h->ws_event, s);
    if (e != hipSuccess) {
        set_error(h, "hipEventRecord", e);
        return XGEMM_ERR_HIP;
    }
    h->ws_recorded = true;
    return XGEMM_OK;
}

// Copy `batch` src_rows x src_cols operands (leading dimension ld, batch
// stride src_stride) into dense rows x cols copies at dst (rows, cols
// multiples of 8 where padded; the copies follow each other).
hipError_t launch_pack(const void *src, int64_t ld, int64_t src_stride, int64_t src_rows, int64_t src_cols, char *dst,
                       int64_t rows, int64_t cols, int64_t batch, hipStream_t s)
{
    const int64_t items = batch * rows * cdiv(cols, xgemm_dev::kPackSeg);  // (problem, row, segment)
    const int grid = (int)(items < 8192 ? items : 8192);
    hipLaunchKernelGGL(xgemm_dev::pack16, dim3(grid), dim3(256), 0, s, (const uint16_t *)src, ld, src_stride,
                       (int)src_rows, (int)src_cols, (uint16_t *)dst, (int64_t)cols, rows * cols, (int)rows,
                       (int)(cols / 8), (int)batch);
    return hipGetLastError();
}

int launch_plan(xgemm_ctx *h, Plan plan, char *ws, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                const void *B, int64_t ldb, float *C, int64_t ldc, int dtype, hipStream_t s);

// The launches of one call: one plan over all of C, or (xgemm_run's body +
// band plans) two plans on sub-matrices, run one after the other.  ws is
// the workspace the larger of them needs.
struct CallPlan {
    int parts = 0;
    Plan plan[2];
    int64_t M[2], N[2];
    const void *A[2];
    const void *B[2];
    float *C[2];
    size_t ws = 0;
};

// Plan a call with K > 0 and M, N > 0 (arguments already checked): the
// forced configuration, or the selected plan, banded or not.  Touches no
// GPU.
int plan_call(int cu_count, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb,
              float *C, int64_t ldc, const xgemm_config *forced, CallPlan *cp, bool allow_sk = true)
{
    BandPlan band;
    if (forced) {
        band.body = *forced;
    } else {
        band = select_band(M, N, K, cu_count, allow_sk);
    }
    if (!allow_sk)
        band.body.stream_k = band.band.stream_k = 0;
    if (!forced && band.body.stream_k > 0) {
        // operands the persistent kernel cannot take as they are (alignment,
        // leading dimensions): the plan without it, banded or not
        Plan probe;
        const int rc = make_plan(M, N, K, A, lda, B, ldb, C, ldc, band.body, cu_count, &probe, true);
        if (rc != XGEMM_OK)
            return rc;
        if (!probe.seg[0].sk)
            band = select_band(M, N, K, cu_count, false);
    }
    if (band.axis == XGEMM_BAND_NONE) {
        cp->parts = 1;
        cp->M[0] = M, cp->N[0] = N, cp->A[0] = A, cp->B[0] = B, cp->C[0] = C;
    } else {
        // body, then band: ordinary calls on sub-matrices of A, B and C
        const int64_t ext = band.extent;
        const bool cols = band.axis == XGEMM_BAND_COLUMNS;
        cp->parts = 2;
        cp->M[0] = cols ? M : ext, cp->N[0] = cols ? ext : N;
        cp->M[1] = cols ? M : M - ext, cp->N[1] = cols ? N - ext : N;
        cp->A[0] = A, cp->B[0] = B, cp->C[0] = C;
        cp->A[1] = cols ? A : (const void *)((const char *)A + 2 * ext * lda);
        cp->B[1] = cols ? (const void *)((const char *)B + 2 * ext) : B;
        cp->C[1] = cols ? C + ext : C + ext * ldc;
    }
    cp->ws = 0;
    for (int i = 0; i < cp->parts; ++i) {
        const int rc = make_plan(cp->M[i], cp->N[i], K, cp->A[i], lda, cp->B[i], ldb, cp->C[i], ldc,
                                 i == 0 ? band.body : band.band, cu_count, &cp->plan[i], true);
        if (rc != XGEMM_OK)
            return rc;
        cp->ws = cp->plan[i].ws > cp->ws ? cp->plan[i].ws : cp->ws;
    }
    return XGEMM_OK;
}

// Enqueue every launch of a planned call, the workspace (cp.ws bytes, or
// unused when 0) at ws.
int launch_call(xgemm_ctx *h, const CallPlan &cp, char *ws, int64_t K, int64_t lda, int64_t ldb, int64_t ldc,
                int dtype, hipStream_t s)
{
    int rc = XGEMM_OK;
    for (int i = 0; i < cp.parts && rc == XGEMM_OK; ++i)
        rc = launch_plan(h, cp.plan[i], ws, cp.M[i], cp.N[i], K, cp.A[i], lda, cp.B[i], ldb, cp.C[i], ldc, dtype, s);
    return rc;
}

// The K == 0 product: C[0:M, 0:N] = 0.
int launch_zero(xgemm_ctx *h, int64_t M, int64_t N, float *C, int64_t ldc, hipStream_t s)
{
    const int64_t n = M * N;
    const int grid = (int)(cdiv(n, 256) < 4096 ? cdiv(n, 256) : 4096);
    hipLaunchKernelGGL(xgemm_dev::fill_zero, dim3(grid), dim3(256), 0, s, C, ldc, (int)M, (int)N);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        set_error(h, "fill_zero launch", e);
        return XGEMM_ERR_HIP;
    }
    return XGEMM_OK;
}

// A call of xgemm_run (forced == nullptr: the selected plan, banded or not)
// or xgemm_run_config (one launch plan with the forced configuration).  All
// parts are planned and the workspace grown before anything is enqueued.
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
    if (K == 0)
        return launch_zero(h, M, N, C, ldc, s);
    CallPlan cp;
    rc = plan_call(h->cu_count, M, N, K, A, lda, B, ldb, C, ldc, forced, &cp, forced || h->persistent);
    if (rc != XGEMM_OK)
        return rc;
    if (cp.ws > 0 && (rc = acquire_workspace(h, cp.ws, s)) != XGEMM_OK)
        return rc;
    rc = launch_call(h, cp, (char *)h->workspace, K, lda, ldb, ldc, dtype, s);
    if (cp.ws > 0) {
        const int rc2 = release_workspace(h, s);
        rc = rc == XGEMM_OK ? rc2 : rc;
    }
    return rc;
}

// Enqueue a plan whose workspace is in place: operand copies, the GEMM
// launches and their split-k reductions.
// The persistent kernel's parameters for a planned segment; flags and part
// are the workspace's counter prefix and its data.
xgemm_dev::SkParams sk_params(const Segment &g, int *flags, float *part)
{
    xgemm_dev::SkParams q;
    q.A = g.p.A;
    q.B = g.p.B;
    q.C = g.p.C;
    q.part = part;
    q.flags = flags;
    q.lda = g.p.lda;
    q.ldb = g.p.ldb;
    q.ldc = g.p.ldc;
    q.M = g.p.M;
    q.N = g.p.N;
    q.K = g.p.K;
    q.tiles_m = g.p.tiles_m;
    q.tiles_n = g.p.tiles_n;
    q.group_m = g.p.group_m;
    q.tiles_per = g.p.tiles_m * g.p.tiles_n;
    q.stride_a = g.p.batch > 1 ? g.p.stride_a : 0;
    q.stride_b = g.p.batch > 1 ? g.p.stride_b : 0;
    q.stride_c = g.p.batch > 1 ? g.p.stride_c : 0;
    q.kt = g.kt;
    q.grid = (int)g.grid;
    q.dp_rounds = g.dp_rounds;
    q.sk_tiles = g.sk_tiles;
    return q;
}

constexpr int kSkBM = 256, kSkBN = 256, kSkWGM = 2, kSkWGN = 4;

hipError_t launch_sk(int dtype, const xgemm_dev::SkParams &q, hipStream_t s)
{
    constexpr int T = kSkWGM * kSkWGN * 64;
    if (dtype == XGEMM_BF16)
        hipLaunchKernelGGL((xgemm_dev::gemm_kernel_sk<kSkBM, kSkBN, kDmaBK, kSkWGM, kSkWGN, 0>), dim3(q.grid), dim3(T),
                           0, s, q);
    else
        hipLaunchKernelGGL((xgemm_dev::gemm_kernel_sk<kSkBM, kSkBN, kDmaBK, kSkWGM, kSkWGN, 1>), dim3(q.grid), dim3(T),
                           0, s, q);
    return hipGetLastError();
}

// Enqueue a plan whose workspace is in place (ws: its start, the counter
// prefix; the plan's data follows it): operand copies, the GEMM launches
// and their split-k reductions.
int launch_plan(xgemm_ctx *h, Plan plan, char *ws, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                const void *B, int64_t ldb, float *C, int64_t ldc, int dtype, hipStream_t s)
{
    hipError_t e;
    int *const flags = (int *)ws;
    ws = ws_data(ws);
    // operand copies for the pipelined kernels
    const Pack &pk = plan.pack;
    if (pk.a && (e = launch_pack(A, lda, 0, M, K, ws + pk.a_off, M, pk.k8, 1, s)) != hipSuccess) {
        set_error(h, "pack A launch", e);
        return XGEMM_ERR_HIP;
    }
    if (pk.b && (e = launch_pack(B, ldb, 0, K, N, ws + pk.b_off, pk.k8, pk.n8, 1, s)) != hipSuccess) {
        set_error(h, "pack B launch", e);
        return XGEMM_ERR_HIP;
    }

    const int vec_c = ((uintptr_t)C % 16 == 0) && (ldc % 4 == 0);
    for (int i = 0; i < plan.nseg; ++i) {
        Segment &g = plan.seg[i];
        if (pk.a)
            g.p.A = (const uint16_t *)(ws + pk.a_off);
        if (pk.b)
            g.p.B = (const uint16_t *)(ws + pk.b_off);
        if (g.reduce)
            g.p.C = (float *)ws;
        e = g.sk ? launch_sk(dtype, sk_params(g, flags, (float *)ws), s)
                 : launch_tile(plan.tile, g.dma, dtype, g.p, (int)g.grid, s);
        if (e != hipSuccess) {
            set_error(h, "gemm launch", e);
            return XGEMM_ERR_HIP;
        }
        if (g.reduce == 1) {
            const int64_t nvec = M * cdiv(N, 4);
            const int grid = (int)(cdiv(nvec, 256) < 8192 ? cdiv(nvec, 256) : 8192);
            hipLaunchKernelGGL(xgemm_dev::splitk_reduce, dim3(grid), dim3(256), 0, s,
                               (const float *)ws, (int64_t)(M * plan.ldw), plan.ldw, g.p.split, C,
                               ldc, (int)M, (int)N, vec_c);
        }
        if (g.reduce) {
            e = hipGetLastError();
            if (e != hipSuccess) {
                set_error(h, "split-k reduce launch", e);
                return XGEMM_ERR_HIP;
            }
        }
    }
    return XGEMM_OK;
}

int run_batched(xgemm_ctx *h, int64_t batch, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                int64_t sa, const void *B, int64_t ldb, int64_t sb, float *C, int64_t ldc, int64_t sc, int dtype,
                void *stream)
{
    if (batch < 0 || sa < 0 || sb < 0 || sc < 0)
        return XGEMM_ERR_INVALID_ARG;
    int rc = check_args(h, M, N, K, A, lda, B, ldb, C, ldc, dtype);
    if (rc != XGEMM_OK)
        return rc;
    if (batch == 0 || M == 0 || N == 0)
        return XGEMM_OK;
    if (batch == 1)
        return run(h, M, N, K, A, lda, B, ldb, C, ldc, dtype, stream, nullptr);
    // outputs of different problems must not overlap; every problem's
    // matrices must stay addressable
    if (sc < (M - 1) * ldc + N)
        return XGEMM_ERR_INVALID_ARG;
    const double last = (double)(batch - 1);
    if (last * sa + (double)M * lda > 9.0e18 || last * sb + (double)K * ldb > 9.0e18 ||
        last * sc + (double)M * ldc > 9.0e18 || batch > 0x7fffffff)
        return XGEMM_ERR_INVALID_ARG;
    h->last_error[0] = '\0';
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    if (K == 0) {
        for (int64_t b = 0; b < batch; ++b) {
            rc = run(h, M, N, 0, A, lda, B, ldb, C + b * sc, ldc, dtype, stream, nullptr);
            if (rc != XGEMM_OK)
                return rc;
        }
        return XGEMM_OK;
    }
    xgemm_config cfg;
    select_config_batched(batch, M, N, K, h->cu_count, &cfg);
    Plan plan;
    rc = make_plan(M, N, K, A, lda, B, ldb, C, ldc, cfg, h->cu_count, &plan, false);
    if (rc != XGEMM_OK)
        return rc;
    // Operands the pipelined kernel cannot read in place (for every problem:
    // alignment, leading dimension, batch stride, N or K) are copied into the
    // workspace, one copy per problem (a single one for a shared operand,
    // stride 0), when that makes the pipelined kernel eligible.
    const bool k_ok = K % 8 == 0;
    Pack pk;
    pk.a = !(k_ok && (uintptr_t)A % 16 == 0 && lda % 8 == 0 && sa % 8 == 0);
    pk.b = !(k_ok && (uintptr_t)B % 16 == 0 && ldb % 8 == 0 && sb % 8 == 0 && N % 8 == 0);
    if (!k_ok)
        pk.a = pk.b = true;
    pk.k8 = cdiv(K, 8) * 8;
    pk.n8 = cdiv(N, 8) * 8;
    const int64_t na = sa == 0 ? 1 : batch, nb = sb == 0 ? 1 : batch;
    Plan packed;
    if ((pk.a || pk.b) &&
        make_plan_with(M, N, K, A, lda, B, ldb, C, ldc, cfg, h->cu_count, pk, &packed) == XGEMM_OK &&
        packed.seg[0].dma) {
        const size_t a_bytes = pk.a ? (size_t)na * (size_t)M * (size_t)pk.k8 * 2 : 0;
        pk.a_off = 0;
        pk.b_off = (a_bytes + 255) / 256 * 256;
        const size_t ws = pk.b ? pk.b_off + (size_t)nb * (size_t)pk.k8 * (size_t)pk.n8 * 2 : a_bytes;
        if (packed.nseg != 1 || packed.seg[0].reduce != 0 || packed.seg[0].p.split != 1 ||
            packed.seg[0].grid * batch > 0x7fffffff)
            return XGEMM_ERR_INVALID_ARG;  // batched plans are single unsplit launches
        rc = acquire_workspace(h, ws, s);
        if (rc != XGEMM_OK)
            return rc;
        char *const w = ws_data(h->workspace);
        e = hipSuccess;
        if (pk.a && (e = launch_pack(A, lda, sa, M, K, w + pk.a_off, M, pk.k8, na, s)) != hipSuccess)
            set_error(h, "pack A launch", e);
        if (e == hipSuccess && pk.b &&
            (e = launch_pack(B, ldb, sb, K, N, w + pk.b_off, pk.k8, pk.n8, nb, s)) != hipSuccess)
            set_error(h, "pack B launch", e);
        if (e != hipSuccess) {
            (void)release_workspace(h, s);
            return XGEMM_ERR_HIP;
        }
        plan = packed;
        if (pk.a) {
            plan.seg[0].p.A = (const uint16_t *)(w + pk.a_off);
            sa = sa == 0 ? 0 : M * pk.k8;
        }
        if (pk.b) {
            plan.seg[0].p.B = (const uint16_t *)(w + pk.b_off);
            sb = sb == 0 ? 0 : pk.k8 * pk.n8;
        }
    } else {
        pk = Pack{};
    }
    Segment &g = plan.seg[0];
    if (plan.nseg != 1 || g.reduce != 0 || g.p.split != 1)
        return XGEMM_ERR_INVALID_ARG;  // batched plans are single unsplit launches
    if (g.grid * batch > 0x7fffffff)
        return XGEMM_ERR_INVALID_ARG;
    g.p.batch = (int)batch;
    g.p.stride_a = sa;
    g.p.stride_b = sb;
    g.p.stride_c = sc;
    // 16-byte vector paths need every problem's matrices aligned
    g.p.vec_ab = g.p.vec_ab && (sa % 8 == 0) && (sb % 8 == 0);
    g.p.vec_c = g.p.vec_c && (sc % 4 == 0);
    g.dma = dma_eligible(g.p, kTiles[plan.tile].bm, pk.b);
    // the persistent kernel over the tiles of all problems, as xgemm_run
    // takes it for one problem with as many tiles
    const TileShape &t256 = kTiles[XGEMM_TILE_256x256];
    if (h->persistent && !pk.a && !pk.b && g.dma && g.p.vec_c && use_persistent(M, N, K, h->cu_count, cfg, batch) &&
        (int64_t)t256.bm * ldc * 4 < ((int64_t)1 << 32) &&
        sk_schedule(g, (M / t256.bm) * (N / t256.bn) * batch, K / t256.bk, h->cu_count)) {
        const size_t ws = sk_workspace(g);
        if (ws > 0 && (rc = acquire_workspace(h, ws, s)) != XGEMM_OK)
            return rc;
        char *const base = ws > 0 ? (char *)h->workspace : nullptr;
        e = launch_sk(dtype, sk_params(g, (int *)base, base ? (float *)ws_data(base) : nullptr), s);
        rc = XGEMM_OK;
        if (e != hipSuccess) {
            set_error(h, "gemm launch", e);
            rc = XGEMM_ERR_HIP;
        }
        if (ws > 0) {
            const int rc2 = release_workspace(h, s);
            rc = rc == XGEMM_OK ? rc2 : rc;
        }
        return rc;
    }
    e = launch_tile(plan.tile, g.dma, dtype, g.p, (int)(g.grid * batch), s);
    rc = XGEMM_OK;
    if (e != hipSuccess) {
        set_error(h, "gemm launch", e);
        rc = XGEMM_ERR_HIP;
    }
    if (pk.a || pk.b) {
        const int rc2 = release_workspace(h, s);
        rc = rc == XGEMM_OK ? rc2 : rc;
    }
    return rc;
}

// ---------------------------------------------------------------------------
// GEMV
// ---------------------------------------------------------------------------

using xgemv_dev::GemvParams;

bool valid_gemv_config(const xgemv_config *c)
{
    return c && (c->rows == 1 || c->rows == 2 || c->rows == 4 || c->rows == 8) &&
           (c->unroll == 1 || c->unroll == 2 || c->unroll == 4) && c->split_k >= 1 && c->split_k <= 256;
}

// K values per split (a multiple of 4, so that every range starts on a
// 16-byte boundary of an aligned row) and the split left after trailing
// empty ranges are dropped.
int gemv_split(int64_t K, int split, int64_t *k_chunk)
{
    *k_chunk = cdiv(cdiv(K, split), 4) * 4;
    while (split > 1 && *k_chunk * (split - 1) >= K) {
        --split;
        *k_chunk = cdiv(cdiv(K, split), 4) * 4;
    }
    return split;
}

// Measured on MI355X (interleaved sweeps over 4096^2 .. 32768^2, 1024 x
// 65536, 65536 x 1024, 131072 x 4096 and 256 x 262144): two rows per
// workgroup with four chunks in flight per row is within 3% of the best
// configuration whenever that still leaves at least four workgroups per CU;
// below that one row per workgroup keeps more CUs streaming (at 256 x
// 262144 it reads 6.2 TB/s against 4.1 TB/s with two chunks in flight).
//
// Fewer than two workgroups per CU leave CUs idle; then K is split so that
// there are about that many, but with at least 65536 values in every range
// (shorter ranges cost more in per-workgroup start-up and partial sums
// than they gain) and at most 256 ranges.  Measured: 64 x 2^20 reads
// 5.6 TB/s split 8 ways against 1.8 TB/s unsplit; 1 x 2^22 2.9 TB/s split
// 64 ways (0.09 TB/s unsplit, 1.6 TB/s split 256 ways).
void select_gemv(int64_t M, int64_t K, int cu_count, xgemv_config *out)
{
    out->rows = M >= 8 * (int64_t)cu_count ? 2 : 1;
    out->unroll = 4;
    const int64_t blocks = cdiv(M, out->rows);
    int64_t split = 1;
    if (blocks < 2 * (int64_t)cu_count) {
        split = cdiv(2 * (int64_t)cu_count, blocks);
        split = split < K / 65536 ? split : K / 65536;
        split = split < 256 ? split : 256;
        split = split > 1 ? split : 1;
    }
    out->split_k = (int)split;
}

template <class F>
auto with_gemv_config(const xgemv_config &c, F &&f)
{
#define XGEMV_CASE(R, U)                                      \
    if (c.rows == R && c.unroll == U)                        \
        return f(std::integral_constant<int, R>{}, std::integral_constant<int, U>{});
    XGEMV_CASE(1, 1) XGEMV_CASE(1, 2) XGEMV_CASE(1, 4)
    XGEMV_CASE(2, 1) XGEMV_CASE(2, 2) XGEMV_CASE(2, 4)
    XGEMV_CASE(4, 1) XGEMV_CASE(4, 2) XGEMV_CASE(4, 4)
    XGEMV_CASE(8, 1) XGEMV_CASE(8, 2)
#undef XGEMV_CASE
    return f(std::integral_constant<int, 8>{}, std::integral_constant<int, 4>{});
}

int check_gemv_args(int64_t M, int64_t K, const float *A, int64_t lda, const float *x, const float *y)
{
    if (M < 0 || K < 0 || M >= kMaxDim || K >= kMaxDim || lda < K || lda < 0)
        return XGEMM_ERR_INVALID_ARG;
    if ((M > 0 && K > 0 && !A) || (K > 0 && M > 0 && !x) || (M > 0 && !y))
        return XGEMM_ERR_INVALID_ARG;
    if ((double)M * (double)lda > 9.0e18)
        return XGEMM_ERR_INVALID_ARG;
    return XGEMM_OK;
}

// Launch parameters of a GEMV with `rows` rows per workgroup; blocks is 0
// when the launch would exceed 2^31 - 1 workgroups (only possible with a
// forced split of a very tall matrix), which callers reject.
GemvParams gemv_params(int64_t M, int64_t K, const float *A, int64_t lda, const float *x, float *y, int rows,
                       int split_k, float *part)
{
    GemvParams p;
    p.A = A;
    p.x = x;
    p.y = y;
    p.part = part;
    p.lda = lda;
    p.M = (int)M;
    p.K = (int)K;
    int64_t kc;
    p.split = gemv_split(K, split_k, &kc);
    p.k_chunk = (int)kc;
    p.vec = ((uintptr_t)A % 16 == 0) && ((uintptr_t)x % 16 == 0) && (lda % 4 == 0);
    const int64_t blocks = cdiv(M, rows) * p.split;
    p.blocks = blocks <= 0x7fffffff ? (int)blocks : 0;
    return p;
}

int run_gemv(xgemm_ctx *h, int64_t M, int64_t K, const float *A, int64_t lda, const float *x, float *y,
             void *stream, const xgemv_config *forced)
{
    if (!h)
        return XGEMM_ERR_INVALID_ARG;
    int rc = check_gemv_args(M, K, A, lda, x, y);
    if (rc != XGEMM_OK)
        return rc;
    if (forced && !valid_gemv_config(forced))
        return XGEMM_ERR_INVALID_ARG;
    h->last_error[0] = '\0';
    hipStream_t s = (hipStream_t)stream;
    if (M == 0)
        return XGEMM_OK;
    if (K == 0) {
        const int grid = (int)(cdiv(M, 256) < 4096 ? cdiv(M, 256) : 4096);
        hipLaunchKernelGGL(xgemm_dev::fill_zero, dim3(grid), dim3(256), 0, s, y, (int64_t)1, (int)M, 1);
    } else {
        xgemv_config cfg;
        if (forced)
            cfg = *forced;
        else
            select_gemv(M, K, h->cu_count, &cfg);
        GemvParams p = gemv_params(M, K, A, lda, x, y, cfg.rows, cfg.split_k, nullptr);
        if (p.blocks == 0)
            return XGEMM_ERR_INVALID_ARG;
        if (p.split > 1) {
            rc = acquire_workspace(h, (size_t)p.split * (size_t)M * sizeof(float), s);
            if (rc != XGEMM_OK)
                return rc;
            p.part = (float *)ws_data(h->workspace);
        }
        with_gemv_config(cfg, [&](auto r, auto u) {
            constexpr int R = decltype(r)::value, U = decltype(u)::value;
            hipLaunchKernelGGL((xgemv_dev::gemv_kernel<R, U>), grid_of(p.blocks), dim3(xgemv_dev::kThreads), 0, s,
                               p);
            return 0;
        });
        if (p.split > 1) {
            const int grid = (int)(cdiv(M, 256) < 1024 ? cdiv(M, 256) : 1024);
            hipLaunchKernelGGL(xgemv_dev::gemv_reduce, dim3(grid), dim3(256), 0, s, (const float *)p.part,
                               p.split, (int)M, y);
            const int rc2 = release_workspace(h, s);
            if (rc2 != XGEMM_OK)
                return rc2;
        }
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        set_error(h, "gemv launch", e);
        return XGEMM_ERR_HIP;
    }
    return XGEMM_OK;
}

// Host stand-in for the device operations of the pipelined kernel: each
// call appends one event to the calling thread's trace instead of touching
// memory.  LDS pointers point into a host buffer of the kernel's LDS size,
// so LDS addresses are byte offsets from its start.
// Where the persistent kernel's trace takes the values of its split-tile
// counters from: `schedule` 0 has every split tile's last steps count in
// first, 1 its first steps; tail and head are this workgroup's two counter
// addresses (slots lw and lw + 1).  Thread 0's hand-over words are recorded
// in order and every thread reads them back in the same order (the threads
// of a workgroup are traced one after another, thread 0 first).
struct TraceSplit {
    int schedule = 0;
    const int *tail = nullptr, *head = nullptr;
    std::vector<int> words;
};

struct TraceOps {
    char *base;
    std::vector<xgemm_trace_event> *ev;
    TraceSplit *split = nullptr;
    mutable size_t word_pos = 0;
    char *lds() const { return base; }
    uint32_t lds_addr(const char *q) const { return (uint32_t)(q - base); }
    int uniform(int x) const { return x; }
    void push(int op, int arg, int64_t lds, int64_t addr) const
    {
        xgemm_trace_event e;
        e.op = op;
        e.arg = arg;
        e.lds = lds;
        e.addr = addr;
        ev->push_back(e);
    }
    void load16(const void *g, uint32_t goff, uint32_t lds) const
    {
        push(XGEMM_TRACE_LDS_LOAD, 16, lds, (int64_t)((uintptr_t)g + goff));
    }
    xgemm_dev::u32x4 read16(const char *q) const
    {
        push(XGEMM_TRACE_LDS_READ, 16, q - base, 0);
        return xgemm_dev::u32x4{0, 0, 0, 0};
    }
    xgemm_dev::v4i16 read_tr8(const char *q) const
    {
        push(XGEMM_TRACE_LDS_READ, 8, q - base, 0);
        return xgemm_dev::v4i16{0, 0, 0, 0};
    }
    template <int DT>
    xgemm_dev::f32x16 mfma(xgemm_dev::u32x4, xgemm_dev::u32x4, xgemm_dev::f32x16 c) const
    {
        return c;
    }
    template <int DT>
    xgemm_dev::f32x4 mfma(xgemm_dev::u32x4, xgemm_dev::u32x4, xgemm_dev::f32x4 c) const
    {
        return c;
    }
    template <int N>
    void wait_vm() const
    {
        push(XGEMM_TRACE_WAIT_VM, N, 0, 0);
    }
    void wait_lgkm0() const { push(XGEMM_TRACE_WAIT_LGKM, 0, 0, 0); }
    void barrier() const { push(XGEMM_TRACE_BARRIER, 0, 0, 0); }
    void fence() const {}
    template <int P>
    void priority() const
    {
    }
    void store4(float *q, xgemm_dev::f32x4) const { push(XGEMM_TRACE_STORE, 16, 0, (int64_t)(uintptr_t)q); }
    void store1(float *q, float) const { push(XGEMM_TRACE_STORE, 4, 0, (int64_t)(uintptr_t)q); }
    xgemm_dev::u32x4 gload16(const uint16_t *q) const
    {
        push(XGEMM_TRACE_LOAD, 16, 0, (int64_t)(uintptr_t)q);
        return xgemm_dev::u32x4{0, 0, 0, 0};
    }
    uint16_t gload2(const uint16_t *q) const
    {
        push(XGEMM_TRACE_LOAD, 2, 0, (int64_t)(uintptr_t)q);
        return 0;
    }
    void lds_write16(char *q, xgemm_dev::u32x4) const { push(XGEMM_TRACE_LDS_WRITE, 16, q - base, 0); }
    void lds_write16(char *q, xgemm_dev::u32x4, bool on) const
    {
        push(XGEMM_TRACE_LDS_WRITE, 16, on ? (int64_t)(q - base) : -1, 0);
    }
    // __syncthreads: the compiler emits s_waitcnt lgkmcnt(0) and s_barrier
    void sync() const
    {
        push(XGEMM_TRACE_WAIT_LGKM, 0, 0, 0);
        push(XGEMM_TRACE_BARRIER, 0, 0, 0);
    }
    // persistent kernel: buffer accesses at base + per-lane + uniform offset
    typedef const char *Rsrc;
    Rsrc rsrc(const void *b) const { return (const char *)b; }
    void buf_store4(Rsrc r, uint32_t voff, uint32_t soff, xgemm_dev::f32x4) const
    {
        push(XGEMM_TRACE_STORE, 16, 0, (int64_t)(uintptr_t)(r + voff + soff));
    }
    void buf_store4_nt(Rsrc r, uint32_t voff, uint32_t soff, xgemm_dev::f32x4 v) const { buf_store4(r, voff, soff, v); }
    // a register exchange between lanes: no memory access, nothing to record
    void line_pair(xgemm_dev::f32x4 &, xgemm_dev::f32x4 &) const {}
    void buf_store4_dev(Rsrc r, uint32_t voff, uint32_t soff, xgemm_dev::f32x4 v) const { buf_store4(r, voff, soff, v); }
    xgemm_dev::f32x4 buf_load4_dev(Rsrc r, uint32_t voff, uint32_t soff) const
    {
        push(XGEMM_TRACE_LOAD, 16, 0, (int64_t)(uintptr_t)(r + voff + soff));
        return xgemm_dev::f32x4{0, 0, 0, 0};
    }
    void stores_done() const { push(XGEMM_TRACE_WAIT_VM, 0, 0, 0); }
    // counter reads and atomic adds are vector-memory loads with a result
    int flag_load(int *f) const
    {
        push(XGEMM_TRACE_LOAD, 4, 0, (int64_t)(uintptr_t)f);
        // the head finds the last steps counted in (schedule 0) or not
        return (split && f == split->head && split->schedule == 0) ? 1 : 0;
    }
    int flag_add(int *f, int) const
    {
        push(XGEMM_TRACE_LOAD, 4, 0, (int64_t)(uintptr_t)f);
        // the piece counting in second finds 1: the tail under schedule 1
        return (split && f == split->tail && split->schedule == 1) ? 1 : 0;
    }
    void flag_store(int *f, int) const { push(XGEMM_TRACE_STORE, 4, 0, (int64_t)(uintptr_t)f); }
    void lds_write4(char *q, int v, bool on) const
    {
        push(XGEMM_TRACE_LDS_WRITE, 4, on ? (int64_t)(q - base) : -1, 0);
        if (on && split)
            split->words.push_back(v);
    }
    int lds_read4(const char *q) const
    {
        push(XGEMM_TRACE_LDS_READ, 4, q - base, 0);
        return split && word_pos < split->words.size() ? split->words[word_pos++] : 0;
    }
};

// Host stand-in for the GEMV kernel's operations.  Lanes whose masked LDS
// access is off record LDS offset -1.
struct TraceGemvOps {
    float *base;
    std::vector<xgemm_trace_event> *ev;
    void push(int op, int arg, int64_t lds, int64_t addr) const
    {
        xgemm_trace_event e;
        e.op = op;
        e.arg = arg;
        e.lds = lds;
        e.addr = addr;
        ev->push_back(e);
    }
    float *lds() const { return base; }
    xgemv_dev::f32x4 load4(const float *q) const
    {
        push(XGEMM_TRACE_LOAD, 16, 0, (int64_t)(uintptr_t)q);
        return xgemv_dev::f32x4{0, 0, 0, 0};
    }
    float load1(const float *q) const
    {
        push(XGEMM_TRACE_LOAD, 4, 0, (int64_t)(uintptr_t)q);
        return 0.0f;
    }
    float wave_sum(float v) const { return v; }
    void lds_write1(float *q, float, bool on) const
    {
        push(XGEMM_TRACE_LDS_WRITE, 4, on ? (int64_t)((char *)q - (char *)base) : -1, 0);
    }
    float lds_read1(const float *q, bool on) const
    {
        push(XGEMM_TRACE_LDS_READ, 4, on ? (int64_t)((const char *)q - (const char *)base) : -1, 0);
        return 0.0f;
    }
    void sync() const
    {
        push(XGEMM_TRACE_WAIT_LGKM, 0, 0, 0);
        push(XGEMM_TRACE_BARRIER, 0, 0, 0);
    }
    void store1(float *q, float) const { push(XGEMM_TRACE_STORE, 4, 0, (int64_t)(uintptr_t)q); }
};

// Plan of a traced call: the same checks and plan as xgemm_run_config.
int trace_plan(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb,
               const float *C, int64_t ldc, const xgemm_config *cfg, int cu_count, int segment, Plan *plan)
{
    if (!valid_config(cfg) || cu_count < 1 || M <= 0 || N <= 0 || K <= 0 || M >= kMaxDim || N >= kMaxDim ||
        K >= kMaxDim || lda < K || ldb < N || ldc < N || !A || !B || !C)
        return XGEMM_ERR_INVALID_ARG;
    const int rc = make_plan(M, N, K, A, lda, B, ldb, C, ldc, *cfg, cu_count, plan, true);
    if (rc != XGEMM_OK)
        return rc;
    if (segment < 0 || segment >= plan->nseg)
        return XGEMM_ERR_INVALID_ARG;
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
    h->ws_stream = nullptr;
    h->ws_used = false;
    h->ws_recorded = false;
    h->ws_multi = false;
    h->ws_limit = 0;
    h->persistent = true;
    h->last_error[0] = '\0';
    h->scratch = nullptr;
    if (dev >= 0 && dev < kMaxDevices) {
        // once per device, with the device current: the address of this
        // device's copy of the scratch array
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        if (!g_scratch_ptr[dev]) {
            void *ptr = nullptr;
            if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
                (void)hipGetLastError();
                delete h;
                return XGEMM_ERR_HIP;
            }
            // its counter prefix starts zero (the persistent kernel leaves it so)
            if (hipMemsetAsync(ptr, 0, kWsPrefix, nullptr) != hipSuccess ||
                hipStreamSynchronize(nullptr) != hipSuccess) {
                (void)hipGetLastError();
                delete h;
                return XGEMM_ERR_HIP;
            }
            g_scratch_ptr[dev] = ptr;
        }
        h->scratch = g_scratch_ptr[dev];
    }
    if (hipEventCreateWithFlags(&h->ws_event, hipEventDisableTiming) != hipSuccess) {
        (void)hipGetLastError();
        delete h;
        return XGEMM_ERR_HIP;
    }
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
    if (hipEventDestroy(h->ws_event) != hipSuccess) {
        (void)hipGetLastError();
        rc = XGEMM_ERR_HIP;
    }
    delete h;
    return rc;
}

int xgemm_set_workspace_limit(xgemm_handle_t h, size_t bytes)
{
    if (!h)
        return XGEMM_ERR_INVALID_ARG;
    h->ws_limit = bytes;
    return XGEMM_OK;
}

int xgemm_set_persistent(xgemm_handle_t h, int enable)
{
    if (!h || (enable != 0 && enable != 1))
        return XGEMM_ERR_INVALID_ARG;
    h->persistent = enable == 1;
    return XGEMM_OK;
}

int xgemm_run(xgemm_handle_t h, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
              const void *B, int64_t ldb, float *C, int64_t ldc, int dtype, void *stream)
{
    return run(h, M, N, K, A, lda, B, ldb, C, ldc, dtype, stream, nullptr);
}

int xgemm_run_noalloc(xgemm_handle_t h, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                      const void *B, int64_t ldb, float *C, int64_t ldc, int dtype, void *stream)
{
    int rc = check_args(h, M, N, K, A, lda, B, ldb, C, ldc, dtype);
    if (rc != XGEMM_OK)
        return rc;
    h->last_error[0] = '\0';
    if (!h->scratch) {
        snprintf(h->last_error, sizeof(h->last_error), "no scratch array on device %d", h->device);
        return XGEMM_ERR_UNSUPPORTED;
    }
    hipStream_t s = (hipStream_t)stream;
    if (M == 0 || N == 0)
        return XGEMM_OK;
    if (K == 0)
        return launch_zero(h, M, N, C, ldc, s);
    CallPlan cp;
    rc = plan_call(h->cu_count, M, N, K, A, lda, B, ldb, C, ldc, nullptr, &cp, h->persistent);
    if (rc == XGEMM_OK && cp.ws + kWsPrefix > kScratchBytes)   // a persistent plan's partials may not fit
        rc = plan_call(h->cu_count, M, N, K, A, lda, B, ldb, C, ldc, nullptr, &cp, false);
    if (rc != XGEMM_OK)
        return rc;
    if (cp.ws + kWsPrefix > kScratchBytes) {
        snprintf(h->last_error, sizeof(h->last_error),
                 "the call needs %zu bytes of scratch, above the static maximum of %zu", cp.ws + kWsPrefix,
                 kScratchBytes);
        return XGEMM_ERR_INVALID_ARG;
    }
    return launch_call(h, cp, (char *)h->scratch, K, lda, ldb, ldc, dtype, s);
}

int xgemm_run_config(xgemm_handle_t h, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                     const void *B, int64_t ldb, float *C, int64_t ldc, int dtype, void *stream,
                     const xgemm_config *cfg)
{
    if (!cfg)
        return XGEMM_ERR_INVALID_ARG;
    return run(h, M, N, K, A, lda, B, ldb, C, ldc, dtype, stream, cfg);
}

int xgemm_run_strided_batched(xgemm_handle_t h, int64_t batch, int64_t M, int64_t N, int64_t K, const void *A,
                              int64_t lda, int64_t stride_a, const void *B, int64_t ldb, int64_t stride_b, float *C,
                              int64_t ldc, int64_t stride_c, int dtype, void *stream)
{
    return run_batched(h, batch, M, N, K, A, lda, stride_a, B, ldb, stride_b, C, ldc, stride_c, dtype, stream);
}

int xgemm_select_config(int64_t M, int64_t N, int64_t K, int dtype, int cu_count, xgemm_config *out)
{
    if (!out || M < 0 || N < 0 || K < 0 || cu_count < 1 || (dtype != XGEMM_BF16 && dtype != XGEMM_FP16))
        return XGEMM_ERR_INVALID_ARG;
    select_config(M, N, K, cu_count, out);
    return XGEMM_OK;
}

int xgemm_select_plan(int64_t M, int64_t N, int64_t K, int dtype, int cu_count, int persistent, xgemm_band *out)
{
    if (!out || M < 0 || N < 0 || K < 0 || cu_count < 1 || (dtype != XGEMM_BF16 && dtype != XGEMM_FP16) ||
        (persistent != 0 && persistent != 1))
        return XGEMM_ERR_INVALID_ARG;
    *out = xgemm_band{};
    if (M == 0 || N == 0 || K == 0 || M >= kMaxDim || N >= kMaxDim || K >= kMaxDim) {
        select_config(M, N, K, cu_count, &out->body);
        return XGEMM_OK;
    }
    const BandPlan b = select_band(M, N, K, cu_count, persistent == 1);
    out->axis = b.axis;
    out->extent = b.extent;
    out->body = b.body;
    if (b.axis != XGEMM_BAND_NONE)
        out->band = b.band;
    return XGEMM_OK;
}

int xgemm_select_band(int64_t M, int64_t N, int64_t K, int dtype, int cu_count, xgemm_band *out)
{
    return xgemm_select_plan(M, N, K, dtype, cu_count, 1, out);
}

int xgemm_tile_info(int tile, int *bm, int *bn, int *bk, int *threads)
{
    if (tile < 0 || tile >= XGEMM_TILE_COUNT || !bm || !bn || !bk || !threads)
        return XGEMM_ERR_INVALID_ARG;
    *bm = kTiles[tile].bm;
    *bn = kTiles[tile].bn;
    *bk = kTiles[tile].bk;
    *threads = tile_threads(tile, true);
    return XGEMM_OK;
}

int xgemm_kernel_family(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B,
                        int64_t ldb, const xgemm_config *cfg)
{
    if (!valid_config(cfg) || M <= 0 || N <= 0 || K <= 0 || M >= kMaxDim || N >= kMaxDim || K >= kMaxDim ||
        lda < K || ldb < N)
        return -1;
    Plan plan;
    // C taken as aligned; the persistent kernel's grid is 256 CUs here
    if (make_plan(M, N, K, A, lda, B, ldb, nullptr, N, *cfg, 256, &plan, true) != XGEMM_OK)
        return -1;
    return plan.seg[0].sk ? XGEMM_KERNEL_PERSISTENT : plan.seg[0].dma ? XGEMM_KERNEL_PIPELINED : XGEMM_KERNEL_GENERAL;
}

size_t xgemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int cu_count, const xgemm_config *cfg)
{
    if (!valid_config(cfg) || M < 0 || N < 0 || K < 0 || cu_count < 1 || M >= kMaxDim || N >= kMaxDim ||
        K >= kMaxDim)
        return 0;
    if (M == 0 || N == 0 || K == 0)
        return 0;
    Plan plan;
    if (make_plan(M, N, K, nullptr, K, nullptr, N, nullptr, N, *cfg, cu_count, &plan, true) != XGEMM_OK)
        return 0;
    return plan.ws > 0 ? plan.ws + kWsPrefix : 0;
}

int xgemm_trace_plan(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb,
                     const float *C, int64_t ldc, const xgemm_config *cfg, int cu_count, int segment,
                     xgemm_trace_info *info)
{
    if (!info)
        return XGEMM_ERR_INVALID_ARG;
    Plan plan;
    const int rc = trace_plan(M, N, K, A, lda, B, ldb, C, ldc, cfg, cu_count, segment, &plan);
    if (rc != XGEMM_OK)
        return rc;
    const Segment &g = plan.seg[segment];
    info->segments = plan.nseg;
    info->family = g.sk ? XGEMM_KERNEL_PERSISTENT : g.dma ? XGEMM_KERNEL_PIPELINED : XGEMM_KERNEL_GENERAL;
    info->reduce = g.reduce;
    info->threads = tile_threads(plan.tile, g.dma);
    info->lds_bytes = g.sk ? xgemm_dev::sk_lds_bytes<kSkBM, kSkBN, kDmaBK>()
                    : g.dma ? with_dma_tile(plan.tile, [](auto t) {
        using T = decltype(t);
        return xgemm_dev::dma_lds_bytes<T::BM, T::BN, T::BK, T::STAGES>();
    }) : with_general_tile(plan.tile, [](auto t) {
        using T = decltype(t);
        return xgemm_dev::general_lds_bytes<T::BM, T::BN, T::BK>();
    });
    info->split = g.p.split;
    info->grid = g.grid;
    info->workspace_bytes = plan.ws > 0 ? (int64_t)(plan.ws + kWsPrefix) : 0;
    info->tile_base = g.p.tile_base;
    info->tile_count = g.p.tile_count;
    const Pack &pk = plan.pack;
    info->packed = (pk.a ? 1 : 0) | (pk.b ? 2 : 0);
    info->k = g.p.K;
    info->lda = g.p.lda;
    info->ldb = g.p.ldb;
    info->a_offset = pk.a ? (int64_t)(kWsPrefix + pk.a_off) : -1;
    info->b_offset = pk.b ? (int64_t)(kWsPrefix + pk.b_off) : -1;
    info->data_offset = (int64_t)kWsPrefix;
    info->dp_rounds = g.dp_rounds;
    info->sk_tiles = g.sk_tiles;
    info->kt = g.kt;
    info->reserved = 0;
    return XGEMM_OK;
}

int xgemm_trace_workgroup(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb,
                          float *C, int64_t ldc, float *W, const xgemm_config *cfg, int cu_count, int segment,
                          int64_t block, int schedule, xgemm_trace_event *out, int64_t capacity, int64_t *counts)
{
    if (!counts || capacity < 0 || (capacity > 0 && !out) || schedule < 0 || schedule > 1)
        return XGEMM_ERR_INVALID_ARG;
    Plan plan;
    int rc = trace_plan(M, N, K, A, lda, B, ldb, C, ldc, cfg, cu_count, segment, &plan);
    if (rc != XGEMM_OK)
        return rc;
    Segment &g = plan.seg[segment];
    if (block < 0 || block >= g.grid)
        return XGEMM_ERR_INVALID_ARG;
    const Pack &pk = plan.pack;
    char *const wdata = W ? ws_data(W) : nullptr;
    if (g.reduce || pk.a || pk.b || (g.sk && g.sk_tiles > 0)) {
        if (!W)
            return XGEMM_ERR_INVALID_ARG;
        if (g.reduce)
            g.p.C = (float *)wdata;
        if (pk.a)
            g.p.A = (const uint16_t *)(wdata + pk.a_off);
        if (pk.b)
            g.p.B = (const uint16_t *)(wdata + pk.b_off);
    }
    const int threads = tile_threads(plan.tile, g.dma);
    TraceSplit split;
    split.schedule = schedule;
    // run `body(ops, tid)` for every thread, collecting each one's events
    auto trace_threads = [&](size_t lds_bytes, auto &&body) {
        std::vector<char> lds(lds_bytes);
        std::vector<xgemm_trace_event> ev;
        for (int tid = 0; tid < threads; ++tid) {
            ev.clear();
            const TraceOps ops{lds.data(), &ev, &split};
            body(ops, tid);
            counts[tid] = (int64_t)ev.size();
            const int64_t n = counts[tid] < capacity ? counts[tid] : capacity;
            if (n > 0)
                memcpy(out + (int64_t)tid * capacity, ev.data(), (size_t)n * sizeof(xgemm_trace_event));
        }
        return (int)XGEMM_OK;
    };
    if (g.sk) {
        const xgemm_dev::SkParams q = sk_params(g, (int *)W, (float *)wdata);
        const int lw = xgemm_dev::sk_logical((int)block, q.grid);
        split.tail = q.flags ? q.flags + lw : nullptr;
        split.head = q.flags ? q.flags + lw + 1 : nullptr;
        return trace_threads(xgemm_dev::sk_lds_bytes<kSkBM, kSkBN, kDmaBK>(), [&](const TraceOps &ops, int tid) {
            xgemm_dev::sk_tile<kSkBM, kSkBN, kDmaBK, kSkWGM, kSkWGN, 0>(ops, q, (int)block, tid);
        });
    }
    if (g.dma)
        return with_dma_tile(plan.tile, [&](auto t) {
            using T = decltype(t);
            return trace_threads(xgemm_dev::dma_lds_bytes<T::BM, T::BN, T::BK, T::STAGES>(),
                                 [&](const TraceOps &ops, int tid) {
                                     xgemm_dev::dma_tile<T::BM, T::BN, T::BK, T::STAGES, T::WGM, T::WGN, 0,
                                                         T::MI, T::KW>(ops, g.p, (int)block, (int)g.grid, tid);
                                 });
        });
    return with_general_tile(plan.tile, [&](auto t) {
        using T = decltype(t);
        return trace_threads(xgemm_dev::general_lds_bytes<T::BM, T::BN, T::BK>(), [&](const TraceOps &ops, int tid) {
            xgemm_dev::general_tile<T::BM, T::BN, T::BK, T::WGM, T::WGN, 0>(ops, g.p, (int)block, (int)g.grid, tid);
        });
    });
}

int xgemv_run(xgemm_handle_t h, int64_t M, int64_t K, const float *A, int64_t lda, const float *x, float *y,
              void *stream)
{
    return run_gemv(h, M, K, A, lda, x, y, stream, nullptr);
}

int xgemv_run_config(xgemm_handle_t h, int64_t M, int64_t K, const float *A, int64_t lda, const float *x,
                     float *y, void *stream, const xgemv_config *cfg)
{
    if (!cfg)
        return XGEMM_ERR_INVALID_ARG;
    return run_gemv(h, M, K, A, lda, x, y, stream, cfg);
}

int xgemv_select_config(int64_t M, int64_t K, int cu_count, xgemv_config *out)
{
    if (!out || M < 0 || K < 0 || cu_count < 1)
        return XGEMM_ERR_INVALID_ARG;
    select_gemv(M, K, cu_count, out);
    return XGEMM_OK;
}

int xgemv_trace_workgroup(int64_t M, int64_t K, const float *A, int64_t lda, const float *x, float *y, float *W,
                          const xgemv_config *cfg, int64_t block, xgemm_trace_event *out, int64_t capacity,
                          int64_t *counts)
{
    if (!counts || capacity < 0 || (capacity > 0 && !out) || !valid_gemv_config(cfg) || M <= 0 || K <= 0 ||
        check_gemv_args(M, K, A, lda, x, y) != XGEMM_OK)
        return XGEMM_ERR_INVALID_ARG;
    const GemvParams p = gemv_params(M, K, A, lda, x, y, cfg->rows, cfg->split_k, W);
    if (p.blocks == 0 || block < 0 || block >= p.blocks || (p.split > 1 && !W))
        return XGEMM_ERR_INVALID_ARG;
    return with_gemv_config(*cfg, [&](auto r, auto u) {
        constexpr int R = decltype(r)::value, U = decltype(u)::value;
        std::vector<float> lds(xgemv_dev::kWaves * R);
        std::vector<xgemm_trace_event> ev;
        for (int tid = 0; tid < xgemv_dev::kThreads; ++tid) {
            ev.clear();
            const TraceGemvOps ops{lds.data(), &ev};
            xgemv_dev::gemv_block<R, U>(ops, p, (int)block, tid);
            counts[tid] = (int64_t)ev.size();
            const int64_t n = counts[tid] < capacity ? counts[tid] : capacity;
            if (n > 0)
                memcpy(out + (int64_t)tid * capacity, ev.data(), (size_t)n * sizeof(xgemm_trace_event));
        }
        return (int)XGEMM_OK;
    });
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
