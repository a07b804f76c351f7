/*
 * xgemm: dense matrix multiply C = A * B on an AMD Instinct MI355X (gfx950).
 *
 * A is M x K and B is K x N, both stored as 16-bit floating point (bfloat16 or
 * IEEE binary16, the same type for both); C is M x N in fp32.  Products are
 * accumulated in fp32 on the matrix (MFMA) units.  All matrices are row-major:
 *
 *     A[i][k] = A[i * lda + k]     B[k][j] = B[k * ldb + j]     C[i][j] = C[i * ldc + j]
 *
 * with leading dimensions counted in elements.  This is the plain sequential
 * GEMM the paper starts every schedule from (Introduction; Section 2.3, chain
 * of equivalence): C[i][j] = sum over k of A[i][k] * B[k][j].  The call
 * overwrites C (no alpha/beta).  The kernels the paper builds from it, a
 * non-split and a split-k GEMM (Section 6), correspond here to split_k = 1
 * and split_k > 1.
 *
 * Accuracy contract: for every (i, j),
 *     |C[i][j] - exact| <= 1e-4 * sum_k |A[i][k] * B[k][j]|
 * where "exact" is the real-number result on the stored input values.
 *
 * Error behaviour: every entry point returns an xgemm_status; no entry point
 * aborts or throws.  A call that fails validation or allocation
 * (XGEMM_ERR_INVALID_ARG, XGEMM_ERR_UNSUPPORTED, XGEMM_ERR_ALLOC) enqueues
 * nothing.  XGEMM_ERR_HIP from a kernel launch may come after launches the
 * same call had already enqueued (operand copies, the body of a banded call);
 * the stream's work is then incomplete and C undefined.
 * Memory ownership: A, B and C are device pointers owned by the caller; the
 * library never frees them nor keeps them past the call.  The library owns
 * only the handle and the workspace inside it (split-k partials and copies
 * of operands the fast kernels cannot read in place).
 */
#ifndef XGEMM_H
#define XGEMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct xgemm_ctx *xgemm_handle_t;

/* Storage type of A and B. */
enum xgemm_dtype {
    XGEMM_BF16 = 0, /* bfloat16: 1 sign, 8 exponent (bias 127), 7 fraction bits */
    XGEMM_FP16 = 1  /* IEEE binary16: 1 sign, 5 exponent (bias 15), 10 fraction bits */
};

enum xgemm_status {
    XGEMM_OK = 0,
    XGEMM_ERR_INVALID_ARG = 1, /* bad size, leading dimension, pointer, dtype or config */
    XGEMM_ERR_UNSUPPORTED = 2, /* the current device is not a gfx950 GPU */
    XGEMM_ERR_ALLOC = 3,       /* the handle's workspace could not be allocated */
    XGEMM_ERR_HIP = 4          /* a HIP runtime call failed; see xgemm_last_error */
};

/* Output-tile shapes the kernels are built for (rows x columns of C per workgroup). */
enum xgemm_tile {
    XGEMM_TILE_256x256 = 0,
    XGEMM_TILE_256x128 = 1,
    XGEMM_TILE_128x128 = 2,
    XGEMM_TILE_COUNT = 3
};

/*
 * A launch configuration.  The paper tries, per problem size, the non-split
 * kernel and split-k factors 1, 2, 4, 8 and 16 and keeps the fastest
 * (Section 6); here the selector picks one from the problem shape and the
 * device's compute-unit count, and xgemm_run_config lets a caller force one.
 */
typedef struct xgemm_config {
    int32_t tile;       /* an xgemm_tile value */
    int32_t split_k;    /* number of K partitions, 1 .. 64; > 1 uses the workspace */
    int32_t group_m;    /* tile rows per group in the launch order, 1 .. 64 (L2 locality) */
    int32_t stream_k;   /* 0: one workgroup per output tile (and K partition).  1: the
                           persistent stream-K kernel with one workgroup per CU; n in
                           2 .. 1023: the same kernel with n workgroups.  Only with split_k == 1
                           and the 256 x 256 tile, for M and N multiples of 256, K a multiple of
                           64, at least as many tiles as workgroups, A and B read in place by the
                           pipelined kernel, C 16-byte aligned with ldc a multiple of 4 and
                           256 * ldc * 4 < 2^32 bytes; otherwise the tile's ordinary kernel runs.
                           See XGEMM_KERNEL_PERSISTENT. */
} xgemm_config;

/*
 * Create a handle bound to the calling thread's current HIP device.  Caches
 * the device's compute-unit count and architecture and creates one HIP event
 * (for ordering workspace users across streams); allocates no device
 * memory.  Returns XGEMM_ERR_UNSUPPORTED if the device is not gfx950,
 * XGEMM_ERR_HIP if no device is usable, XGEMM_ERR_INVALID_ARG if out is NULL.
 * The caller owns *out and releases it with xgemm_destroy.
 */
int xgemm_create(xgemm_handle_t *out);

/*
 * Release a handle, its workspace and its event.  NULL is accepted (no-op).
 * Work that uses the handle's workspace must have completed (synchronize
 * the streams it was enqueued on first).
 */
int xgemm_destroy(xgemm_handle_t h);

/*
 * Cap the device memory the handle's workspace may hold at `bytes` (0, the
 * default: no cap).  A later call that needs a larger workspace returns
 * XGEMM_ERR_ALLOC and enqueues nothing, as when hipMalloc fails; a
 * workspace already larger than the cap is kept.  For callers that budget
 * device memory.  XGEMM_ERR_INVALID_ARG for a NULL handle.
 */
int xgemm_set_workspace_limit(xgemm_handle_t h, size_t bytes);

/*
 * enable = 0: the plans this handle selects (xgemm_run, xgemm_run_noalloc,
 * xgemm_run_strided_batched) never use the persistent kernel, and take the
 * plan they would take without it (banded or not); enable = 1 (the
 * default): they use it where xgemm_select_band says.  For callers that
 * budget workspace (the persistent kernel's shared tiles need 2 x 256 KiB of
 * partial sums per CU) or compare plans.  xgemm_run_config is not affected.
 * XGEMM_ERR_INVALID_ARG for a NULL handle or another value of enable.
 */
int xgemm_set_persistent(xgemm_handle_t h, int enable);

/*
 * C = A * B, row-major, enqueued asynchronously on `stream` (a hipStream_t;
 * NULL means the default stream).  C is complete once the stream has been
 * synchronized.  Arguments:
 *   M, N, K      sizes, each >= 0.  M == 0 or N == 0: no-op.  K == 0: C is
 *                set to zero (the empty sum).
 *   A, lda       device pointer to M x K values, lda >= K
 *   B, ldb       device pointer to K x N values, ldb >= N
 *   C, ldc       device pointer to M x N floats, ldc >= N; C must not overlap
 *                A or B
 *   dtype        XGEMM_BF16 or XGEMM_FP16 (applies to A and B)
 * A pointer may be NULL only when its matrix has no elements.  Aligned fast
 * path: A, B 16-byte aligned, lda, ldb, K and N multiples of 8 (C: 16-byte
 * aligned with ldc a multiple of 4 for vector stores).  Any other layout is
 * still correct: the operands that miss these conditions are first copied,
 * zero-padded, into the handle's workspace (M x K rounded up to 8 for A, K x N
 * both rounded up to 8 for B; both when K is not a multiple of 8), or, where
 * K is too short for the pipelined kernels (under about 3 steps of 64 per
 * split), read in place by a slower element-wise kernel.  Sizes are limited
 * to M, N, K < 2^31 with every matrix addressable in 64-bit element offsets.  A handle holds one workspace
 * (split-k partials and operand copies), grown on demand with hipMalloc
 * (XGEMM_ERR_ALLOC if that fails).  Calls that share a handle may be
 * enqueued on different streams, and never overlap on the workspace: while
 * all of a handle's workspace users come on one stream its order suffices;
 * the first such call on another stream waits on the host for the device to
 * finish its work (hipDeviceSynchronize, so not inside a graph capture);
 * from then on each such call records an event on its stream and the next
 * one on another stream makes its stream wait for it.  A buffer being grown
 * is freed only after its last user has completed.  Calls on different
 * streams run concurrently only with one handle per stream.  A handle must not be used by two host threads at
 * once.  The configuration comes from the problem shape and the
 * device's CU count (xgemm_select_band: one plan, or a body and a band of C
 * launched one after the other).
 */
int xgemm_run(xgemm_handle_t h, int64_t M, int64_t N, int64_t K,
              const void *A, int64_t lda, const void *B, int64_t ldb,
              float *C, int64_t ldc, int dtype, void *stream);

/*
 * For callers that cannot allocate device memory: code being captured into
 * a HIP graph, tight serving loops, harnesses that forbid hipMalloc.  The
 * same product as xgemm_run, with the same plan, kernels and arguments, and
 * the same result bit for bit, but the split-k partials, the persistent
 * kernel's partial sums and counters, and operand copies live in a static
 * array of the library (XGEMM_NOALLOC_SCRATCH_BYTES per GPU, held from the
 * first xgemm_create on that GPU until the process ends) instead of the
 * handle's workspace.  One exception: where xgemm_run's plan is the
 * persistent kernel with shared tiles whose partial sums do not fit the
 * array, the call takes the plan xgemm_run would take without that kernel
 * (banded or not); its result agrees with xgemm_run's within the accuracy
 * contract, not necessarily in the last bits.  The call allocates nothing
 * and frees nothing; the library keeps the array's counters at zero between
 * calls, and nothing else in it needs to start at zero.  Every call of this
 * entry point on one GPU shares that GPU's array, so calls that overlap in
 * time on one GPU (on different streams, or through different handles) race
 * and must be ordered by the caller.  Returns XGEMM_ERR_INVALID_ARG, with
 * nothing enqueued and the reason in xgemm_last_error, when the call needs
 * more than XGEMM_NOALLOC_SCRATCH_BYTES of scratch (a split-k plan or
 * operand copies too large for it); other errors as xgemm_run.
 */
#define XGEMM_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int xgemm_run_noalloc(xgemm_handle_t h, int64_t M, int64_t N, int64_t K,
                      const void *A, int64_t lda, const void *B, int64_t ldb,
                      float *C, int64_t ldc, int dtype, void *stream);

/*
 * As xgemm_run, with the launch configuration forced to *cfg (validated:
 * XGEMM_ERR_INVALID_ARG for an unknown tile, split_k, group_m or stream_k
 * out of range, or stream_k > 0 together with split_k > 1).  Results agree
 * with xgemm_run within the accuracy contract; only the summation grouping
 * differs.
 */
int xgemm_run_config(xgemm_handle_t h, int64_t M, int64_t N, int64_t K,
                     const void *A, int64_t lda, const void *B, int64_t ldb,
                     float *C, int64_t ldc, int dtype, void *stream,
                     const xgemm_config *cfg);

/*
 * Strided batched product: for b = 0 .. batch-1,
 *     C + b*stride_c  =  (A + b*stride_a) * (B + b*stride_b)
 * each problem M x N x K as in xgemm_run (row-major, leading dimensions
 * lda, ldb, ldc).  Strides are in elements; stride_a or stride_b may be 0
 * (one A or B shared by every problem), but the outputs must not overlap:
 * stride_c >= (M-1)*ldc + N when batch > 1.  batch == 0: no-op.  The
 * paper's benchmarks include such batched products (its comparison uses a
 * strided-batched vendor GEMM with batch count L, Section 6).  All problems
 * run in one launch without split-k; the pipelined path additionally needs
 * stride_a and stride_b multiples of 8 (vector stores of C: stride_c a
 * multiple of 4).  Operands that miss the layout are copied into the
 * handle's workspace as in xgemm_run, one copy per problem (one in all for
 * a stride of 0), which needs batch times the operand's padded size.
 * Errors as xgemm_run, plus XGEMM_ERR_INVALID_ARG for negative batch or
 * strides, overlapping outputs or batch > 2^31 - 1.
 */
int xgemm_run_strided_batched(xgemm_handle_t h, int64_t batch, int64_t M, int64_t N, int64_t K,
                              const void *A, int64_t lda, int64_t stride_a,
                              const void *B, int64_t ldb, int64_t stride_b,
                              float *C, int64_t ldc, int64_t stride_c, int dtype, void *stream);

/*
 * The configuration xgemm_run would use for this problem on a device with
 * `cu_count` compute units (host-only; touches no GPU).  Returns
 * XGEMM_ERR_INVALID_ARG for negative sizes, an unknown dtype, cu_count < 1 or
 * out == NULL.
 */
int xgemm_select_config(int64_t M, int64_t N, int64_t K, int dtype, int cu_count,
                        xgemm_config *out);

/*
 * Body + band plans.  xgemm_run may cut C in two when the selected
 * configuration would end in a partial round of workgroups: a body of whole
 * rounds of one tile shape, and a band (the columns on the right or the rows
 * at the bottom) with a configuration of its own.  The two run one after the
 * other on the stream, each as xgemm_run_config would run it on that
 * sub-matrix, so each output element is still a single sum over K.
 * xgemm_run_config never bands.
 */
enum xgemm_band_axis {
    XGEMM_BAND_NONE = 0,    /* one plan over all of C */
    XGEMM_BAND_COLUMNS = 1, /* body: columns [0, extent); band: columns [extent, N) */
    XGEMM_BAND_ROWS = 2     /* body: rows [0, extent); band: rows [extent, M) */
};

typedef struct xgemm_band {
    int32_t axis;       /* an xgemm_band_axis value */
    int32_t reserved;   /* 0 */
    int64_t extent;     /* columns or rows of C in the body (0 with XGEMM_BAND_NONE) */
    xgemm_config body;  /* the body's configuration; with XGEMM_BAND_NONE, the whole call's
                           (as xgemm_select_config, with stream_k = 1 where the call runs the
                           persistent kernel: the 256 x 256 tile in four or more whole
                           rounds of CUs, or three or more and a half) */
    xgemm_config band;  /* the band's configuration (zeros with XGEMM_BAND_NONE) */
} xgemm_band;

/*
 * The plan xgemm_run would use for this problem on a device with cu_count
 * compute units (host-only; touches no GPU).  A persistent plan
 * (body.stream_k = 1) becomes the plan without the persistent kernel when
 * the operands' alignment or leading dimensions do not suit that kernel.  XGEMM_ERR_INVALID_ARG for
 * negative sizes, an unknown dtype, cu_count < 1 or out == NULL.
 */
int xgemm_select_band(int64_t M, int64_t N, int64_t K, int dtype, int cu_count, xgemm_band *out);

/*
 * As xgemm_select_band, for a handle whose persistent kernel is switched on
 * (persistent = 1: the same as xgemm_select_band) or off (0, see
 * xgemm_set_persistent).  XGEMM_ERR_INVALID_ARG as xgemm_select_band, or for
 * another value of persistent.
 */
int xgemm_select_plan(int64_t M, int64_t N, int64_t K, int dtype, int cu_count, int persistent, xgemm_band *out);

/*
 * Workgroup tile of a tile id: rows (bm), columns (bn), K step (bk) and
 * threads per workgroup of its pipelined kernel (the general kernel, taken
 * for shapes or alignments the pipelined one does not cover, may use another
 * count: xgemm_trace_plan reports the launched one).  Host-only.
 * XGEMM_ERR_INVALID_ARG for an unknown id or a NULL output pointer.
 */
int xgemm_tile_info(int tile, int *bm, int *bn, int *bk, int *threads);

/* Kernel families (see xgemm_kernel_family). */
enum xgemm_kernel_family_id {
    XGEMM_KERNEL_GENERAL = 0,    /* any shape and alignment; element-wise edge handling */
    XGEMM_KERNEL_PIPELINED = 1,  /* direct global-to-LDS loads, multi-stage LDS pipeline */
    XGEMM_KERNEL_PERSISTENT = 2  /* the pipelined 256 x 256 schedule as a persistent stream-K
                                    kernel.  The paper's kernels are persistent, handing out
                                    output tiles from a task generator (Section 4.2), and it
                                    blames the variation on small and long-K problems on wave
                                    quantisation (Section 6).  Each workgroup takes whole tiles in
                                    rounds, then an equal share of the remaining tiles' K steps, so
                                    no CU idles in a partial last round; a tile split between two
                                    workgroups is finished by whichever completes second, which
                                    adds the other's partial sum in a fixed order (the tile's first
                                    K steps plus its last), without waiting on it.  The LDS
                                    pipeline runs across a workgroup's tiles and a finished tile's
                                    stores overlap the next tile's first MFMAs.  The workspace
                                    holds two partial sums per workgroup (2 x 256 x 256 floats)
                                    when tiles are split. */
};

/*
 * Which kernel family xgemm_run_config would launch for these arguments
 * (host-only; A and B are only inspected for their alignment).  The
 * pipelined family reads A and B 16-byte aligned with lda, ldb, N and K
 * multiples of 8 (B's rows readable to a multiple of 8 columns) and needs
 * at least 3 K steps of 64 in every split, a partial last step counting;
 * operands that miss the layout are first copied into the workspace
 * (xgemm_run), so the general family remains only for too few K steps or
 * tiles whose byte offsets exceed 32 bits.  Returns -1 for M, N or K <= 0,
 * leading dimensions too small, or an invalid cfg.
 */
int xgemm_kernel_family(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                        const void *B, int64_t ldb, const xgemm_config *cfg);

/*
 * Bytes of workspace xgemm_run_config allocates for this problem and cfg on
 * a device with cu_count compute units, for 16-byte aligned A and B with
 * lda = K and ldb = N: a 4096-byte prefix of counters (for the persistent
 * kernel's split tiles, zeroed when the workspace is allocated and left zero
 * by every call), then split_k * M * ceil(N/4)*4 floats when split_k > 1, the
 * persistent kernel's partial sums when it splits tiles, plus the operand
 * copies when K or N is not a multiple of 8 (each 256-byte aligned, after the
 * partials); 0 when nothing is needed.  Host-only.  Returns 0 for invalid
 * arguments.
 */
size_t xgemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int cu_count, const xgemm_config *cfg);

/*
 * Synchronisation traces (host-only; touch no GPU).
 *
 * The paper checks its kernels' synchronisation by running an abstract
 * machine over the program with concrete sizes: every shared-memory access
 * leaves a read or mutate record, and fences, arrivals and waits raise the
 * visibility of those records (Section 5, Abstract Machine).  These entry
 * points provide the input for such a check of this library: they run the
 * kernels' own bodies on the host, for one workgroup of a planned launch
 * (either kernel family), with every hardware operation recorded as an
 * event instead of executed.  A, B, C and W are only used as addresses
 * (never dereferenced), so any values that satisfy the alignment of a real
 * call may be passed.
 */

/* Event kinds of a workgroup trace. */
enum xgemm_trace_op {
    XGEMM_TRACE_LDS_LOAD = 0,  /* direct global-to-LDS load (vector-memory counter): the lane's
                                  `arg` bytes at global address `addr` land at LDS offset
                                  lds + arg * lane (lane = thread id % 64) */
    XGEMM_TRACE_LDS_READ = 1,  /* LDS read (LDS counter) of `arg` bytes at LDS offset `lds` */
    XGEMM_TRACE_WAIT_VM = 2,   /* s_waitcnt vmcnt(arg): all but the arg most recent vector-memory
                                  operations of the wave have completed */
    XGEMM_TRACE_WAIT_LGKM = 3, /* s_waitcnt lgkmcnt(arg), likewise for LDS operations */
    XGEMM_TRACE_BARRIER = 4,   /* s_barrier across the workgroup */
    XGEMM_TRACE_STORE = 5,     /* global store (vector-memory counter) of `arg` bytes at `addr` */
    XGEMM_TRACE_LDS_WRITE = 6, /* LDS write from registers (LDS counter) of `arg` bytes at `lds` */
    XGEMM_TRACE_LOAD = 7       /* global load into registers (vector-memory counter) of `arg` bytes
                                  at `addr` */
};
/* A lane that takes no part in a lane-masked LDS_READ or LDS_WRITE records lds = -1. */

/* One event of one thread.  LDS offsets count bytes from the start of the
   workgroup's LDS allocation; global addresses are byte addresses. */
typedef struct xgemm_trace_event {
    int32_t op;   /* an xgemm_trace_op */
    int32_t arg;  /* bytes per lane (accesses) or the wait count (waits) */
    int64_t lds;  /* LDS offset (LDS_LOAD: the wave's base; LDS_READ: this lane's) */
    int64_t addr; /* global byte address (LDS_LOAD source, STORE destination) */
} xgemm_trace_event;

/* One kernel launch of a planned call.  Offsets count bytes from W, the
   start of the workspace (its counter prefix comes first). */
typedef struct xgemm_trace_info {
    int32_t segments;        /* GEMM launches in the plan (1) */
    int32_t family;          /* xgemm_kernel_family_id of this launch */
    int32_t reduce;          /* 0: writes C (the persistent kernel: also partial sums in W);
                                1: full-matrix split partials in W, summed by a later launch */
    int32_t threads;         /* threads per workgroup */
    int32_t lds_bytes;       /* LDS bytes per workgroup of the pipelined kernel (else 0) */
    int32_t split;           /* split-k factor of this launch */
    int64_t grid;            /* workgroups in this launch */
    int64_t workspace_bytes; /* bytes of W the whole plan writes */
    int32_t tile_base;       /* the launch covers logical tiles [tile_base, tile_base + tile_count) */
    int32_t tile_count;
    int32_t packed;          /* bit 0: A, bit 1: B is read from a copy in W (see xgemm_run) */
    int32_t k;               /* K as the GEMM kernel sees it (K rounded up to 8 when packed) */
    int64_t lda, ldb;        /* leading dimensions the kernel reads A and B with */
    int64_t a_offset;        /* byte offset of the packed A (M x k, leading dimension lda) in W, or -1 */
    int64_t b_offset;        /* byte offset of the packed B (k x ldb) in W, or -1 */
    int64_t data_offset;     /* byte offset of the workspace's data after the counter prefix: the
                                split partials, or the persistent kernel's partial sums (two of
                                256 x 256 floats per workgroup, in the accumulators' layout) */
    int32_t dp_rounds;       /* persistent kernel: rounds of whole tiles per workgroup */
    int32_t sk_tiles;        /* persistent kernel: tiles shared out as K-step ranges */
    int32_t kt;              /* persistent kernel: K steps per tile */
    int32_t reserved;
} xgemm_trace_info;

/*
 * Launch `segment` (0 .. segments-1) of the plan xgemm_run_config would
 * make for these arguments on a device with cu_count CUs.
 * XGEMM_ERR_INVALID_ARG for invalid arguments (including M, N or K == 0,
 * which launch no GEMM kernel), a segment out of range or info == NULL.
 */
int xgemm_trace_plan(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb,
                     const float *C, int64_t ldc, const xgemm_config *cfg, int cu_count, int segment,
                     xgemm_trace_info *info);

/*
 * Trace of workgroup `block` (0 .. grid-1) of launch `segment`: for each
 * thread t (0 .. threads-1), its events in program order are written to
 * out[t * capacity ...], at most `capacity` of them, and their number to
 * counts[t] (counts has `threads` entries, the caller owns both arrays).  A
 * count above capacity means the trace was cut; call again with a larger
 * capacity (capacity 0 with out == NULL only counts).  W is the workspace
 * address (its start) for launches that write partials (reduce != 0, or the
 * persistent kernel with sk_tiles > 0) or read packed operands
 * (packed != 0), else unused.  `schedule` (0 or 1) matters only to the
 * persistent kernel, whose path through a split tile depends on which
 * workgroup counts in first: 0 traces every split tile's last K steps
 * counting in first (the usual order: they start a workgroup's range while
 * the first steps end the previous one's), 1 its first steps.  Counter reads
 * and atomic adds appear as 4-byte LOAD events, counter resets as STORE.
 * Every kernel family is traced.  XGEMM_ERR_INVALID_ARG as
 * xgemm_trace_plan, or for a block out of range, a schedule other than 0 or
 * 1, counts == NULL, or W == NULL where it is needed.
 */
int xgemm_trace_workgroup(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb,
                          float *C, int64_t ldc, float *W, const xgemm_config *cfg, int cu_count, int segment,
                          int64_t block, int schedule, xgemm_trace_event *out, int64_t capacity, int64_t *counts);

/*
 * Matrix-vector product (GEMV): y = A * x in fp32.
 *
 * The paper's second benchmark beside its GEMMs is a full-precision fp32
 * GEMV that uses no matrix instructions (Section 6).  A is M x K, row-major
 * with leading dimension lda (A[i][k] = A[i * lda + k]); x holds K floats and
 * y receives M floats, both contiguous:
 *
 *     y[i] = sum over k of A[i][k] * x[k]
 *
 * Products and sums are fp32 (fused multiply-adds); the summation is
 * grouped (per-thread partial sums, then a tree, then, with a K split
 * into s ranges, a sum over the ranges), so for every i, with
 * n = 4 * ceil(K / 1024) + 10 roundings on the longest path (which bounds
 * the path 4 * ceil(K / (1024 s)) + 10 + s - 1 of a split, since s never
 * exceeds ceil(K / 1024)),
 *     |y[i] - exact| <= n * 2^-24 * sum_k |A[i][k] x[k]| + (K + 256 s) * 2^-150
 * (up to second-order terms; the last term bounds rounding in the
 * subnormal range, summed over the K + 256 s - 1 operations that form y[i]),
 * where "exact" is the real-number result on the stored inputs.  Subnormal
 * inputs and results are kept, not flushed to zero.
 */

/* GEMV launch configuration: rows of A per 256-thread workgroup (1, 2, 4 or
   8), 16-byte chunks of x each thread loads per loop iteration (1, 2 or 4;
   A's rows are loaded the same number of chunks ahead), and the number of K
   ranges (1 .. 256): with split_k > 1 each workgroup sums one range of its
   rows into the handle's workspace and a second launch adds the ranges'
   partial sums in ascending order, which keeps the GPU busy when M is
   small. */
typedef struct xgemv_config {
    int32_t rows;
    int32_t unroll;
    int32_t split_k;
} xgemv_config;

/*
 * y = A * x, enqueued asynchronously on `stream` (a hipStream_t; NULL means
 * the default stream); y is complete once the stream has been synchronized.
 *   M, K     sizes, each >= 0 and < 2^31.  M == 0: no-op.  K == 0: y = 0.
 *   A, lda   device pointer to M x K floats, lda >= K
 *   x        device pointer to K floats
 *   y        device pointer to M floats; must not overlap A or x
 * A pointer may be NULL only when it addresses no element.  16-byte loads
 * need A and x 16-byte aligned and lda a multiple of 4; any other alignment
 * is still correct through 4-byte loads.  The handle supplies the device's
 * CU count, and its workspace holds the partial sums of a K split
 * (split_k * M floats; ordered across streams as for xgemm_run).  Errors:
 * XGEMM_ERR_INVALID_ARG for a NULL handle, bad sizes or pointers, or a
 * forced configuration whose launch would exceed 2^31 - 1 workgroups
 * (ceil(M / rows) * split_k); XGEMM_ERR_ALLOC if the workspace cannot grow;
 * XGEMM_ERR_HIP if a launch fails.  Nothing is enqueued on a validation or
 * allocation error.
 */
int xgemv_run(xgemm_handle_t h, int64_t M, int64_t K, const float *A, int64_t lda, const float *x, float *y,
              void *stream);

/* As xgemv_run with the configuration forced (XGEMM_ERR_INVALID_ARG for an
   unsupported one).  For a given split_k the result is the same bit for bit
   for every rows and unroll: they change only which workgroup computes a
   row and how far ahead it loads, not its arithmetic. */
int xgemv_run_config(xgemm_handle_t h, int64_t M, int64_t K, const float *A, int64_t lda, const float *x,
                     float *y, void *stream, const xgemv_config *cfg);

/* The configuration xgemv_run uses on a device with cu_count CUs
   (host-only).  XGEMM_ERR_INVALID_ARG for negative sizes, cu_count < 1 or
   out == NULL. */
int xgemv_select_config(int64_t M, int64_t K, int cu_count, xgemv_config *out);

/*
 * Trace of GEMV workgroup `block` (0 .. ceil(M / cfg->rows) * s - 1, s the
 * split left after empty K ranges are dropped) in the format of
 * xgemm_trace_workgroup (256 threads; A, x, y and W, the partial sums of a
 * split, are only used as addresses).  M and K must be > 0.
 * XGEMM_ERR_INVALID_ARG for invalid arguments, a block out of range,
 * counts == NULL, W == NULL with a split, or an unsupported cfg.
 */
int xgemv_trace_workgroup(int64_t M, int64_t K, const float *A, int64_t lda, const float *x, float *y, float *W,
                          const xgemv_config *cfg, int64_t block, xgemm_trace_event *out, int64_t capacity,
                          int64_t *counts);

/* Static description of a status code; never NULL. */
const char *xgemm_strerror(int status);

/*
 * Detail of the last failure recorded on a handle (e.g. the HIP error text),
 * or "" if none.  The string is owned by the handle and valid until the next
 * call on it.  NULL handle: a static string.
 */
const char *xgemm_last_error(xgemm_handle_t h);

#ifdef __cplusplus
}
#endif

#endif /* XGEMM_H */
