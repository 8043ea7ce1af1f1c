/*
 * nnjit.h -- C-ABI of the lite-space, per-shape tuned MatMul / BatchMatMul /
 * GEMV library for MI355X (gfx950, CDNA4).
 *
 * The operation is the paper's MatMul and BatchMatMul (kernel table, Table 3:
 * "MatMul M,K,N", "BatchMatMul B,M,K,N"): one kernel per operator shape that
 * computes C = A . B.  Which kernel runs is picked from a small, resource-
 * driven "lite" space of tiling configurations and tuned just in time per
 * shape on the device (Sec. 5.2 and its Table 1 formulas and heuristics;
 * candidates are measured on the device and the fastest is kept, Sec. 3).
 *
 * Conventions for every entry point below
 *   - All matrices are row-major.  Element (i, j) of X lives at
 *     X[i * ldx + j]; batch b of a batched operand starts at X + b * strideX
 *     (strides and leading dimensions are in ELEMENTS, not bytes).
 *   - C[i][j] = sum_k A[i][k] * B[k][j]; C is overwritten (no alpha/beta).
 *   - Shapes are passed as (M, N, K): A is M x K, B is K x N, C is M x N.
 *     (The paper writes shapes as [M, K, N]; the order here differs.)
 *   - dtype NNJIT_F32: A, B, C are fp32; products are accumulated in fp32 on
 *     the fp32 matrix cores (v_mfma_f32_*_f32), or in fp32 FMAs for GEMV.
 *     dtype NNJIT_F16: A and B are IEEE binary16, C is fp32, accumulation is
 *     fp32.
 *   - A, B, C are DEVICE pointers owned by the caller; the library never
 *     allocates, frees or retains them beyond the call.
 *   - stream is a hipStream_t (NULL = the default stream).  Launches are
 *     asynchronous on that stream; a fault inside a kernel surfaces at the
 *     caller's next synchronisation, not as a return code.
 *   - Preconditions: M, N, K >= 0 (and < 2^31); batch >= 0; lda >= max(1, K);
 *     ldb >= max(1, N); ldc >= max(1, N); strides >= 0; a NULL pointer is
 *     allowed only for an operand with no elements.  M == 0, N == 0 or
 *     batch == 0 is a no-op that returns NNJIT_OK without touching the GPU;
 *     K == 0 writes zeros to C.  Overlap between C and A/B, or between the C
 *     slices of a batch, is the caller's error and is not detected.
 *   - Arguments are validated before any HIP call, so a process without a GPU
 *     gets an error code (NNJIT_EINVAL / NNJIT_EDTYPE for bad arguments,
 *     NNJIT_EHIP otherwise), never an abort.
 *   - Operands whose base pointers are not 16-byte aligned, or whose leading
 *     dimensions, batch strides, K or N are not multiples of 16 bytes' worth
 *     of elements, run on an element-load fallback configuration (correct,
 *     slower); this is not an error.
 *   - Thread safety: all entry points may be called from several host
 *     threads.  Split-K scratch is kept per (device, stream), so concurrent
 *     calls on different streams do not share it; calls on one stream are
 *     ordered by the stream.  A tune in progress on one thread does not hold
 *     up calls on other threads (it times candidates on its own stream and
 *     scratch).
 *   - Stream capture: a call may be recorded into a HIP graph.  A call whose
 *     configuration needs more split-K scratch than any earlier call on that
 *     stream allocates a larger buffer; the outgrown one is retired, not
 *     freed, so queued launches and graphs captured earlier on the stream stay
 *     valid.  Retired buffers are released by nnjit_cache_clear() (after a
 *     device synchronisation); graphs captured before that call must be
 *     captured again.  During capture a call that would need to grow the
 *     scratch enqueues nothing and returns NNJIT_EHIP: run each shape once on
 *     the stream before capturing it.  Graphs captured on one stream share
 *     that stream's scratch, so they must not be replayed concurrently (on
 *     several streams at once).
 *   - A launch is limited to 2^31 - 1 workgroups (tiles x split x batch slices
 *     of up to 65535): larger problems return NNJIT_EINVAL.
 *   - Errors: a negative return code; nnjit_last_error() gives a message.
 *
 * Environment variables (none is needed; read when the library first
 * initialises a device and again by nnjit_cache_clear(), never per call)
 *   NNJIT_TUNE_BUDGET_MS  wall-time budget of one shape's tuning (default 900)
 *   NNJIT_TUNE_REPS       timed bursts per candidate (default 3)
 *   NNJIT_TUNE_RUNOFF     0 skips the re-timing of the near-best candidates
 *   NNJIT_TUNE_GRAPH      0 times candidates with eager launches instead of
 *                         captured graph bursts
 *   NNJIT_RETUNE          non-zero: tune a shape again even if it is cached
 *   NNJIT_FORCE_CONFIG    configuration id used for every call of its family
 *                         (for experiments; results are the same, speed not)
 *   NNJIT_GROUP_M         tile rows per group of a GEMM's tile order
 *                         (default: chosen per launch; any value gives the
 *                         same results)
 *   NNJIT_LOG, NNJIT_TRACE  non-zero: print each tuned shape / each timed
 *                         candidate to stderr
 *   NNJIT_FAULT_CONFIG    configuration id whose launches fail with
 *                         NNJIT_EHIP before any GPU work (tests of the
 *                         tuner's failure handling)
 */
#ifndef NNJIT_H
#define NNJIT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum nnjit_dtype { NNJIT_F32 = 0, NNJIT_F16 = 1 };

/* Operator kinds: the key "t" (kernel type) of the paper's kernel database
 * (Sec. 5.3).  GEMV is the M == 1, batch == 1 case of MatMul.  GEMV_Q4 is
 * the GEMV of a 4-bit weight-only quantised matrix (nnjit_gemv_q4); every
 * function below that takes (kind, dtype, batch, M, N, K) identifies such a
 * shape as (NNJIT_KIND_GEMV_Q4, NNJIT_F16, group, 1, N, K): the group size
 * stands in the batch position (the product has no batch dimension). */
enum nnjit_kind { NNJIT_KIND_GEMM = 0, NNJIT_KIND_BATCHED = 1, NNJIT_KIND_GEMV = 2, NNJIT_KIND_GEMV_Q4 = 3 };

#define NNJIT_OK 0
#define NNJIT_EINVAL (-1)  /* bad dimension, leading dim, stride, NULL pointer, config id */
#define NNJIT_EDTYPE (-2)  /* dtype is not NNJIT_F32 / NNJIT_F16                         */
#define NNJIT_ENOCFG (-3)  /* no configuration fits (not expected: fallbacks exist)      */
#define NNJIT_EHIP (-4)    /* HIP runtime error, including "no GPU"                     */
#define NNJIT_ENOMEM (-5)  /* device scratch allocation failed                           */

/* C = A . B for one product (MatMul; GEMV when M == 1).  Uses the tuned
 * configuration of this (kind, M, N, K, dtype) on the current device if
 * nnjit_tune() ran for it, else the first configuration of the shape's lite
 * space in evaluation order (the paper's predefined kernel that serves until
 * just-in-time tuning finds a better one, Sec. 3).  Never tunes implicitly.
 * Returns NNJIT_OK or a negative error code. */
int nnjit_matmul(int64_t M, int64_t N, int64_t K,
                 const void *A, int64_t lda,
                 const void *B, int64_t ldb,
                 void *C, int64_t ldc, int dtype, void *stream);

/* C_b = A_b . B_b for b in [0, batch) (BatchMatMul, Table 3).  Operand b
 * starts at A + b * strideA (elements), likewise B and C.  Same rules as
 * nnjit_matmul; the tuned configuration is looked up under kind BATCHED
 * (batch == 1 behaves exactly like nnjit_matmul). */
int nnjit_batched_matmul(int64_t batch, int64_t M, int64_t N, int64_t K,
                         const void *A, int64_t lda, int64_t strideA,
                         const void *B, int64_t ldb, int64_t strideB,
                         void *C, int64_t ldc, int64_t strideC,
                         int dtype, void *stream);

/* nnjit_batched_matmul for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  Same arguments, results and dispatch (tuned, else default
 * configuration; a shape being tuned online is served by its registered
 * configuration without measuring), but split-K partials go to a fixed
 * scratch array of 128 MiB that the library holds on each GPU for the life
 * of the process, and the call makes no allocating HIP call
 * (the first call on a device initialises it, which only takes that array's
 * address).  A configuration that needs more partials than 128 MiB
 * (split-K: S x batch x M x N x 4 bytes; stream-K: 2 x workgroups x Mt x Nt
 * x 4 bytes) is refused with NNJIT_ENOMEM before any launch.  All calls on one GPU share the array: calls that overlap in time
 * on that GPU (on different streams, or replays of captured graphs that run
 * concurrently) race on it and must be ordered by the caller.  Nothing in
 * the scratch needs to start at zero: each call writes every partial it
 * reads. */
int nnjit_batched_matmul_noalloc(int64_t batch, int64_t M, int64_t N, int64_t K,
                                 const void *A, int64_t lda, int64_t strideA,
                                 const void *B, int64_t ldb, int64_t strideB,
                                 void *C, int64_t ldc, int64_t strideC,
                                 int dtype, void *stream);

/* Just-in-time tuning of one shape (Sec. 3 JIT phase, Sec. 5.2 lite space;
 * the problem statement: one kernel per operator shape, Sec. 3):
 * builds the shape's lite space (enumerate the compiled configurations of
 * the kind and dtype, drop those with another setting of a primitive fixed
 * offline, compute each one's Table 1 resource use on this device, prune by
 * the heuristics, order by workgroups per CU, most first, at most 96),
 * times every survivor on device scratch of this exact shape (1 untimed
 * warm-up, 1 single timed launch, then 3 timed bursts of back-to-back
 * launches, each captured as a HIP graph of about 500 us of device work,
 * whose per-launch median is the candidate's cost; a candidate whose single
 * launch is more than 1.5x the fastest single launch so far is dropped; the
 * candidates within 15% of the best are timed again, in turns, and the best
 * of that run-off is kept; about 900 ms of evaluation at most; an M = 1
 * (GEMV) shape is timed on weights streamed from HBM: the weight operand
 * rotates over scratch copies of >= 512 MiB together), keeps the fastest in
 * the per-shape cache and returns its configuration id (>= 0).  The scratch
 * operands hold near-normal values scaled like activations (A) and weights
 * (B).  Synchronous; the stream and the scratch it times on are created and
 * allocated by the call and released before it returns; other threads'
 * calls are not held up meanwhile.  Re-tuning a cached shape replaces the
 * incumbent only if the new winner is at least 3% faster.  Wall time and
 * counts: nnjit_last_tune_stats().  Negative return: error code. */
int nnjit_tune(int64_t M, int64_t N, int64_t K, int dtype);

/* As nnjit_tune, for BatchMatMul shapes (contiguous operands: strideA = M*K,
 * strideB = K*N, strideC = M*N).  batch == 1 is nnjit_tune. */
int nnjit_tune_batched(int64_t batch, int64_t M, int64_t N, int64_t K, int dtype);

/* Run one forced configuration `cfg` -- one point of the kernel space, a
 * setting of each primitive of Table 2 (tiling, staging, unroll, vectorize)
 * plus a split-K factor (split 0 = stream-K, see nnjit_config_info) -- (test
 * and report helper; the candidates the tuner measures, Sec. 5.2): any kind's
 * configuration may be forced as long as it belongs to this dtype; GEMV
 * configurations additionally need batch == 1 and M == 1; a vector-load
 * configuration needs the 16-byte alignment described above.  A mismatch,
 * or a configuration of the 4-bit GEMV family, is NNJIT_EINVAL. */
int nnjit_matmul_config(int cfg, int64_t batch, int64_t M, int64_t N, int64_t K,
                        const void *A, int64_t lda, int64_t strideA,
                        const void *B, int64_t ldb, int64_t strideB,
                        void *C, int64_t ldc, int64_t strideC,
                        int dtype, void *stream);

/* y = x . W for a 4-bit weight-only quantised W (the 4-bit Llama-2-7B
 * decode workload of Sec. 7, whose quantisation format the paper does not
 * give; this library reads it as a linear layer's weight: one row per output
 * n, symmetric 4-bit codes with one fp16 scale per output and group of
 * `group` consecutive inputs):
 *     W[k][n] = (q[n][k] - 8) * scales[n * lds + k / group]
 *     q[n][k] = (Wq[n * ldq + k / 8] >> (4 * (k % 8))) & 15
 *     y[n]    = sum_k x[k] * W[k][n],   0 <= n < N,  0 <= k < K
 * x: IEEE binary16 [K]; Wq: uint32 words, N rows of ldq words, eight codes
 * per word along k, low nibble first; scales: binary16, N rows of lds;
 * y: fp32 [N], overwritten.  Products are exact, sums in fp32 in a fixed
 * order, so results are deterministic.
 * Preconditions: N, K >= 0 (< 2^31); group >= 1; ldq >= ceil(K / 8);
 * lds >= ceil(K / group); NULL only for an operand with no elements.  N == 0
 * is a no-op; K == 0 writes zeros.  All pointers are DEVICE pointers owned by
 * the caller.  Errors: NNJIT_EINVAL for bad arguments, as for nnjit_matmul.
 * 16-byte loads are used when group % 32 == 0, ldq % 4 == 0 and x, Wq are
 * 16-byte aligned; otherwise a word-load configuration runs (correct,
 * slower).  Uses the tuned configuration of (N, K, group) if
 * nnjit_tune_gemv_q4 ran for it, else the first of its lite space; online
 * tuning (nnjit_set_online) applies as for nnjit_matmul. */
int nnjit_gemv_q4(int64_t N, int64_t K, int64_t group, const void *x, const void *Wq, int64_t ldq,
                  const void *scales, int64_t lds, void *y, void *stream);

/* Just-in-time tuning of a 4-bit GEMV shape, as nnjit_tune (the weights
 * and scales are timed streamed from HBM, rotating over copies of >= 512 MiB
 * together).  Returns the chosen configuration id or an error code. */
int nnjit_tune_gemv_q4(int64_t N, int64_t K, int64_t group);

/* nnjit_gemv_q4 with a forced configuration `cfg` of the 4-bit GEMV family
 * (test and report helper); another family's id, or a 16-byte-load
 * configuration for operands that do not meet its conditions, is
 * NNJIT_EINVAL. */
int nnjit_gemv_q4_config(int cfg, int64_t N, int64_t K, int64_t group, const void *x, const void *Wq, int64_t ldq,
                         const void *scales, int64_t lds, void *y, void *stream);

/* Number of compiled configurations (ids are 0 .. n-1, fixed for a build):
 * the offline-compiled set from which every shape's lite space is drawn
 * (Sec. 5.1: consistent primitives fixed offline; Sec. 5.2: the per-shape
 * lite space). */
int nnjit_num_configs(void);

/* Writes a one-line description of configuration `cfg` -- its primitive
 * settings (Table 2: tile extents, K slab, staging, LDS layout, unroll,
 * vector width) and its Table 1 inputs -- into buf (at most len bytes
 * including the terminating NUL); split=0 marks a stream-K configuration
 * (the tiles' K slabs cut evenly over one workgroup per resident slot,
 * shared tiles summed by a fix-up kernel in workgroup order), e.g.
 * "id=12 family=gemm_f32 name=... mfma=32x32x2 Mt=128 Nt=64 Kt=16 waves=2x2
 *  stages=2 prefetch=2 vec=16 split=4 threads=256 lds=...".  Returns the full length of the
 * description, or NNJIT_EINVAL. */
int nnjit_config_info(int cfg, char *buf, int64_t len);

/* Device description used by the resource model (Table 1's hardware
 * constants, mapped to one CDNA4 compute unit). */
typedef struct nnjit_device_limits {
    int num_cus;             /* compute units (MI355X: 256)                      */
    int simds_per_cu;        /* 4                                                */
    int vgprs_per_lane;      /* unified VGPR+AGPR file per SIMD lane (gfx950: 512) */
    int vgpr_granule;        /* allocation granule (8)                           */
    int max_waves_per_simd;  /* wave slots per SIMD (8)                          */
    int wave_size;           /* 64                                               */
    int64_t lds_per_cu;      /* bytes (gfx950: 163840)                           */
    int64_t lds_per_wg;      /* bytes a workgroup may allocate (163840)          */
    int max_threads_per_wg;  /* 1024                                             */
} nnjit_device_limits;

/* Table 1 quantities of one configuration on a device. */
typedef struct nnjit_resources {
    int regs_per_lane;   /* Reg_thread: VGPR+AGPR per lane (measured if available) */
    int regs_measured;   /* 1 if regs_per_lane came from the compiled kernel      */
    int64_t lds_per_wg;  /* L1_block: LDS bytes of one workgroup                  */
    int threads_per_wg;  /* Thread_block                                         */
    int waves_per_wg;    /* Warp_block                                           */
    int reg_limit;       /* RegLimit:  workgroups per CU the register file allows */
    int lds_limit;       /* L1Limit:   workgroups per CU the LDS allows           */
    int wave_limit;      /* WarpLimit: workgroups per CU the wave slots allow     */
    int wg_per_cu;       /* Block_core = min(RegLimit, L1Limit, WarpLimit)        */
} nnjit_resources;

/* Resource use of configuration `cfg` on `dev` (NULL: the current GPU, which
 * also supplies the compiled kernel's measured register count).  Host-only
 * when dev != NULL: no HIP call is made. */
int nnjit_config_resources(int cfg, const nnjit_device_limits *dev, nnjit_resources *out);

/* The lite space of a shape: writes up to `cap` configuration ids, in
 * evaluation order, into `ids` and returns the size of the lite space (the
 * survivors of pruning, at most the first 96 in evaluation order; may exceed
 * cap).  *n_enumerated (if not NULL) receives the number of
 * compiled configurations of the kind and dtype that were considered, and
 * *n_naive the size of the unpruned space over the same parameter axes.
 * With dev != NULL this is pure host code (no GPU needed) and uses estimated
 * register counts; with dev == NULL it uses the current GPU's limits and the
 * compiled kernels' measured registers, as nnjit_tune does. */
int nnjit_lite_space(int kind, int dtype, int64_t batch, int64_t M, int64_t N, int64_t K,
                     const nnjit_device_limits *dev, int *ids, int cap,
                     int *n_enumerated, int64_t *n_naive);

/* Statistics of the last nnjit_tune / nnjit_tune_batched / nnjit_tune_gemv_q4
 * call on this thread (the paper reports tuning time per shape and the size
 * of the space searched, Sec. 7.3 and Table 6): *wall_ms = wall time of the
 * whole call (scratch set-up, evaluation, syncs; 0 on a cache hit beyond the
 * lookup), *n_enum = compiled configurations of the kind and dtype that were
 * considered, *n_pruned = the size of the pruned (lite) space, *n_timed =
 * candidates fully timed.  Any pointer may be NULL.  Returns NNJIT_OK. */
int nnjit_last_tune_stats(double *wall_ms, int *n_enum, int *n_pruned, int *n_timed);

/* The same statistics in full. */
typedef struct nnjit_tune_stats {
    double wall_ms;       /* whole call, including scratch set-up and syncs       */
    double eval_ms;       /* the candidate evaluation loop only                   */
    int n_enumerated;     /* compiled configurations of the kind and dtype        */
    int n_lite;           /* survivors of pruning (the lite space)               */
    int n_timed;          /* candidates fully timed                              */
    int n_aborted;        /* dropped after the warm-up (> 1.5x best)             */
    int n_failed;         /* launch failures (skipped)                           */
    int chosen;           /* configuration id returned                           */
    double best_us;       /* its per-launch time in a burst (median of 3)        */
    double default_us;    /* the same for the first lite-space candidate          */
    int cache_hit;        /* 1 if the shape was already tuned (nothing timed)     */
} nnjit_tune_stats;

/* Copies the full statistics of the last tune on this thread into *out.
 * Returns NNJIT_OK, or NNJIT_EINVAL if out is NULL. */
int nnjit_last_tune_stats_ex(nnjit_tune_stats *out);

/* Best-so-far curve of the last tune on this thread: for the i-th evaluated
 * candidate, its id, its per-launch time in us (or -1 if aborted/failed) and the
 * wall-clock ms since the start of the call.  Returns the number of entries
 * (may exceed cap). */
int nnjit_last_tune_trace(int *ids, double *us, double *at_ms, int cap);

/* Configuration id cached for a shape on the current device, or NNJIT_ENOCFG. */
int nnjit_cached_config(int kind, int dtype, int64_t batch, int64_t M, int64_t N, int64_t K);

/* The ranked candidates kept for a tuned shape (Sec. 5.3: the best kernels of
 * a device are shared with identical devices): up to 5 configuration ids and
 * their measured per-launch times in us, the registered configuration first,
 * then the fastest other candidates.  Writes min(count, cap) entries to ids
 * and us (either may be NULL); returns the count, or NNJIT_ENOCFG if the
 * shape is not tuned on the current device. */
int nnjit_cached_ranked(int kind, int dtype, int64_t batch, int64_t M, int64_t N, int64_t K, int *ids, double *us,
                        int cap);

/* Online just-in-time tuning (Sec. 3: while the application runs, candidates
 * are measured between inferences and a significantly faster one is
 * re-registered).  With enable = 1, an untuned shape is not served by its
 * default configuration alone: each nnjit_matmul / nnjit_batched_matmul call
 * on it runs the next candidate of its lite space -- every configuration
 * computes the same product, so the call's result is the caller's result --
 * timed by HIP events on the caller's stream and read back by a later call
 * (never waited for).  A candidate at least 3% faster than the registered one
 * replaces it; once every candidate has been measured the shape is cached as
 * if nnjit_tune had run.  Calls during stream capture, calls whose operands
 * need the element-load path and calls made while a measurement is still in
 * flight are served by the registered configuration without measuring.  With
 * enable = 0 no new measurement starts (shapes in progress keep their
 * registered configuration).  Off by default.  Returns the previous setting. */
int nnjit_set_online(int enable);

/* Online progress of a shape on the current device: 0 while it is being tuned
 * online (*measured candidates of *total so far, *registered = the
 * configuration serving calls), 1 once it is tuned (*registered = its cached
 * configuration), NNJIT_ENOCFG if neither.  Output pointers may be NULL. */
int nnjit_online_status(int kind, int dtype, int64_t batch, int64_t M, int64_t N, int64_t K, int *measured,
                        int *total, int *registered);

/* Forget every tuned shape (the per-shape cache of Sec. 5.3), release the
 * outgrown split-K buffers (after a device synchronisation; graphs captured
 * before must be captured again) and read the environment overrides again.
 * Returns NNJIT_OK. */
int nnjit_cache_clear(void);

/* Persistent kernel database (the paper's kernel database keyed by kernel
 * type, shape and device, Sec. 5.3): write every tuned shape of every
 * initialised device to a text file at `path` (one line per shape: device
 * signature = architecture name and CU count, kind, dtype, batch, M, N, K,
 * then up to 5 ranked candidates as configuration name, split, measured
 * time -- the registered one first).  Configurations are stored by name,
 * not id, so a file stays valid across builds that reorder the table.
 * Returns the number of entries written, or NNJIT_EINVAL / NNJIT_EHIP. */
int nnjit_cache_save(const char *path);

/* Read such a file into the per-shape cache of the current device: entries
 * for another device signature, unknown configuration names, configurations
 * that do not fit the entry's kind and dtype, and malformed lines are skipped
 * (a line whose first candidate is unknown is skipped whole; unknown later
 * candidates are dropped).  Loading merges: a shape already in the cache
 * keeps whichever entry has the faster measured time, so databases from
 * identical devices can be loaded one after another.  Returns the number of
 * valid entries read (>= 0), or NNJIT_EINVAL (unreadable file) / NNJIT_EHIP. */
int nnjit_cache_load(const char *path);

/* Measurement helper: reads `bytes` of device memory at `src` once, with
 * 16-byte non-temporal loads (the GEMVs read their weights the same way)
 * from `workgroups` workgroups of 256 threads, and writes
 * (practically) nothing -- at most one word per workgroup into `sink`
 * (device memory of `workgroups` 32-bit words).  Timed around it, this is
 * what one launch can stream from HBM, the reference against which the
 * bandwidth-bound GEMV launches are set.  Preconditions: bytes >= 0 and a
 * multiple of 16; src 16-byte aligned (NULL only when bytes == 0);
 * 1 <= workgroups <= 2^20.  Asynchronous on stream.  Returns NNJIT_OK,
 * NNJIT_EINVAL or NNJIT_EHIP. */
int nnjit_stream_read(const void *src, int64_t bytes, void *sink, int workgroups, void *stream);

/* Message for the last error on this thread ("" if none).  The pointer stays
 * valid until the next nnjit_* call on the same thread. */
const char *nnjit_last_error(void);

/* Library version, (major << 16) | minor. */
int nnjit_version(void);

#ifdef __cplusplus
}
#endif

#endif /* NNJIT_H */
