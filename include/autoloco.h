/*
 * autoloco.h — C ABI of the AutoLoCo synchronisation-round library for AMD
 * Instinct MI355X (gfx950).
 *
 * One synchronisation round of AutoLoCo (arxiv 2609.36662, "AutoLoCo:
 * Communication Efficient Distributed LLM Training via Adaptive
 * Synchronization") on one GPU that holds all K worker replicas:
 *
 *   Delta_k   = theta - theta_k                       pseudo-gradient of worker k
 *   Delta_bar = (1/K) sum_k Delta_k                   the synchronised average
 *   D = (1/K) sum_k ||Delta_k||^2                     local-drift energy
 *   C = K ||Delta_bar||^2 / (D + eps)                 aggregation coherence
 *   Delta_tilde = Delta_bar / rho  (if normalising)   normalised pseudo-gradient
 *   v' = mu v + Delta_tilde;  d = Delta_tilde + mu v';  theta' = theta - eta d
 *   theta_k <- theta'                                 every worker restarts from theta'
 *
 * (Sec. "Adaptive Interval Selection", eq. adaptive-h-core-diagnostics;
 * Sec. "Outer Optimizer Correction", eqs. normalized-pseudo-gradient and
 * autoloco-corrected-nesterov; Alg. "AutoLoCo outer interval"; App. C.1 for
 * the endpoint disagreement.)  The paper writes the worker count as N; this
 * interface calls it k and uses n for the number of parameters.
 *
 * Device calls run on the HIP stream bound to the context.  Host-only calls
 * (schedule, correction, controller) touch no device.  Device calls that do not
 * return sums to the host only launch kernels on that stream and may be
 * captured into a HIP graph; calls that return sums wait for them and may not.
 *
 * Conventions for every call:
 *   - Return value: AUTOLOCO_OK or a negative autoloco_status.  No call throws,
 *     aborts or exits.  When argument validation fails, no device work is
 *     launched and the outputs are left untouched; autoloco_last_error()
 *     describes the failure.
 *   - Ownership: the caller owns every buffer it passes (device or host) and
 *     keeps it alive until the call's device work has finished.  The library
 *     owns only the context's scratch memory.
 *   - Device buffers are flat, contiguous arrays of n elements, 16-byte
 *     aligned, and must not overlap one another.
 *   - Non-finite values in the data are not an error: they propagate through
 *     the update and are reported as finite = 0 in the statistics.  Values
 *     narrowed to bf16 round to nearest, ties to even; a NaN stays a quiet
 *     NaN (its payload bits are not specified).
 */
#ifndef AUTOLOCO_H
#define AUTOLOCO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Largest worker count: the paper runs 4, 8 and 16 workers. */
#define AUTOLOCO_MAX_K 16

typedef enum {
    AUTOLOCO_OK = 0,
    AUTOLOCO_E_INVALID = -1, /* null pointer, k or n out of range, unknown dtype or flag, or a
                                buffer that is not device memory of the context's device */
    AUTOLOCO_E_ALIGN = -2,   /* a device pointer is not 16-byte aligned */
    AUTOLOCO_E_ALIAS = -3,   /* two device buffers overlap */
    AUTOLOCO_E_DEVICE = -4,  /* the HIP runtime reported an error */
    AUTOLOCO_E_NOMEM = -5,   /* an allocation failed */
    AUTOLOCO_E_STATE = -6    /* call out of order (e.g. controller after its budget) */
} autoloco_status;

typedef enum { AUTOLOCO_F32 = 0, AUTOLOCO_BF16 = 1 } autoloco_dtype;

/* Text of a status code (static storage). */
const char* autoloco_status_string(int status);

/* ------------------------------------------------------------------------ */
/* Context                                                                   */
/* ------------------------------------------------------------------------ */

/* A context binds one device and one HIP stream and owns the scratch memory of
 * the two-stage statistics reduction (per-block fp64 partial sums and the
 * final sums) plus a pinned, coherent host buffer that the reduction writes
 * them to.  One context
 * serves one stream; calls on one context must not overlap.
 *   device: HIP device ordinal.  stream: a hipStream_t of that device, or NULL
 *   for the default stream.  *out receives the context.
 * Errors: E_INVALID (null out, bad ordinal), E_DEVICE, E_NOMEM. */
typedef struct autoloco_ctx autoloco_ctx;
int autoloco_create(int device, void* stream, autoloco_ctx** out);
void autoloco_destroy(autoloco_ctx* ctx);
/* Message of the last failed call on ctx ("" if none).  Valid until the next call. */
const char* autoloco_last_error(const autoloco_ctx* ctx);

/* Record HIP events around the device work of every call made through ctx (on
 * the context's stream: the streaming kernel and, when the call returns sums,
 * the one-workgroup kernel that adds the per-workgroup partials after it) so
 * that autoloco_last_kernel_ms() can report the device time of the most recent
 * call.  Off by default. */
int autoloco_set_timing(autoloco_ctx* ctx, int enable);
/* Device milliseconds of the last timed launch; waits for it to finish.
 * Errors: E_INVALID (null argument), E_STATE (timing off, no timed launch yet,
 * or the last call that launched device work failed after it began),
 * E_DEVICE. */
int autoloco_last_kernel_ms(autoloco_ctx* ctx, float* ms);
/* Cap on the number of workgroups of the streaming kernels, 0..16384 (0 = the
 * default: one workgroup per compute unit from k = 5 with fp32 replicas and
 * from k = 6 with bf16, below that three, or fewer
 * if the fused kernel's register use fits fewer).  The statistics
 * are bit-identical between runs with the same n, k, replica type, device and
 * cap, and between the standalone and the fused call. */
int autoloco_set_grid_limit(autoloco_ctx* ctx, int max_blocks);
/* Workgroups and threads per workgroup a round over n parameters with k
 * replicas of the given type uses. */
int autoloco_launch_shape(const autoloco_ctx* ctx, int64_t n, int32_t k, int32_t replica_dtype,
                          int32_t* blocks, int32_t* threads);

/* ------------------------------------------------------------------------ */
/* Placement of the streamed buffers                                         */
/* ------------------------------------------------------------------------ */

/* Allocates `count` device buffers of `bytes` each (16-byte aligned, not
 * overlapping) for buffers that one kernel streams through at the same time,
 * such as theta, the momentum and the k replicas of a round, placed far apart
 * in the device's physical memory.  On MI355X, streams whose pages lie close
 * together in physical memory collide in the DRAM address mapping: the round's
 * ten concurrent streams (k = 8) run at ~5.1 TB/s when adjacent and at
 * ~6.2 TB/s when spread over the device.  The call fills the free device
 * memory (leaving headroom) with equal slots, keeps `count` slots evenly spaced
 * among them and frees the rest before returning, so other allocations made at
 * the same time may fail transiently; call it at set-up.  With too little free
 * memory to spread, it allocates plainly.  *spread (may be NULL) reports
 * which.  Each buffer is freed with autoloco_free.
 * Errors: E_INVALID (null pointers, count outside 1..64, bytes == 0), E_NOMEM. */
int autoloco_alloc_spread(autoloco_ctx* ctx, int32_t count, size_t bytes, void** out, int32_t* spread);
/* Frees one buffer from autoloco_alloc_spread (NULL is a no-op).  The buffers
 * are not owned by the context that made them: destroying it frees none of
 * them, and any context of the same device may free them.
 * Errors: E_INVALID (null context), E_DEVICE (hipFree failed). */
int autoloco_free(autoloco_ctx* ctx, void* ptr);

/* ------------------------------------------------------------------------ */
/* Device buffers of one round                                               */
/* ------------------------------------------------------------------------ */

/* Every buffer argument of the device calls below must be device (or managed)
 * memory of the context's device; host memory and memory of another device are
 * rejected with E_INVALID before anything is launched.  Element counts n lie in
 * 0..2^56 (E_INVALID otherwise), so no byte count or address the library forms
 * from them overflows. */

typedef struct {
    int64_t n;             /* parameters per buffer, 0 <= n <= 2^56 */
    int32_t k;             /* worker replicas, 1..AUTOLOCO_MAX_K */
    int32_t replica_dtype; /* autoloco_dtype of every replica */
    float* theta;          /* [n] fp32: synchronised parameters theta_t (in/out) */
    float* momentum;       /* [n] fp32: outer momentum v (in/out); unused by stats/reset */
    void* replicas[AUTOLOCO_MAX_K]; /* k x [n] worker endpoints theta_k (read; written by a reset) */
} autoloco_buffers;

/* Sums over all n parameters and the diagnostics derived from them. */
typedef struct {
    double sq_norm[AUTOLOCO_MAX_K]; /* ||Delta_k||^2 */
    double sq_dev[AUTOLOCO_MAX_K];  /* ||Delta_k - Delta_bar||^2 */
    double sq_mean;                 /* ||Delta_bar||^2 */
    double D;                       /* (1/k) sum_k sq_norm[k] */
    double C;                       /* k sq_mean / (D + eps) */
    double disagreement;            /* (1/k) sum_k sq_dev[k]  (= D - sq_mean, App. C.1) */
    int32_t finite;                 /* 1 if every value above is finite */
    int32_t k;
} autoloco_stats;

/* Coefficients of one corrected Nesterov step (see autoloco_outer_correction). */
typedef struct {
    double mu;         /* momentum retention mu_t */
    double eta_out;    /* outer learning rate eta_t */
    double rho;        /* interval ratio rho_t >= 1 */
    double kappa;      /* bounded outer-step scale (reported; not used by the step) */
    int32_t normalize; /* 1: Delta_tilde = Delta_bar / rho; 0: Delta_tilde = Delta_bar */
} autoloco_outer_coeffs;

#define AUTOLOCO_FUSE_STATS 1u /* also compute the round statistics of theta_t */
#define AUTOLOCO_FUSE_RESET 2u /* also write theta_{t+1} into every replica */

/* Statistics of one round (eq. adaptive-h-core-diagnostics; App. C.1):
 * reads theta and the k replicas once, writes nothing but *out.  Blocks until
 * the sums are on the host.  eps > 0 (finite) is the constant in C, so that
 * D = 0 (every replica equal to theta) gives C = 0.  Stats of the same
 * buffers are bit-identical from run to run (fixed reduction order).
 * Errors: E_INVALID, E_ALIGN, E_ALIAS, E_DEVICE. */
int autoloco_round_stats(autoloco_ctx* ctx, const autoloco_buffers* bufs, double eps,
                         autoloco_stats* out);

/* Corrected Nesterov outer step (eq. autoloco-corrected-nesterov, with the
 * normalisation of eq. normalized-pseudo-gradient) in one pass over the
 * buffers: theta and momentum are updated in place from theta_t, v_{t-1} and
 * Delta_bar.  With AUTOLOCO_FUSE_STATS the statistics of theta_t are computed
 * in the same pass (out required; the call then blocks until they are on the
 * host).  With AUTOLOCO_FUSE_RESET every replica is overwritten with
 * theta_{t+1} (bf16 replicas: rounded to nearest even), as each worker starts
 * the next interval from the synchronised parameters (Alg. "AutoLoCo outer
 * interval").  Without FUSE_STATS the call is asynchronous on the stream.
 * The coefficients are applied in fp32 (mu, eta_out and 1/rho rounded once).
 * Errors: E_INVALID (incl. unknown flags, null out with FUSE_STATS, null
 * momentum), E_ALIGN, E_ALIAS, E_DEVICE. */
int autoloco_outer_step(autoloco_ctx* ctx, const autoloco_buffers* bufs,
                        const autoloco_outer_coeffs* coeffs, uint32_t flags, double eps,
                        autoloco_stats* out);

/* The same corrected Nesterov step, with the worker average taken through the
 * INT8 blockwise pseudo-gradient codec of App. G.1 ("Low-precision
 * communication configuration"): every Delta_k is encoded per block of 4,096
 * parameters (FP32 scale = max|Delta_k| / 127, 1 for a zero block and at
 * least 2^-126; codes round-to-nearest-even, clipped to +-127), decoded in
 * FP32, averaged (float64 sum in worker order times 1/K, rounded once to
 * FP32), and the mean is encoded and decoded once more; the step uses that
 * decoded aggregate.  Statistics (FUSE_STATS): sq_norm from the
 * pre-quantisation Delta_k (D), sq_mean from the decoded aggregate (C),
 * sq_dev = ||Delta_k - aggregate||^2.  Blocks run over the flat buffer; the
 * last one is shorter.  mean_codes ([n] int8) and mean_scales
 * ([ceil(n / 4096)] fp32) receive the encoded mean, the payload every worker
 * would receive; pass both or neither (NULL).  Non-finite data propagates and
 * is reported as finite = 0; the codes of such blocks are unspecified.
 * Errors: as autoloco_outer_step, plus E_INVALID for only one payload buffer,
 * E_ALIGN / E_ALIAS for the payload buffers. */
int autoloco_outer_step_int8(autoloco_ctx* ctx, const autoloco_buffers* bufs,
                             const autoloco_outer_coeffs* coeffs, uint32_t flags, double eps,
                             autoloco_stats* out, int8_t* mean_codes, float* mean_scales);

/* The same corrected Nesterov step, with the worker average taken as the
 * paper's main runs communicate it: BF16 pseudo-gradients (Table "Quality and
 * communication cost": payload in full-model BF16 tensors per worker; App.
 * G.1: master parameters, outer reference and momentum stay FP32).  Per
 * parameter: Delta_k = theta - theta_k in FP32, each rounded to BF16 (nearest
 * even); their sum in float64 in worker order times 1/K, rounded to FP32 and
 * then to BF16, is the mean every worker receives, and the step uses it.
 * Statistics (FUSE_STATS): sq_norm from the unrounded Delta_k (D), sq_mean
 * from the received mean (C), sq_dev = ||Delta_k - received mean||^2.
 * mean_bf16 ([n] bf16 bit patterns, 16-byte aligned) receives the received
 * mean, or NULL.  Flags, blocking and non-finite data as autoloco_outer_step.
 * Errors: as autoloco_outer_step, plus E_ALIGN / E_ALIAS for mean_bf16. */
int autoloco_outer_step_bf16(autoloco_ctx* ctx, const autoloco_buffers* bufs,
                             const autoloco_outer_coeffs* coeffs, uint32_t flags, double eps,
                             autoloco_stats* out, uint16_t* mean_bf16);

/* The corrected outer step of autoloco_outer_step, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): no context, and no allocation of any kind
 * (no hipMalloc, no pinned host memory).  The statistics' reduction scratch
 * (per-workgroup partial sums and the final sums: 1,024 workgroups x 33 sums
 * plus 33, 270 KB) is a static device array of the library, one copy per
 * device, held until the process ends; the first call on a device looks up its
 * address with that device current.  The call runs the kernels, launch shape
 * and reduction order of autoloco_outer_step on the same device, so theta',
 * v', the replicas and the statistics equal that call's bit for bit.
 *   device: HIP device ordinal (the call makes it current and restores the
 *     previous one); stream: a hipStream_t of that device, or NULL.
 *   bufs, coeffs, flags, eps, out: as autoloco_outer_step.  With FUSE_STATS the
 *     sums are copied to the calling thread's stack and the call waits for
 *     them; without it the call only launches kernels on the stream.
 * Every call on a device uses that device's one array, and each call writes
 * every word of it that it reads, so nothing needs clearing between calls;
 * calls that overlap in time on one device (from several threads or streams)
 * race on the array and give wrong statistics: serialise them.
 * Errors: E_INVALID (as autoloco_outer_step, a bad device ordinal, or a launch
 * shape of more than 1,024 workgroups, which a device of more than 341
 * compute units would need below k = 8), E_ALIGN, E_ALIAS, E_DEVICE.  There is
 * no context, so no message is kept. */
int autoloco_outer_step_static(int device, void* stream, const autoloco_buffers* bufs,
                               const autoloco_outer_coeffs* coeffs, uint32_t flags, double eps,
                               autoloco_stats* out);

/* Replica reset alone: theta_k <- theta for every replica (Alg. "AutoLoCo
 * outer interval", start of the local loop).  Asynchronous on the stream.
 * Errors: E_INVALID, E_ALIGN, E_ALIAS, E_DEVICE. */
int autoloco_broadcast_reset(autoloco_ctx* ctx, const autoloco_buffers* bufs);

/* Measurement reference for the fused round (no operation of the paper): the
 * memory traffic of autoloco_outer_step with FUSE_STATS | FUSE_RESET and none
 * of its arithmetic.  Same launch shape, same loads and stores in the same
 * order: theta, the momentum and every replica are read once and each word
 * is written back unchanged, so all buffers hold their old contents afterwards
 * (the last n mod 4 parameters are not touched).  Its device time (timing on,
 * autoloco_last_kernel_ms) is what the device sustains for the round's access
 * pattern on these buffers: the practical ceiling of the fused round.
 * Asynchronous on the stream.  Buffers as autoloco_outer_step.
 * Errors: E_INVALID, E_ALIGN, E_ALIAS, E_DEVICE. */
int autoloco_traffic_reference(autoloco_ctx* ctx, const autoloco_buffers* bufs);

/* Streaming-pattern probe (measurement only, no operation of the paper): moves
 * the bytes of `count` streams with no arithmetic, so its device time is what
 * the device sustains for that access pattern on those buffers — for instance
 * the round's ten streams in place, the same buffers read only or written
 * only, or the loads and stores of the reset and of the per-GPU kernels.
 *   streams[s].ptr: device buffer of n elements of streams[s].elem_bytes (4 or
 *     2); 16-byte aligned; no two overlap.
 *   streams[s].access: AUTOLOCO_PROBE_READ, AUTOLOCO_PROBE_WRITE or both (both:
 *     4-byte streams only; each word is written back unchanged).  Written-only
 *     streams receive the words of stream 0 (2-byte streams: the upper halves
 *     of its words) when stream 0 is read, else the index of each run of 4, so
 *     they lose their contents.
 *   The streams come in this order of classes: 4-byte read and written, 4-byte
 *     read, 2-byte read, 2-byte written, 4-byte written; only the class counts
 *     the library instantiates are accepted (E_INVALID otherwise): with
 *     AUTOLOCO_PROBE_RUN1 (the fp32 round's window loop, one run of 4 elements
 *     per lane per window) 1, 2, 4, 6 or 10 streams in place, 1, 2, 4 or 10
 *     read, 1 or 10 written, 5 read and 5 written, 1 read and 1, 2, 4, 8 or 16
 *     written; with AUTOLOCO_PROBE_RUN2 (two runs per lane, 256 runs apart: the
 *     bf16 round's and the per-GPU kernels' shape) 10 in place or read, one 4-byte read
 *     and 1, 4, 8 or 16 2-byte written, two 4-byte read (or one 4-byte and one
 *     2-byte) and one 2-byte written, two 4-byte in place with 1, 2, 4, 8 or 16
 *     2-byte read and one 2-byte written (or, for 4 and 8, none); with
 *     AUTOLOCO_PROBE_RUN8 (eight runs per lane, 256 runs apart: 32 KB of every
 *     4-byte stream per workgroup and window, the standalone reset's shape
 *     with three or more fp32 replicas) 10 in place, read or written, and one
 *     read and 4, 8 or 16 written; with
 *     AUTOLOCO_PROBE_SERIAL (every workgroup stages 16 KB of each read stream
 *     in LDS with direct loads, stream after stream, at most two streams'
 *     loads in flight, then stores stream by stream) and AUTOLOCO_PROBE_TILE
 *     (the same tiles with all streams' loads in flight at once) 10 streams in
 *     place, read, or written; with AUTOLOCO_PROBE_PHASED (read and write
 *     phases of the whole grid: every workgroup loads a tile of 7,168
 *     elements of each stream, 3/7 into LDS and 4/7 into registers, then all
 *     workgroups meet at a grid barrier, store, and meet again; a cooperative
 *     launch, so blocks may not exceed the workgroups resident at once, one
 *     per compute unit) 10 streams in place.  Run shapes skip the last n mod 4
 *     elements, tile shapes the elements past the last whole tile of 4,096,
 *     the phased shape those past the last whole round of tiles over the grid.
 *   blocks: workgroups (256 threads), 0 = one per compute unit.
 *   *bytes (may be NULL) receives the bytes moved (reads plus writes).
 * Asynchronous on the stream and timed like the other calls, except the phased
 * shape: it waits for the kernel, whose grid barriers give up (E_STATE) rather
 * than wait without bound.
 * Errors: E_INVALID, E_ALIGN, E_ALIAS, E_DEVICE, E_STATE. */
#define AUTOLOCO_PROBE_READ 1
#define AUTOLOCO_PROBE_WRITE 2
#define AUTOLOCO_PROBE_RUN1 0
#define AUTOLOCO_PROBE_RUN2 1
#define AUTOLOCO_PROBE_SERIAL 2
#define AUTOLOCO_PROBE_TILE 3
#define AUTOLOCO_PROBE_PHASED 4
#define AUTOLOCO_PROBE_RUN8 5
typedef struct {
    void* ptr;
    int32_t elem_bytes;
    int32_t access;
} autoloco_probe_stream;
int autoloco_traffic_probe(autoloco_ctx* ctx, int64_t n, const autoloco_probe_stream* streams, int32_t count,
                           int32_t shape, int32_t blocks, double* bytes);

/* Hash of the source files this library was built from (static storage).  A
 * binding compares it with the sources beside it to refuse a stale build. */
const char* autoloco_build_id(void);

/* ------------------------------------------------------------------------ */
/* One GPU's share of a round with one worker replica per GPU                */
/* ------------------------------------------------------------------------ */

/* In the paper's topology every worker's replica lives on its own GPU and the
 * pseudo-gradients travel as BF16 payloads.  A round then is, on GPU r:
 *   1. autoloco_rank_payload: Delta_r = theta - theta_r (FP32) as a BF16
 *      payload, and ||Delta_r||^2 (D = the mean over workers of these);
 *   2. an all-to-all of payload shards (GPU s receives shard s of every
 *      worker's payload; not part of this library);
 *   3. autoloco_shard_step on GPU r's shard: the received mean and the
 *      corrected Nesterov step of theta and v on that shard, and the shard's
 *      ||mean||^2 (C = K * (sum over shards) / (D + eps));
 *   4. an all-gather of theta' shards into theta, and autoloco_broadcast_reset
 *      for the worker's replica.
 * Steps 1 and 3 use the arithmetic of autoloco_outer_step_bf16, so theta',
 * v' and the received mean equal that call's bit for bit. */

/* Step 1 for one worker.  theta: [n] fp32; replica: [n] fp32 or bf16
 * (replica_dtype); payload: [n] bf16 bit patterns, written.  All 16-byte
 * aligned and disjoint.  sq_norm (or NULL) receives ||Delta_r||^2 (float64, deterministic
 * order); with it the call blocks, without it it is asynchronous.
 * Errors: E_INVALID, E_ALIGN, E_ALIAS, E_DEVICE. */
int autoloco_rank_payload(autoloco_ctx* ctx, int64_t n, const float* theta, const void* replica,
                          int32_t replica_dtype, uint16_t* payload, double* sq_norm);

/* Buffers of one GPU's shard: n parameters of theta and v (fp32, read and
 * written) and the K workers' payload shards for them (bf16, read). */
typedef struct {
    int64_t n;
    int32_t k;
    float* theta;
    float* momentum;
    const uint16_t* payloads[AUTOLOCO_MAX_K];
} autoloco_shard_buffers;

/* Step 3 on one shard: mean = bf16(fp32(sum_k payload_k in float64, worker
 * order, times 1/K)); the corrected Nesterov step with it (coefficients as
 * autoloco_outer_step); mean_bf16 ([n], or NULL) receives the mean's bits;
 * sq_mean (or NULL) receives the shard's ||mean||^2 and makes the call block.
 * Errors: E_INVALID (k outside 1..16, null or non-finite arguments),
 * E_ALIGN, E_ALIAS, E_DEVICE. */
int autoloco_shard_step(autoloco_ctx* ctx, const autoloco_shard_buffers* bufs,
                        const autoloco_outer_coeffs* coeffs, uint16_t* mean_bf16, double* sq_mean);

/* ------------------------------------------------------------------------ */
/* Inner AdamW step of the K workers                                         */
/* ------------------------------------------------------------------------ */

/* Each worker's state for its local inner loop (Alg. "AutoLoCo outer
 * interval", local inner loops; App. G.1 keeps master parameters and AdamW
 * states in FP32 and computes the model in BF16).  All buffers are device
 * memory owned by the caller, [n] elements, 16-byte aligned, pairwise
 * disjoint.  params, exp_avg and exp_avg_sq are read and written; grads are
 * read; model_bf16 (bf16 bit patterns) is written iff set: set all k of them
 * or none. */
typedef struct {
    int64_t n;
    int32_t k;
    float* params[AUTOLOCO_MAX_K];       /* worker k's FP32 master parameters */
    float* exp_avg[AUTOLOCO_MAX_K];      /* first moment m */
    float* exp_avg_sq[AUTOLOCO_MAX_K];   /* second moment v */
    const float* grads[AUTOLOCO_MAX_K];  /* this step's gradient of worker k */
    void* model_bf16[AUTOLOCO_MAX_K];    /* BF16 compute copy of the new params, or NULL */
} autoloco_adamw_buffers;

/* Settings of one step, shared by all workers (Table "Training settings":
 * C4 uses beta = (0.9, 0.95), weight decay 0.1, clipping 1.0; SFT
 * (0.9, 0.999), 0, 1.0).  lr is the schedule's value at this step
 * (autoloco_inner_lr); step counts from 1 and sets the bias corrections;
 * max_grad_norm = 0 turns clipping off. */
typedef struct {
    double lr, beta1, beta2, eps, weight_decay, max_grad_norm;
    int64_t step;
} autoloco_adamw_coeffs;

/* Per-worker gradient norms of the step and the clipping factors applied. */
typedef struct {
    double grad_norm[AUTOLOCO_MAX_K];
    double clip_coef[AUTOLOCO_MAX_K];
    int32_t k;
    int32_t finite;   /* every gradient norm is finite */
} autoloco_adamw_stats;

/* One AdamW step of every worker, each clipped by its own global gradient
 * norm: c_k = min(1, max_grad_norm / (||g_k|| + 1e-6)), g <- c_k g, then
 * decoupled weight decay theta <- theta (1 - lr wd), m <- beta1 m +
 * (1 - beta1) g, v <- beta2 v + (1 - beta2) g^2 and theta <- theta - lr
 * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps).  With clipping (or
 * out) a first pass sums each worker's g^2 (fp64, deterministic order); the
 * update pass reads those sums on the device.  With out the call blocks until
 * the norms are on the host; without, it is asynchronous on the stream.
 * Element arithmetic is fp32 with the step's scalars rounded once to fp32.
 * A non-finite gradient is not an error: it propagates into the state and
 * finite = 0.
 * Errors: E_INVALID (k outside 1..16, n outside 0..2^56, null buffer, partial model_bf16,
 * step < 1, lr / eps / weight_decay / max_grad_norm negative or not finite,
 * beta outside [0, 1)), E_ALIGN, E_ALIAS, E_DEVICE. */
int autoloco_inner_adamw(autoloco_ctx* ctx, const autoloco_adamw_buffers* bufs,
                         const autoloco_adamw_coeffs* coeffs, autoloco_adamw_stats* out);

/* Device milliseconds of the two passes of the last timed autoloco_inner_adamw
 * call (norm_ms = 0 if the norm pass did not run); waits for them to finish. */
int autoloco_last_adamw_ms(autoloco_ctx* ctx, float* norm_ms, float* update_ms);

/* Measurement, no operation of the paper: the traffic reference of the AdamW
 * update pass.  It runs that pass's kernel on the same grid with the same
 * loads and stores and none of the arithmetic: params, exp_avg and exp_avg_sq
 * keep their bits, grads are read, and each model_bf16 (if set) receives the
 * BF16 rounding of the unchanged params, which is what the last AdamW step
 * wrote there.  Asynchronous on the stream; timed like a round
 * (autoloco_last_kernel_ms).  Errors: as autoloco_inner_adamw's buffer
 * checks. */
int autoloco_adamw_traffic_reference(autoloco_ctx* ctx, const autoloco_adamw_buffers* bufs);

/* ------------------------------------------------------------------------ */
/* Host-only scalar routines                                                 */
/* ------------------------------------------------------------------------ */

/* Inner learning-rate schedule: linear warm-up then cosine decay, the recipe
 * of Table "Training settings".  eta(s) = peak (s+1)/warmup for s < warmup,
 * else min_lr + (peak - min_lr)(1 + cos(pi min(1, (s - warmup)/(total - warmup))))/2,
 * with s the 0-based global inner step. */
typedef struct {
    double peak, min_lr;
    int64_t warmup, total;
} autoloco_schedule;
double autoloco_inner_lr(const autoloco_schedule* sched, int64_t step);

/* Learning-rate mass sum_{h=1..steps} eta(start_step + h - 1): the exact
 * scheduler preview of eq. app-outer-correction-lr-masses.  Returns NaN for a
 * null schedule or negative arguments. */
double autoloco_lr_mass(const autoloco_schedule* sched, int64_t start_step, int64_t steps);

/* Outer Optimizer Correction (eqs. outer-correction-ratio,
 * adjusted-outer-learning-rate; App. B.2-B.4):
 *   rho = max(lambda_sel / (lambda_base + eps), 1), mu = clip(mu_base^rho, mu_min, mu_max),
 *   kappa = min(rho, kappa_max), eta_out = eta_base kappa (1 - mu)/(1 - mu_base).
 * Errors: E_INVALID (null pointers, non-finite masses, mu_base outside (0,1),
 * mu_min > mu_max, kappa_max < 1). */
typedef struct {
    double eta_base, mu_base, mu_min, mu_max, kappa_max, eps;
    int32_t normalize;
} autoloco_outer_cfg;
int autoloco_outer_correction(const autoloco_outer_cfg* cfg, double lambda_sel,
                              double lambda_base, autoloco_outer_coeffs* out);

/* ------------------------------------------------------------------------ */
/* Adaptive interval controller (host)                                       */
/* ------------------------------------------------------------------------ */

/* Settings of the controller and token mapper (Table "AutoLoCo
 * configuration"; App. A).  Horizons h_* are token-equivalent horizons. */
typedef struct {
    int64_t h_base, h_min, h_max, q_h, budget_steps;
    double beta_tok;      /* token-density EMA coefficient (0.9) */
    double eps;           /* numerical constant of the residuals and the mapper, > 0 */
    double thr_cand, thr_mod, thr_sev; /* z_max class limits 1.5 / 2.5 / 4.0 */
    double cand_exposure; /* candidate LR-exposure multiplier 1.15 */
    double retire_frac;   /* rejected-bound retirement fraction 0.90 */
    double red_moderate, red_severe; /* reduction divisors 1.20 / 1.50 */
    double ref_ema;       /* log-space EMA coefficient of D_ref, C_ref */
    double mad_scale, scale_floor; /* robust scale = max(mad_scale * MAD, scale_floor) */
    int32_t n_mapper_boot, n_ref_boot, n_var, hist_max;   /* 3, 2, 3, 16 */
    int32_t moderate_confirm, fallback_count;             /* 2, 2 */
    autoloco_schedule sched;
    autoloco_outer_cfg outer;
} autoloco_controller_cfg;

/* Fills *out with the C4 column of Table "AutoLoCo configuration" and the C4
 * training recipe (50,000 steps, 1,000 warm-up steps, peak 4e-4, outer
 * learning rate 0.7, momentum 0.9, no normalisation). */
void autoloco_controller_default_cfg(autoloco_controller_cfg* out);

/* What the trainer observed over the interval just completed. */
typedef struct {
    double D, C;          /* diagnostics of the round (autoloco_stats) */
    double lambda_done;   /* learning-rate mass of the executed steps */
    double tokens;        /* non-padding tokens processed (M_t) */
    int64_t h_step_done;  /* executed local steps */
    int32_t finite;       /* 0 if any required statistic was non-finite */
} autoloco_observation;

typedef enum {
    AUTOLOCO_ASSESS_NONE = -1, AUTOLOCO_ASSESS_SUPPORTED = 0, AUTOLOCO_ASSESS_CONSISTENT = 1,
    AUTOLOCO_ASSESS_MODERATE = 2, AUTOLOCO_ASSESS_SEVERE = 3, AUTOLOCO_ASSESS_INVALID = 4
} autoloco_assessment;

typedef enum {
    AUTOLOCO_PHASE_WARMUP = 0, AUTOLOCO_PHASE_REF_BOOT = 1, AUTOLOCO_PHASE_INIT = 2,
    AUTOLOCO_PHASE_VAR = 3, AUTOLOCO_PHASE_MONITOR = 4, AUTOLOCO_PHASE_CAND1 = 5,
    AUTOLOCO_PHASE_CAND2 = 6, AUTOLOCO_PHASE_DONE = 7
} autoloco_phase;

/* The next interval: where it starts, its horizons, the previewed LR masses,
 * the outer coefficients to use after it, and the assessment of the interval
 * just observed. */
typedef struct {
    int64_t start_step, h_tok, h_step, h_ref;
    double lambda_sel, lambda_base;
    double z_max;          /* NaN when the observed interval was not assessed */
    int32_t assessment;    /* autoloco_assessment of the observed interval */
    int32_t phase;         /* autoloco_phase of the next interval */
    int32_t done;          /* 1: the budget is spent, no next interval */
    int32_t reserved;
    autoloco_outer_coeffs coeffs;
} autoloco_decision;

/* The adaptive interval controller of Sec. "Adaptive Interval Selection" and
 * App. A: residuals r_D, r_C against the accepted-horizon reference profile
 * (eqs. adaptive-h-lr-mass, adaptive-h-core-residuals), robust deviation
 * z_max (eq. adaptive-h-core-deviation), the assessment classes of Table
 * "Interval assessments", candidate search and evaluation, rejected-horizon
 * bound, reductions, and the token mapper (eq. adaptive-h-token-mapping).
 * Not thread-safe; one controller per training run.
 * create errors: E_INVALID (inconsistent settings), E_NOMEM. */
typedef struct autoloco_controller autoloco_controller;
int autoloco_controller_create(const autoloco_controller_cfg* cfg, autoloco_controller** out);
void autoloco_controller_destroy(autoloco_controller* ctrl);

/* First call: obs = NULL, returns the first interval.  Every later call:
 * obs describes the interval returned by the previous call.  Once a decision
 * with done = 1 has been returned, further calls fail with E_STATE.
 * Errors: E_INVALID (null ctrl/next, missing or unexpected obs), E_STATE. */
int autoloco_select_interval(autoloco_controller* ctrl, const autoloco_observation* obs,
                             autoloco_decision* next);

/* Current reference profile (D_ref, C_ref, Lambda_ref); zeros before it exists. */
int autoloco_controller_reference(const autoloco_controller* ctrl, double* d_ref,
                                  double* c_ref, double* lambda_ref);

/* Checkpoint of the whole controller state.  save: with buf = NULL sets *len
 * to the size needed; otherwise writes *len bytes (E_INVALID if *len is too
 * small).  load: restores a state saved by the same library version into a
 * controller created with any configuration (the saved configuration wins).
 * Errors: E_INVALID (null pointers, bad size, bad magic or version). */
int autoloco_controller_save(const autoloco_controller* ctrl, void* buf, size_t* len);
int autoloco_controller_load(autoloco_controller* ctrl, const void* buf, size_t len);

#ifdef __cplusplus
}
#endif

#endif /* AUTOLOCO_H */
