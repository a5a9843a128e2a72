/*
 * zero_shard.h -- C ABI of libzeroshard: the per-rank optimizer step that ZeRO's
 * P_os+g partitioning leaves on every data-parallel rank, for AMD Instinct
 * MI355X (gfx950).
 *
 * Paper: ZeRO: Memory Optimizations Toward Training Trillion Parameter Models
 * (Rajbhandari et al., arXiv 1910.02054).  Sec. 5.1: the optimizer state is
 * split into N_d equal partitions and rank i updates only partition i, then
 * the updated parameters are all-gathered.  Sec. 5.2: the gradients are
 * reduce-scattered so that each rank holds only its partition's reduced
 * gradients.  Sec. 3.1: mixed-precision Adam keeps fp16 parameters and
 * gradients and fp32 master parameters, momentum and variance.
 *
 * Conventions shared by every entry point:
 *   - Plain C types only; no exception crosses the ABI.
 *   - Return value 0 = success (for zero_shard_step: 0 = applied, 1 = skipped),
 *     negative = error (ZERO_E*); zero_last_error() then describes it.
 *   - Array arguments are DEVICE pointers owned by the caller.  The library
 *     never allocates, frees or retains them and touches exactly [0, n).
 *   - The library owns a small per-(device, stream) workspace (per-workgroup
 *     partial sums, one result record, a barrier counter, one pinned host
 *     record: about 64 KiB of device memory), allocated on a stream's first
 *     call and held until zero_stream_release(stream) or the process ends, so
 *     the library's memory grows with the number of distinct streams it has
 *     seen.  Its size does not depend on n (constant-size buffers, Sec. 6.2).
 *   - `stream` is a hipStream_t passed as void*; NULL is the null stream.  The
 *     device is the current HIP device of the calling thread; a stream of
 *     another device is rejected with ZERO_EINVAL.
 *   - Concurrent calls are serialised per (device, stream) by the library.
 *     The workspace is keyed by the stream handle: do not destroy a stream
 *     while calls on it are in flight, and release its workspace
 *     (zero_stream_release) before destroying a stream, since a new stream may
 *     be handed the same handle.
 */
#ifndef ZERO_SHARD_H
#define ZERO_SHARD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ZERO_OK 0
#define ZERO_SKIPPED 1
#define ZERO_EINVAL (-1) /* invalid argument: nothing was launched or written    */
#define ZERO_EHIP (-2)   /* a HIP runtime call failed                             */
#define ZERO_ENOMEM (-3) /* the library's own workspace could not be allocated    */

/* ------------------------------------------------------------------------ */
/* Partition layout                                                         */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t shard_numel;  /* S = ceil(total / nd): every rank's shard length      */
    int64_t offset;       /* rank * S: first flat index of the shard              */
    int64_t valid_numel;  /* clamp(total - rank*S, 0, S): elements holding state */
    int64_t padded_total; /* nd * S: length of the padded flat buffer             */
} zero_layout_t;

/* Sec. 5.1 (N_d equal partitions, rank i owns partition i).  The paper does not
 * say what happens when nd does not divide total_numel; here the flat index
 * space is padded at its tail, so the last rank(s) are short and a rank may
 * hold no valid elements.  Host-only integer arithmetic, exact in int64.
 * total_numel in [0, 2^62], nd >= 1, 0 <= rank < nd, out != NULL, else
 * ZERO_EINVAL (out untouched). */
int zero_partition_layout(int64_t total_numel, int32_t nd, int32_t rank, zero_layout_t* out);

/* ------------------------------------------------------------------------ */
/* The shard step                                                           */
/* ------------------------------------------------------------------------ */

/* One mixed-precision Adam step over one rank's shard (Sec. 3.1, Sec. 5.1-5.2;
 * Adam with bias correction as in Kingma & Ba, which Sec. 3.1 cites):
 *
 *   grad16       [n] binary16 gradients as the reduce-scatter delivers them:
 *                averaged over ranks and still multiplied by loss_scale.
 *                Read only.  Alignment: 2 bytes.
 *   master32     [n] fp32 master parameters, updated in place.  4-byte aligned.
 *   m32, v32     [n] fp32 first and second moments, updated in place.
 *   param16_out  [n] binary16 copy of the updated master parameters (rounded
 *                to nearest even): the slice the all-gather publishes.  Write
 *                only.  Alignment: 2 bytes.
 *   n            elements of the shard that hold state (the layout's
 *                valid_numel); n == 0 returns 0 and touches nothing.
 *   lr, beta1, beta2, eps, weight_decay
 *                Adam hyper-parameters; beta1, beta2 in [0, 1); lr, eps >= 0
 *                and weight_decay finite.  weight_decay != 0 adds decoupled
 *                decay (AdamW): u += weight_decay * master before the update.
 *   step         t >= 1: number of applied updates INCLUDING this one (bias
 *                correction 1 - beta^t).  Skipped steps must not advance it.
 *   loss_scale   > 0 and finite; the gradient is divided by it.
 *   clip         global-norm clipping threshold of the unscaled gradient; the
 *                shard's own norm is the global norm (one rank).  <= 0 disables.
 *   stream       hipStream_t (void*), NULL = null stream.
 *
 * The step: overflow = any grad16 element is inf or NaN; norm =
 * sqrt(sum grad16^2) / loss_scale; coef = clip/norm if clip > 0 and norm >
 * clip, else 1; every element uses g = (float)grad16 * (float)(coef /
 * loss_scale) and, in fp32,
 *   m = b1*m + (1-b1)*g;  v = b2*v + (1-b2)*g*g;
 *   u = (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps)  [+ wd*master];
 *   master -= lr*u;  param16_out = binary16(master).
 * On overflow nothing is written and the call returns ZERO_SKIPPED (1); the
 * caller then lowers its loss scale and does not advance t.
 *
 * All five arrays must be distinct, non-overlapping ranges; base pointers of
 * any element alignment are accepted (when all five share one misalignment
 * the vectorised path runs after a few scalar head elements).  Placement
 * affects speed, not results: separate allocations, or arrays packed into one
 * buffer each on its own 2 MiB boundary, run fastest; arrays offset from one
 * another by a few hundred bytes run about 5 % slower.  Shards small enough
 * for one resident grid (a quarter of the device's co-resident capacity for
 * the kernel, or 1/q with q = GPU_MAX_HW_QUEUES when that is larger: about
 * 1.5 million elements on MI355X with the default four queues) whose arrays share one
 * misalignment take a single launch (statistics, a grid barrier and the
 * update in one kernel, the gradient read once); larger ones take the
 * statistics kernels and the update kernel.  The barrier relies on the whole
 * grid being resident at once; its wait is bounded, and should the device
 * not run the grid together within seconds, the step writes nothing and
 * returns ZERO_EHIP.  The call
 * blocks until the skip decision is known (the statistics kernels publish it
 * in host-mapped memory, which the calling thread polls); the update kernel
 * may still be running on `stream` when it returns.  Returns 0 applied,
 * 1 skipped, ZERO_EINVAL / ZERO_EHIP / ZERO_ENOMEM on error (on ZERO_EINVAL
 * nothing is launched). */
int zero_shard_step(const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                    int64_t n, double lr, double beta1, double beta2, double eps, double weight_decay,
                    int64_t step, double loss_scale, double clip, void* stream);

/* For callers that cannot allocate memory (tight serving or training loops,
 * harnesses that forbid the allocator): zero_shard_step with the same
 * arguments, checks, kernels, results and return values, that calls no
 * hipMalloc, hipFree or other allocating routine.  Its workspace (statistics
 * partials for up to 4096 workgroups, the one-launch step's barrier words and
 * two result records: 73 KiB) is one fixed device array per GPU, held by
 * every GPU the library runs on until the process ends; n up to 2^40 (the
 * library's limit, ZERO_EINVAL above it) needs no more.  Differences: the call
 * returns once the whole step (update included) has completed on `stream`,
 * since the skip decision is copied back after it; no kernel timing is
 * sampled.  All calls on one GPU share its array: calls from several threads
 * are serialised on the host, but calls whose work overlaps on the GPU (on
 * different streams, or queued behind other work so that two steps' kernels
 * run together) race on it and must not be made. */
int zero_shard_step_noalloc(const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                            int64_t n, double lr, double beta1, double beta2, double eps, double weight_decay,
                            int64_t step, double loss_scale, double clip, void* stream);

/* ------------------------------------------------------------------------ */
/* Split-phase step: local statistics, then the update with global ones      */
/* ------------------------------------------------------------------------ */

/* With N_d ranks (Sec. 5.1-5.2) clipping and the skip decision need the norm
 * of the WHOLE gradient, so each rank first computes its shard's local sum of
 * squares, the ranks combine the N_d values (an all-reduce of 8 bytes per
 * rank; summing them in rank order gives every rank the same bits), and each
 * rank then applies the update with the global value.  zero_shard_step is the
 * one-rank composition of the two phases.
 *
 * zero_shard_stats: *local_sumsq = sum of grad16^2 over [0, n) (loss-scaled,
 * accumulated in fp64; +inf or NaN iff some element is inf or NaN).  Blocks
 * until the value is known.  n == 0 gives 0.  grad16: device, 2-byte aligned,
 * read only.  Returns 0 or ZERO_E*. */
int zero_shard_stats(const uint16_t* grad16, int64_t n, double* local_sumsq, void* stream);

/* zero_shard_apply: the update of zero_shard_step with the global sum of
 * squares supplied by the caller (the sum over all ranks of their
 * local_sumsq).  Overflow = global_sumsq is not finite: then nothing is
 * written and ZERO_SKIPPED is returned.  Otherwise norm =
 * sqrt(global_sumsq)/loss_scale and the rest is exactly zero_shard_step's
 * update (same kernels).  Arguments and errors as for zero_shard_step;
 * global_sumsq must not be negative.  Does not block: the skip decision is
 * known on the host from global_sumsq, and the kernels are queued on
 * `stream`.  Does not change zero_shard_last_stats. */
int zero_shard_apply(const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                     int64_t n, double global_sumsq, double lr, double beta1, double beta2, double eps,
                     double weight_decay, int64_t step, double loss_scale, double clip, void* stream);

/* Asynchronous split phase: the same kernels as zero_shard_stats /
 * zero_shard_apply, with the scalars in DEVICE memory and no host wait, so both
 * calls only enqueue work on `stream` and return.  A device-side exchange of
 * the per-rank sums (an all-reduce or all-gather on the same stream, summed in
 * rank order so that every rank holds the same bits) can sit between them, and
 * the step never makes the host wait for the GPU.
 *   zero_shard_stats_async writes this shard's sum of grad16^2 (fp64; +inf or
 *   NaN on overflow, as zero_shard_stats returns it) to *local_sumsq (device,
 *   8-byte aligned); n = 0 writes 0.
 *   zero_shard_apply_async reads the global sum from *global_sumsq (device) when
 *   its kernels run; a non-finite, negative or NaN value skips the update (no
 *   state byte written) exactly as an overflow does.  The skip decision (1 or
 *   0) is stored to *skipped when skipped is not NULL (device memory, or
 *   mapped host memory from hipHostMalloc that the host reads after the stream
 *   has reached this call).  The loss scaler is the caller's, with that flag.
 * Argument checks, the allocation checks included, are those of the
 * synchronous calls; returns ZERO_OK (enqueued) or an error. */
int zero_shard_stats_async(const uint16_t* grad16, int64_t n, double* local_sumsq, void* stream);
int zero_shard_apply_async(const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                           int64_t n, const double* global_sumsq, double lr, double beta1, double beta2, double eps,
                           double weight_decay, int64_t step, double loss_scale, double clip, int32_t* skipped,
                           void* stream);

/* Resident step: the whole step, loss scaler included, driven by a state
 * record in DEVICE memory, so a call only enqueues kernels and never waits;
 * the enqueued work can be captured into a HIP graph and replayed, each replay
 * being the next optimizer step.  The caller owns the record: it fills it with
 * zero_resident_state_init (a host copy, checked there) and copies it to the
 * device before the first step or between steps, and reads t / loss_scale /
 * skipped whenever it needs them.  Per step, on the device:
 *   statistics of grad16 (as zero_shard_step) -> scalars from the record's
 *   loss_scale and clip -> the fp32 constants from lr, betas, eps, weight
 *   decay and t (each computed in double and rounded once, the bias
 *   corrections as zero_bias_corrections defines them) -> the scaler: on a
 *   skip halve loss_scale (not below min_scale), good = 0; else t += 1,
 *   good += 1 and double loss_scale when good reaches window (> 0), good = 0
 *   -> skip or the update.  The record is updated before the update kernel
 *   runs (which reads only the scalars and constants taken from it before);
 *   once the step's work on the stream is complete the record describes the
 *   step just taken.  A record whose hyperparameters are outside the ranges
 *   zero_shard_step accepts (or min_scale not finite and > 0) is not a valid
 *   step: nothing is written and only its `skipped` field changes, to -1.
 * Workspace: each state record has its own (statistics partials, result
 * record, constants; about 64 KiB of device memory), allocated on the first
 * step taken with it and held until zero_resident_release(state) or the
 * process ends.  Eager calls and graph replays with that record use it, and
 * nothing else does; so steps with one record must not overlap each other
 * (they also read and advance its t and loss scale), while steps with
 * different records, graph replays included, may run concurrently on any
 * streams.  Same arrays, checks and skip semantics as zero_shard_step.  Make
 * one eager call with the arrays and the record before capturing: while the
 * stream is capturing, the allocation checks and the sampled timing
 * (zero_profile_enable) are left out.  `state` must be 8-byte aligned device
 * memory (or mapped host memory) that no array overlaps. */
typedef struct {
    double lr, beta1, beta2, eps, weight_decay, clip; /* hyperparameters (caller)          */
    double loss_scale;                                /* current loss scale                */
    double min_scale;                                 /* floor of the halving               */
    int64_t window;                                   /* growth window; <= 0: never grow    */
    int64_t t;                                        /* t of the next applied update, >= 1 */
    int64_t good;                                     /* applied steps since skip or growth */
    int64_t steps;                                    /* steps taken, applied or skipped    */
    int32_t skipped;                                  /* last step: 1 skipped, 0 applied,
                                                         -1 record out of range             */
    int32_t pad_;
} zero_resident_state_t;

/* Fills a HOST record for the resident step after checking the values as
 * zero_shard_step checks its arguments (lr, eps >= 0 finite, weight_decay
 * finite, beta1, beta2 in [0, 1), t >= 1, loss_scale finite > 0, clip not
 * NaN) and min_scale finite > 0; good, steps and skipped start at 0.
 * ZERO_EINVAL (out untouched) otherwise. */
int zero_resident_state_init(zero_resident_state_t* out, double lr, double beta1, double beta2, double eps,
                             double weight_decay, double clip, double loss_scale, double min_scale, int64_t window,
                             int64_t t);

int zero_shard_step_resident(const uint16_t* grad16, float* master32, float* m32, float* v32,
                             uint16_t* param16_out, int64_t n, zero_resident_state_t* state, void* stream);

/* Frees the workspace the resident step holds for `state` on the current
 * device (nothing to do if it holds none).  Graph replays may use it on any
 * stream, so this first waits for the device to finish its queued work
 * (hipDeviceSynchronize): call it while no stream of the device is being
 * captured, since such a wait ends a capture in progress with an error.  A
 * later step with the record allocates a new workspace; graphs captured with
 * it must not be replayed after the release.  Returns 0 or ZERO_EHIP. */
int zero_resident_release(const zero_resident_state_t* state);

/* The array checks of zero_shard_step without launching anything: n range,
 * NULL pointers, alignment, that each array [p, p + n*size) lies inside one
 * GPU-accessible allocation (hipMemGetAddressRange), then overlap.
 * zero_shard_step, zero_shard_apply and zero_shard_stats make the same
 * allocation check on every call (a lookup costs well under a microsecond), so
 * an n that overruns its allocation or a pageable host pointer is rejected with
 * ZERO_EINVAL rather than faulting the GPU.  Limit: the allocation is what the
 * HIP runtime handed out, so a caching allocator's segment (larger than the
 * tensor carved from it) bounds the check.
 * Returns 0 or ZERO_EINVAL. */
int zero_shard_validate(const uint16_t* grad16, const float* master32, const float* m32, const float* v32,
                        const uint16_t* param16_out, int64_t n);

/* Statistics of the calling thread's last successful zero_shard_step (or
 * zero_lamb_step). */
typedef struct {
    double sumsq;     /* sum of grad16^2 (loss-scaled), accumulated in fp64;
                         non-finite iff overflow                                  */
    double norm;      /* sqrt(sumsq) / loss_scale                                 */
    double coef;      /* clipping coefficient in (0, 1]; 1 when skipped           */
    float mult;       /* fp32 multiplier applied to grad16: (float)(coef/scale)   */
    int32_t overflow; /* 1 if any grad16 element was inf or NaN                   */
    int32_t skipped;  /* equals overflow                                          */
    int32_t path;     /* 1: the one-launch small-shard step; 0: statistics kernels
                         and update kernel                                        */
    int64_t n;        /* elements of that call                                    */
} zero_step_stats_t;

/* The clipping diagnostics of the calling thread's last successful step
 * (Sec. 3.2: the norm over the gradient; the clipping multiplier and the
 * overflow flag of the mixed-precision step): *norm = sqrt(sum grad16^2) /
 * loss_scale (+inf on overflow), *mult = the fp32 multiplier applied to
 * grad16, *overflow = 1 if some element was inf or NaN.  Host pointers; any
 * of them may be NULL (not all three).  ZERO_EINVAL if all are NULL or this
 * thread has made no successful step yet. */
int zero_shard_last_stats(double* norm, float* mult, int* overflow);

/* The same step's whole record (sum of squares, norm, clipping coefficient,
 * multiplier, overflow, skip flag, n) into *out (host); ZERO_EINVAL if out is
 * NULL or this thread has made no successful step yet. */
int zero_shard_last_step_stats(zero_step_stats_t* out);

/* The fp32 bias corrections 1 - beta1^t and 1 - beta2^t that every Adam and
 * LAMB update uses (Adam's bias-corrected moments, Kingma & Ba, cited in
 * Sec. 3.1): beta^t is the double nearest the exact power, 1 - beta^t is
 * taken in double and rounded once to fp32.  The host calls and the resident
 * step's kernel evaluate this one definition and get the same bits.  Host
 * only (no GPU needed).  beta1, beta2 in [0, 1), step >= 1, bc1 and bc2
 * non-NULL host pointers, else ZERO_EINVAL. */
int zero_bias_corrections(double beta1, double beta2, int64_t step, float* bc1, float* bc2);

/* ------------------------------------------------------------------------ */
/* Dynamic loss scaling (host state owned by the caller)                     */
/* ------------------------------------------------------------------------ */

typedef struct {
    double scale;      /* current loss scale                                  */
    double min_scale;  /* floor after repeated overflow                       */
    int64_t window;    /* applied steps between doublings (<= 0: never grow)  */
    int64_t applied;   /* updates applied so far; the next step uses t = applied + 1 */
    int64_t good;      /* applied steps since the last overflow or growth     */
} zero_scaler_t;

/* Mixed-precision loss scaling as cited by Sec. 3.1: after a skipped step the
 * scale halves (not below min_scale) and applied/good do not advance (good
 * restarts); after an applied step applied and good advance and the scale
 * doubles once good reaches window.  scale > 0 finite, min_scale > 0. */
int zero_scaler_init(zero_scaler_t* s, double scale, int64_t window, double min_scale);
int zero_scaler_update(zero_scaler_t* s, int32_t skipped);

/* The arguments of zero_shard_step that stay fixed over a training loop: the
 * shard's five arrays (DEVICE pointers with zero_shard_step's rules), n, the
 * hyperparameters and the stream (NULL: the default stream). */
typedef struct {
    const uint16_t* grad16;
    float* master32;
    float* m32;
    float* v32;
    uint16_t* param16_out;
    int64_t n;
    double lr, beta1, beta2, eps, weight_decay, clip;
    void* stream;
} zero_step_args_t;

/* One step of a mixed-precision training loop (Sec. 3.1) in one call: the
 * shard step of *args at t = scaler->applied + 1 and loss_scale =
 * scaler->scale, then zero_scaler_update(scaler, skipped).  For loops over
 * small shards, where the host call is most of the step.  Returns what
 * zero_shard_step returns (0 applied, 1 skipped); ZERO_EINVAL if args or
 * scaler is NULL or scaler->applied is negative or INT64_MAX.  On any error
 * the scaler is left as it was. */
int zero_shard_step_scaled(const zero_step_args_t* args, zero_scaler_t* scaler);

/* ------------------------------------------------------------------------ */
/* Model-state memory per device (Sec. 3.1, Sec. 5.1-5.3, Table 1)           */
/* ------------------------------------------------------------------------ */

#define ZERO_STAGE_DP 0       /* (2 + 2 + K) * Psi               */
#define ZERO_STAGE_OS 1       /* 2*Psi + 2*Psi + K*Psi/N_d       */
#define ZERO_STAGE_OS_G 2     /* 2*Psi + (2 + K)*Psi/N_d         */
#define ZERO_STAGE_OS_G_P 3   /* (2 + 2 + K)*Psi/N_d             */

/* Bytes of model state per device (Sec. 3.1: fp16 parameters and gradients
 * take 2 bytes each per parameter and the optimizer state K bytes, K = 12 for
 * mixed-precision Adam; Sec. 5.1-5.3 and Table 1: P_os divides the optimizer
 * state by N_d, P_os+g also the gradients, P_os+g+p everything) for psi
 * parameters, data-parallel degree nd >= 1 and multiplier k >= 0 (bytes per
 * parameter of optimizer state), written to *bytes (host).  Evaluated in
 * double; psi >= 0 and finite.  ZERO_EINVAL for an unknown stage, nd < 1,
 * k < 0, a bad psi or bytes == NULL. */
int zero_memory_bytes(double psi, int32_t nd, int32_t stage, int32_t k, double* bytes);

/* zero_memory_bytes with nd and k as doubles (fractional K for optimizers whose
 * state is not a whole number of bytes per parameter): nd > 0 and k finite,
 * psi >= 0 finite, else ZERO_EINVAL. */
int zero_model_state_bytes(double psi, double nd, int32_t stage, double k, double* out);

/* ------------------------------------------------------------------------ */
/* LAMB: the same mixed-precision shard step with a per-layer trust ratio    */
/* ------------------------------------------------------------------------ */

/* LAMB (You et al., layer-wise adaptive moments for large batches) is among
 * the adaptive optimizers that ZeRO's related work (Sec. 2.3) says its
 * partitioning of optimizer state makes affordable.  Its fp32 state is Adam's
 * (K = 12, Sec. 3.1); only the update differs.  With the moments and the
 * direction u of zero_shard_step (unscale + clip, bias correction, eps outside
 * the square root, decoupled weight decay), each layer L of the shard moves by
 *     theta_L <- theta_L - step_L * u_L,
 *     step_L   = (float)(lr * trust_L)   (computed in double, rounded once),
 *     trust_L  = phi(||theta_L||) / ||u_L||, or 1 if either norm is zero,
 *     phi(z)   = min(max(z, phi_lo), phi_hi)   (phi_lo = 0, phi_hi = +inf:
 *                identity),
 * where the norms are over the layer's old parameters and its whole u.
 *
 * A plan holds the shard's layer table and the work decomposition built from
 * it.  seg_off (HOST memory, n_seg + 1 int64 offsets, copied) must rise
 * strictly from seg_off[0] = 0 to seg_off[n_seg] = n: layer s is elements
 * [seg_off[s], seg_off[s+1]) of the shard.  n = 0 requires n_seg = 0.  A
 * layer that continues on a neighbouring rank's shard appears clipped to this
 * shard; its norms then need the split-phase calls below.  The plan is tied to
 * the device current at creation and owns device memory (about 16 bytes per
 * 256 elements plus 32 bytes per layer, and the work lists, built per array
 * alignment on first use); zero_lamb_plan_destroy waits for the plan's own
 * queued work and frees it.  Calls on one plan are serialised by the library:
 * each call records a plan-owned event after its kernels, and a call on a
 * different stream from the plan's previous one makes its stream wait for
 * that event on the device (no host wait, no other stream affected; the
 * event stays valid if the previous stream has been destroyed).
 * Returns ZERO_OK, ZERO_EINVAL (bad table, n outside [0, 2^40], NULL out) or
 * ZERO_ENOMEM / ZERO_EHIP. */
typedef struct zero_lamb_plan zero_lamb_plan_t;

int zero_lamb_plan_create(const int64_t* seg_off, int32_t n_seg, int64_t n, zero_lamb_plan_t** out);
int zero_lamb_plan_destroy(zero_lamb_plan_t* plan);

/* One LAMB step on a shard whose layers all lie in it (N_d = 1, or a caller
 * that cuts its flat buffer at layer boundaries).  Arrays, checks, skip
 * semantics, return values and zero_shard_last_stats as for zero_shard_step,
 * with n taken from the plan; phi_lo >= 0, phi_hi >= phi_lo (may be +inf),
 * neither NaN.  The library's per-layer sums live in the plan. */
int zero_lamb_step(const zero_lamb_plan_t* plan, const uint16_t* grad16, float* master32, float* m32, float* v32,
                   uint16_t* param16_out, double lr, double beta1, double beta2, double eps, double weight_decay,
                   int64_t step, double loss_scale, double clip, double phi_lo, double phi_hi, void* stream);

/* Split phase for layers that straddle shards (Sec. 5.1 cuts the flat buffer
 * without regard to layers):
 *   1. zero_shard_stats -> the ranks combine the gradient sums (global_sumsq);
 *   2. zero_lamb_moments writes m and v and, into layer_sumsq (DEVICE, 2*n_seg
 *      doubles, 16-byte aligned, caller-owned), this shard's sum theta^2 and
 *      sum u^2 of each local layer;
 *   3. the caller adds, for every layer shared with a neighbouring rank, the
 *      neighbours' entries of that layer (rank order), in place;
 *   4. zero_lamb_apply updates theta and the fp16 copy from the moments
 *      stored in step 2 and the completed layer sums.
 * Both calls take the same hyperparameters and global_sumsq; a non-finite
 * global_sumsq (gradient overflow on some rank) returns ZERO_SKIPPED from both
 * without launching anything. */
int zero_lamb_moments(const zero_lamb_plan_t* plan, const uint16_t* grad16, const float* master32, float* m32,
                      float* v32, double global_sumsq, double beta1, double beta2, double eps, double weight_decay,
                      int64_t step, double loss_scale, double clip, double* layer_sumsq, void* stream);
int zero_lamb_apply(const zero_lamb_plan_t* plan, float* master32, const float* m32, const float* v32,
                    uint16_t* param16_out, double global_sumsq, const double* layer_sumsq, double lr, double beta1,
                    double beta2, double eps, double weight_decay, int64_t step, double phi_lo, double phi_hi,
                    void* stream);

/* Kernel timing of sampled zero_lamb_step calls (the sampling period is the
 * one zero_profile_enable sets): events before the statistics, moments,
 * layer-sum and apply kernels and after the last.  zero_lamb_profile_read
 * waits for the recorded work, returns the sums since the last read and resets
 * them; a deferred profiling failure is reported as by zero_profile_read. */
typedef struct {
    int64_t steps;      /* steps timed                                  */
    double stats_ms;    /* statistics + finalize kernels                */
    double moments_ms;  /* k_lamb_moments                               */
    double layer_ms;    /* k_lamb_layer                                 */
    double apply_ms;    /* k_lamb_apply                                 */
} zero_lamb_profile_t;

int zero_lamb_profile_read(zero_lamb_profile_t* out);

/* ------------------------------------------------------------------------ */
/* Diagnostics                                                              */
/* ------------------------------------------------------------------------ */

/* Message of the calling thread's last error ("" if none).  Valid until the
 * thread's next call into the library. */
const char* zero_last_error(void);

/* Kernel timing with HIP events on the call's own stream.  With every = k > 0,
 * one zero_shard_step in k on each stream records its own three events:
 * before its statistics kernels, before its update kernel and after it (each
 * event marker costs the GPU a few microseconds, hence the sampling; for the
 * one-launch small-shard step the whole kernel counts as the update);
 * zero_shard_apply, zero_shard_apply_async and eager resident calls are
 * sampled the same way, their statistics interval covering only the
 * one-workgroup kernel; every = 0 disables.  zero_profile_read waits for the
 * recorded work, then returns the summed durations and the number of
 * profiled steps since enabling (or the last read) and resets them.  A
 * profiling failure after a step's kernels were queued never fails that step:
 * the sample is dropped and the next zero_profile_read returns ZERO_EHIP with
 * the message (the totals of the other samples are still written).
 * ZERO_EINVAL for every < 0. */
typedef struct {
    int64_t steps;      /* steps timed                                        */
    double stats_ms;    /* total time of the statistics + finalize kernels    */
    double update_ms;   /* total time of the fused update kernel              */
} zero_profile_t;

int zero_profile_enable(int32_t every);
int zero_profile_read(zero_profile_t* out);

/* Frees the per-(device, stream) workspace of `stream` on the current device
 * after waiting for the work queued on that stream (nothing to do if the
 * library holds none for it).  Call it before destroying a stream the library
 * has been used on; a later call on the stream allocates a new workspace.
 * Calls on the stream from other threads wait for the release or run on a
 * fresh workspace, never on freed memory.  Returns 0, ZERO_EINVAL (a stream of
 * another device) or ZERO_EHIP. */
int zero_stream_release(void* stream);

/* The number of per-stream workspaces and of resident-record workspaces the
 * library holds (all devices), for leak checks; either pointer may be NULL
 * (not both). */
int zero_workspace_count(int64_t* streams, int64_t* records);

/* Device-to-device copy of `bytes` bytes with the library's own streaming
 * kernel (16-byte vectors): the achievable-bandwidth reference for the update
 * kernel and the calibration kernel for hardware byte counters.  src and dst
 * must be 16-byte aligned, bytes a multiple of 16, ranges disjoint, each inside
 * one GPU-accessible allocation; ZERO_EINVAL otherwise, before any launch. */
int zero_probe_copy(const void* src, void* dst, int64_t bytes, void* stream);

/* Byte-mix probe of the Adam update: one launch over the shard's arrays with
 * the launch shape, tile walk, vector width and cache policy of the update
 * kernel, reading grad16, master32, m32, v32 and writing master32, m32, v32,
 * param16_out (28 bytes per element, as the update) with three adds and a
 * conversion per element instead of Adam: the achievable time of the
 * update's streams on this device.  The arrays it writes get meaningless
 * values.  fp32 arrays 16-byte aligned, fp16 arrays 8-byte aligned, each
 * inside one GPU allocation, no overlaps, 0 <= n <= 2^40; ZERO_EINVAL
 * otherwise, before any launch.  Enqueues only. */
int zero_probe_adam_mix(const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                        int64_t n, void* stream);

/* Byte-mix probes of the LAMB passes: one launch over the shard's arrays with
 * the launch shape, tile walk, vector width and cache policy of
 * k_lamb_moments (pass 0: reads grad16, master32, m32, v32; writes m32, v32)
 * or k_lamb_apply (pass 1: reads master32, m32, v32; writes master32,
 * param16_out), doing one or two adds per element instead of the pass's
 * arithmetic: the achievable time of that pass's streams on this device.
 * The arrays it writes get meaningless values.  fp32 arrays 16-byte aligned,
 * fp16 arrays 8-byte aligned (the array a pass does not touch may be NULL),
 * each inside one GPU allocation, no overlaps; ZERO_EINVAL otherwise, before
 * any launch.  Enqueues only. */
int zero_probe_lamb_pass(int32_t pass, const uint16_t* grad16, float* master32, float* m32, float* v32,
                         uint16_t* param16_out, int64_t n, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ZERO_SHARD_H */
