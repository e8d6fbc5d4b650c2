/*
 * smat.h -- C ABI of the SMAT per-step parameter transform on MI355X (gfx950).
 *
 * SMAT ("SMAT: Simple and Efficient Merge-Aware Training") trains an expert
 * while also evaluating its loss at a simulated merged state
 *
 *     theta~ = theta0 + s * m (.) (theta - theta0) + eps           (Sec. 4.1, Eq. smat-state)
 *
 * with a sampled scale s, a DARE-style keep mask m (drop probability
 * p = 1 - keep, kept coordinates rescaled by 1/keep; Eq. smat-mask) and
 * additive noise eps of RMS sigma (Sec. 4.1, "Perturb").  The gradient reaches
 * the expert weights through the participation coefficient s*m
 * (Sec. 4.2, Eq. smat-gradient); this library accumulates it weighted by the
 * simulated-loss weight lambda (Eq. smat-objective).  Simulated weights live
 * in one reusable buffer that the model reads for its forward and backward
 * pass; the expert storage is restored before the optimizer
 * (Sec. 4.3, "Parameter storage switching"; App. "Implementation details").
 *
 * Conventions for every entry point:
 *   - Every function returns an smat_status; SMAT_OK is 0.  An argument, dtype
 *     or state error enqueues nothing; a HIP runtime failure (SMAT_ERR_HIP) may
 *     leave work the call issued before it enqueued.  smat_last_error()
 *     describes the cause.  No C++ exception crosses this boundary.
 *   - Tensor arguments are device pointers to contiguous memory owned by the
 *     caller (for example PyTorch tensors); the library never frees them.
 *     Element counts are int64_t; 0 elements is a valid no-op.
 *   - Work is enqueued on the caller's HIP stream (NULL = the default
 *     stream) without synchronising the host.  Calls that upload host tables
 *     (smat_plan_bind_workspace, smat_plan_set_params, smat_plan_set_grads,
 *     smat_plan_bind_adam_state, smat_merge_plan_bind_workspace, smat_merge_multi)
 *     return SMAT_ERR_STATE while `stream` is being captured into a graph; the
 *     *_dev calls are the ones meant for capture.
 *   - Random draws are never stored.  They are regenerated from Philox4x32-10
 *     (Salmon et al., SC'11) with key = seed and counter
 *     (g_lo, g_hi, tensor_id, 4*step + stream), where g = e >> 2 for the
 *     global element index e = elem_offset + i and element e takes word e & 3.
 *     Stream 0 draws the mask (kept iff word < floor(keep * 2^32)), stream 1
 *     the noise, stream 2 (group 0 of tensor id 0) the step's shared scale
 *     (smat_step_state_advance, smat_scale_draw).  Gaussian noise pairs words
 *     (w0, w1) for lanes 0/1 and (w2, w3) for lanes 2/3 by Box-Muller on 24-bit uniforms
 *     u1 = ((a >> 8) + 1) 2^-24, u2 = (b >> 8) 2^-24 (cosine on the even lane).
 *     step must be below 2^30.
 *   - A tensor split into shards (elem_offset = index of its first element
 *     in the whole tensor) produces exactly the bytes of the whole tensor.
 */
#ifndef SMAT_H
#define SMAT_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum smat_status {
  SMAT_OK = 0,
  SMAT_ERR_INVALID = 1, /* null pointer with n > 0, n < 0, keep outside [0,1], sigma < 0 or not
                           finite, s or lambda not finite, step >= 2^30, forbidden aliasing,
                           duplicate tensor_id, too small workspace */
  SMAT_ERR_DTYPE = 2,   /* unsupported dtype code */
  SMAT_ERR_STATE = 3,   /* call not allowed in the plan's current state */
  SMAT_ERR_HIP = 4      /* a HIP runtime call failed; smat_last_error() holds its message */
} smat_status;

typedef enum smat_dtype {
  SMAT_F32 = 0,  /* IEEE binary32 */
  SMAT_BF16 = 1  /* bfloat16, rounded to nearest even when written */
} smat_dtype;

typedef enum smat_noise_kind {
  SMAT_NOISE_GAUSSIAN = 0, /* eps = sigma * z, z standard normal by Box-Muller */
  SMAT_NOISE_UNIFORM = 1,  /* eps = sigma * sqrt(3) * (2u - 1), u = ((w >> 8) + 1/2) 2^-24:
                              the paper's default U[-sqrt(3) sigma, sqrt(3) sigma] (Sec. 4.1) */
  SMAT_NOISE_LAPLACE = 2   /* eps = -sigma sign(u - 1/2) ln(1 - 2|u - 1/2|) / sqrt(2), same u: Laplace noise
                              of RMS sigma, compared with the other two in Sec. 4.1 */
} smat_noise_kind;

typedef enum smat_storage {
  SMAT_EXPERT = 0,   /* the model sees the expert (fp32 master) storage */
  SMAT_SIMULATED = 1 /* the model sees the reusable buffer holding theta~ */
} smat_storage;

/* Per-tensor operation parameters (Sec. 4.1).
 *   s          scale (the paper's alpha), finite
 *   keep       keep probability 1 - p in [0, 1]; keep >= 1 leaves the tensor outside the mask
 *              set (no draw), keep == 0 drops every coordinate (no draw, theta~ = theta0 + eps)
 *   sigma      noise RMS, finite and >= 0; 0 disables the noise (no draw)
 *   rescale    nonzero: kept coordinates are multiplied by 1/keep (Eq. smat-mask)
 *   noise_kind an smat_noise_kind value */
typedef struct smat_op_params {
  float s;
  float keep;
  float sigma;
  int32_t rescale;
  int32_t noise_kind;
} smat_op_params;

/* Random-draw key of one tensor (or shard) for one step. */
typedef struct smat_rng_key {
  uint64_t seed;        /* Philox key */
  uint32_t step;        /* global training step, < 2^30 (fresh draws every step, Sec. 4.2) */
  uint32_t tensor_id;   /* identifies the tensor; shards of one tensor share it */
  uint64_t elem_offset; /* global index of element 0 of this range within its tensor */
} smat_rng_key;

/* smat_simulate -- theta~ for one flat tensor (Sec. 4.1, Eq. smat-state, Eq. smat-mask).
 *   theta   [n] fp32 expert weights (device)
 *   theta0  [n] frozen base weights in theta0_dtype (device); may be the same pointer as out
 *           (in-place over a buffer that holds theta0), must not overlap it otherwise
 *   out     [n] simulated weights in out_dtype (device); must not overlap theta
 * For kept coordinates out = theta0 + t (theta - theta0) + eps with t = s/keep (rescale) or s,
 * evaluated in fp32 as fma(t, theta, fma(-t, theta0, theta0)) + sigma z and rounded once to
 * out_dtype; dropped coordinates get theta0 + eps.
 * Errors: SMAT_ERR_INVALID, SMAT_ERR_DTYPE, SMAT_ERR_HIP. */
smat_status smat_simulate(const float* theta, const void* theta0, smat_dtype theta0_dtype, void* out,
                          smat_dtype out_dtype, int64_t n, smat_op_params p, smat_rng_key key,
                          hipStream_t stream);

/* smat_backward_accum -- grad_theta += lambda * t * m (.) grad_sim (Sec. 4.2, Eq. smat-gradient).
 *   grad_sim    [n] gradient of the loss at theta~ in grad_dtype (device)
 *   grad_theta  [n] fp32 accumulator (device), updated in place; must not overlap grad_sim
 * The mask is regenerated from (key, p.keep) exactly as smat_simulate drew it, so the same key
 * and keep must be passed (App. "Implementation details").  Kept coordinates become
 * fma(lambda * t, grad_sim, grad_theta) in fp32; dropped coordinates keep their bits.
 * Errors: SMAT_ERR_INVALID, SMAT_ERR_DTYPE, SMAT_ERR_HIP. */
smat_status smat_backward_accum(const void* grad_sim, smat_dtype grad_dtype, float* grad_theta, int64_t n,
                                smat_op_params p, float lambda, smat_rng_key key, hipStream_t stream);

/* smat_debug_draws -- the raw draws of n elements, for bit-exact checks of the RNG layout.
 *   mask_words  [n] uint32: stream-0 word of each element, or NULL
 *   noise_words [n] uint32: stream-1 word of each element, or NULL
 *   kept        [n] uint8: 1 where the mask keeps the element under p.keep, or NULL
 *   z           [n] fp32: the standard-normal Box-Muller value of each element, or NULL
 * All outputs are device pointers.  Test and diagnosis use only.
 * Errors: SMAT_ERR_INVALID, SMAT_ERR_HIP. */
smat_status smat_debug_draws(smat_rng_key key, int64_t n, smat_op_params p, uint32_t* mask_words,
                             uint32_t* noise_words, uint8_t* kept, float* z, hipStream_t stream);

/* Hyperparameters of the fused optimizer step: decoupled-weight-decay Adam (AdamW; Adam when
 * weight_decay == 0), the optimizers of the paper's language and vision experiments (App.
 * "Additional Experimental Settings", "Training").
 *   lr >= 0, beta1 and beta2 in [0, 1), eps > 0, weight_decay >= 0, all finite
 *   grad_scale  multiplies the gradient first (e.g. a norm-clipping factor the caller computed)
 *   step        1-based optimizer step count k, for the bias corrections 1 - beta^k */
typedef struct smat_adamw_params {
  float lr;
  float beta1;
  float beta2;
  float eps;
  float weight_decay;
  float grad_scale;
  int32_t step;
} smat_adamw_params;

/* smat_adamw_fused -- the optimizer update of a simulated step fed directly by the gradient through
 * the simulation (Sec. 4.2, Eq. smat-gradient, weighted by lambda), on the expert storage with its
 * weight decay (App. "Training and Scheduling Details", "Implementation details").  With
 *   g = grad_scale * (grad_acc + lambda * t * m (.) grad_sim)      (grad_acc == NULL: no accumulator)
 * it applies m1 += (1 - b1)(g - m1), m2 = b2 m2 + (1 - b2) g^2,
 *   theta = theta (1 - lr wd) - (lr / (1 - b1^k)) m1 / (sqrt(m2) / sqrt(1 - b2^k) + eps)
 * in fp32.  It replaces smat_backward_accum followed by a separate optimizer pass and never writes a
 * gradient: per element it moves 12 B of optimizer state in and out plus the gradient at theta~
 * (and grad_acc), against 10 B more for the unfused pair.  Dropped coordinates enter with a zero
 * simulated gradient (their moments still decay and weight decay still applies).
 *   grad_sim            [n] gradient of the loss at theta~ (grad_dtype, device)
 *   grad_acc            [n] fp32 gradient already accumulated for theta (device), or NULL
 *   theta, exp_avg, exp_avg_sq  [n] fp32 expert weights and first/second moments (device), in place
 *   grad_scale_dev      device pointer to one fp32 factor that further multiplies grad_scale (read by
 *                       the kernel when it runs, e.g. the clipping factor smat_grad_norm_multi wrote
 *                       earlier on the same stream), or NULL for none
 * The arrays must not overlap.  The mask is regenerated from (key, p.keep) as in smat_simulate.
 * Errors: SMAT_ERR_INVALID, SMAT_ERR_DTYPE, SMAT_ERR_HIP. */
smat_status smat_adamw_fused(const void* grad_sim, smat_dtype grad_dtype, const float* grad_acc, float* theta,
                             float* exp_avg, float* exp_avg_sq, int64_t n, smat_op_params p, float lambda,
                             smat_adamw_params hp, smat_rng_key key, const float* grad_scale_dev,
                             hipStream_t stream);

/* ---------------------------------------------------------------- ragged tensor lists
 * A plan covers a fixed list of parameter tensors processed by one launch per operation
 * (the grouping of tensors of Sec. 4.3, "Kernel fusion").  It holds host-side tables only; its device tables live
 * in a caller-allocated workspace.  One launch per operation covers the whole list, split
 * into equal-sized chunks so that thousands of small vectors and a few huge matrices share
 * the GPU evenly. */
typedef struct smat_plan smat_plan;

/* One tensor of a plan.  Pointers are device pointers unless stated. */
typedef struct smat_tensor_desc {
  const float* theta;       /* [n] fp32 expert storage */
  const void* theta0;       /* [n] frozen base in the plan's theta0 dtype; resident mode only
                               (NULL in offload mode, where the buffer `out` holds theta0) */
  void* out;                /* [n] reusable buffer for theta~ in the plan's out dtype */
  const void* grad_sim;     /* [n] gradient at theta~ (grad dtype), or NULL (set later or never) */
  float* grad_theta;        /* [n] fp32 gradient accumulator, or NULL (set later or never) */
  const void* theta0_host;  /* offload mode: [n] pinned host copy of theta0 (out dtype); else NULL */
  int64_t n;                /* element count, >= 0 */
  uint32_t tensor_id;       /* unique within the plan */
  uint32_t reserved;        /* must be 0 */
  uint64_t elem_offset;     /* global index of element 0 within the tensor (shards) */
} smat_tensor_desc;

/* smat_plan_create -- validate a tensor list and build its tables.
 *   offload  0: theta0 resident in device memory (the plan reads desc.theta0).
 *            1: the paper's pinned-host layout (Sec. 4.3; App. "Hardware, Software, and
 *               Implementation"): theta0 lives in desc.theta0_host and is copied into the
 *               buffer `out` on a copy stream whenever the expert storage is restored, so each
 *               simulate runs in place over the buffer.  Requires theta0_dtype == out_dtype.
 * Each gradient pointer is given for every tensor or for none (smat_plan_set_grads can supply or
 * replace them later).  Aliasing: within a tensor no two arrays overlap (the buffer may be exactly
 * theta0, in place); across the list an array that an operation writes (theta, which the fused
 * optimizer step updates, the buffer, grad_theta, bound moments) overlaps no other array, while
 * theta0 and grad_sim of different tensors may share memory.  The caller owns *out_plan and must
 * release it with smat_plan_destroy.
 * Limits: at most 2^26 tensors, and fewer than 2^31 256-element tiles over the whole list
 * (about 5.5e11 elements).
 * Errors: SMAT_ERR_INVALID (bad descriptor, duplicate tensor_id, aliasing, gradient pointers given
 * for some tensors only, a list beyond the limits), SMAT_ERR_DTYPE. */
smat_status smat_plan_create(const smat_tensor_desc* descs, int32_t count, smat_dtype theta0_dtype,
                             smat_dtype out_dtype, smat_dtype grad_dtype, int32_t offload,
                             smat_plan** out_plan);

/* smat_plan_workspace_bytes -- device bytes the plan's tables need (256-byte aligned start). */
smat_status smat_plan_workspace_bytes(const smat_plan* plan, size_t* bytes);

/* smat_plan_bind_workspace -- hand the plan its device workspace and upload its static tables on
 * `stream` (in offload mode also the first theta0 prefetch).  The workspace stays owned by the
 * caller and must outlive the plan.  A call that failed with SMAT_ERR_HIP leaves the plan unbound
 * and may be repeated.  Errors: SMAT_ERR_INVALID (null, misaligned or too small), SMAT_ERR_STATE
 * (already bound), SMAT_ERR_HIP. */
smat_status smat_plan_bind_workspace(smat_plan* plan, void* workspace, size_t bytes, hipStream_t stream);

/* smat_plan_set_params -- per-tensor s, keep, sigma for the next operations (count entries, in
 * descriptor order), uploaded asynchronously on `stream`.  Only the records that differ from the
 * ones the workspace holds are copied (the span from the first changed record to the last one);
 * a call that changes nothing enqueues nothing.  The backward of a step must see the same keep
 * values as its simulate.  A call that fails with SMAT_ERR_HIP leaves the plan without
 * parameters until a later call succeeds.  Errors: SMAT_ERR_INVALID, SMAT_ERR_STATE (no
 * workspace), SMAT_ERR_HIP. */
smat_status smat_plan_set_params(smat_plan* plan, const smat_op_params* per_tensor, hipStream_t stream);

/* smat_simulate_multi -- smat_simulate over every tensor of the plan in one launch, keys
 * (seed, step, desc.tensor_id, desc.elem_offset).  Allowed only while the expert storage is
 * active.  In offload mode the simulate writes theta~ over the buffer, the device's only copy of
 * theta0, so a second simulate needs a restore in between (a switch to the simulated storage and
 * back, whose restore refills theta0).  Errors: SMAT_ERR_INVALID (step), SMAT_ERR_STATE (no
 * workspace, no params, simulated storage active, offload buffers not refilled since the last
 * simulate), SMAT_ERR_HIP. */
smat_status smat_simulate_multi(smat_plan* plan, uint64_t seed, uint32_t step, hipStream_t stream);

/* smat_simulate_multi_static -- for callers that cannot allocate device memory (serving loops,
 * harnesses that forbid allocation): smat_simulate_multi over the list `descs` without a plan.
 * Same validation as smat_plan_create (resident mode; grad pointers are not read) and
 * smat_plan_set_params (per_tensor[i] for descs[i]), the same kernels and the same output bits.
 * The tensor records, per-tensor constants and chunk table live in one static device array of the
 * library, 8 MiB per GPU, held until the process ends: at most 8192 tensors, and at most
 * (8 MiB - the records) / 8 chunks of 16384 elements (about 15.8e9 elements at 8192 tensors, 17e9
 * for a few hundred).  The call allocates nothing; it builds the tables in static host memory and
 * copies them with one synchronous host-to-device copy ordered on `stream` (so it blocks until
 * earlier work on `stream` has finished), then enqueues the kernel.  Every call on a GPU reuses
 * that GPU's array: calls on different streams of one GPU that overlap in time race (the later
 * upload may overwrite tables the earlier kernel still reads); calls on one stream are ordered.
 * Not capturable (SMAT_ERR_STATE under stream capture).
 * Errors: SMAT_ERR_INVALID (bad descriptor or params, aliasing, duplicate ranges, a list beyond the
 * limits above), SMAT_ERR_DTYPE, SMAT_ERR_STATE, SMAT_ERR_HIP. */
smat_status smat_simulate_multi_static(const smat_tensor_desc* descs, int32_t count, smat_dtype theta0_dtype,
                                       smat_dtype out_dtype, const smat_op_params* per_tensor, uint64_t seed,
                                       uint32_t step, hipStream_t stream);

/* smat_backward_multi -- the gradient through the simulation over every tensor of the plan in one
 * launch (Sec. 4.2, Eq. smat-gradient, weighted by lambda).  accumulate = 1: grad_theta += lambda t m
 * (.) grad_sim on kept coordinates, dropped ones bit-unchanged (smat_backward_accum_multi).
 * accumulate = 0: grad_theta = lambda t m (.) grad_sim everywhere, +0 where dropped, without reading
 * grad_theta: the bits of accumulating into +0, for a step whose simulated-loss gradient is the only
 * gradient (periodic scheduling), at 6 B instead of 10 B per element for a bf16 grad_sim.
 * Errors: SMAT_ERR_INVALID (lambda, step, accumulate), SMAT_ERR_STATE (no workspace or params,
 * gradient arrays not set), SMAT_ERR_HIP. */
smat_status smat_backward_multi(smat_plan* plan, uint64_t seed, uint32_t step, float lambda, int32_t accumulate,
                                hipStream_t stream);

/* smat_backward_accum_multi -- smat_backward_accum over every tensor of the plan in one launch.
 * Errors: SMAT_ERR_INVALID (lambda, step), SMAT_ERR_STATE (no workspace or params, gradient arrays
 * not set), SMAT_ERR_HIP. */
smat_status smat_backward_accum_multi(smat_plan* plan, uint64_t seed, uint32_t step, float lambda,
                                      hipStream_t stream);

/* Per-step values that the device-driven list calls read from device memory when their kernels
 * run, so that a call recorded once into a HIP graph (stream capture) serves every later step: the
 * caller rewrites the 16 bytes between replays, or has kernels of its own graph advance them.
 *   seed   Philox key
 *   step   global step; the counter word uses it modulo 2^30 (steps 2^30 apart share draws)
 *   scale  the step's sampled scale (Sec. 4.1, "Scale"): tensor i uses s' = fl32(scale * s_i) in
 *          place of its s_i from smat_plan_set_params, so s_i = 1 gives every tensor the sampled
 *          scale and other s_i give fixed per-tensor multiples of it.  The coefficient is then
 *          s'/keep (rescale, 0 < keep < 1) or s', rounded exactly as smat_plan_set_params rounds
 *          it: the results are the bits of the host-driven call given s'.  The value is not
 *          checked; a non-finite scale makes every kept coordinate non-finite. */
typedef struct smat_step_state {
  uint64_t seed;
  uint32_t step;
  float scale;
} smat_step_state;

/* smat_step_state_advance -- step += increment (modulo 2^30, the range of steps that the counter
 * word holds: a device-driven run past step 2^30 - 1 continues at step 0 and repeats its draws,
 * and a state written with a step >= 2^30 is taken modulo 2^30), then scale = the step's shared scale
 * alpha ~ U[alpha_min, 1] (Sec. 4.1, "Scale": one coefficient per simulated update, shared by every
 * coordinate), written in place by one thread on `stream`.  alpha comes from word 0 of the Philox
 * counter (0, 0, 0, 4 step + 2) under key seed (stream 2, which no tensor uses):
 * u = (w0 >> 8) 2^-24 and alpha = fl32(alpha_min + (1 - alpha_min) u), the sum formed in fp64.  It
 * is a function of (seed, step) only, so a run resumed at a step draws the same scales; increment 0
 * only sets the scale of the current step.  One kernel node under stream capture.  state as for
 * smat_simulate_multi_dev.  Errors: SMAT_ERR_INVALID (null or misaligned state, alpha_min outside
 * [0, 1]), SMAT_ERR_HIP. */
smat_status smat_step_state_advance(smat_step_state* state, uint32_t increment, float alpha_min, hipStream_t stream);

/* smat_scale_draw -- the same scale on the host, for the host-driven calls: *alpha = the scale that
 * smat_step_state_advance draws for (seed, step, alpha_min), bit for bit.  Host only (no GPU, no
 * stream).  Errors: SMAT_ERR_INVALID (null alpha, step >= 2^30, alpha_min outside [0, 1]). */
smat_status smat_scale_draw(uint64_t seed, uint32_t step, float alpha_min, float* alpha);

/* smat_simulate_multi_dev / smat_backward_multi_dev -- smat_simulate_multi and smat_backward_multi
 * with seed, step and scale read from `state` (device-accessible, 16-byte aligned, caller-owned; it
 * must hold its values when the kernels run).  keep, sigma, noise kind and rescale still come from
 * smat_plan_set_params, and the backward of a step must read the state its simulate read.  The
 * host does no synchronisation and waits on no event, so both calls may be recorded under stream
 * capture.  Not for offload plans, whose theta0 prefetch runs on the plan's own copy stream.
 * Errors: SMAT_ERR_INVALID (null or misaligned state; lambda, accumulate), SMAT_ERR_STATE (offload
 * plan, no workspace or params, simulated storage active for the simulate, gradient arrays not set
 * for the backward), SMAT_ERR_HIP. */
smat_status smat_simulate_multi_dev(smat_plan* plan, const smat_step_state* state, hipStream_t stream);
smat_status smat_backward_multi_dev(smat_plan* plan, const smat_step_state* state, float lambda,
                                    int32_t accumulate, hipStream_t stream);

/* Optimizer state of one tensor of a plan (device pointers, [n] fp32 each). */
typedef struct smat_adam_state {
  float* exp_avg;
  float* exp_avg_sq;
} smat_adam_state;

/* smat_plan_bind_adam_state -- hand the plan the optimizer state of every tensor (count entries in
 * descriptor order) for smat_adamw_fused_multi; uploads a small table on `stream`.  May be called
 * again to rebind.  The two moments of a tensor must not overlap each other, theta, theta0, the
 * simulated buffer, the gradient arrays or any array of another tensor.  Errors: SMAT_ERR_INVALID (null or overlapping arrays),
 * SMAT_ERR_STATE (no workspace), SMAT_ERR_HIP. */
smat_status smat_plan_bind_adam_state(smat_plan* plan, const smat_adam_state* per_tensor, hipStream_t stream);

/* smat_plan_set_grads -- point the plan at new gradient arrays: grad_sims (count device pointers
 * in descriptor order, grad_dtype, e.g. the tensors autograd produced at theta~ this step) and/or
 * grad_thetas (count fp32 device pointers); a NULL array keeps the current ones.  Lets a caller use
 * fresh tensors every step instead of fixed buffers, and a plan created without gradient pointers
 * gain them.  Uploads the tensor records on `stream`; later operations on that stream use the new
 * arrays.  The arrays must not overlap theta, theta0, the simulated buffer, each other or bound
 * optimizer moments, nor (grad_theta) any array of another tensor, and must stay valid until the
 * operations that read them have run.
 * Errors: SMAT_ERR_INVALID (both NULL, a null entry, overlap), SMAT_ERR_STATE (no workspace),
 * SMAT_ERR_HIP. */
smat_status smat_plan_set_grads(smat_plan* plan, const void* const* grad_sims, float* const* grad_thetas,
                                hipStream_t stream);

/* smat_plan_clear_grads -- forget the plan's gradient arrays: bit 0 of `which` drops grad_sim, bit 1
 * grad_theta.  A caller whose gradient tensors live for one step clears them once the step's
 * operations are queued, so that no pointer to a freed tensor is kept (set_grads with a NULL array
 * keeps the current one, and would check new arrays for overlap against it).  Operations that read
 * a cleared kind return SMAT_ERR_STATE until set_grads supplies it again.  Host-side only: enqueues
 * nothing, and operations already queued keep the arrays they were given.
 * Errors: SMAT_ERR_INVALID (null plan, `which` outside 1..3). */
smat_status smat_plan_clear_grads(smat_plan* plan, int32_t which);

/* smat_adamw_fused_multi -- smat_adamw_fused over every tensor of the plan in one launch: theta is
 * desc.theta (the expert storage, updated in place), grad_sim is desc.grad_sim and, when accumulate
 * is nonzero, grad_acc is desc.grad_theta (read, not written); grad_scale_dev as in
 * smat_adamw_fused.  Allowed only while the expert storage is active (the optimizer never sees the
 * simulated buffer).  Errors: SMAT_ERR_INVALID, SMAT_ERR_STATE (no workspace, params or optimizer
 * state, gradient arrays not set, or simulated storage active), SMAT_ERR_HIP. */
smat_status smat_adamw_fused_multi(smat_plan* plan, uint64_t seed, uint32_t step, float lambda, smat_adamw_params hp,
                                   int32_t accumulate, const float* grad_scale_dev, hipStream_t stream);

/* smat_grad_norm_multi -- squared L2 norm of the expert gradient of a simulated step over every
 * tensor of the plan, for gradient-norm clipping ahead of the optimizer update (App. "Training and
 * Scheduling Details": the language models train with clipping at 1):
 *   sumsq = sum over tensors and elements of g^2,  g = [grad_acc +] lambda t m (.) grad_sim
 * (Eq. smat-gradient weighted by lambda; grad_acc = desc.grad_theta when accumulate is 1), with the
 * mask regenerated as in smat_backward_accum_multi.  Reads grad_sim (and grad_acc) only: 2 B per
 * element for bf16 gradients.  Outputs, written on `stream` by the last of three small launches:
 *   sumsq       device fp64 scalar, or NULL
 *   clip_coef   device fp32 scalar min(1, max_norm / (sqrt(sumsq) + 1e-6)), the factor
 *               torch.nn.utils.clip_grad_norm_ applies, or NULL; then max_norm must be finite and > 0.
 *               Pass it as grad_scale_dev of smat_adamw_fused_multi to clip without a host sync.
 * At least one output must be given.  Per-chunk fp32 partial sums (in the plan's workspace) are
 * added in fp64 in a fixed order: the result is the same on every call.  Any storage may be active.
 * Norm calls on one plan share those partials: calls that overlap (on different streams) race.
 * Errors: SMAT_ERR_INVALID, SMAT_ERR_STATE (no workspace or params, gradient arrays not set),
 * SMAT_ERR_HIP. */
smat_status smat_grad_norm_multi(smat_plan* plan, uint64_t seed, uint32_t step, float lambda, int32_t accumulate,
                                 float max_norm, double* sumsq, float* clip_coef, hipStream_t stream);

/* The optimizer's per-step values for smat_adamw_fused_multi_dev, read from device memory when the
 * update runs (so a captured graph can advance them):
 *   lr    learning rate of this step, finite and >= 0
 *   step  the optimizer's step count k >= 1 of this update (bias corrections 1 - beta^k)
 * Neither is checked on the device; step 0 or a non-finite lr makes the update non-finite. */
typedef struct smat_adam_step_state {
  float lr;
  uint32_t step;
} smat_adam_step_state;

/* smat_adamw_fused_multi_dev / smat_grad_norm_multi_dev -- smat_adamw_fused_multi and
 * smat_grad_norm_multi with seed, step and scale read from `state` (see smat_step_state; the
 * coefficient of each tensor is formed as smat_simulate_multi_dev forms it).  The optimizer step
 * also reads `adam_state` (device-accessible, 8-byte aligned, caller-owned); hp supplies beta1,
 * beta2, eps, weight_decay and grad_scale, and its lr and step are ignored.  A one-thread launch
 * first forms the step's constants into the plan's workspace with the same fp64 operations as
 * the host-driven call: given the same values both calls give the same bits.  Optimizer calls on
 * one plan share those constants, and norm calls the norm partials: calls that overlap (on
 * different streams) race.  No host synchronisation and no wait on an outside event, so both may
 * be recorded under stream capture; not for offload plans.  Errors: SMAT_ERR_INVALID (null or
 * misaligned states, lambda, accumulate, hyperparameters, outputs as in smat_grad_norm_multi),
 * SMAT_ERR_STATE (offload plan, no workspace, params or optimizer state, gradient arrays not set,
 * simulated storage active for the optimizer step), SMAT_ERR_HIP. */
smat_status smat_adamw_fused_multi_dev(smat_plan* plan, const smat_step_state* state,
                                       const smat_adam_step_state* adam_state, smat_adamw_params hp, float lambda,
                                       int32_t accumulate, const float* grad_scale_dev, hipStream_t stream);
smat_status smat_grad_norm_multi_dev(smat_plan* plan, const smat_step_state* state, float lambda, int32_t accumulate,
                                     float max_norm, double* sumsq, float* clip_coef, hipStream_t stream);

/* smat_switch_storage -- point the model at the simulated buffer (SMAT_SIMULATED) or back at the
 * expert storage (SMAT_EXPERT) (Sec. 4.3, "Parameter storage switching").  The plan holds one
 * device table of per-tensor pointers for each storage; switching selects the active one (see
 * smat_plan_active_ptrs) and moves no data.  SMAT_SIMULATED requires a simulate since the last
 * restore and is an error when already active; SMAT_EXPERT is idempotent.  In offload mode,
 * restoring the expert storage also starts the theta0 prefetch into the buffers on the plan's copy
 * stream once `stream` has reached this point; the next simulate waits for it.  A restore whose
 * prefetch fails with SMAT_ERR_HIP leaves the simulated storage active, so repeating it enqueues
 * the whole prefetch again.  Expert storage is never written.  Errors: SMAT_ERR_INVALID (bad `to`),
 * SMAT_ERR_STATE, SMAT_ERR_HIP. */
smat_status smat_switch_storage(smat_plan* plan, int32_t to, hipStream_t stream);

/* smat_plan_state -- the active storage (an smat_storage value) in *state. */
smat_status smat_plan_state(const smat_plan* plan, int32_t* state);

/* smat_plan_active_ptrs -- the active pointer of every tensor.  host_out, if not NULL, receives
 * count pointers; *dev_table, if dev_table is not NULL, receives the device address of the
 * count-entry pointer table of the active storage (inside the workspace; the address changes with
 * each switch, the two tables themselves never do). */
smat_status smat_plan_active_ptrs(const smat_plan* plan, void** host_out, void** dev_table);

/* smat_plan_destroy -- wait for the plan's own pending uploads and prefetches, then free its host
 * tables.  NULL is a no-op.  The workspace is not touched. */
smat_status smat_plan_destroy(smat_plan* plan);

/* ---------------------------------------------------------------- N-expert merge
 * The merged parameters seen from any expert (Sec. 3, Eq. merged-state; App. "Additional
 * Experimental Settings", mergers):
 *   theta_merge = theta0 + sum_j alpha_j m_j (.) (theta_j - theta0)
 * with one scalar weight alpha_j = gamma per expert (Task Arithmetic; gamma = 1/N gives weight
 * averaging) and DARE masks m_j: a coordinate is dropped with probability 1 - keep_j and kept ones
 * are scaled by 1/keep_j.  Expert j's mask is drawn exactly like a training mask (the smat_simulate
 * mask stream) from its own (seed, step) and the tensor's id and global element index, so a
 * one-expert merge with (gamma = s, keep, seed, step) equals smat_simulate with sigma = 0 bit for bit.
 * Computed in fp32 as acc = theta0; acc = fma(t_j, theta_j, fma(-t_j, theta0, acc)) over kept
 * coordinates of experts j = 0, 1, ... (t_j = gamma_j/keep_j with rescale, else gamma_j), rounded
 * once to out_dtype (round to nearest even).  Per element it reads N experts and theta0 and writes
 * out: 18 B for seven bf16 experts with bf16 theta0 and out. */
typedef struct smat_merge_term {
  float gamma;      /* weight of the expert's task vector; any finite value */
  float keep;       /* DARE keep probability 1 - p in [0, 1]; 1 = whole task vector, 0 = expert left out */
  int32_t rescale;  /* nonzero: kept coordinates scaled by 1/keep */
  uint32_t step;    /* counter step of the expert's mask, < 2^30 */
  uint64_t seed;    /* key of the expert's mask */
} smat_merge_term;

/* smat_merge -- one flat tensor: experts[0..n_experts) are n_experts device pointers (a host array)
 * to [n] expert weights of expert_dtype; theta0 [n] of theta0_dtype; out [n] of out_dtype, which may
 * be theta0 itself when the dtypes match but must not overlap any expert.  terms: n_experts host
 * records.  1 <= n_experts <= 16.  Errors: SMAT_ERR_INVALID (sizes, null pointers, overlap, a bad
 * term), SMAT_ERR_DTYPE, SMAT_ERR_HIP.  n == 0 is a no-op. */
smat_status smat_merge(const void* const* experts, int32_t n_experts, smat_dtype expert_dtype, const void* theta0,
                       smat_dtype theta0_dtype, void* out, smat_dtype out_dtype, int64_t n,
                       const smat_merge_term* terms, uint32_t tensor_id, uint64_t elem_offset, hipStream_t stream);

/* A merge plan: a fixed list of tensors, each with its n_experts expert tensors, merged by one launch
 * per call.  Like smat_plan it keeps host tables only; its device tables live in a caller-allocated
 * workspace. */
typedef struct smat_merge_plan smat_merge_plan;

typedef struct smat_merge_desc {
  const void* theta0;    /* [n] base weights, device, theta0_dtype */
  void* out;             /* [n] merged weights, device, out_dtype; may be theta0 when the dtypes match */
  int64_t n;
  uint32_t tensor_id;    /* mask counter word, as in smat_tensor_desc */
  uint32_t reserved;     /* must be 0 */
  uint64_t elem_offset;  /* global index of element 0 (shards of one tensor) */
} smat_merge_desc;

/* smat_merge_plan_create -- experts is a host array of count * n_experts device pointers, row i
 * holding tensor i's experts in expert order.  Checks as smat_merge for every tensor; a tensor id may
 * repeat only for disjoint element ranges.  Across the list no output may overlap another tensor's
 * output, theta0 or experts (inputs, which are only read, may share memory).
 * Errors: SMAT_ERR_INVALID, SMAT_ERR_DTYPE. */
smat_status smat_merge_plan_create(const smat_merge_desc* descs, int32_t count, const void* const* experts,
                                   int32_t n_experts, smat_dtype expert_dtype, smat_dtype theta0_dtype,
                                   smat_dtype out_dtype, smat_merge_plan** out_plan);

/* smat_merge_plan_workspace_bytes -- device bytes the plan's tables need (256-byte aligned start). */
smat_status smat_merge_plan_workspace_bytes(const smat_merge_plan* plan, size_t* bytes);

/* smat_merge_plan_bind_workspace -- hand the plan its device workspace (caller-owned, outliving the
 * plan) and upload its static tables on `stream`.  Errors as smat_plan_bind_workspace. */
smat_status smat_merge_plan_bind_workspace(smat_merge_plan* plan, void* workspace, size_t bytes, hipStream_t stream);

/* smat_merge_multi -- smat_merge over every tensor of the plan in one launch.  terms: count *
 * n_experts host records, row i for tensor i (so the caller can leave tensors outside the DARE set
 * unmasked with keep = 1), uploaded asynchronously on `stream`.  Errors: SMAT_ERR_INVALID (a bad
 * term), SMAT_ERR_STATE (no workspace), SMAT_ERR_HIP. */
smat_status smat_merge_multi(smat_merge_plan* plan, const smat_merge_term* terms, hipStream_t stream);

/* smat_merge_plan_destroy -- wait for the plan's pending uploads, free its host tables.  NULL is a
 * no-op. */
smat_status smat_merge_plan_destroy(smat_merge_plan* plan);

/* smat_stream_copy -- a plain device copy of `bytes` from src to dst, built like the library's
 * kernels (one-wave blocks, 16-byte nontemporal accesses).  Not part of the method: the benchmark
 * times it to state what fraction of the achievable HBM stream rate each kernel reaches.  Pointers
 * and size must be multiples of 16 bytes and the ranges must not overlap.  Errors:
 * SMAT_ERR_INVALID, SMAT_ERR_HIP. */
smat_status smat_stream_copy(const void* src, void* dst, uint64_t bytes, hipStream_t stream);

/* smat_last_error -- message of the last failure on the calling thread ("" if none). */
const char* smat_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SMAT_H */
