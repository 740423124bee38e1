/*
 * uad.h - C ABI of the Urgency-Aware Denoising (UAD) action-expert library
 * for AMD Instinct MI355X (gfx950).
 *
 * The library evaluates the flow-matching action expert F_theta jointly over
 * an action chunk whose tokens each carry their own flow time, attends every
 * chunk token to a cached vision-language prefix K/V and to the chunk, and
 * applies the per-token Euler update that freezes released urgent actions
 * while tail actions keep refining (Sec. 3 Eqs. 1-2; Sec. 4.2 Eqs. 3-5;
 * App. C.1 "Per-Action Time Conditioning").
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every call returns a uad_status; nothing aborts or prints.  On a non-OK
 *    status uad_last_error(ctx) holds a message naming the offending argument
 *    or tensor.  Validation happens before any device work is enqueued.
 *  - Device work is enqueued asynchronously on the context's HIP stream.
 *    Caller-owned device buffers (x, t, dt, masks, outputs) are borrowed
 *    only for the duration of that enqueued work; keep them alive until
 *    uad_synchronize() or an equivalent synchronisation of that stream.
 *  - Token order: token m = b * chunk + i for environment b and action i.
 *    Flow time runs from t = 1 (noise) to t = 0; the Euler step is
 *    x <- x + dt * v with dt = -1/N_i for an action with budget N_i.
 *  - A context is not thread-safe; use one per host thread.
 *  - Errors of enqueued device work are reported by uad_synchronize: a
 *    device status word collects them while the work runs.
 *
 * Where this interface differs from the bare statement of the problem (the
 * four calls load_weights / set_prefix_kv / denoise_step / denoise_schedule):
 *  - uad_denoise_schedule reports device wall-clock ticks (step_ticks, n_steps
 *    + 1 entries, with uad_tick_rate_hz) instead of host nanoseconds per step,
 *    because only the device can stamp the end of a step without a sync;
 *  - uad_set_prefix_kv takes a dtype, so an fp32 prefix can be handed over
 *    without a host-side bf16 conversion;
 *  - uad_build_schedule takes max_steps, the capacity of the caller's tables;
 *  - UAD_E_UNSUPPORTED and UAD_E_RANGE are added: the first for model
 *    dimensions the kernels cannot tile, the second for fp16 operand overflow
 *    found while the work ran.
 *  - Weights are named tensors in PyTorch Linear layout [out][in], row-major:
 *      action_in.w [d][Da], action_in.b [d],
 *      time_mlp_in.w [d][2d], time_mlp_in.b [d],
 *      time_mlp_out.w [d][d], time_mlp_out.b [d],
 *      layers.<l>.attn_norm [d], layers.<l>.wq [Hq*hd][d],
 *      layers.<l>.wk [Hkv*hd][d], layers.<l>.wv [Hkv*hd][d],
 *      layers.<l>.wo [d][Hq*hd], layers.<l>.mlp_norm [d],
 *      layers.<l>.w_gate [F][d], layers.<l>.w_up [F][d], layers.<l>.w_down [d][F],
 *      final_norm [d], action_out.w [Da][d], action_out.b [Da].
 *    The action expert is a pre-norm transformer: per-token time embedding
 *    e_j = sin(w_j t), e_{j+d/2} = cos(w_j t), w_j = 1000 * 10000^(-j/(d/2)),
 *    concatenated to the projected action and passed through a SiLU MLP; then
 *    per layer RMSNorm -> Q/K/V -> attention over [prefix ; chunk] (no mask,
 *    query head j uses KV head floor(j*Hkv/Hq), scale 1/sqrt(hd)) -> output
 *    projection + residual -> RMSNorm -> GeGLU (tanh GELU) MLP + residual;
 *    final RMSNorm and action projection give the velocity.
 *  - With UAD_FLAG_ADARMS (adaptive-norm time conditioning, the pi0.5-style
 *    expert of App. C.1) the time embedding no longer enters the action token:
 *    h_0 = W_in x + b_in, and c = SiLU(W_t2 SiLU(W_t1 e(t) + b_t1) + b_t2) per
 *    token modulates every norm: for each norm site (a, b, g) = W c + b gives
 *    n = RMSNorm_unit(h) * (1 + a) + b and the branch enters the residual as
 *    h += g * branch; the final norm takes (a, b) only.  Weight names then are
 *      time_mlp_in.w [d][d] (instead of [d][2d]),
 *      layers.<l>.attn_mod.w [3d][d], layers.<l>.attn_mod.b [3d],
 *      layers.<l>.mlp_mod.w [3d][d], layers.<l>.mlp_mod.b [3d],
 *      final_mod.w [2d][d], final_mod.b [2d],
 *    rows ordered (a | b | g), replacing attn_norm, mlp_norm and final_norm.
 */
#ifndef UAD_H
#define UAD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct uad_ctx uad_ctx; /* opaque, owned by the library */

typedef enum {
  UAD_OK = 0,
  UAD_E_INVALID = 1,     /* null pointer, non-positive size, bad dtype/flag */
  UAD_E_SHAPE = 2,       /* size beyond the context's maxima, tensor shape mismatch */
  UAD_E_STATE = 3,       /* weights or prefix not loaded yet */
  UAD_E_MISSING = 4,     /* a required weight tensor is absent or duplicated */
  UAD_E_HIP = 5,         /* a HIP runtime call failed (message has hipGetErrorString) */
  UAD_E_OOM = 6,         /* device allocation failed */
  UAD_E_UNSUPPORTED = 7, /* model dimensions the kernels do not support */
  UAD_E_RANGE = 8        /* (from uad_synchronize) an fp16 operand of the enqueued work was not finite */
} uad_status;

enum { UAD_DTYPE_F32 = 0, UAD_DTYPE_BF16 = 1 };

typedef struct {
  int32_t n_layers;   /* L */
  int32_t d_model;    /* d, multiple of 32 */
  int32_t n_heads;    /* Hq */
  int32_t n_kv_heads; /* Hkv, divides Hq */
  int32_t head_dim;   /* hd in {64, 128, 256} */
  int32_t d_ff;       /* F, multiple of 32 */
  int32_t action_dim; /* Da, 1..64 */
  int32_t max_batch;  /* largest batch B of any later call */
  int32_t max_chunk;  /* largest chunk H of any later call */
  int32_t max_prefix; /* largest prefix length P */
  float rms_eps;      /* RMSNorm epsilon (1e-6 in the bundled workloads) */
  int32_t flags;      /* 0 or UAD_FLAG_ADARMS */
} uad_model_config;

/* uad_model_config.flags: adaptive-norm time conditioning (see the top). */
enum { UAD_FLAG_ADARMS = 1 };

typedef struct {
  const char *name;  /* one of the names listed above */
  const void *data;  /* host or device pointer, row-major, dense */
  int32_t dtype;     /* UAD_DTYPE_F32 or UAD_DTYPE_BF16 */
  int32_t ndim;      /* 1 or 2 */
  int64_t shape[4];
  int32_t on_device; /* 1 if data is a device pointer */
} uad_tensor;

/* Create a context on HIP device `device`.  `hip_stream` is the hipStream_t
 * on that device the context enqueues its work on; NULL selects the device's
 * null stream, so the work is ordered with everything else the caller (or
 * PyTorch's default stream) queues there.  Allocates the
 * weight store, the prefix/chunk K/V store and all activation workspace for
 * the configured maxima, including the split-K partial tiles of the batched
 * residual projections (128 KiB per compute unit) and their arrival counters,
 * which every call of the context reuses (so its calls run in stream order,
 * never overlapping).  Errors: UAD_E_INVALID (null/negative fields),
 * UAD_E_UNSUPPORTED (dimension the kernels cannot tile), UAD_E_OOM, UAD_E_HIP.
 * On error *out is set to NULL. */
uad_status uad_create(const uad_model_config *cfg, int32_t device, void *hip_stream, uad_ctx **out);

/* Free every device buffer of the context (after synchronising its stream). */
void uad_destroy(uad_ctx *ctx);

/* Message for the last non-OK status returned for this context (empty if none).
 * With ctx == NULL: the message of the last failed uad_create on this thread. */
const char *uad_last_error(const uad_ctx *ctx);

/* Re-target the context at another stream of the same device (NULL: the
 * null stream), after its queued work is done. */
uad_status uad_set_stream(uad_ctx *ctx, void *hip_stream);

/* Load the action-expert parameters theta of F_theta (Sec. 3 Eq. 1).
 * `tensors` must name every weight listed at the top exactly once, with the
 * listed shape; dtype F32 or BF16.  The large projections (time MLP, QKV, O,
 * gate/up, down) are rounded once to bf16 (nearest-even; a no-op for BF16
 * input) and held as fp16, which represents every bf16 value of magnitude in
 * [2^-14, 65504] exactly; smaller magnitudes round to the nearest fp16
 * subnormal (absolute error <= 2^-25).  Norm gains, biases and the action
 * in/out projections are kept in fp32.  The data are COPIED into
 * library-owned device memory in the kernels' packed layout; the caller may
 * free its buffers on return.  Synchronous: waits for the context's queued
 * work first, which may still read the weights being replaced.  Errors: UAD_E_MISSING (absent or
 * duplicated name, named in the message), UAD_E_SHAPE, UAD_E_INVALID (bad
 * dtype, or a projection weight that is NaN or beyond +-65504), UAD_E_HIP. */
uad_status uad_load_weights(uad_ctx *ctx, const uad_tensor *tensors, int32_t n_tensors);

/* Set the cached context of the action expert: the per-layer key/value
 * vectors of the P vision-language prefix tokens (the o, L conditioning of
 * Sec. 3 Eq. 1), for `batch` environments.  k and v are dense
 * [L][batch][P][Hkv][hd] arrays of `dtype` (F32 rounded to bf16, nearest-even),
 * host memory (on_device = 0) or device memory (on_device = 1).  COPIED into
 * the library's K/V store, where each step appends the chunk's own keys and
 * values after the prefix.  Synchronous: waits for the context's queued work
 * first, which may still read the K/V being replaced.  Errors: UAD_E_INVALID,
 * UAD_E_SHAPE (batch > max_batch, P > max_prefix), UAD_E_HIP. */
uad_status uad_set_prefix_kv(uad_ctx *ctx, const void *k, const void *v, int32_t dtype,
                             int32_t batch, int32_t prefix_len, int32_t on_device);

/* One denoising step (Sec. 3 Eq. 1 with per-token time, App. C.1; Sec. 4.2
 * Eq. 5): ONE joint evaluation v = F_theta(x, t) over all batch*chunk tokens
 * -- frozen tokens included, they remain keys/values of the others -- then the
 * per-token Euler update x_i <- x_i + dt_i * v_i for tokens with
 * mask_i == 0 and dt_i != 0; other tokens are copied unchanged (bit-identical).
 *   x      device fp32 [batch][chunk][Da], in/out
 *   t, dt  device fp32 [batch][chunk]
 *   mask   device uint8 [batch][chunk], 1 = released/frozen
 *   v_out  device fp32 [batch][chunk][Da] or NULL: receives the velocity
 * Environment b attends to prefix environment b.  Requires weights and a
 * prefix set for >= batch environments (else UAD_E_STATE).  Errors:
 * UAD_E_INVALID (null pointer, batch/chunk < 1), UAD_E_SHAPE (beyond maxima),
 * UAD_E_STATE, UAD_E_HIP. */
uad_status uad_denoise_step(uad_ctx *ctx, float *x, const float *t, const float *dt,
                            const uint8_t *mask, float *v_out, int32_t batch, int32_t chunk);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * joint step as uad_denoise_step, with the same arguments, results (bit for
 * bit) and errors, that allocates nothing.  Its kernels are launched directly
 * on the context's stream (no graph is captured or instantiated) and the
 * attention's split-KV partials use a static device array of 8 MiB per GPU,
 * held until the process ends, instead of the context's workspace.  A call
 * whose batch, chunk and prefix need more than that is refused with
 * UAD_E_SHAPE before any work.  Every context on a GPU shares that GPU's
 * array: calls that overlap on one GPU (other streams, other contexts) race;
 * the array needs no clearing between calls. */
uad_status uad_denoise_step_static(uad_ctx *ctx, float *x, const float *t, const float *dt,
                                   const uint8_t *mask, float *v_out, int32_t batch, int32_t chunk);

/* A whole per-token schedule (Sec. 4.2 Eqs. 4-5): n_steps joint steps, step k
 * using the k-th slice of the tables.
 *   x                     device fp32 [batch][chunk][Da], in/out (x_0 in, final out)
 *   t_sched, dt_sched     device fp32 [n_steps][batch][chunk]
 *   mask_sched            device uint8 [n_steps][batch][chunk]
 *   released              device fp32 [batch][chunk][Da] or NULL: a^i = x^i right
 *                         after token i's release step
 *   release_step          device int32 [batch][chunk] or NULL: that step (0-based),
 *                         left untouched for a token that is never active
 *   step_ticks            pinned host uint64 [n_steps + 1] or NULL: device
 *                         wall-clock ticks at the schedule start and after each
 *                         step (see uad_tick_rate_hz)
 * A token's release step is the last step at which it is updated: the step k
 * with mask==0 and dt!=0 whose next step has mask==1, or the final step.
 * Errors as uad_denoise_step. */
uad_status uad_denoise_schedule(uad_ctx *ctx, float *x, const float *t_sched, const float *dt_sched,
                                const uint8_t *mask_sched, int32_t n_steps, int32_t batch, int32_t chunk,
                                float *released, int32_t *release_step, uint64_t *step_ticks);

/* A whole per-token schedule from integer budgets N_i (Sec. 4.2 Eqs. 4-5),
 * with the step tables built by the library (as uad_build_schedule) and
 * finished environments compacted away: joint step k evaluates only the
 * environments that still have a token with N_i > k.  An environment whose
 * tokens are all released takes no further part (the paper's per-token
 * update leaves its states, released actions and release steps final), so
 * the results are those of uad_denoise_schedule on the same tables, to
 * rounding order (smaller steps may run other kernel variants).  The
 * adaptive-norm expert evaluates every environment every step.
 *   x                 device fp32 [batch][chunk][Da], in/out (x_0 in, final out)
 *   budgets           host int32 [batch][chunk], each in 1..64; the tables are
 *                     rebuilt and uploaded (waiting for the context's queued work)
 *                     only when the budgets differ from the previous call's
 *   released, release_step, step_ticks  as uad_denoise_schedule
 *                     (step_ticks has max N_i + 1 entries)
 * Errors: UAD_E_INVALID (null x/budgets, a budget outside 1..64), UAD_E_SHAPE,
 * UAD_E_STATE, UAD_E_HIP. */
uad_status uad_denoise_budgets(uad_ctx *ctx, float *x, const int32_t *budgets, int32_t batch, int32_t chunk,
                               float *released, int32_t *release_step, uint64_t *step_ticks);

/* Urgency-aware release of one chunk per environment (Sec. 4.2-4.4, App. C).
 * Tokens i < U are urgent: they take K steps of size 1/K while the tail takes
 * the canonical N* steps of 1/N*, all in ONE joint evaluation per step (N*
 * evaluations in total, none extra).  After step K the urgent actions
 * a^i = x_K^i are released; then, by mode:
 *   UAD_RELEASE_UAER  plain early release: urgent tokens stay frozen (t = 0) as
 *                     context for the remaining N* - K steps;
 *   UAD_RELEASE_TR    Trajectory Reconciliation (Sec. 4.3 Eqs. 6-7): their
 *                     states are rebuilt from the cached velocities,
 *                     x'_K = x_0 + (1/N*) sum_{k<=K} v_k (flow-time convention
 *                     of the integrator: dt* = -1/N*), and continue as ghost
 *                     states at the tail's flow time 1 - k/N*; with K = 1 the
 *                     tail and the ghosts reproduce the uniform N*-step
 *                     schedule bit for bit.
 * Ghost Action Correction (Sec. 4.4 Eqs. 8-9, TR only): with executed_out,
 * E = sum_{i<U} (a'^i - a^i) over the ghost actions a'^i = x'^i_{N*}, and
 * the executed chunk is a^0..a^{U-1} (released, unchanged) followed by
 * x^i_{N*} + E/(S - U) for i = U .. S-1 on the dimensions gac_mask selects.
 *   x             device fp32 [batch][chunk][Da]: x_0 in; final states out
 *                 (ghost states x'_{N*} for i < U with TR, frozen x_K without)
 *   U, K, N*, S   1 <= U < S <= chunk, 1 <= K < N* <= 64
 *   urgent_out    device fp32 [batch][U][Da]: the released urgent actions
 *   executed_out  device fp32 [batch][S][Da] or NULL (requires UAD_RELEASE_TR)
 *   gac_mask      device uint8 [Da] or NULL: 1 = additive dimension corrected,
 *                 0 = left as denoised (e.g. a gripper); NULL corrects all
 *   urgent_host   pinned host fp32 [batch][U][Da] or NULL: receives a copy of
 *                 the urgent actions as soon as step K is done, while the
 *                 tail keeps denoising on the context's stream (App. C,
 *                 asynchronous execution).  Page-locked memory (hipHostMalloc,
 *                 torch pin_memory) is written by the release kernel itself
 *                 through its device address; other host memory gets a copy
 *                 on a separate release stream (slower)
 *   release_event hipEvent_t or NULL: recorded when the urgent actions (and
 *                 their host copy, if requested) are final; a controller waits
 *                 on it instead of on the whole chunk
 *   step_ticks    pinned host uint64 [N* + 1] or NULL, as uad_denoise_schedule
 * Asynchronous like uad_denoise_schedule; caller buffers must outlive the
 * work.  Errors: UAD_E_INVALID (null x/urgent_out, bad U, K, N* or S, bad mode, GAC
 * without TR), UAD_E_SHAPE, UAD_E_STATE, UAD_E_HIP. */
enum { UAD_RELEASE_UAER = 0, UAD_RELEASE_TR = 1 };
uad_status uad_denoise_release(uad_ctx *ctx, float *x, int32_t batch, int32_t chunk, int32_t U, int32_t K,
                               int32_t Nstar, int32_t S, int32_t mode, float *urgent_out, float *executed_out,
                               const uint8_t *gac_mask, float *urgent_host, void *release_event,
                               uint64_t *step_ticks);

/* Build the per-step tables from integer budgets N_i (Sec. 4.2 Eq. 4): pure
 * host code, no context needed.  budgets: host int32 [batch][chunk], each in
 * 1..max_steps.  Outputs (host, caller-allocated, capacity max_steps slices):
 * *n_steps = max N_i; t[k] = (N_i - min(k, N_i)) / N_i (fp32 division of
 * integers); dt[k] = -(1/N_i) while k < N_i, else 0; mask[k] = (k >= N_i).
 * Errors: UAD_E_INVALID (null pointer, size < 1, a budget outside 1..max_steps). */
uad_status uad_build_schedule(const int32_t *budgets, int32_t batch, int32_t chunk, int32_t max_steps,
                              int32_t *n_steps, float *t, float *dt, uint8_t *mask);

/* Average action-availability latency of a controller that executes actions in
 * order, each for t_act, starting each action as soon as it is released and
 * the previous one finished (App. B timing model, App. C.3 measurement):
 * AAL = (sum of waits) / n.  release[j] is the release time of executed
 * action j measured from the request.  Pure host code. */
uad_status uad_aal(const double *release, int32_t n, double t_act, double *aal_out);

/* Block the host until all work enqueued on the context's stream is done,
 * then read and clear the context's device status word: UAD_E_RANGE when a
 * GEMM or attention operand rounded to fp16 was not finite (|value| > 65504,
 * or NaN) since the last call, UAD_E_HIP when an in-kernel wait gave up; the
 * results of that work are then invalid.  Errors: UAD_E_HIP, UAD_E_RANGE. */
uad_status uad_synchronize(uad_ctx *ctx);

/* Device wall-clock tick rate (Hz) of the counter written to step_ticks. */
uad_status uad_tick_rate_hz(uad_ctx *ctx, double *hz);

/* Test hook: when enabled, steps skip F_theta and use the synthetic velocity
 * field v = alpha * x + beta, so the integrator and schedule can be checked
 * against the closed-form Euler solution. */
uad_status uad_debug_velocity_field(uad_ctx *ctx, int32_t enable, float alpha, float beta);

/* Measurement hook: while enabled, every kernel launch of a step is bracketed
 * by a pair of HIP events recorded on the context's stream, grouped by kernel
 * class.  Enabling resets the totals. */
uad_status uad_profile_enable(uad_ctx *ctx, int32_t enable);

/* Read the totals of kernel class `index` (0-based; UAD_E_INVALID past the
 * last class): its name (NUL-terminated, truncated to name_cap), the summed
 * event-measured duration in milliseconds and the number of launches.
 * Synchronises the context's stream first. */
uad_status uad_profile_read(uad_ctx *ctx, int32_t index, char *name, int32_t name_cap, double *total_ms,
                            int64_t *launches);

#ifdef __cplusplus
}
#endif

#endif /* UAD_H */
