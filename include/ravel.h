/*
 * ravel.h -- C ABI of the MI355X rolling-denoise-step library (libravel.so).
 *
 * One call of ravel_step performs one control step of rolling flow denoising
 * for B independent environments:
 *   - one pass of the flow-matching action expert over every env's H-slot
 *     action buffer, each slot at its own flow time, conditioned on the
 *     env's latest VLM context (layer-wise prefix K/V caches) and its age,
 *     and on Fast-Observation-Pathway tokens (paper Sec. 3.1 Eq. 3, Sec. 3.2
 *     Eq. 4, App. A.1);
 *   - a per-slot Euler update, release of the now-clean first slot as the
 *     env's action, and a fresh N(0, I) action appended in its place by
 *     advancing a ring index (the rule stated right after Eq. 3).
 *
 * Time convention: logical slot i = 0..H-1 holds the action executed i+1
 * steps from now at flow time tau_i = (i+1)/H (1 = noise, 0 = clean), and a
 * step applies a_i <- a_i - (1/H) v_i.  This is the paper's Eq. 3 mirrored
 * (tau_paper = 1 - tau, v_paper = -v, K = H).
 *
 * Threading: ravel_set_context / ravel_context_acquire (the VLM worker, paper
 * Sec. 3.2 and Sec. 4.3's separate workers) may run on another host thread
 * concurrently with ravel_step (the control loop).  Two ravel_step calls on
 * one buffer must not overlap, and consecutive steps must be ordered (same
 * stream, or the caller orders them).
 *
 * Errors: every entry point returns a ravel_status and never throws; the
 * message of the calling thread's last failure is in ravel_last_error().
 * Shape and argument errors are returned synchronously.  Asynchronous device
 * faults surface as RAVEL_E_HIP on a later call that synchronises.  A failed
 * launch of the persistent layers' kernel (a grid barrier or split meeting
 * that timed out) is not left silent: that step and every step enqueued after
 * it release NaN actions and leave the ring and t unchanged, and the next
 * ravel_step / ravel_step_state / ravel_full_denoise / ravel_train_loss call
 * that finds the release kernel's pinned host flag raised (read without
 * synchronising), or the next ravel_buffer_sync / ravel_debug_state, waits for
 * the device, re-arms the kernel's counters and returns RAVEL_E_HIP; the call
 * after that runs normally from the unchanged state.
 *
 * Streams are hipStream_t values passed as void* (NULL = the default stream).
 */
#ifndef RAVEL_H
#define RAVEL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RAVEL_OK = 0,
  RAVEL_E_INVALID = -1, /* bad argument (null pointer, out-of-range value)   */
  RAVEL_E_NOMEM = -2,   /* device or host allocation failed                   */
  RAVEL_E_HIP = -3,     /* a HIP runtime call or kernel failed                */
  RAVEL_E_SHAPE = -4,   /* tensor shape or config inconsistent                */
  RAVEL_E_STATE = -5    /* call not valid in the current state (no context,
                           t_obs going backwards, missing weight, ...)        */
} ravel_status;

enum { RAVEL_F32 = 0, RAVEL_BF16 = 1 };

/* Velocity model.  TRANSFORMER is the action expert.  The two analytic fields
 * need no weights beyond one tensor and exist to pin the rolling scheduler:
 *   ANALYTIC_OT:     v_i = (x_i - a*) / tau_i      weight "analytic.target" [D_a]
 *   ANALYTIC_LINEAR: v_i = lambda * x_i            weight "analytic.lambda" [1]   */
enum { RAVEL_TRANSFORMER = 0, RAVEL_ANALYTIC_OT = 1, RAVEL_ANALYTIC_LINEAR = 2 };

typedef struct {
  int32_t layers;      /* L transformer blocks                                  */
  int32_t width;       /* w residual width (even, multiple of 8)                */
  int32_t n_q_heads;   /* query heads                                           */
  int32_t n_kv_heads;  /* KV heads (divides n_q_heads), grouped-query attention */
  int32_t head_dim;    /* hd (multiple of 32, <= 256)                           */
  int32_t mlp_dim;     /* F gated-GeLU hidden size (multiple of 16)             */
  int32_t horizon;     /* H buffer slots (the paper's K), 1..128                 */
  int32_t action_dim;  /* D_a per slot (the paper's h low-level actions folded)  */
  int32_t prefix_len;  /* P prefix tokens of the VLM context per layer (>= 0)    */
  int32_t n_fop;       /* FOP tokens per env (0 disables adapters)              */
  int32_t fop_obs_dim; /* observation size of the FOP stand-in encoder          */
  int32_t fop_stride;  /* adapter in layers l with l % stride == stride - 1     */
  int32_t dtype;       /* RAVEL_F32 or RAVEL_BF16 (bf16 weights/activations,
                          fp32 accumulation, fp32 residual stream and ring)     */
  int32_t model_kind;  /* RAVEL_TRANSFORMER / RAVEL_ANALYTIC_OT / _LINEAR        */
  float delta_bias;    /* delta_0 added to the offset p/H (Sec. 4.4, App. B.1)   */
  float rms_eps;       /* RMSNorm epsilon (1e-6)                                 */
  int32_t offset_mode; /* how the offset delta enters the expert (App. A.1):
                          RAVEL_OFFSET_MLP    an MLP of delta added to the flow-time
                                              embedding (the pi0.5 expert);
                          RAVEL_OFFSET_CONCAT delta concatenated to every slot's noisy
                                              action at the action encoder (the X-VLA
                                              expert): in.w is [w, D_a + 1], its last
                                              column multiplies delta, and the
                                              conditioning is silu(c_tau(i)) alone;
                          RAVEL_OFFSET_ADAPTER delta concatenated with the action and
                                              flow-time embeddings before an
                                              action-time MLP, whose tokens then pass
                                              a gated residual adapter conditioned on
                                              delta's sinusoidal embedding (the
                                              DynamicVLA expert, App. A.1):
                                              e_i = in.w a_i + in.b,
                                              g_i = at.w2 silu(at.w1 [e_i; emb(tau_i);
                                              delta] + at.b1) + at.b2,
                                              h_i = g_i + tanh(ta.alpha) ta.w2
                                              silu(ta.w1 [g_i; emb(delta)] + ta.b1),
                                              emb the flow-time sinusoid; the
                                              conditioning is silu(c_tau(i)) alone;
                                              w a multiple of 32                     */
  float rope_base;     /* 0: no positional encoding of the buffer tokens (the
                          paper's expert); > 0: rotary embedding of their
                          self-attention queries and keys, rotate-half pairs
                          (d, d + hd/2) turned by (P + i) base^(-2d/hd) for
                          logical slot i, the prefix keys used as given        */
} ravel_config;

enum { RAVEL_OFFSET_MLP = 0, RAVEL_OFFSET_CONCAT = 1, RAVEL_OFFSET_ADAPTER = 2 };

/* A named host or device tensor, row-major, [out, in] for linear layers.
 * dtype RAVEL_F32 or RAVEL_BF16 (raw bf16 bits).  Names and shapes:
 *   in.w [w,D_a] ([w,D_a+1] with RAVEL_OFFSET_CONCAT)  in.b [w]
 *   time.w1 [w,w] time.b1 [w] time.w2 [w,w] time.b2 [w]
 *   delta.w1 [w,1] delta.b1 [w] delta.w2 [w,w] delta.b2 [w]  (RAVEL_OFFSET_MLP only)
 *   at.w1 [w,2w+1] at.b1 [w] at.w2 [w,w] at.b2 [w]
 *   ta.w1 [w/4,2w] ta.b1 [w/4] ta.w2 [w,w/4] ta.alpha [1]     (RAVEL_OFFSET_ADAPTER only)
 *   layers.<l>.mod.w [6w,w] .mod.b [6w] .qkv.w [(nq+2nkv)hd,w] .o.w [w,nq hd]
 *   layers.<l>.gate.w [F,w] .up.w [F,w] .down.w [w,F]
 *   adapter layers: layers.<l>.fop.gamma [w] .fop.q.w [nq hd,w]
 *                   .fop.kv.w [2 nkv hd,w] .fop.o.w [w,nq hd] .fop.alpha [1]
 *   final.mod.w [3w,w] final.mod.b [3w] (third chunk unused)  out.w [D_a,w] out.b [D_a]
 *   FOP encoder (optional): fop.w1 [w,d_obs] fop.b1 [w] fop.w2 [n_fop w,w] fop.b2 [n_fop w]
 * The modulation rows of layers.<l>.mod are the chunks (s1,b1,g1,s2,b2,g2) of
 * w rows each: attention-norm scale/shift/gate, MLP-norm scale/shift/gate.  */
typedef struct {
  const char* name;
  int32_t dtype;
  int32_t rank;
  int64_t dims[4];
  const void* data;
} ravel_tensor;

typedef struct ravel_model ravel_model;
typedef struct ravel_buffer ravel_buffer;

/* Build a model on the current HIP device.  Copies every tensor (the caller
 * keeps ownership), converts to the model dtype (bf16 round-to-nearest-even)
 * and lays weights out for the kernels; precomputes each slot's flow-time
 * conditioning c_tau(i), fixed because tau_i is fixed (Sec. 3.1 after Eq. 1).
 * Synchronous.  Errors: E_SHAPE (config or tensor shape), E_STATE (missing
 * weight), E_NOMEM, E_HIP. */
ravel_status ravel_create(const ravel_config* cfg, const ravel_tensor* weights, int32_t n_weights,
                          ravel_model** out);
void ravel_destroy(ravel_model* model);

/* Bytes of device memory held by the model's weights (for roofline accounting). */
int64_t ravel_model_weight_bytes(const ravel_model* model);

/* Create the rolling state of `batch` environments.  Every slot starts as
 * pure N(0, I) noise: initial action r = 0..H-1 of env e sits in physical
 * slot r mod H and is Philox noise for (seed, e, r) (App. A.1: no additional
 * initialisation).  Noise is Philox4x32-10 (Salmon et al., SC'11) keyed by
 * (seed lo, seed hi) with counter (j/4, env, r lo, r hi) and Box-Muller in
 * float64 rounded to float32.  Synchronous.
 * Environment variables read here (each "1" to apply), for tests and comparisons:
 *   RAVEL_NO_PERSISTENT   the per-kernel path even where the persistent kernel fits;
 *   RAVEL_NO_FUSED_XATTN  a separate attention phase for the FOP adapters in the
 *                         persistent kernel (default for one env with 256-dim heads
 *                         and <= 16 FOP tokens: computed inside the output projection);
 *   RAVEL_NO_SIDE_MOD     the modulation of every layer in one launch before the
 *                         persistent kernel (default: layer 0's only, the others
 *                         computed by blocks the kernel's phases leave idle);
 *   RAVEL_NO_FUSED_PROLOGUE  the persistent step's offset conditioning, input
 *                         projection, layer-0 modulation and FOP keys/values in
 *                         separate launches (default: two launches, same results);
 *   RAVEL_NO_WHOLE_K      split-K items instead of whole-K items for the persistent
 *                         kernel's phases with K <= 1024;
 *   RAVEL_NO_WHOLE_K_GEMM (read once per process) few-row GEMMs with K <= 1024 split
 *                         K across blocks instead of one block per 32 columns;
 *   RAVEL_SYNC_CONTEXT    RAVEL_OPT_SYNC_CONTEXT on;  RAVEL_NO_GRAPH  RAVEL_OPT_USE_GRAPH off;
 *   RAVEL_COOPERATIVE     not supported: set to a nonzero value, buffer creation
 *                         fails with RAVEL_E_INVALID (the persistent kernel is
 *                         launched ordinarily; its waits are bounded). */
ravel_status ravel_buffer_create(ravel_model* model, int32_t batch, uint64_t seed, ravel_buffer** out);
void ravel_buffer_destroy(ravel_buffer* buf);

/* Options (ravel_buffer_set_option):
 *   RAVEL_OPT_SYNC_CONTEXT  1: a published context is applied at the very next
 *                           step, which waits on the GPU (not the host) for its
 *                           data; 0 (default): applied at the first step whose
 *                           host-side event query finds the data ready.
 *   RAVEL_OPT_USE_GRAPH     1 (default): replay a captured hipGraph per step (the
 *                           whole step after the host's publish check, on either
 *                           execution path; one graph per pointer set); 0: launch
 *                           the step's kernels eagerly.
 *   RAVEL_OPT_DEBUG         1: synchronise and check for NaN/Inf after each kernel.
 *   RAVEL_OPT_PERSISTENT    1 (default where available): run the transformer layers
 *                           of a bf16 model whose B*H rows fit one 64-row tile as a
 *                           single persistent kernel (one block per CU, grid
 *                           barriers between phases) between the few kernels around
 *                           it; 0: one kernel per operation.  E_STATE if the buffer
 *                           does not qualify.
 *   RAVEL_OPT_FAIL_LAYERS   test hook, 1: mark the persistent layers' kernel as failed
 *                           (synchronises, then sets its error word as a grid barrier
 *                           that timed out would; every later launch then returns at
 *                           once and the error handling described at the top of this
 *                           file takes over).  E_STATE on a buffer without the
 *                           persistent kernel. */
enum { RAVEL_OPT_SYNC_CONTEXT = 1, RAVEL_OPT_USE_GRAPH = 2, RAVEL_OPT_DEBUG = 3, RAVEL_OPT_PERSISTENT = 4,
       RAVEL_OPT_FAIL_LAYERS = 5 };
ravel_status ravel_buffer_set_option(ravel_buffer* buf, int32_t option, int64_t value);

/* Context plane (paper Sec. 3.2: the latest available context is reused
 * across steps until a newer one is ready; refreshing never blocks a step).
 *
 * Each env owns two device context slots; steps read the active one.
 * ravel_context_acquire returns device pointers to the env's inactive slot,
 * K and V each [L, P, n_kv, hd] in the model dtype, after making `producer`
 * wait (on the GPU) until no enqueued step still reads that slot.  The
 * producer writes the new context there (e.g. its own kernels), then calls
 * ravel_set_context with k = v = NULL.  Acquiring cancels a publish of this
 * env that has not yet been applied.
 *
 * ravel_set_context publishes a context for env (0..B-1) computed from the
 * observation of control step t_obs.  With non-NULL k and v (host or device,
 * [L, P, n_kv, hd] model dtype) it first copies them into the inactive slot
 * on `producer` (acquire + copy); the sources must stay valid until that copy
 * has run.  env = -1 publishes one context per env at once: k and v are then
 * [B, L, P, n_kv, hd] (env e's block at offset e * L*P*n_kv*hd) and must not be
 * NULL; t_obs is checked for every env before anything is copied (E_STATE for
 * all if one env's would decrease).  The swap happens at a later ravel_step: the slot index flips in
 * device memory and the step's offset becomes p = t - t_obs.  t_obs must not
 * decrease per env (E_STATE).  Never blocks on the GPU. */
ravel_status ravel_context_acquire(ravel_buffer* buf, int32_t env, void** k_slot, void** v_slot,
                                   void* producer_stream);
ravel_status ravel_set_context(ravel_buffer* buf, int32_t env, const void* k, const void* v,
                               int64_t t_obs, void* producer_stream);

/* One rolling denoise step for all envs, enqueued on `stream` (asynchronous).
 *   fop_tokens: device [B, n_fop, w] in the model dtype (NULL only when the
 *               model has no adapters);
 *   action_out: device float [B, D_a], the action released by this step.
 * The step number t lives in device memory (starts at 0, +1 per step).
 * Errors: E_STATE if some env has no context yet (transformer model). */
ravel_status ravel_step(ravel_buffer* buf, const void* fop_tokens, float* action_out, void* stream);

/* FOP stand-in encoder z = reshape(W_f2 gelu_tanh(W_f1 obs + b_f1) + b_f2)
 * (paper Eq. 4 with a 2-layer MLP in place of the image encoder).
 *   obs: device float [B, d_obs]; fop_tokens: device [B, n_fop, w] model dtype. */
ravel_status ravel_fop_encode(ravel_buffer* buf, const float* obs, void* fop_tokens, void* stream);

/* ravel_fop_encode for callers that cannot allocate device memory -- code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc: the
 * same encoder (same kernels, same results as ravel_fop_encode on a buffer of
 * `batch` envs) without a buffer, its staging rows, split-K partials and tickets
 * kept in a fixed device array of 16 MiB that the library holds on every GPU it
 * runs on until the process ends (set up by ravel_create on the device current
 * then).  Calls no allocating routine; enqueued on `stream` (its tickets are
 * cleared with a kernel, not a memset).
 *   obs: device float [batch, d_obs]; fop_tokens: device [batch, n_fop, w] model dtype.
 * Every call on one GPU shares that GPU's array (the last call's contents stay):
 * calls that overlap on one GPU (different streams or threads without ordering)
 * race and must be serialised by the caller.  Errors: E_INVALID (null pointer, or
 * a batch whose workspace exceeds the fixed array -- the message gives both sizes),
 * E_SHAPE (batch < 1), E_STATE (no FOP encoder weights, or no model created on
 * the current device). */
ravel_status ravel_fop_encode_noalloc(const ravel_model* model, int32_t batch, const float* obs, void* fop_tokens,
                                      void* stream);

/* Wait until every enqueued step and context copy of this buffer finished. */
ravel_status ravel_buffer_sync(ravel_buffer* buf);

/* Synchronises, then copies the state out (any pointer may be NULL):
 *   X_host float [B, H, D_a] ring in PHYSICAL slot order (slot (t+i) mod H is
 *   logical slot i); t = step counter; t_obs_host int64 [B]. */
ravel_status ravel_debug_state(ravel_buffer* buf, float* X_host, int64_t* t, int64_t* t_obs_host);

/* Facts about a buffer's execution (for tests and tooling):
 *   RAVEL_Q_GRAPHS      step graphs captured so far (one per (fop, state, action)
 *                       pointer set and execution path while RAVEL_OPT_USE_GRAPH is on);
 *   RAVEL_Q_PERSISTENT  1 if the transformer layers run as the persistent kernel;
 *   RAVEL_Q_PHASES      phases of that kernel's list (0 on the per-kernel path);
 *   RAVEL_Q_STEPS       steps enqueued (the host's copy of t).
 * Errors: E_INVALID (null pointer, unknown key). */
enum { RAVEL_Q_GRAPHS = 1, RAVEL_Q_PERSISTENT = 2, RAVEL_Q_PHASES = 3, RAVEL_Q_STEPS = 4 };
ravel_status ravel_buffer_query(ravel_buffer* buf, int32_t key, int64_t* value);

/* Publish log: entries (env, t_apply, t_obs) as int64 triples, oldest first.
 * On input *n is the capacity in entries; on output the number written. */
ravel_status ravel_publish_log(ravel_buffer* buf, int64_t* entries, int32_t* n);

/* Bit-exact checkpoint of the rolling state (ring, t, seed, per-env t_obs and
 * active context).  Call with host_blob = NULL to get the size in *n.
 * Synchronises.  Load requires a buffer of the same model and batch. */
ravel_status ravel_buffer_save(ravel_buffer* buf, void* host_blob, size_t* n);
ravel_status ravel_buffer_load(ravel_buffer* buf, const void* host_blob, size_t n);

/* Relative actions (App. B.1, pi0.5 on RoboTwin 2.0; App. B.3, DynamicVLA): a model that
 * predicts actions relative to the robot state keeps its buffer across a moving state by
 * holding the clean targets absolute, converting them relative to the latest state before
 * each expert pass and back afterwards, with the paired noise in model coordinates.  On the
 * buffer of noisy actions this is a shift of every slot i by (1 - tau_i) * (s_prev - s) on
 * the relative dimensions before the pass (s_prev: the state of the env's previous step; no
 * shift at its first step), and the released action is slot 0 plus s on those dimensions.
 * ravel_set_relative_dims marks the relative dimensions: mask [D_a] host int32, nonzero =
 * relative (NULL or all zero: absolute actions, the default); only before the first step
 * (RAVEL_E_STATE after).  With relative dimensions set, every step is ravel_step_state:
 * ravel_step with state [B, D_a] fp32 device, the latest robot state in the actions'
 * normalised units (ravel_step is then RAVEL_E_STATE, as is ravel_step_state without
 * relative dimensions).  The analytic OT field's target is then absolute. */
ravel_status ravel_set_relative_dims(ravel_buffer* buf, const int32_t* mask);
ravel_status ravel_step_state(ravel_buffer* buf, const void* fop_tokens, const float* state, float* action_out,
                              void* stream);

/* Full-horizon synchronous denoising: the baseline rolling inference is compared with
 * (Sec. 4.1 synchronous evaluation and App. B.1: the same budget of expert passes spent on
 * full-horizon denoising steps, and the first-action latency table of Sec. 4.1).  A fresh
 * chunk of H slots per env starts as the given noise at flow time 1; every slot shares one
 * flow time, and `steps` Euler steps of size 1/steps -- step k evaluates the expert with
 * every slot at tau = (steps - k)/steps and applies chunk -= v / steps -- bring it to 0.
 * Each step is one expert pass over the chunk with the buffer's contexts at age 0 (offset
 * delta = delta_bias) and the given FOP tokens (as in ravel_step; NULL only for a model
 * without adapters).  Context publications are applied first exactly as ravel_step applies
 * them (and logged at the current step index).  Analytic models use their velocity field
 * at the shared tau.
 *   noise: [B, H, D_a] fp32, device; chunk_out: [B, H, D_a] fp32, device (may be noise
 *   itself); chunk_out holds the denoised chunk when the stream reaches the end of the call.
 *   steps: 1 .. 1024.
 * Does not touch the rolling ring or the step counter t; it shares the buffer's
 * activations with ravel_step, so it must not overlap a step (or
 * another call of this) on the same buffer.  The first call with a given step count builds
 * that count's flow-time conditioning table on the device and synchronises; later calls
 * enqueue on `stream` and return.  Errors: RAVEL_E_INVALID (null pointers, missing FOP
 * tokens), RAVEL_E_SHAPE (steps), RAVEL_E_STATE (an env without a context). */
ravel_status ravel_full_denoise(ravel_buffer* buf, int32_t steps, const void* fop_tokens, const float* noise,
                                float* chunk_out, void* stream);

/* Streaming-aligned training objective, forward and loss (Sec. 3.3, Eq. 5 and 6): for
 * every sample e of the batch, the training buffer at the rolling flow-time profile,
 * slot i = tau_i * noise + (1 - tau_i) * target with tau_i = (i+1)/H (this build's time
 * direction: the paper's (1 - tau_k) eps + tau_k a_hat), one expert pass with the buffer's
 * context of sample e as the observation-time context and offset delta = ages[e] / H
 * (no lead bias delta_0), and loss[e] = (1/H) sum_i ||v_i - (noise_i - target_i)||^2 (the
 * paper's ||v - (a_hat - eps)||^2 with velocities of the opposite sign).
 *   target, noise: [B, H, D_a] fp32, device (slot i = the action i+1 steps after t_a);
 *   ages: [B] int64, device, context age p = t_a - t_o per sample;
 *   fop_tokens: as ravel_step; loss_out: [B] fp32, device;
 *   v_out: optional [B, H, D_a] fp32, device: the predicted velocities (NULL: none).
 * Context publications are applied first as ravel_step applies them.  Does not touch the
 * ring or t; shares the buffer's activations with ravel_step (no overlap on one buffer).
 * No backward pass.  Errors: RAVEL_E_INVALID (null pointers, missing FOP tokens),
 * RAVEL_E_STATE (a sample without a context). */
ravel_status ravel_train_loss(ravel_buffer* buf, const float* target, const float* noise, const int64_t* ages,
                              const void* fop_tokens, float* loss_out, float* v_out, void* stream);

/* Per-kernel timing of one eagerly launched step (HIP events around every
 * launch on `stream`; synchronises).  Each record: kernel class name,
 * algorithmic bytes and flops of that launch, and its duration.  With the
 * persistent path on, further records "persistent/<phase class>" split the
 * "persistent_layers" record by phase class (time between the kernel's grid
 * barriers as seen by its first block, summed over layers), followed by one
 * record "phase/<index>/<phase class>" per phase in launch order; neither kind
 * is an additional launch.  Launches whose row count is decided on the device
 * (the modulation GEMMs run on the rows of distinct offset conditionings,
 * class "gemm_rows") carry bytes = flops = 0.  On input *n is the
 * capacity; on output the number of records. */
typedef struct {
  char name[48];
  double bytes;
  double flops;
  float ms;
} ravel_kernel_record;
ravel_status ravel_profile_step(ravel_buffer* buf, const void* fop_tokens, float* action_out,
                                void* stream, ravel_kernel_record* records, int32_t* n);

/* Message of the calling thread's last non-OK status ("" if none). */
const char* ravel_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RAVEL_H */
