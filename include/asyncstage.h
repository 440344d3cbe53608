/*
 * asyncstage.h - C ABI of one pipeline stage's training step under a one-step gradient delay,
 * for AMD Instinct MI355X (gfx950).
 *
 * The method (One-Step Gradient Delay is Not a Barrier for Large-Scale Asynchronous Pipeline
 * Parallel LLM Pretraining):
 *   - §2, Alg. 1 (Delayed Gradient Update): iteration t computes g_t at x_t, feeds g_{t-1} to the
 *     optimizer statistics and sets x_{t+1} = x_t - u_{t-1}(g_{t-1}); g_{-1} = 0, u_{-1} = 0.
 *   - §3.2, Error-Feedback equation: x_{t+1} = x_t - 2 u_{t-1}(g_{t-1}) + u_{t-2}(g_{t-2}) for
 *     t >= 2, and App. A.4 its lambda-scaled form x_{t+1} = x_t - u_{t-1} - lambda (u_{t-1} - u_{t-2}).
 *   - §2 and App. E.1: u is decoupled AdamW, betas (0.9, 0.95), weight decay 0.1, global-norm
 *     gradient clipping at 1.0; Alg. 2 (§4) puts the weight decay on the current weights x_t.
 *   - §2 / App. F.1: PipeDream-2BW keeps one stashed weight version, so a stage holds two compute
 *     copies of its weights (versions t mod 2) and two gradient buffers (g_t being accumulated,
 *     g_{t-1} being consumed).
 *   - App. C (delayed method with prev(k) = k - tau): a fixed delay tau >= 2 consumes g_{t-tau},
 *     with Error Feedback against the update formed tau iterations earlier, x_{t+1} = x_t - u -
 *     lambda (u - u_{t-tau}) (lambda = tau: the coefficients tau + 1 and tau of its proof); the
 *     stage then holds tau + 1 gradient buffers and tau EF buffers.
 *   - App. E.2: the stage is a stack of Llama-style decoder blocks (pre-norm RMSNorm, grouped-query
 *     causal attention with RoPE, SwiGLU feed-forward, no biases); a first stage owns the token
 *     embedding, a last stage the LM head with next-token cross-entropy (App. E) - tied to the
 *     embedding when one stage holds both ends, else its own matrix.
 *
 * Conventions
 *   - Every function returns a stage_status; no C++ exception crosses the ABI.  On error,
 *     stage_last_error() returns a message (thread-local, valid until the next call).
 *   - The library never allocates device memory.  The caller allocates one arena of
 *     stage_required_bytes() and every input/output buffer; all pointers stay owned by the caller.
 *   - All device work is enqueued asynchronously on the HIP stream given to stage_init (or to
 *     delayed_update_flat), with one exception: delayed_update runs its kernels on a stream of
 *     the stage's own (non-blocking, default priority).  It waits there only for the backwards
 *     whose gradient it consumes and for the last use of the weight version it overwrites, so
 *     it overlaps forward / backward work the caller enqueued before it; the stage stream then
 *     waits for it, so everything enqueued after delayed_update returns sees its results.
 *     Host pointers are never retained.  The caller synchronises.
 *   - The caller may write master weights and optimizer state (stage_tensor views) only when no
 *     update is in flight, and then calls stage_sync_weights() before the next delayed_update.
 *   - Device pointers must be 16-byte aligned.  Layouts are row-major, last index contiguous.
 *   - Token ids are int32; an id outside [0, vocab) is never used as an index (see
 *     stage_forward).
 *   - One stage_t per host thread; calls on one stage_t must not overlap.
 */
#ifndef ASYNCSTAGE_H
#define ASYNCSTAGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct stage stage_t; /* opaque */

typedef enum {
  STAGE_OK = 0,
  STAGE_EINVAL = -1,     /* bad argument or shape                                  */
  STAGE_ENOSPACE = -2,   /* arena smaller than stage_required_bytes()              */
  STAGE_EHIP = -3,       /* a HIP runtime call failed                              */
  STAGE_ESTATE = -4,     /* call out of the documented order                       */
  STAGE_ENONFINITE = -5  /* reported by stage_poll_nonfinite                       */
} stage_status;

typedef enum { STAGE_DT_F32 = 0, STAGE_DT_BF16 = 1, STAGE_DT_I32 = 2 } stage_dtype;

/* Largest delay a stage can be shaped for (stage_shape_t.max_delay). */
enum { STAGE_MAX_DELAY = 8 };

/* Shape of one stage.  dtype 0: fp32 compute and storage; 1: bf16 compute copies, bf16
 * activations, fp32 accumulation, fp32 master weights / optimizer state / gradients.
 * vocab > 0 sizes the token embedding [vocab, d_model] of a first stage (vocab < 2^17) and the
 * head of a last stage (vocab < 2^20): logits = RMSNorm(x) W^T with W the embedding when
 * tie_embedding (which needs first_stage and last_stage), else the stage's "head" matrix
 * [vocab, d_model].  The head keeps fp32 logits [tokens, vocab] per activation slot.  head_dim in {32, 64, 128};
 * n_heads a multiple of n_kv_heads; d_model a multiple of 64.  max_inflight >= 1 is the number
 * of activation slots (microbatches whose backward is pending).  optimizer 0: AdamW only;
 * 1: the arena also holds the Newton-Schulz workspace of delayed Muon (Alg. 2 of §4), 8 to 12 (fp32
 * stage: 8) bytes per element of the blocks' weight matrices plus their Gram matrices, so that
 * delayed_update accepts update_hparams_t.optimizer = 1; 2: the arena also holds Adan's two extra
 * state vectors (8 bytes per parameter), so that delayed_update accepts optimizer = 4.  max_delay
 * in [0, 8] (0 is read as 1):
 * the largest delay delayed_update accepts; the arena holds max_delay + 1 gradient buffers and
 * max_delay EF buffers. */
typedef struct {
  int32_t n_blocks, d_model, n_heads, n_kv_heads, head_dim, d_ffn;
  int32_t vocab, first_stage, last_stage, tie_embedding;
  int32_t seq_len, micro_batch, max_inflight;
  int32_t dtype;
  float rms_eps, rope_theta;
  int32_t optimizer;
  int32_t max_delay;
} stage_shape_t;

/* Hyper-parameters of one update.  clip_norm <= 0 disables clipping.  ef_lambda = 0 is standard
 * delayed training, 1 the Error-Feedback equation of §3.2.  delay 1 is Alg. 1; delay 0 is the
 * synchronous optimizer (requires ef_lambda = 0); delay tau in [2, max_delay] consumes g_{t-tau}
 * with EF against the update formed tau iterations earlier (ef_lambda = tau reproduces the
 * appendix's x_k - (tau + 1) u_k + tau u_{k-tau}).  The delay of a stage stays fixed over a run.
 * optimizer 0: AdamW (beta1, beta2, eps) on every parameter.  optimizer 1: delayed Muon (Alg. 2
 * of §4) on every 2-D weight matrix of a block (wq, wk, wv, wo, wgate, wup, wdown, each on its
 * own) and AdamW on the embedding and the gains: M <- momentum M + (1 - momentum) c g;
 * O = Newton-Schulz(M) (ns_steps >= 1 quintic iterations on M / ||M||_F in the orientation with
 * rows <= cols, coefficients (3.4445, -4.7750, 2.0315); on a bf16 stage the iterate is held in
 * fp32 or as a hi + lo pair of bf16 matrices and the product P X uses the pair, while
 * A = hi hi^T and P = b A + c A A are bf16);
 * u = lr (update_rms sqrt(max(rows, cols)) O + weight_decay x_t); then the same standard or
 * Error-Feedback step as AdamW.  Needs a stage shaped with optimizer 1.
 * optimizer 2: Lion (§3.3's optimizer list) on every parameter, u = lr (sign(beta1 m + (1 - beta1)
 * c g) + weight_decay x_t), m <- beta2 m + (1 - beta2) c g (v unused).  optimizer 3: NAdam with the
 * momentum-decay schedule mu_k = beta1 (1 - 0.5 0.96^(k nadam_psi)): m, v as AdamW and u = lr
 * ((1 - mu_k) / (1 - P_k) c g + mu_{k+1} / (1 - P_k mu_{k+1}) m) / (sqrt(v / (1 - beta2^k)) + eps)
 * + lr weight_decay x_t, P_k = mu_1 ... mu_k.  optimizer 4: Adan (§3.3's optimizer list; the rule of
 * the cited Adan work, betas as averaging weights, the paper's beta1 = 0.98) on every parameter,
 * with diff = c g - c g_last (0 at the first update; g_last the clipped gradient the previous update
 * consumed): m <- beta1 m + (1 - beta1) c g, d <- beta2 d + (1 - beta2) diff, n <- beta3 n + (1 -
 * beta3) (c g + beta2 diff)^2 (n in the v slot), u = lr ((m / (1 - beta1^k) + beta2 d / (1 - beta2^k))
 * / (sqrt(n / (1 - beta3^k)) + eps) + weight_decay x_t); needs a stage shaped with optimizer 2.
 * predict 1 (AdamW, delay 1, ef_lambda 0 only): SAPipe weight prediction with the updated
 * optimizer state (App. B.1) - the master takes the standard delayed step x_{t+1} = x_t -
 * u_{t-1}(g_{t-1}) while the compute copy receives x_{t+1} - u_t(g_{t-1}), AdamW fed g_{t-1} once
 * more from the updated state (bias correction k + 1; the predicted state is not kept). */
typedef struct {
  float lr, beta1, beta2, eps, weight_decay, clip_norm, ef_lambda;
  int32_t delay;
  int32_t optimizer;
  float momentum, update_rms;
  int32_t ns_steps;
  int32_t predict;
  float nadam_psi;
  float beta3;
} update_hparams_t;

/* Bytes of device memory the stage needs (weights, optimizer state, max_delay + 1 gradient
 * buffers, max_delay EF buffers, two compute versions, the activation ring and scratch).  0 on an
 * invalid shape. */
size_t stage_required_bytes(const stage_shape_t* shape);

/* Carve the arena (device memory, >= stage_required_bytes, 256-byte aligned) and zero the
 * optimizer state.  The master weights are left for the caller to fill through stage_tensor(),
 * followed by stage_sync_weights().  hip_stream: a hipStream_t (NULL = default stream). */
int stage_init(const stage_shape_t* shape, void* arena, size_t arena_bytes, void* hip_stream,
               stage_t** out);

/* Number of named tensors exposed by stage_tensor. */
int stage_num_tensors(const stage_t* s, int32_t* count);

/* Tensor idx: name, device pointer, element count and dtype (stage_dtype).  Names:
 *   "embed", "blk{i}.attn_norm|wq|wk|wv|wo|ffn_norm|wgate|wup|wdown", "final_norm", "head" - fp32
 *   master weights [out, in]; the same names prefixed "m.", "v.", "u_prev." (fp32 optimizer
 *   state, EF buffer), "u_prev{j}." for j in [1, max_delay) (the further EF buffers: iteration t
 *   of a delay-tau run uses buffer t mod tau, "u_prev." being buffer 0), "grad{j}." for j in
 *   [0, max_delay] (gradient buffers: step s accumulates into buffer s mod (max_delay + 1)) and
 *   "w0.", "w1." (the two compute versions, bf16 or fp32); "flat.master|m|v|u_prev|u_prev{j}|
 *   grad{j}|w0|w1" for the whole flat vectors (padding between tensors is zero and stays zero);
 *   "act{slot}.blk{i}.{x|rstd1|n1|qkv|o|lse|h|rstd2|n2|gu|z}" (on a bf16 stage also "o32", the
 *   attention output in fp32) and "act{slot}.{x0|y|logits}"
 *   for the saved activations of an activation slot. */
int stage_tensor(const stage_t* s, int32_t idx, const char** name, void** dev_ptr,
                 int64_t* numel, int32_t* dtype);

/* Look a tensor up by name; STAGE_EINVAL if absent. */
int stage_tensor_by_name(const stage_t* s, const char* name, void** dev_ptr, int64_t* numel,
                         int32_t* dtype);

/* Copy the fp32 master weights into both compute versions (after the caller wrote them). */
int stage_sync_weights(stage_t* s);

/* Forward of one microbatch of optimizer step `step` at the weights x_step (compute version
 * step mod 2), saving activations in slot `slot` (0 <= slot < max_inflight).
 *   tokens  [micro_batch, seq_len] int32, device  (first stage; else NULL).  Ids outside
 *           [0, vocab) are not read: such a position embeds as a zero row and adds nothing to
 *           the embedding gradient.
 *   x_in    [micro_batch, seq_len, d_model] bf16/fp32 per dtype, device (non-first; else NULL)
 *   targets [micro_batch, seq_len] int32, device  (last stage; else NULL).  A target outside
 *           [0, vocab) is ignored: zero loss and zero gradient at that position (the mean still
 *           divides by micro_batch*seq_len).
 *   y_out   [micro_batch, seq_len, d_model] device (non-last; may be NULL to keep it in the slot)
 *   loss_dev one float, device (last stage: mean cross-entropy of this microbatch; else NULL)
 * STAGE_ESTATE if compute version step mod 2 does not hold x_step. */
int stage_forward(stage_t* s, int32_t slot, int64_t step, const int32_t* tokens, const void* x_in,
                  const int32_t* targets, void* y_out, float* loss_dev);

/* Backward of the microbatch saved in `slot`; its parameter gradient is added to gradient buffer
 * (step mod (max_delay + 1)) - the first backward of a step overwrites it; STAGE_ESTATE if that
 * buffer still holds a gradient no update has consumed.  dy: upstream gradient
 * [micro_batch, seq_len, d_model] (non-last stage; NULL on a last stage, whose loss is the mean
 * cross-entropy divided by microbatches_per_step).  dx_out: gradient w.r.t. x_in (non-first
 * stage; may be NULL).  STAGE_ESTATE if the slot holds no pending forward. */
int stage_backward(stage_t* s, int32_t slot, const void* dy, void* dx_out,
                   int32_t microbatches_per_step);

/* Second half of iteration t of Alg. 1: with delay tau >= 1 consume g_{t-tau} (the gradient of
 * step t-tau, complete), with delay 0 consume g_t; clip by the global norm; AdamW (or Muon);
 * standard or lambda-EF update of the master weights (EF once tau earlier updates exist: the
 * "t <= 1" rule for tau = 1; the EF buffer of iteration t is t mod tau); write x_{t+1} to compute
 * version (t+1) mod 2.  Must be called once per t in increasing order; for t < tau (no pending
 * gradient) the weights are unchanged (u_{-1} = 0).  A non-finite
 * gradient norm leaves x, m, v and the EF buffer untouched (x_{t+1} = x_t, the compute copy is
 * written from x_t) and is counted on the device; see stage_poll_nonfinite.  Such an iteration still
 * counts as having consumed its gradient: the bias-correction index of every update is
 * k = t - tau + 1 (t + 1 with delay 0) whether or not earlier gradients were skipped, Error Feedback
 * starts once tau gradients have been consumed, and an EF buffer the skipped iteration would have
 * written keeps its contents.  The norm (two deterministic passes over the gradient) runs whether
 * or not clipping is on, since it is also the non-finite check.  STAGE_ESTATE on out-of-order t or
 * an incomplete gradient. */
int delayed_update(stage_t* s, int64_t t, const update_hparams_t* hp);

/* Resume a run at iteration next_t of a fixed-delay run (Alg. 1 carries x_t, the optimizer
 * statistics, the EF buffers and the gradients not yet consumed from one iteration to the next).
 * On a fresh stage (no delayed_update yet, no pending microbatch), after the caller has written
 * through stage_tensor views the master weights x_next_t, m, v, every EF buffer ("u_prev.",
 * "u_prev{j}.") and, for delay tau >= 1, the gradients g_s of steps s = next_t - tau .. next_t - 1
 * into their buffers "grad{s mod (max_delay + 1)}.": marks those gradients complete and unconsumed,
 * sets the count of consumed gradients to next_t - tau (next_t with delay 0) and copies the master
 * weights into both compute versions (stage_sync_weights).  The next calls are stage_forward(...,
 * step next_t, ...) and delayed_update(next_t).  delay in [0, max_delay] is the delay of the run
 * being resumed.  STAGE_ESTATE when the stage has run an update or holds a pending microbatch. */
int stage_resume(stage_t* s, int64_t next_t, int32_t delay);

/* Stateless fused update (AdamW, Lion, NAdam or the AdamW weight prediction of hp; not Muon) over
 * flat device vectors of n elements:
 * iteration t of a delay-tau run (tau = hp->delay >= 1) consumes g_prev (= g_{t-tau}; fp32, or
 * bf16 when g_is_bf16), with k = t - tau + 1 the AdamW bias-correction index and EF from
 * t >= 2 tau; t < tau only writes x_shadow.  x, m, v, u_prev fp32 (read and written; u_prev holds
 * the update formed tau iterations earlier - the caller keeps a ring of tau buffers, slot t mod
 * tau - and may be NULL when ef_lambda = 0); x_shadow (written, bf16 when shadow_is_bf16 else
 * fp32; may be NULL; required with predict, which writes the predicted point there).
 * clip_scale_dev: device float multiplying g_prev, or NULL for 1. */
int delayed_update_flat(int64_t n, float* x, const void* g_prev, int32_t g_is_bf16, float* m,
                        float* v, float* u_prev, void* x_shadow, int32_t shadow_is_bf16,
                        int64_t t, const update_hparams_t* hp, const float* clip_scale_dev,
                        void* hip_stream);

/* delayed_update_flat for Adan (hp->optimizer 4), whose rule keeps two more state vectors: d (the
 * average of gradient differences) and g_last (the clipped gradient of the previous update), fp32,
 * 16-byte aligned, read and written; v holds Adan's second moment n.  Every other argument and the
 * delay / EF / shadow conventions as delayed_update_flat. */
int delayed_update_flat_adan(int64_t n, float* x, const void* g_prev, int32_t g_is_bf16, float* m, float* v,
                             float* d, float* g_last, float* u_prev, void* x_shadow, int32_t shadow_is_bf16,
                             int64_t t, const update_hparams_t* hp, const float* clip_scale_dev, void* hip_stream);

/* Device bytes of the workspace grad_norm_flat needs (partial sums of the first pass). */
size_t grad_norm_flat_workspace_bytes(void);

/* Global L2 norm of a flat gradient vector and its clip coefficient (the gradient clipping of §2 /
 * App. E.1, c = min(1, clip_norm / (||g|| + 1e-6)), 1 when clip_norm <= 0 or the norm is not
 * finite), the pass delayed_update runs over the stage's gradient, for a caller-held flat vector
 * (with delayed_update_flat, whose clip_scale_dev can be out_dev + 1).  Two deterministic passes:
 * contiguous ranges summed in double per block, then the partials in a fixed order.
 *   g          n elements, fp32 or bf16 (g_is_bf16), device, 16-byte (bf16: 8-byte) aligned
 *   out_dev    two floats, device: ||g||, c
 *   nonfinite_dev  one int32, device, set to 1 when ||g|| is not finite and 0 otherwise; may be NULL
 *   workspace  device scratch of >= grad_norm_flat_workspace_bytes(), 8-byte aligned, owned by
 *              the caller; calls that share a workspace must not overlap
 * Enqueued on hip_stream. */
int grad_norm_flat(int64_t n, const void* g, int32_t g_is_bf16, float clip_norm, float* out_dev,
                   int32_t* nonfinite_dev, void* workspace, size_t workspace_bytes, void* hip_stream);

/* grad_norm_flat for callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the same two passes, with the partial sums
 * in a static device array of the library (1024 doubles, 8 KiB per GPU, held until the process
 * ends) instead of a caller workspace.  It calls no hipMalloc, hipFree or allocating routine.  The
 * first pass runs at most 1024 blocks whatever n is, so n has no scratch-imposed maximum; a grid that
 * would need more partials is refused with STAGE_EINVAL.  Every call on a GPU shares that GPU's
 * array (each call overwrites every partial it reads): calls that overlap on one GPU race.
 * Arguments, results and alignment as grad_norm_flat. */
int grad_norm_flat_noalloc(int64_t n, const void* g, int32_t g_is_bf16, float clip_norm, float* out_dev,
                           int32_t* nonfinite_dev, void* hip_stream);

/* Measurement reference, not a step of the method: a streaming device copy of `bytes` (a multiple
 * of 16; both pointers 16-byte aligned) with 16-byte non-temporal loads and stores, four chunks in
 * flight per thread - the practical HBM ceiling the update pass's bandwidth is reported against. */
int hbm_stream_copy(void* dst, const void* src, size_t bytes, void* hip_stream);

/* Ascending unique token ids of the microbatch in `slot` and their counts (after its backward
 * on a first stage).  ids, counts: device int32 arrays of >= micro_batch*seq_len entries;
 * n_unique: device int32. */
int stage_embed_indices(stage_t* s, int32_t slot, int32_t* ids, int32_t* counts,
                        int32_t* n_unique);

/* Synchronise the stream and report how many updates were skipped for a non-finite gradient
 * norm since the last poll (STAGE_ENONFINITE if any). */
int stage_poll_nonfinite(stage_t* s, int64_t* skipped);

/* Overlap mode (off by default).  Off: everything enqueued on the stage stream after
 * delayed_update(t) returns runs after that update.  On: the stage stream waits for update t only
 * where the one-step delay needs it - the first stage_forward of step t+1 (it reads compute
 * version (t+1) mod 2, which the update writes) and the first stage_backward that overwrites the
 * gradient buffer the update read (stage_sync_weights and stage_join_update wait for every
 * update).  A caller may then issue delayed_update(t) before step t's forwards and backwards, and
 * the update runs beside them on the stage's own stream (Alg. 1: x_{t+1} depends only on x_t and
 * g_{t-1}).  Reads of the master weights or optimizer state through stage_tensor() views must
 * follow stage_join_update() or a device synchronisation.  Turning it off joins.
 * on = 2: as 1, and the elementwise pass of each delayed_update (AdamW, Lion, NAdam, the
 * prediction; not Muon's or Adan's) is deferred in chunks, one per attention backward the stage
 * runs in a step (n_blocks x the microbatches_per_step of the last stage_backward; chunks of at
 * least 2^16 elements): each stage_backward launches the next chunk on the update stream as a
 * block's attention backward starts, so that the pass's HBM traffic runs beside work bound by the
 * matrix cores instead of beside the forward's products.  The results are those of mode 1
 * (elementwise pass, bit for bit).  Chunks not launched by then are launched by the first call that
 * needs the update: the forward that reads the version it writes, the backward that overwrites the
 * gradient buffer it reads, the next delayed_update, stage_join_update, stage_sync_weights, or a
 * change of mode; view reads must follow stage_join_update() (a device synchronisation alone does
 * not launch them).  Other values: STAGE_EINVAL. */
int stage_set_update_overlap(stage_t* s, int32_t on);

/* The stage stream waits for every delayed_update issued so far (no-op when none is owed). */
int stage_join_update(stage_t* s);

/* Global L2 norm of gradient buffer `which` (0 <= which <= max_delay), computed on device into
 * norm_dev (float). */
int stage_grad_norm(stage_t* s, int32_t which, float* norm_dev);

/* Kernel-class timing.  While enabled, the stage records a HIP event pair on the launching
 * stream around every launch of a class and, when read, adds up the elapsed times and the algorithmic work of
 * those launches: GEMM and attention in flops (2 M N K per product; causal attention forward
 * 4 B Hq hd s(s+1)/2, backward twice that), the delayed update and the gradient norm in bytes of
 * HBM traffic, the Newton-Schulz products of Muon (STAGE_PROF_NS) in flops.  Reading synchronises the stream and resets the counters.  Meant for measurement
 * passes; it adds two event records per launch. */
typedef enum {
  STAGE_PROF_GEMM = 0, STAGE_PROF_ATTN_FWD = 1, STAGE_PROF_ATTN_BWD = 2, STAGE_PROF_UPDATE = 3,
  STAGE_PROF_NORM = 4, STAGE_PROF_OTHER = 5, STAGE_PROF_NS = 6, STAGE_PROF_NCLASS = 7
} stage_prof_class;
int stage_profile_enable(stage_t* s, int32_t on);
int stage_profile_read(stage_t* s, int32_t cls, double* ms, int64_t* launches, double* work);

const char* stage_last_error(void);
void stage_destroy(stage_t* s);

#ifdef __cplusplus
}
#endif
#endif /* ASYNCSTAGE_H */
