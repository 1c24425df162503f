/*
 * tadm.h -- C ABI of the MI355X (gfx950) implementation of the reverse-diffusion
 * step of Time-Anchored Diffusion Models (TADM).
 *
 * The method (Sec. 3.1, eq. DenoiserOp): a shared network S maps the current
 * canvas z_t to c_t = S(z_t); an expensive anchor network A produces
 * h_t' = A(S(z_t')) only at refresh steps and the result is cached; every reverse
 * step runs the fusion module h~ = Phi(c_t, h_t'), the lightweight denoiser D and
 * the vocabulary head, then the masked-diffusion reverse step.  Anchor-cache
 * inference (Algorithm 1) refreshes the cache at reverse step i iff
 * (T - i) mod K == 0.
 *
 * Conventions shared by every call:
 *  - Array arguments named *_dev are device pointers (HIP device memory of the
 *    model's device).  Token ids are int32, hidden states and logits float32.
 *  - The mask token id is cfg.vocab; real token ids are in [0, cfg.vocab).
 *  - All work is enqueued on the model's stream (tadm_set_stream); calls return
 *    without synchronising unless stated.  Inputs must stay valid until the
 *    enqueued work completes.  Outputs are caller-allocated.
 *  - Arguments are validated on the host before anything is enqueued; an invalid
 *    argument returns TADM_ERR_INVALID and has no side effects.  A cache or
 *    context built for another model or shape returns TADM_ERR_STATE.  HIP
 *    failures return TADM_ERR_DEVICE.  tadm_last_error() then describes the
 *    failure.  No call aborts the process.
 *  - Objects (model, cache, context) are opaque, created and destroyed by the
 *    caller.  A cache or context must be destroyed before its model.
 */
#ifndef TADM_H
#define TADM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TADM_OK = 0,
  TADM_ERR_INVALID = 1,      /* bad argument (shape, range, null pointer)          */
  TADM_ERR_OOM = 2,          /* device allocation failed                           */
  TADM_ERR_DEVICE = 3,       /* HIP runtime error                                  */
  TADM_ERR_STATE = 4,        /* object mismatch, weights missing, wrong model      */
  TADM_ERR_UNSUPPORTED = 5   /* valid request the library does not implement       */
} tadm_status;

enum { TADM_DTYPE_F32 = 0, TADM_DTYPE_BF16 = 1 };
enum { TADM_FFN_GELU = 0, TADM_FFN_SWIGLU = 1, TADM_FFN_GEGLU = 2 };
/* Fusion Phi: gated residual MLP (App. C.2) or paired attention (App. C.1). */
enum { TADM_FUSION_GATED_MLP = 0, TADM_FUSION_PAIRED = 1 };

/* Model shape.  Layers are numbered shared [0, n_shared), anchor, then denoiser.
 * dtype is the storage/operand type of weights and GEMM/attention operands; the
 * residual stream, norm statistics, softmax, logits and the sampler are float32.
 * max_batch x max_seq bounds every call (positions include any context).
 * vocab is at most 262144 (the sampler keeps one partial per 64 entries on chip). */
typedef struct {
  int32_t vocab, d_model, n_heads, n_kv_heads, head_dim, d_ffn, ffn_kind;
  int32_t n_shared, n_anchor, n_denoise, fusion_kind, fusion_rank, paired_heads;
  int32_t dtype, max_batch, max_seq;
  float rms_eps;     /* RMSNorm epsilon of the transformer layers / paired scales */
  float ln_eps;      /* LayerNorm epsilon of the gated-MLP fusion                  */
  float rope_theta;  /* rotary base                                               */
} tadm_config;

typedef struct tadm_model tadm_model;
typedef struct tadm_cache tadm_cache;
typedef struct tadm_context tadm_context;

/* Arguments of one reverse step (Sec. 2.1 time grid t(i) = i/T). */
typedef struct {
  int32_t i, T;        /* reverse step i in [1, T]                                   */
  int32_t n_unmask;    /* masked positions revealed per row (clamped per row)        */
  uint32_t step_id;    /* Philox counter word: block * T + (T - i) in tadm_generate  */
  uint64_t seed;       /* Philox key                                                 */
  float inv_temp;      /* 1 / temperature, > 0                                       */
  const int32_t* n_unmask_rows;  /* nullable device [B]: per-row counts (each >= 0, clamped
                                    to the row's masked count) used instead of n_unmask  */
  int32_t mode;        /* TADM_STEP_RANKED: confidence-ranked unmasking (n_unmask);
                          TADM_STEP_REMASK: remasking posterior (p_unmask, sigma)    */
  float p_unmask;      /* REMASK: probability that a masked position takes its token  */
  float sigma;         /* REMASK: probability that a decoded position is remasked     */
  float top_p;         /* in (0, 1): tokens come from the top-p nucleus (exact fixed-point
                          weights, ties at the boundary kept); 0 or 1: the whole vocabulary */
  float entropy_eta;   /* ENTROPY: the entropy bound eta >= 0                          */
  const float* sc_in;  /* ENTROPY: nullable device [B, L - canvas_off, d] float32, the
                          self-conditioning signal added to the canvas embeddings      */
  float* sc_out;       /* ENTROPY: nullable device [B, L - canvas_off, d] float32,
                          receives s = softmax(logits * inv_temp) E (may alias sc_in)  */
} tadm_step_args;

/* Reverse-step kinds.  REMASK is the posterior of eq. inf-post-TADM (the ReMDM form,
 * Sec. 3 and App. B): per canvas position, one uniform u from Philox4x32-10 word 0 at
 * counter (2^31, absolute position, row, step_id); a masked position becomes its
 * Gumbel-max token iff u < p_unmask, a decoded one becomes the mask iff u < sigma. */
/* ENTROPY is a step of the uniform-state entropy-bound sampler (Algorithm 2, App. C.1):
 * every canvas position gets x_hat = argmax of its logits, x_tilde = the Gumbel-max
 * draw at inv_temp (the counters of the masked sampler) and the entropy H of
 * softmax(logits * inv_temp), summed in 2^-40 fixed point (A = sum rint(e 2^40),
 * B = sum rint(-y e 2^40), e = exp(y), y = l' - max l'; H = log(A 2^-40) + B / A).
 * Positions in ascending (H, position) order are accepted while the entropies ranked
 * before them sum to at most eta (exact integer sums of rint(H 2^40)); accepted
 * positions take x_tilde, the others a uniform token ((w V) >> 32, w = Philox word 0
 * at counter (2^31 + 1, absolute position, row, step_id)); at i = 1 every position
 * takes x_hat.  The decoder adds sc_in to the canvas embeddings of its passes (the
 * reading of Decoder(z, s)), and sc_out receives the next step's signal. */
enum { TADM_STEP_RANKED = 0, TADM_STEP_REMASK = 1, TADM_STEP_ENTROPY = 2 };

/* ---------------------------------------------------------------- model ---- */
/* Number of weight tensors of a configuration, and the shape of tensor `index`
 * (matrices [rows = out features, cols = in features]; vectors cols = 0).
 * Order: embed [V+1, d], final_norm [d], w_out [V, d], the fusion tensors, then
 * per layer attn_norm, wq, wk, wv, wo, ffn_norm, (w_gate,) w_up, w_down. */
int32_t tadm_weight_count(const tadm_config* cfg);
tadm_status tadm_weight_info(const tadm_config* cfg, int32_t index, int64_t* rows, int64_t* cols);

/* Creates a model on the current HIP device and allocates its weight arena. */
tadm_status tadm_model_create(const tadm_config* cfg, tadm_model** out);
/* Copies weight `index` (elements of cfg.dtype, row-major, `bytes` long) from
 * host (src_on_device = 0) or device memory into the model's own layout.
 * Synchronous.  Every tensor must be loaded before a compute call. */
tadm_status tadm_model_load_weight(tadm_model* m, int32_t index, const void* src, size_t bytes,
                                   int32_t src_on_device);
tadm_status tadm_model_destroy(tadm_model* m);
/* Stream for all later work of this model (a hipStream_t; NULL = default stream). */
tadm_status tadm_set_stream(tadm_model* m, void* hip_stream);

/* ---------------------------------------------------------------- cache ---- */
/* Anchor cache for B rows x L positions (Algorithm 1's h^cache plus refresh index).
 * Fields: TADM_CACHE_H   anchor output h' = A(c')            float32 [B, L, d]
 *         TADM_CACHE_C   shared state c' at the refresh      float32 [B, L, d]
 *         TADM_CACHE_A   LN_a(h') (gated-MLP fusion input)   dtype   [B, L, d] */
enum { TADM_CACHE_H = 0, TADM_CACHE_C = 1, TADM_CACHE_A = 2 };
tadm_status tadm_cache_create(tadm_model* m, int32_t B, int32_t L, tadm_cache** out);
tadm_status tadm_cache_destroy(tadm_cache* c);
/* Enqueues a copy of one field into dst_dev (bytes must equal the field size). */
tadm_status tadm_cache_read(const tadm_cache* c, int32_t field, void* dst_dev, size_t bytes);
/* Reverse step index i of the last refresh (0 = never refreshed). */
int32_t tadm_cache_refresh_step(const tadm_cache* c);

/* -------------------------------------------------------------- context ---- */
/* Block diffusion with an encoder/decoder split (App. C.1, architecture details of the
 * post-trained model): the encoder pass prefills a KV context from the prompt, the
 * decoder denoises one block at a time attending to that context, and each finished
 * block is appended to the context by the encoder.  Here the context holds per-layer
 * K, V of the prompt and the finished blocks; attention is bidirectional within a
 * block and causal across blocks (the prompt is block 0).
 *
 * tadm_context_create: a context for B rows and at most max_ctx positions
 * (1 <= B <= max_batch, 1 <= max_ctx <= max_seq), owned by the caller and destroyed
 * with tadm_context_destroy; device memory n_layers x 2 x B x Hkv x cap x head_dim
 * elements of the model dtype (cap = max_ctx rounded up to 64).  TADM_ERR_INVALID for
 * sizes outside those bounds, TADM_ERR_OOM when the allocation fails. */
tadm_status tadm_context_create(tadm_model* m, int32_t B, int32_t max_ctx, tadm_context** out);
/* The encoder pass: a fresh pass (a refresh step: S, A, Phi with the fresh anchor, D)
 * over n clean tokens per row, tokens_dev device int32 [B, n] (borrowed until the
 * stream work completes), at positions [len, len + n), attending to the context and
 * bidirectionally among themselves; appends every layer's K, V and advances len by n.
 * Token ids are not read on the host: an id outside [0, vocab] is clamped into that
 * range by the embedding gather (memory safety only; the result is then meaningless).
 * TADM_ERR_INVALID when n < 1 or the positions exceed max_seq or the context's
 * capacity; TADM_ERR_STATE for a context of another model or another B. */
tadm_status tadm_context_append(tadm_model* m, tadm_context* ctx, const int32_t* tokens_dev,
                                int32_t B, int32_t n);
/* Committed positions (len); 0 after create or reset (and for NULL).  reset empties
 * the context without freeing it.  destroy waits for the device, then frees it. */
int32_t tadm_context_length(const tadm_context* ctx);
tadm_status tadm_context_reset(tadm_context* ctx);
tadm_status tadm_context_destroy(tadm_context* ctx);

/* ------------------------------------------------------------ the step ---- */
/* Anchor refresh (Alg. 1): c = S(canvas), h = A(c), written to `cache`.
 * canvas_dev [B, L] is the window at positions [ctx_len, ctx_len + L) (ctx may be
 * NULL: positions [0, L)).  (i, T) is recorded as the refresh step. */
tadm_status tadm_anchor_forward(tadm_model* m, const tadm_context* ctx, const int32_t* canvas_dev,
                                int32_t B, int32_t L, int32_t i, int32_t T, tadm_cache* cache);
/* The same with a self-conditioning signal sc_dev [B, L - canvas_off, d] float32 added to
 * the embeddings of the canvas columns [canvas_off, L) (the decoder input of Algorithm 2;
 * NULL: none). */
tadm_status tadm_anchor_forward_sc(tadm_model* m, const tadm_context* ctx, const int32_t* canvas_dev,
                                   int32_t B, int32_t L, int32_t i, int32_t T, const float* sc_dev,
                                   int32_t canvas_off, tadm_cache* cache);

/* One reverse step on a stale (or fresh) cache (Sec. 3.1, eq. DenoiserOp;
 * MDLM posterior with carry-over, App. B.1.1):
 * c = S(canvas), h~ = Phi(c, cache), x = D(h~), logits = head(x) for the canvas
 * columns [canvas_off, L), then tadm_sample.  logits_dev (float32
 * [B, L - canvas_off, V]) may be NULL: then the head runs only on the masked
 * positions (the only ones whose logits the reverse step uses; in ENTROPY mode every
 * canvas position goes through the head).  next_canvas_dev
 * [B, L] receives the canvas after the step (it may alias canvas_dev).  The cache
 * is read only. */
tadm_status tadm_denoise_step(tadm_model* m, const tadm_context* ctx, const int32_t* canvas_dev,
                              int32_t B, int32_t L, int32_t canvas_off, const tadm_cache* cache,
                              const tadm_step_args* args, float* logits_dev,
                              int32_t* next_canvas_dev);

/* Masked-diffusion reverse step from given logits [B, L - canvas_off, V]
 * (MDLM zero-masking and carry-over, App. B.1.1, with sigma_t = 0).
 * For every masked position (absolute position pos0 + column): Gumbel-max token
 * from softmax(logits * inv_temp) with Philox4x32-10 noise, and its confidence
 * (log-probability at that temperature; the normaliser is summed in 2^-40 fixed
 * point per group of 64 vocabulary entries relative to the group maximum, and the
 * groups' integer sums are rescaled to the row maximum and added as integers, so the
 * result does not depend on summation order).  Logits must be finite.
 * Per row, the n_unmask (or n_unmask_rows[b]) masked positions of highest
 * (confidence, then lowest position) take their token; every other entry of
 * canvas_dev is copied.
 * choice_dev / conf_dev ([B, L - canvas_off], nullable) receive the sampled token
 * and confidence (-1 / -inf where not masked).
 * In ENTROPY mode every position is sampled: choice_dev receives x_tilde and conf_dev
 * the entropy H; the rest follows TADM_STEP_ENTROPY (sc_in is not used here, the
 * self-conditioning signal needs the model's embedding; L - canvas_off <= 8192). */
tadm_status tadm_sample(tadm_model* m, const float* logits_dev, const int32_t* canvas_dev,
                        int32_t B, int32_t L, int32_t canvas_off, int32_t pos0,
                        const tadm_step_args* args, int32_t* next_canvas_dev,
                        int32_t* choice_dev, float* conf_dev);

/* tadm_sample for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same arguments,
 * results bit-identical to tadm_sample, but it calls no hipMalloc/hipFree and never
 * touches the model's workspace: the per-position tokens, confidences and nucleus
 * thresholds that pass between its kernels live in a fixed device array of the
 * library, one per GPU (TADM_NOALLOC_MAX_POSITIONS entries, about 2 MB, held until the
 * process ends; its address is looked up on the first call on each device).
 * Limits: B * (L - canvas_off) <= TADM_NOALLOC_MAX_POSITIONS, else TADM_ERR_INVALID;
 * ENTROPY mode returns TADM_ERR_UNSUPPORTED (its statistics need the workspace).  The
 * stage timers are not used.  Every call on one GPU shares that array: calls that
 * overlap on one GPU (on different streams, or from several threads) race and must be
 * serialised by the caller; nothing in it needs clearing between calls. */
#define TADM_NOALLOC_MAX_POSITIONS 65536
tadm_status tadm_sample_noalloc(tadm_model* m, const float* logits_dev, const int32_t* canvas_dev,
                                int32_t B, int32_t L, int32_t canvas_off, int32_t pos0,
                                const tadm_step_args* args, int32_t* next_canvas_dev,
                                int32_t* choice_dev, float* conf_dev);

/* Whole generation (Algorithm 1 with the linear unmask schedule
 * n_i = floor(M0 i / T) - floor(M0 (i-1) / T)).  prompt_dev [B, P]; tokens_dev
 * [B, P + gen_len] receives prompt and generated tokens.  block_len == gen_len:
 * one bidirectional canvas; block_len < gen_len (must divide gen_len): block
 * diffusion with a context KV.  Returns after enqueueing. */
tadm_status tadm_generate(tadm_model* m, const int32_t* prompt_dev, int32_t B, int32_t P,
                          int32_t gen_len, int32_t T, int32_t K, int32_t block_len, uint64_t seed,
                          float temperature, int32_t* tokens_dev);

/* Pure host helper: n_i of the linear schedule. */
int32_t tadm_unmask_count(int32_t M0, int32_t i, int32_t T);

/* Sampler of a whole generation.  kind TADM_STEP_RANKED: confidence-ranked unmasking
 * with the linear schedule (the default of tadm_generate).  kind TADM_STEP_REMASK:
 * the remasking posterior with sigma_i = min(eta, (1 - alpha_s) / alpha_t), the
 * largest remasking probability that keeps the posterior's mask probability
 * 1 - alpha_s - sigma alpha_t non-negative (ReMDM-Cap's form; eta = 0 is the plain
 * absorbing posterior), on the linear schedule alpha_t = 1 - t.
 * kind TADM_SAMPLER_LOOP: the ReMDM-Loop schedule (the paper's sampler for T >= L,
 * App. C.2 sampler details, with eta = 0.02, t_on = 0.55, t_off = 0.05, alpha_on = 0.9):
 * alpha rises linearly from 0 at t = 1 to alpha_on at t_on, stays at alpha_on down to
 * t_off and rises linearly to 1 at t = 0; steps wholly inside [t_off, t_on] remask with
 * sigma = min(eta, (1 - alpha_s) / alpha_t), the others have sigma = 0.  Its steps run
 * in TADM_STEP_REMASK mode.  Needs 0 < t_off < t_on < 1 and 0 < alpha_on < 1. */
enum { TADM_SAMPLER_LOOP = 2 };
/* kind TADM_SAMPLER_ENTROPY: uniform-state generation with the entropy-bound sampler
 * (Algorithm 2; the paper's settings eta = 0.1, tau 0.8 -> 0.4, T = 48, canvas blocks of
 * 256): each block starts from uniform tokens ((w V) >> 32, w = Philox word 0 at
 * counter (2^31 + 2, absolute position, row, block index)) and a zero self-conditioning
 * signal; step n runs at 1 / tau_n = tadm_entropy_inv_temp(n, T, tau_max, tau_min) in
 * TADM_STEP_ENTROPY mode with eta the entropy bound, feeding each step's signal s = pE
 * to the next.  The result is the last step's argmax canvas; `temperature` is unused. */
enum { TADM_SAMPLER_ENTROPY = 3 };
typedef struct {
  int32_t kind;
  float eta;
  float top_p;  /* nucleus of the sampled tokens (0 or 1: off); the paper's runs use 0.9 */
  double t_on, t_off, alpha_on;  /* TADM_SAMPLER_LOOP only */
  float tau_max, tau_min;        /* TADM_SAMPLER_ENTROPY only: 0 < tau_min <= tau_max */
} tadm_sampler;

/* Pure host helper: (sigma, p_unmask) of reverse step i under the capped schedule,
 * computed in double and rounded to float. */
void tadm_remask_probs(int32_t i, int32_t T, float eta, float* sigma, float* p_unmask);
/* Pure host helper: (sigma, p_unmask) of reverse step i (t = i/T, s = (i-1)/T) under the
 * ReMDM-Loop schedule described above, computed in double and rounded to float. */
void tadm_loop_probs(int32_t i, int32_t T, float eta, double t_on, double t_off, double alpha_on, float* sigma,
                     float* p_unmask);

/* Pure host helper: float32(1 / tau_n), tau_n = tau_min + (tau_max - tau_min) n / T
 * computed in double (the temperature schedule of Algorithm 2). */
float tadm_entropy_inv_temp(int32_t n, int32_t T, float tau_max, float tau_min);

/* tadm_generate with a sampler (NULL: confidence-ranked). */
tadm_status tadm_generate_sampler(tadm_model* m, const int32_t* prompt_dev, int32_t B, int32_t P,
                                  int32_t gen_len, int32_t T, int32_t K, int32_t block_len, uint64_t seed,
                                  float temperature, const tadm_sampler* sampler, int32_t* tokens_dev);

/* ------------------------------------------------------------- training ---- */
/* Training objective of TADM:Pretraining (Sec. 5, Theorem T-ANELBO with gamma = 0 and
 * sigma = 0; training details of App. C.2), forward pass.  Per row b of the clean tokens
 * x_dev [B, L] (ids < vocab), with times t_dev[b] in (0, 1] and t_stale_dev[b] in
 * [t_b, 1] (device float32 [B]):
 *   z_t, z_t': position l is masked in z_t iff u < float((1 - eps) t_b), in z_t' iff
 *     u < float((1 - eps) t'_b), u = (2 (w >> 9) + 1) 2^-24 with w Philox4x32-10 word 0
 *     at counter (2^31 + 3, l, b, step) (the log-linear schedule alpha_t = 1 - (1-eps) t;
 *     z_t' is z_t further corrupted, eq. fwd_t_t');
 *   logits = head(D(Phi(S(z_t), (A(S(z_t')), S(z_t'))))) on the positions masked in z_t;
 *   loss_dev[b] = (1 / t_b) sum over those positions of -log softmax(logits)[x] (the
 *     continuous-time weight of lambda_t for this schedule).
 * n_masked_dev [B], zt_dev / zs_dev [B, L] are optional outputs (NULL: not written).
 * Positions [0, L) of one sequence, no context; B <= max_batch, L <= max_seq. */
tadm_status tadm_train_loss(tadm_model* m, const int32_t* x_dev, int32_t B, int32_t L, const float* t_dev,
                            const float* t_stale_dev, float eps, uint64_t seed, uint32_t step, float* loss_dev,
                            int32_t* n_masked_dev, int32_t* zt_dev, int32_t* zs_dev);
/* Pure host helper: the training times of a batch (App. C.2): with (w0, w1, w2, w3) =
 * Philox4x32-10 at counter (2^31 + 4, b, step, 0) and u0 = (2 (w0 of row 0 >> 9) + 1) 2^-24,
 * t_b = float(eps + (1 - eps) frac(u0 + b / B)) (antithetic), K_b = {1, 2, 4, 8}[w1 >> 30],
 * T_b = {128, 256, 512, 1024, 2048, 4096}[(6 w2) >> 32], k_b = (K_b w3) >> 32 (the cache age),
 * t'_b = float(min(1, t_b + k_b / T_b)); arithmetic in double.  Outputs are host arrays
 * [B]; K, T, k may be NULL. */
void tadm_stale_times(int32_t B, uint64_t seed, uint32_t step, float eps, float* t, float* t_stale, int32_t* K,
                      int32_t* T, int32_t* k);

/* -------------------------------------------------------- observability ---- */
/* Copies (float32) a buffer of the last step into dst_dev:
 *   TADM_TAP_EMBED  c = S(z)          [B, L, d]
 *   TADM_TAP_FUSED  h~ = Phi(c, h')   [B, L, d]
 *   TADM_TAP_FINAL  final-normed D output of the canvas columns [B, L - off, d]
 *                   (only after a step that was given logits_dev)
 *   TADM_TAP_CHOICE sampled token of every canvas column [B, L - off] (int32 bits;
 *                   -1 where the entry was not masked)
 *   TADM_TAP_CONF   its confidence [B, L - off] (float32; -inf where not masked) */
enum { TADM_TAP_EMBED = 0, TADM_TAP_FUSED = 1, TADM_TAP_FINAL = 2, TADM_TAP_CHOICE = 3, TADM_TAP_CONF = 4 };
/* Keep a copy of h~ for TADM_TAP_FUSED (one extra [B, L, d] copy per step; off by default). */
tadm_status tadm_debug_taps(tadm_model* m, int32_t enable);
/* Per-layer capture for layer-by-layer checks: from now on every transformer layer li
 * that runs (in any call) copies the residual stream entering it to slot 3 li, the
 * stream after its attention half to slot 3 li + 1 and the stream leaving it to slot
 * 3 li + 2 of dst_dev, each slot [B, L, d] float32 of that call (caller-owned, bytes =
 * capacity; a layer whose slots do not fit is skipped).  A slot holds the last call
 * that ran the layer.  dst_dev = NULL turns capture off.  Costs three device copies per
 * layer; for tests. */
tadm_status tadm_debug_layers(tadm_model* m, float* dst_dev, size_t bytes);
/* Enqueues copies of one layer's context K [B, Hkv, cap, head_dim] (rotary embedding
 * applied) and V transposed [B, Hkv, head_dim, cap], in the model dtype; positions
 * [0, tadm_context_length) are committed.  bytes is the size of each array
 * (TADM_ERR_INVALID otherwise). */
tadm_status tadm_context_read(const tadm_context* ctx, int32_t layer, void* k_dev, void* vt_dev, size_t bytes);
/* cap of a context: max_ctx rounded up to a multiple of 64 (0 for NULL). */
int32_t tadm_context_capacity(const tadm_context* ctx);
tadm_status tadm_debug_read(tadm_model* m, int32_t tap, float* dst_dev, size_t bytes);

/* Per-stage timing on the model stream for each stage whose bit is set in stage_mask
 * (bit s = stage s; 0 = off, -1 = all).  Stages nest.  A single-kernel stage (HEAD,
 * SAMPLE and QKV..FUSION2; with fp32 weights FFN_UP times its GEMM only, with a nucleus
 * SAMPLE times the draw and not the threshold kernel) hands a pair of
 * events to its kernel launch (hipExtLaunchKernel), which stamps the kernel's own start
 * and end and adds nothing to the stream; the other stages record events before and
 * after their launches.  read synchronises the stream and sums the intervals recorded
 * since the last reset; reset also drops stages left open by a failed call.  Stage ids: */
enum {
  TADM_STAGE_EMBED = 0, TADM_STAGE_ANCHOR = 1, TADM_STAGE_FUSION = 2, TADM_STAGE_DENOISE = 3,
  TADM_STAGE_HEAD = 4, TADM_STAGE_SAMPLE = 5, TADM_STAGE_SELECT = 6, TADM_STAGE_CONTEXT = 7,
  /* single-kernel stages inside the layers and the gated-MLP fusion (every layer of
   * every pass): q/k/v projection (with rotary epilogue), attention, output projection,
   * feed-forward up (gate+up) and down projections, fusion GEMM 1 and 2 */
  TADM_STAGE_QKV = 8, TADM_STAGE_ATTN = 9, TADM_STAGE_OPROJ = 10, TADM_STAGE_FFN_UP = 11,
  TADM_STAGE_FFN_DOWN = 12, TADM_STAGE_FUSION1 = 13, TADM_STAGE_FUSION2 = 14,
  /* the self-conditioning product s = pE of the entropy-bound sampler (its K-split
   * GEMM and ordered reduction); in that sampler SAMPLE is the statistics kernel and
   * SELECT the acceptance */
  TADM_STAGE_SELFCOND = 15,
  TADM_STAGE_COUNT = 16
};
tadm_status tadm_profile_enable(tadm_model* m, int32_t stage_mask);
tadm_status tadm_profile_read(tadm_model* m, int32_t stage, double* total_ms, int64_t* count);
tadm_status tadm_profile_reset(tadm_model* m);

/* Message of the last failure on the calling thread ("" if none). */
const char* tadm_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* TADM_H */
