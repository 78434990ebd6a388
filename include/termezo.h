/*
 * termezo.h -- C ABI of the MI355X (gfx950) TerMeZO sparse zeroth-order step.
 *
 * TerMeZO (Sec. 3 and Algorithm 1 of the paper) fine-tunes the latent weights
 * w of a BitNet model's ternary linear projections with two-point SPSA
 * (eq. spsa), perturbing and updating only a mask of latents that lie close
 * to the ternary quantiser's decision boundaries (eq. distance,
 * eq. selection_init, eq. selection_).  This library holds the hot path of one
 * step on one GPU: mask construction, seed-regenerated perturbation with
 * absmean requantisation, BitLinear forward (per-token absmax int8 activations
 * x ternary weights, int32 accumulation, rescale) and the masked update.
 *
 * Conventions shared by every call
 *   - All functions return a termezo_status; no C++ exception crosses the ABI.
 *     A call that fails validation changes no state; termezo_last_error()
 *     returns a message for the last failure on a context.
 *   - A context is not thread-safe.  All device work is ordered on the HIP
 *     stream given at creation.  Only the calls that return host values
 *     (build_mask, update with k_out, mse_loss, model_loss, sync and the
 *     exports) wait for the stream; they also report a deferred error
 *     raised by an earlier kernel on that context (NUMERIC, or INVALID_ARG for
 *     a token id out of range).
 *   - Device pointers are plain device addresses of memory owned by the
 *     caller (for example PyTorch tensors); host pointers are noted as such.
 *   - Latent weights are BORROWED: the caller owns them and they must outlive
 *     the context.  The library writes them only in termezo_update, and only
 *     at the active indices.
 *   - Global ids: layers are enumerated in registration order; inside a layer
 *     the latent matrix is row-major [d_out][d_in]; gid = (sum of the sizes
 *     of the earlier layers) + row * d_in + col.
 *   - Gaussian directions z are regenerated from the 64-bit seed with
 *     Philox4x32-10 (counter = (gid >> 2, stream 0)) and the Box-Muller
 *     transform; they are never stored.
 */
#ifndef TERMEZO_H_
#define TERMEZO_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TERMEZO_OK = 0,
  TERMEZO_ERR_INVALID_ARG = 1, /* bad argument; nothing was done            */
  TERMEZO_ERR_STATE = 2,       /* call not valid in the current state       */
  TERMEZO_ERR_DEVICE = 3,      /* no usable HIP device / HIP runtime error  */
  TERMEZO_ERR_OOM = 4,         /* device allocation failed                  */
  TERMEZO_ERR_NUMERIC = 5      /* non-finite value or |w| >= 4 in a latent  */
} termezo_status;

typedef enum {
  TERMEZO_F32 = 0,
  TERMEZO_BF16 = 1,
  TERMEZO_I8 = 2,
  TERMEZO_I32 = 3
} termezo_dtype;

/* One ternary linear projection (Sec. 3: q, k, v, o and every MLP linear).
 * latent: device pointer to d_out * d_in latent weights, row-major, 16-byte
 * aligned, of the context's latent dtype.  d_in must be a multiple of 16 and
 * d_out * d_in must not exceed 2^25 (the fixed-point |w| sum stays exact). */
typedef struct {
  void* latent;
  int64_t d_out;
  int64_t d_in;
} termezo_layer;

typedef struct termezo_ctx termezo_ctx;

/* Register the latent weights of n_layers projections (latent_dtype F32 or
 * BF16) and allocate the library-owned state: packed 2-bit ternary codes
 * (d_out * d_in / 4 bytes per layer), per-layer thresholds and fixed-point
 * sums, and mask storage.  hip_stream: a hipStream_t (NULL = default stream).
 * At most 2048 layers per context; each layer at most 2^25 weights.
 * Errors: INVALID_ARG (null pointers, n_layers <= 0 or > 2048, d_in % 16 != 0,
 * misaligned latent, layer too large, bad dtype), DEVICE, OOM. */
termezo_status termezo_create(const termezo_layer* layers, int32_t n_layers,
                              termezo_dtype latent_dtype, void* hip_stream,
                              termezo_ctx** out);

/* Free every library-owned buffer.  Never frees the latents.  NULL is a no-op. */
void termezo_destroy(termezo_ctx* ctx);

/* Message describing the last failure on ctx ("" if none).  Owned by ctx. */
const char* termezo_last_error(const termezo_ctx* ctx);

/* Initial mask (Sec. 3, eq. distance and eq. selection_init; the initial
 * threshold and selection of Algorithm 1).  Computes tau^l = 0.5 (mean|w^l| + delta) per layer,
 * the distance d_i = min(|w_i - tau|, |w_i + tau|) of every latent, the global
 * budget k0 = floor(rho0 * D) and xi0, the k0-th smallest distance over all
 * layers (ties at xi0 broken by ascending gid; tie_inclusive != 0 keeps every
 * distance <= xi0 instead).  Also sets the current codes to Q(w) (clean).
 * k0_out, xi0_out: host pointers (nullable) receiving the mask size and xi0.
 * Waits for the stream.  Rebuilding discards the previous mask.
 * Errors: INVALID_ARG (rho0 not in (0, 1], delta <= 0 or not finite),
 * STATE (k0 == 0), NUMERIC (a latent non-finite or |w| >= 4). */
termezo_status termezo_build_mask(termezo_ctx* ctx, float rho0, float delta,
                                  int32_t tie_inclusive, int64_t* k0_out,
                                  float* xi0_out);

/* Perturbed evaluation point (Algorithm 1: w +/- eps m (.) z).  Sets the
 * current ternary codes and scales of every layer to the requantisation of
 * w' = w + sign * eps * m (.) z(seed): w'_i = fma(sign * eps, z_i, w_i) on the
 * active set, w'_i = w_i elsewhere; tau' and beta' = 2 tau' are recomputed from
 * w' (the quantiser is applied on the fly to the perturbed latents, eq.
 * objective).  The latents themselves are not modified.  sign = 0 gives the
 * clean codes.  Registered theta tensors are perturbed too (see the theta
 * section below).  Records (seed, eps) for the following termezo_update.
 * Perturbation pairs: the first call with a (seed, eps) and sign +-1 also forms
 * the perturbed values of the other sign (list order, 4 bytes per active latent
 * of library memory; z itself is never stored); a following call with the same
 * seed and eps and either sign reuses them.  Any other seed or eps, sign 0, an
 * update or a mask rebuild starts afresh; the caller must not write the latents
 * in between (they are borrowed).
 * Errors: INVALID_ARG (sign not in {-1, 0, 1}; eps <= 0 or not finite),
 * STATE (no mask).  A perturbed |w'| >= 4 raises a deferred NUMERIC. */
termezo_status termezo_perturb(termezo_ctx* ctx, uint64_t seed, float eps,
                               int32_t sign);

/* Requantisation strategy of termezo_perturb (the codes are the same either way).
 * By default a perturbation rewrites only the codes of the active latents while
 * no frozen code can change: every frozen latent is tracked to lie at least a
 * bound m^l (exactly, from xi0 and the threshold drift) from the threshold its
 * code was computed with, and a layer whose perturbed threshold tau' moves by
 * less than m^l keeps its frozen codes (the actives' codes are rewritten one by
 * one, or, above 1/256 active, tile by tile over the code words); other layers
 * are requantised densely.
 * always_dense != 0 requantises every latent of every layer on each call
 * (for measurement).  Errors: INVALID_ARG (null ctx). */
termezo_status termezo_set_dense_requant(termezo_ctx* ctx, int32_t always_dense);

/* BitLinear forward of one projection on its current codes (Sec. 1 and 3:
 * ternary weights with 8-bit activations).  x: device [M][d_in] (F32 or BF16);
 * y: device [M][d_out] (F32 or BF16).  Per token row m: a_m = max_k |x[m][k]|,
 * s_m = 127 / max(a_m, 1e-5), x_q = clamp(round_half_even(x * s_m), -128, 127);
 * acc[m][n] = sum_k x_q[m][k] * c[n][k] exactly in int32;
 * y[m][n] = float(acc) * (beta' / s_m) (rounded to bf16 if y is BF16).
 * xq_out [M][d_in] int8, xscale_out [M] fp32 (s_m), acc_out [M][d_out] int32:
 * optional device outputs (nullable) for inspection.
 * Errors: INVALID_ARG (layer out of range, M <= 0, bad dtype, null x or y),
 * STATE (no current codes: before build_mask or after update). */
termezo_status termezo_bitlinear_forward(termezo_ctx* ctx, int32_t layer,
                                         const void* x, termezo_dtype x_dtype,
                                         int64_t M, void* y, termezo_dtype y_dtype,
                                         int8_t* xq_out, float* xscale_out,
                                         int32_t* acc_out);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): the same BitLinear
 * forward as termezo_bitlinear_forward (same kernels, same results) without the
 * inspection outputs, whose activation-quantisation scratch (int8 x_q, the
 * per-token scales and the per-token sums of x_q) lives in a fixed 16 MiB device
 * array inside the library instead of context buffers grown on demand.  The call
 * allocates nothing.  Limit: M * d_in bytes rounded up to 256, plus 4 * M rounded
 * up to 256, plus 4 * M, at most 16 MiB (for example M <= 6533 at d_in = 2560,
 * M <= 2424 at d_in = 6912).  Each GPU holds
 * one copy of the array, shared by every context and call on that GPU: calls
 * whose work overlaps on one GPU (different streams, or different host
 * threads) race on it; calls ordered on one stream do not.  Nothing in the
 * array needs to start at zero.  Errors: as termezo_bitlinear_forward, and
 * INVALID_ARG when M exceeds the limit; DEVICE if the array's address could
 * not be obtained at context creation. */
termezo_status termezo_bitlinear_forward_noalloc(termezo_ctx* ctx, int32_t layer, const void* x,
                                                 termezo_dtype x_dtype, int64_t M, void* y,
                                                 termezo_dtype y_dtype);

/* Masked projected-gradient update (Algorithm 1, last loop, K = 1) followed by
 * the shrink-only set update (eq. selection_).  With the seed of the last
 * termezo_perturb: for every active i, w_i <- round(fma(-(lr * g), z_i, w_i))
 * (round = to nearest-even bf16 for BF16 latents, identity for F32); unmasked
 * latents are untouched.  Then tau^l is recomputed from the updated latents and
 * the active set keeps only the i with d_i <= xi0 (order preserved).
 * Registered theta tensors are updated with the same g (theta section below).
 * proj_grad is g = (F+ - F-) / (2 eps) (eq. spsa).  k_out: host pointer
 * (nullable) receiving the new mask size; when non-NULL the call waits.
 * Invalidates the current codes.  Errors: INVALID_ARG (g or lr not finite),
 * STATE (no perturbation since the last update or mask build). */
termezo_status termezo_update(termezo_ctx* ctx, float proj_grad, float lr,
                              int64_t* k_out);

/* Device-side projected gradient and update (Algorithm 1: g = (F+ - F-) / (2 eps),
 * then the same update and shrink as termezo_update) without a host round
 * trip: loss_plus and loss_minus are device fp32 scalars (for example written
 * by termezo_model_loss).  g is formed in fp32 on the device as
 * (F+ - F-) / (2 eps).  A non-finite g skips the latent update and raises a
 * deferred NUMERIC.  Never waits.  Errors: INVALID_ARG (null pointers, eps or
 * lr not positive/finite), STATE as for termezo_update. */
termezo_status termezo_update_from_losses(termezo_ctx* ctx, const float* loss_plus,
                                          const float* loss_minus, float eps, float lr);

/* ---- memory-optimal storage (Sec. 5 eq. memory: frozen weights as 2-bit codes) ----
 * After the mask is built, termezo_compact copies the active latents into a
 * library-owned array in list order; from then on the context never reads or
 * writes the caller's latent tensors (they may be freed).  Frozen latents live
 * on only as their ternary codes.  Perturbation, update and shrink work on the
 * compact array (contiguous instead of scattered accesses).  The codes are
 * those of the dense semantics while every layer's threshold stays within its
 * frozen margin (see termezo_set_dense_requant); if a perturbed threshold ever
 * moves farther, the frozen codes are kept and a deferred NUMERIC error names
 * the condition.  termezo_build_mask then fails with STATE (it needs the full
 * latents).  Errors: STATE (no mask, already compact, pending perturbation),
 * OOM.  Waits for the stream. */
termezo_status termezo_compact(termezo_ctx* ctx);

/* Values (fp32, host) of one layer's active latents in list order (ascending
 * local index); *n receives the count.  Works with and without compact mode.
 * Errors: INVALID_ARG (layer, null n, cap below the count), STATE (no mask).
 * Waits for the stream. */
termezo_status termezo_active_values(termezo_ctx* ctx, int32_t layer, float* values,
                                     int64_t cap, int64_t* n);

/* Device memory of the method's state (host values, nullable): library_bytes =
 * the library-owned buffers (codes, mask lists, thresholds, tile tables, the
 * list-order copy of the active latents -- kept for sets of at most 1/8 of the
 * latents and in compact mode --, theta copies, the codes snapshot once taken,
 * scratch); latent_bytes = the caller's latent tensors the context still needs
 * (0 in compact mode). */
termezo_status termezo_memory_footprint(termezo_ctx* ctx, int64_t* library_bytes,
                                        int64_t* latent_bytes);

/* K perturbation directions per step (Algorithm 1: the K two-point estimates
 * are all taken at w_t, then the K updates are applied).  After the caller has
 * evaluated F+_k and F-_k for every seed s_k (termezo_perturb(s_k, eps, +1),
 * loss, termezo_perturb(s_k, eps, -1), loss), one call applies, at every active
 * latent (and every registered theta value),
 *   v = fma(a_K, z_K, ... fma(a_1, z_1, w) ...) in fp32,  w <- round(v),
 * with a_k = -((lr / K) * g_k) in fp32 and z_k regenerated from s_k, then the
 * shrink of termezo_update.  With fp32 storage this equals the K updates of
 * Algorithm 1 applied one after another; with bf16 storage the sum is rounded
 * once.  seeds, proj_grads: host arrays of K entries, 1 <= K <= 32.
 * k_out as for termezo_update.  Errors: INVALID_ARG (K out of range, null
 * arrays, non-finite g or lr), STATE (no perturbation since the last update). */
termezo_status termezo_update_multi(termezo_ctx* ctx, const uint64_t* seeds,
                                    const float* proj_grads, int32_t K, float lr,
                                    int64_t* k_out);

/* The same with the projected gradients formed on the device from the losses
 * (device fp32 [2K]: F+_1, F-_1, F+_2, F-_2, ...): g_k = (F+_k - F-_k) / (2 eps)
 * in fp32; seeds is a host array.  Never waits.  A non-finite g_k skips the
 * update and raises a deferred NUMERIC.  Errors as above (eps must be > 0). */
termezo_status termezo_update_multi_from_losses(termezo_ctx* ctx, const uint64_t* seeds,
                                                const float* losses, int32_t K, float eps,
                                                float lr);

/* ---- evolution strategies on the mask (appendix on RL-based fine-tuning) -------
 * The RL variant evaluates N one-sided perturbations w + sigma m (.) z_n
 * (termezo_perturb(s_n, sigma, +1), then the caller's reward R_n) and updates
 * with the reward-weighted sum of the directions, restricted to the mask:
 *   v = fma(a_N, z_N, ... fma(a_1, z_1, w) ...) in fp32,  w <- round(v),
 * a_n = (lr / N) * Rt_n in fp32 (lr / N one fp32 division), at every active
 * latent (and every registered theta value, stream 1), then the shrink of
 * termezo_update.  standardize != 0: Rt_n = fp32((R_n - mu) / sd) with mu and
 * the population deviation sd computed in fp64 in index order (all Rt zero when
 * sd = 0, so N = 1 or equal rewards leave the weights unchanged); standardize
 * = 0: Rt_n = R_n.  seeds: host array of N entries, 1 <= N <= 32.  A negative
 * lr descends instead of ascends (rewards = losses).
 * Errors: INVALID_ARG (N out of range, null arrays, non-finite reward, lr or
 * coefficient), STATE (no perturbation since the last update). */
termezo_status termezo_es_update(termezo_ctx* ctx, const uint64_t* seeds, const float* rewards,
                                 int32_t N, float lr, int32_t standardize, int64_t* k_out);

/* The same with the rewards in device memory (fp32 [N]); never waits.  A
 * non-finite coefficient skips the update and raises a deferred NUMERIC. */
termezo_status termezo_es_update_from_rewards(termezo_ctx* ctx, const uint64_t* seeds,
                                              const float* rewards, int32_t N, float lr,
                                              int32_t standardize);

/* ---- full-precision parameters theta (Sec. 3; Algorithm 1) ---------------------
 * Algorithm 1 perturbs and updates the full-precision parameters (embeddings,
 * normalisation weights, LM head) densely, together with the masked latents,
 * with directions drawn from the same seed.  Registering theta switches this on;
 * without registration theta is frozen.
 *   - theta ids: the registered tensors are enumerated in registration order,
 *     each flat; id = (sum of the sizes of the earlier tensors) + index.
 *     z_theta(id) is drawn like z (Philox4x32-10 + Box-Muller, same seed) on
 *     counter stream 1: counter = (id >> 2, stream 1).
 *   - termezo_perturb(seed, eps, sign != 0) makes the forward read
 *     theta' = round(fma(sign * eps, z_theta, theta)) (round = to nearest-even
 *     bf16 for BF16 tensors, identity for F32), held in library-owned copies;
 *     theta itself is not modified.  Both signs of a (seed, eps) pair are
 *     produced by the first of the two calls; sign = 0 reads theta itself.
 *   - termezo_update / termezo_update_from_losses apply, after the latent
 *     update, theta <- round(fma(-(lr * g), z_theta, theta)) in place (a
 *     non-finite g leaves theta untouched), and the forward reads theta again.
 * The tensors are BORROWED (caller-owned device memory that must outlive the
 * context); the caller must not write them while a perturbation is pending. */
typedef struct {
  void* data;              /* device pointer, 16-byte aligned                 */
  int64_t n;               /* number of elements                              */
  termezo_dtype dtype;     /* F32 or BF16                                     */
} termezo_theta;

/* Register n tensors as theta (once per context).  Allocates two copies of each
 * (the +eps and -eps values).  Errors: INVALID_ARG (null or misaligned data,
 * n <= 0, bad dtype), STATE (already registered), OOM. */
termezo_status termezo_theta_register(termezo_ctx* ctx, const termezo_theta* params,
                                      int32_t n);

/* *values receives the device pointer the forward pass must read for tensor i
 * now: the perturbed copy after termezo_perturb with sign +1 or -1, else the
 * caller's tensor.  Errors: INVALID_ARG (i out of range, null values). */
termezo_status termezo_theta_current(termezo_ctx* ctx, int32_t i, void** values);

/* Copy (device to device, ordered on the context's stream, no wait) the values
 * termezo_theta_current points to for tensor i into the caller's device buffer
 * dst (n elements of the tensor's dtype).  Inspection support.
 * Errors: INVALID_ARG (i out of range, null dst), DEVICE. */
termezo_status termezo_theta_copy(termezo_ctx* ctx, int32_t i, void* dst);

/* ---- BitNet decoder around the registered projections (Sec. 3) ----------------
 * The context's layers must be the ternary projections of n_blocks decoder
 * blocks in the order q, k, v, o, gate, up, down (shapes [n_heads*hd][d],
 * [n_kv_heads*hd][d] twice, [d][n_heads*hd], [d_ffn][d] twice, [d][d_ffn],
 * hd = d_model / n_heads).  The full-precision parameters are the token
 * embedding (tied to the LM head), the caller's device matrix [vocab][d_model]
 * in act_dtype, and the RMSNorm weights (one unless set with
 * termezo_model_set_norm_weights).  Either may be a registered theta tensor;
 * the forward then reads its current values.  Blocks are pre-norm:
 * h += o(attn(rope(q(x)), rope(k(x)), v(x))), x = rmsnorm(h); then
 * h += down(silu(gate(x)) * up(x)).  Attention is causal grouped-query with
 * scale 1/sqrt(hd); rotary pairs are (i, i + hd/2) with angle
 * p * rope_base^(-2i/hd).  Activations are stored in act_dtype between kernels;
 * BitLinear inputs are quantised per token as in termezo_bitlinear_forward. */
typedef struct {
  int32_t n_blocks, d_model, n_heads, n_kv_heads, d_ffn, vocab;
  float rope_base;          /* e.g. 10000 */
  float norm_eps;           /* e.g. 1e-5  */
  termezo_dtype act_dtype;  /* F32 or BF16 */
} termezo_model_config;

typedef struct termezo_model termezo_model;

/* Bind a decoder to ctx (which must outlive it).  embedding: device pointer,
 * 16-byte aligned, borrowed.  Errors: INVALID_ARG (shapes do not match the
 * registered layers, unsupported head_dim for BF16 (64, 96, 128), d_model or
 * d_ffn above 8192, bad dtype). */
termezo_status termezo_model_create(termezo_ctx* ctx, const termezo_model_config* cfg,
                                    const void* embedding, termezo_model** out);
/* RMSNorm weights of the model: norm_weights is a device [2 n_blocks + 1][d_model]
 * array in act_dtype, 16-byte aligned, borrowed (row 2 b scales the attention
 * input of block b, row 2 b + 1 its MLP input, the last row the LM-head input);
 * NULL restores weights one.  Errors: INVALID_ARG (misaligned pointer). */
termezo_status termezo_model_set_norm_weights(termezo_model* model, const void* norm_weights);

/* Free the model's activation buffers (it does not touch the context, which
 * may already have been destroyed).  NULL is a no-op. */
void termezo_model_destroy(termezo_model* model);

/* Batch loss of eq. objective_est with next-token cross-entropy: the mean over
 * the batch * (seq - 1) labelled positions of logsumexp(logits) - logit[next
 * token], with the current codes (clean or perturbed).  tokens: device int32
 * [batch][seq]; every id must lie in [0, vocab).  Outputs (all optional):
 * loss_dev (device fp32 scalar), row_loss_dev (device fp32 [batch*seq], 0 at
 * each sequence's last position), loss_host (host; the call then waits and
 * reports deferred errors).  An id outside [0, vocab) is read as id 0 (the
 * embedding is never read out of bounds) and raises a deferred INVALID_ARG,
 * reported by this call when loss_host is given, else by the next waiting
 * call (termezo_sync, ...); the losses of that call are then meaningless.
 * Errors: INVALID_ARG, STATE (no current codes), OOM. */
termezo_status termezo_model_loss(termezo_model* model, const int32_t* tokens, int32_t batch,
                                  int32_t seq, float* loss_dev, float* row_loss_dev,
                                  float* loss_host);

/* The two evaluations of a perturbation pair, F(w + eps z) and F(w - eps z) on the
 * same batch (Algorithm 1), depend on nothing but the pair's codes, so they may run
 * at the same time.  termezo_codes_snapshot copies the current codes and output
 * scales (those of the last termezo_perturb) into a library-owned buffer (allocated
 * on the first call: 4 bytes per 16 latents plus 4 per layer), stream-ordered on the
 * context's stream; a model set to read the snapshot (termezo_model_use_snapshot)
 * evaluates that perturbation while the next termezo_perturb rewrites the current
 * codes.  termezo_model_set_stream runs a model's forwards on a stream of the
 * caller's (NULL: the context's stream, the default): each termezo_model_loss then
 * starts after the work queued on the context's stream, and termezo_model_join
 * makes the context's stream wait for the model's work before anything queued after
 * it (the update that reads the losses).  A snapshot stays valid until the next
 * snapshot; the caller orders a snapshot after the forwards that read the previous
 * one (a join does).  Errors: INVALID_ARG (null), STATE (no current codes; a
 * snapshot model before any snapshot), OOM, DEVICE. */
termezo_status termezo_codes_snapshot(termezo_ctx* ctx);
termezo_status termezo_model_set_stream(termezo_model* model, void* hip_stream);
termezo_status termezo_model_use_snapshot(termezo_model* model, int32_t on);
termezo_status termezo_model_join(termezo_model* model);

/* Event timing of the model's matrix-core kernels, for measurement: with
 * enable != 0 every following termezo_model_loss records a HIP event pair on
 * the context's stream for each launch of class 0 (BitLinear int8 GEMM) and 2
 * (LM head with cross-entropy partials), whose events take the kernel's own
 * start and end (hipExtLaunchKernel), and around each launch pair of class 1
 * (attention: K/V preparation, then the attention kernel); enabling or
 * disabling clears the records.  termezo_model_timing waits for the stream and
 * returns, for one class, the summed kernel time in ms, the number of launches
 * and their algorithmic operation count (2 M K N per GEMM; 4 B H hd S(S+1)/2
 * for causal attention; 2 M d V for the LM head). */
termezo_status termezo_model_set_timing(termezo_model* model, int32_t enable);
termezo_status termezo_model_timing(termezo_model* model, int32_t cls, double* ms,
                                    int64_t* launches, double* ops);

/* ---- inspection and support calls (not part of the four hot-path calls) ---- */

/* Wait for the context's stream; reports a deferred NUMERIC error. */
termezo_status termezo_sync(termezo_ctx* ctx);

/* Copy one layer's ascending active local indices (row * d_in + col) to the
 * host buffer idx (capacity cap entries); *n receives the count.
 * Errors: INVALID_ARG (layer range, null n, cap < count), STATE (no mask). */
termezo_status termezo_mask_export(termezo_ctx* ctx, int32_t layer, uint32_t* idx,
                                   int64_t cap, int64_t* n);

/* Unpack one layer's current ternary codes to host int8 [d_out][d_in]. */
termezo_status termezo_codes_export(termezo_ctx* ctx, int32_t layer, int8_t* codes);

/* Host copies of one layer's clean (tau, beta, fixed-point sum) and current
 * (tau', beta') scales; any pointer may be NULL. */
termezo_status termezo_layer_stats(termezo_ctx* ctx, int32_t layer, float* tau,
                                   float* beta, int64_t* abs_sum_fix,
                                   float* tau_cur, float* beta_cur);

/* Mean squared error of device fp32 y against device fp32 target over n
 * elements: e = y - t and e*e in fp32, the sum in fp64, mean rounded to fp32.
 * out: host pointer.  Waits for the stream. */
termezo_status termezo_mse_loss(termezo_ctx* ctx, const float* y, const float* target,
                                int64_t n, float* out);

/* The same mean squared error written to a device fp32 scalar (loss_dev), e.g.
 * for termezo_update_from_losses; never waits.  Errors: INVALID_ARG. */
termezo_status termezo_mse_loss_dev(termezo_ctx* ctx, const float* y, const float* target,
                                    int64_t n, float* loss_dev);

/* Gaussian directions z_i for n global ids (device uint64 gids, device fp32
 * z), exactly as the perturbation and the update regenerate them from seed.
 * hip_stream: a hipStream_t (NULL = default stream); no synchronisation. */
termezo_status termezo_gauss(void* hip_stream, uint64_t seed, const uint64_t* gids, int64_t n,
                             float* z);

/* Number of active latents (host value; waits for the stream). */
termezo_status termezo_active_count(termezo_ctx* ctx, int64_t* k);

#ifdef __cplusplus
}
#endif

#endif /* TERMEZO_H_ */
