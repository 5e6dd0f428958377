/*
 * tim.h -- batch-invariant fused LM-head token log-probabilities and
 * training-inference mismatch statistics on AMD MI355X (gfx950).
 *
 * The quantities follow "Diagnosing Training Inference Mismatch in LLM
 * Reinforcement Learning" (VeXact):
 *   - the token log-probability log pi(a_t | s_t) that the rollout engine and
 *     the trainer must agree on (Section 2; the two sides of Eq. 1), computed
 *     with kernels whose tiling and reduction order do not depend on how rows
 *     are batched (the batch-invariance principle of Section 3.1);
 *   - the per-token discrepancy delta_t of Eq. 1, the K3 estimator of
 *     Section 4.1 and the truncated importance weight of Eq. 6 (Section 4.2).
 *
 * Conventions shared by every entry point:
 *   - All array arguments are DEVICE pointers owned by the caller. The library
 *     allocates nothing, keeps no state between calls and never synchronises:
 *     every kernel is enqueued on `stream` (0 = the null stream) and the call
 *     returns as soon as the launches are enqueued.
 *   - Argument errors are detected on the host, before anything is enqueued,
 *     and reported by the return value; on any error no output is written.
 *   - T == 0 is a successful no-op (pointers are not inspected).
 *   - A failed kernel launch returns TIM_ERR_HIP; outputs are then undefined.
 *   - Calls that overlap in time must not share a workspace.
 */
#ifndef TIM_H
#define TIM_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TIM_OK = 0,
  TIM_ERR_NULL = 1,      /* a required pointer is NULL */
  TIM_ERR_SHAPE = 2,     /* T < 0, d not a positive multiple of 128 (256 for TIM_ORDER_SPLITK4),
                            V outside [1, TIM_MAX_VOCAB] */
  TIM_ERR_VALUE = 3,     /* temperature or C not finite or <= 0, unknown mode/order,
                            micro_batch < 0, hidden or w_vocab not 16-byte aligned */
  TIM_ERR_WORKSPACE = 4, /* workspace NULL or smaller than tim_logprobs_workspace_size() */
  TIM_ERR_HIP = 5        /* a HIP runtime call or kernel launch failed */
} tim_status;

/* Launch shape only: both modes compute every row with identical arithmetic,
 * so their outputs are bitwise equal for any batching of the same rows. */
typedef enum {
  TIM_MODE_ROLLOUT = 0,  /* one call per decode step: a ragged batch of rows, one launch */
  TIM_MODE_TRAINING = 1  /* packed token stream, processed in micro-batches of micro_batch rows (each
                            micro-batch in launches of at most tim_logprobs_rows_per_launch rows) */
} tim_mode;

/* Reduction order. TIM_ORDER_SPLITK4 is a deliberately different order of the
 * same mathematics (the hidden dimension summed as four separately accumulated
 * quarters, the vocabulary partials folded left to right instead of by a
 * balanced tree). It models a second engine whose kernels reduce in another
 * order -- the second source of mismatch named in Section 3.1 -- and exists to
 * produce controlled, small mismatches for tim_mismatch. */
typedef enum {
  TIM_ORDER_INVARIANT = 0,
  TIM_ORDER_SPLITK4 = 1
} tim_order;

/* Vocabulary entries per softmax partial (the fixed vocab tile width). */
#define TIM_VOCAB_TILE 256
/* Largest supported vocabulary: 2048 tiles. */
#define TIM_MAX_VOCAB (2048 * TIM_VOCAB_TILE)

/* Rows tim_logprobs hands to one kernel launch: T in rollout mode; in training
 * mode min(T, micro_batch) (micro_batch 0 means T), at most
 * max(8192, floor((224 MiB / (2 d) - 8192) / 8192) * 8192) rows: the largest
 * multiple of 8192 whose bf16 hidden block, beside the 16384 d bytes of weight
 * tiles the GPU's eight XCDs stream at once, fits 224 MiB of the 256 MB
 * memory-side cache (16384 rows at d = 4096, 8192 at d = 5120). A training
 * micro-batch longer than that runs as consecutive launches; rows are
 * independent, so no result changes. Callers composing tim_logprobs_partials
 * and tim_logprobs_merge themselves take the same launches from this. Returns
 * 0 for T <= 0, d not a positive multiple of 128, a bad mode or
 * micro_batch < 0. Pure host function. */
int64_t tim_logprobs_rows_per_launch(int64_t T, int32_t d, int32_t mode, int64_t micro_batch);

/* Bytes of device workspace tim_logprobs needs for these arguments:
 * rows_per_launch * ceil(V / TIM_VOCAB_TILE) * 16, with rows_per_launch from
 * tim_logprobs_rows_per_launch; in rollout mode with T <= 128 (a decode batch,
 * whose partials may be taken over half tiles)
 * T * ceil(V / (TIM_VOCAB_TILE / 2)) * 16. Returns 0 for invalid arguments or
 * T == 0. Pure host function. */
size_t tim_logprobs_workspace_size(int64_t T, int32_t d, int32_t V, int32_t mode, int64_t micro_batch);

/* Token log-probabilities and entropies of T rows (Section 2, Eq. 1's terms).
 *
 * For row i, with z_v = (sum_k hidden[i,k] * w_vocab[v,k]) * (1/temperature):
 *   logp[i]    = z_{tokens[i]} - log sum_v exp(z_v)
 *   entropy[i] = - sum_v p_v log p_v,  p_v = softmax(z)_v   (nats)
 *   lse[i]     = log sum_v exp(z_v)
 *
 * hidden   bf16 [T, d] row-major, 16-byte aligned (final hidden states).
 * w_vocab  bf16 [V, d] row-major, 16-byte aligned (LM-head weight, vocab-major).
 * tokens   int32 [T]; tokens[i] is the token sampled from row i's distribution
 *          (no label shift is applied). A token outside [0, V) yields
 *          logp[i] = NaN; entropy[i] and lse[i] are still computed.
 * temperature  finite and > 0; the logits are multiplied by the fp32 value
 *          (float)(1.0 / temperature) in every mode and order.
 * mode, micro_batch  see tim_mode; micro_batch is ignored in rollout mode.
 * order    tim_order.
 * logp     fp32 [T] out (required); entropy, lse fp32 [T] out, may be NULL.
 * workspace, workspace_bytes  device scratch of at least
 *          tim_logprobs_workspace_size(T, d, V, mode, micro_batch) bytes.
 *
 * Arithmetic: bf16 x bf16 products accumulated in fp32 by MFMA with the
 * hidden dimension in ascending order; fp32 softmax partials per tile of
 * TIM_VOCAB_TILE vocabulary entries, each the merge of its two halves' (lower
 * half first); partials merged by a fixed balanced tree over the tile index.
 * None of this depends on T, mode, micro_batch or a row's position in the
 * batch (a decode batch of at most 128 rows may write the halves' partials
 * and merge each pair in the merge pass, which gives the same bits), so with
 * TIM_ORDER_INVARIANT a row's outputs are bitwise identical however it is
 * batched. NaN or Inf in the inputs
 * propagates to that row's outputs. */
tim_status tim_logprobs(const void* hidden, const void* w_vocab, const int32_t* tokens,
                        int64_t T, int32_t d, int32_t V, float temperature,
                        int32_t mode, int64_t micro_batch, int32_t order,
                        float* logp, float* entropy, float* lse,
                        void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Size of the device scratch array behind tim_logprobs_noalloc: 64 MiB, held
 * by every GPU the library runs on until the process ends. */
#define TIM_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/* tim_logprobs for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc. Same
 * arguments, outputs and errors as tim_logprobs, without the workspace: the
 * softmax partials go to a file-scope device array of
 * TIM_NOALLOC_SCRATCH_BYTES per GPU, whose address is looked up once per
 * device on that device's first call. The call allocates nothing (no
 * hipMalloc / hipFree, no allocating library routine) and gives exactly the
 * bits of tim_logprobs on the same arguments.
 *
 * Limit: tim_logprobs_workspace_size(T, d, V, mode, micro_batch) must not
 * exceed TIM_NOALLOC_SCRATCH_BYTES, else TIM_ERR_WORKSPACE before anything is
 * enqueued (at V = 151936: up to 7061 rows per launch -- a rollout batch of
 * that many rows, or training micro-batches of at most that many tokens).
 * TIM_ERR_HIP if the device array's address cannot be obtained.
 *
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * partials (each launch writes every partial it reads, so nothing needs
 * clearing). Calls that overlap in time on one GPU (on different streams or
 * from different host threads) race on the array: serialise them. */
tim_status tim_logprobs_noalloc(const void* hidden, const void* w_vocab, const int32_t* tokens,
                                int64_t T, int32_t d, int32_t V, float temperature,
                                int32_t mode, int64_t micro_batch, int32_t order,
                                float* logp, float* entropy, float* lse, hipStream_t stream);

/* The two stages of tim_logprobs, for callers that schedule them themselves
 * (a profiler timing one kernel, or a vocabulary-sharded deployment that
 * exchanges partials between the stages). tim_logprobs over one launch's rows
 * gives exactly the outputs of tim_logprobs_partials followed by
 * tim_logprobs_merge (whose partials are always per whole tile).
 *
 * tim_logprobs_partials: one launch over all T rows (no micro-batching; mode
 * only picks the row tile). Writes T * ceil(V / TIM_VOCAB_TILE) partials of
 * 16 bytes (running max, sum of exponentials, sum of exponential-weighted
 * logit offsets, gathered token logit) into `workspace`, which must hold
 * tim_logprobs_workspace_size(T, d, V, TIM_MODE_ROLLOUT, 0) bytes. Arguments
 * and errors as tim_logprobs.
 *
 * tim_logprobs_merge: reduces those partials to logp / entropy / lse (same
 * definitions as tim_logprobs). `tokens`, T, V and `order` must be the ones
 * given to the partials call; TIM_ORDER_SPLITK4 folds the partials left to
 * right instead of by the balanced tree. Errors: TIM_ERR_SHAPE for T < 0 or V
 * out of range, TIM_ERR_NULL for a NULL workspace / tokens / logp,
 * TIM_ERR_VALUE for an unknown order. */
tim_status tim_logprobs_partials(const void* hidden, const void* w_vocab, const int32_t* tokens,
                                 int64_t T, int32_t d, int32_t V, float temperature,
                                 int32_t mode, int32_t order,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream);
tim_status tim_logprobs_merge(const void* workspace, const int32_t* tokens, int64_t T, int32_t V,
                              int32_t order, float* logp, float* entropy, float* lse,
                              hipStream_t stream);

/* Token-level mismatch statistics between two evaluations of the same tokens
 * (Section 2, Eq. 1; Section 4.1 K3; Section 4.2 r_corr and Eq. 6):
 *   log_ratio[i] = logp_a[i] - logp_b[i]          (delta_t; a = trainer, b = rollout)
 *   k3[i]        = expm1(delta) - delta            ((r - 1) - log r with r = exp(delta))
 *   is_weight[i] = min(exp(delta), C)              (truncated correction ratio)
 * All fp32 device arrays of length T; any output may be NULL (not written).
 * C must be finite and > 0 (the paper's tau_tok is 2). */
tim_status tim_mismatch(const float* logp_a, const float* logp_b, int64_t T, float C,
                        float* log_ratio, float* k3, float* is_weight, hipStream_t stream);

/* Estimator of the sequence-level score (Section 4.1): K1(r) = -log r,
 * K3(r) = (r - 1) - log r. */
typedef enum {
  TIM_EST_K1 = 1,
  TIM_EST_K3 = 3
} tim_estimator;

/* Sequence-level mismatch score, rejection mask and token weights
 * (Section 4.2: token-level truncation min(r_corr, tau_tok) and sequence-level
 * rejection 1[S_seq <= tau_seq] with S_seq = sum over the response of
 * K(r_corr,t); the appendix's tis-srs-k1/k3-corr objectives weight each token's
 * PPO term by both).
 *
 * The stream of T tokens packs n_seq responses: response j is the tokens
 * [cu_seqlens[j], cu_seqlens[j+1]). With delta_t = logp_a[t] - logp_b[t]
 * (a = trainer, b = rollout, as in tim_mismatch) and r_corr = exp(delta):
 *   score[j]  = sum over response j of K(delta_t), K1 = -delta,
 *               K3 = expm1(delta) - delta; delta and the sum are fp64, summed in
 *               a fixed order that depends only on the response's length (a
 *               response's score is bitwise the same wherever it sits);
 *   keep[j]   = 1 if score[j] <= tau_seq, else 0 (a NaN score rejects);
 *   weight[t] = keep[j] ? min(exp(delta_t), C) : 0 for t in response j, in
 *               fp32 (tim_mismatch's is_weight, zeroed in rejected responses).
 *
 * cu_seqlens  int64 [n_seq + 1] DEVICE array: non-decreasing, cu_seqlens[0] = 0,
 *             cu_seqlens[n_seq] = T. It is only read on the device: bounds are
 *             clamped into [0, T] and reversed bounds give an empty response
 *             (score 0), so malformed offsets cannot make the kernel touch
 *             memory outside the arrays (overlapping responses are not
 *             detected; their weights are then unspecified).
 * estimator   TIM_EST_K1 or TIM_EST_K3.
 * C           finite and > 0 (tau_tok; 2 in the paper); tau_seq must not be NaN
 *             (0.001 in the paper).
 * score fp64 [n_seq], keep uint8 [n_seq], weight fp32 [T]: device outputs, any
 *             may be NULL (not written). Tokens outside every response are not
 *             written.
 * n_seq == 0 is a no-op. Errors: TIM_ERR_SHAPE for T < 0, n_seq < 0 or
 * n_seq > 2^31 - 1; TIM_ERR_NULL for NULL cu_seqlens, or NULL logp_a / logp_b
 * with T > 0; TIM_ERR_VALUE for an unknown estimator, a bad C or a NaN tau_seq. */
tim_status tim_mismatch_seq(const float* logp_a, const float* logp_b, int64_t T,
                            const int64_t* cu_seqlens, int64_t n_seq, int32_t estimator,
                            float C, double tau_seq,
                            double* score, uint8_t* keep, float* weight, hipStream_t stream);

/* Gradients of the token log-probabilities and entropies (the trainer's side
 * of Section 2's Eq. 1: the PPO / GRPO objectives of Section 4 differentiate
 * log pi_train through the ratio, and entropy regularisers the entropy).
 *
 * For a scalar loss L with grad_logp[t] = dL/dlogp[t] and grad_entropy[t] =
 * dL/dentropy[t], and z, p, lse, entropy as in tim_logprobs (same hidden,
 * w_vocab, tokens, temperature), the gradient with respect to the LM-head
 * contraction acc = hidden . w_v of row t is
 *   dlogits[t,v] = ( g ([v == tokens[t]] - p_v) - e p_v (z_v - lse + H) ) / temperature
 * (g = grad_logp[t], or 0 when tokens[t] is outside [0, V); e = grad_entropy[t];
 * H = entropy[t]), and
 *   grad_hidden[t, :] = sum_v dlogits[t,v] w_vocab[v, :]       fp32 [T, d]
 *   grad_w[v, :]      = sum_t dlogits[t,v] hidden[t, :]        fp32 [V, d]
 *
 * lse, entropy  fp32 [T] as returned by tim_logprobs for these inputs (the
 *          logits are recomputed with the forward's own contraction, so p is
 *          exactly the forward's); entropy may be NULL when grad_entropy is.
 * grad_logp fp32 [T] (required); grad_entropy fp32 [T] or NULL (zero).
 * micro_batch  0 (all T in one pass) or a positive multiple of 128: tokens per
 *          pass, bounding the workspace; at most 2^22 tokens per pass.
 * grad_hidden, grad_w  fp32 device outputs, 16-byte aligned; either may be NULL
 *          (not computed). With accumulate_grad_w = 1 the weight gradient is
 *          added to grad_w's contents (gradient accumulation), else it
 *          overwrites them.
 * workspace  at least tim_logprobs_backward_workspace_size(T, d, V,
 *          micro_batch) bytes, 16-byte aligned: about
 *          2 * d * V_pad + 4 * step * V_pad + 2 * d * step bytes with
 *          V_pad = ceil(V / 256) * 256 and step = min(T, micro_batch) (d and
 *          step rounded up to multiples of 256 in the first and second terms).
 *
 * Arithmetic: dlogits is formed in fp32 from the recomputed fp32 logits and
 * rounded once to bf16 (round to nearest even); the two products run on bf16
 * MFMA with one fp32 accumulation chain per output element, the vocabulary
 * (for grad_hidden) and the tokens (for grad_w) in ascending order. A row's
 * grad_hidden is bitwise independent of T, micro_batch and the row's position;
 * grad_w is bitwise independent of micro_batch (the chain over tokens continues
 * across passes) and deterministic, with no atomics. Errors: as tim_logprobs;
 * TIM_ERR_VALUE also for a bad micro_batch or accumulate_grad_w, a misaligned
 * output, or a pass of more than 2^22 tokens; TIM_ERR_NULL for a missing
 * lse / grad_logp, or grad_entropy without entropy. T == 0 writes zeros to
 * grad_w (unless accumulating). */
size_t tim_logprobs_backward_workspace_size(int64_t T, int32_t d, int32_t V, int64_t micro_batch);
tim_status tim_logprobs_backward(const void* hidden, const void* w_vocab, const int32_t* tokens,
                                 int64_t T, int32_t d, int32_t V, float temperature,
                                 const float* lse, const float* entropy,
                                 const float* grad_logp, const float* grad_entropy,
                                 int64_t micro_batch, float* grad_hidden, float* grad_w,
                                 int32_t accumulate_grad_w, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/* The first pass of tim_logprobs_backward on its own, for checking it element
 * by element: writes dlogits (definition above) as bf16 [T, ceil(V / 256) * 256]
 * row-major (entries past V are 0) into `dlogits` (16-byte aligned). The
 * workspace holds T * 16 bytes of per-row coefficients. Arguments and errors
 * as tim_logprobs_backward. */
tim_status tim_logit_grads(const void* hidden, const void* w_vocab, const int32_t* tokens,
                           int64_t T, int32_t d, int32_t V, float temperature,
                           const float* lse, const float* entropy,
                           const float* grad_logp, const float* grad_entropy,
                           void* dlogits, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Clipped PPO / GRPO token loss over a packed stream of n_seq responses
 * (Section 4.1: Eq. 2's surrogate on Eq. 3's ratio, Eq. 5's zero-centred
 * contribution; Section 4.2's token weights), summed over each response and
 * averaged over the responses:
 *   r_t          = exp(logp[t] - logp_old[t])    (logp_old: the trainer's recomputed
 *                                                 or the rollout's old log-probs)
 *   L_t          = -min(r_t A_t, clip(r_t, 1 - eps_low, 1 + eps_high) A_t)
 *   token_loss[t]= w_t L_t                        (w = weight[t], or 1 when NULL)
 *   seq_loss[j]  = sum over response j of token_loss      (fp64, fixed order)
 *   batch_loss[0]= (1 / n_seq) sum_j seq_loss[j]          (fp64)
 *   grad_logp[t] = d batch_loss / d logp[t] = w_t (-A_t r_t) / n_seq where the
 *                  unclipped term is the minimum, else 0 (feeds tim_logprobs_backward)
 *   contribution[t] = -(r_t - 1) A_t               (C(r), the same gradient as -r A)
 *   clipped[t]   = 1 where the clipped term is strictly the minimum (zero gradient)
 * delta = logp - logp_old is formed exactly in fp64, r and the losses in fp64
 * (token outputs rounded once to fp32); the clip decision is taken on delta
 * against log1p(eps_high) / log1p(-eps_low), which is exact. Responses are
 * given by cu_seqlens (int64 [n_seq + 1], DEVICE, clamped into [0, T] as in
 * tim_mismatch_seq); tokens outside every response are not written. A
 * response's outputs are bitwise the same wherever it sits in the stream.
 * advantages fp32 [T] (GRPO: the response's advantage on each of its tokens).
 * All outputs are device pointers and may be NULL, except that batch_loss needs
 * seq_loss. eps_low in [0, 1), eps_high >= 0 (the paper's single eps is both).
 * n_seq == 0 is a no-op. Errors: TIM_ERR_SHAPE for T < 0 or a bad n_seq;
 * TIM_ERR_VALUE for bad eps; TIM_ERR_NULL for NULL cu_seqlens, NULL inputs with
 * T > 0, or batch_loss without seq_loss. */
tim_status tim_ppo_loss(const float* logp, const float* logp_old, const float* advantages, const float* weight,
                        int64_t T, const int64_t* cu_seqlens, int64_t n_seq, float eps_low, float eps_high,
                        double* seq_loss, double* batch_loss, float* token_loss, float* grad_logp,
                        float* contribution, uint8_t* clipped, hipStream_t stream);

/* Final RMS normalisation in front of the LM head (Section 3.1 lists RMSNorm
 * among the batch-invariant kernels; root-mean-square layer normalisation).
 * Row t of x (bf16 [T, d] row-major, 16-byte aligned, d a multiple of 8):
 *   rstd[t] = 1 / sqrt(mean_k x[t,k]^2 + eps)                       (fp32)
 *   h[t,k]  = bf16(gamma[k] * bf16(x[t,k] * rstd[t]))              (bf16(x * rstd) if gamma is NULL)
 * rounding to nearest even, the arithmetic of the model implementation the
 * engine follows (fp32 scale, a cast to bf16, a bf16 multiply by the weight).
 * The sum of squares is reduced in one fixed order that depends only on d, so
 * a row's outputs are bitwise independent of T and of its position. h (bf16
 * [T, d], 16-byte aligned) feeds tim_logprobs as `hidden`; rstd (fp32 [T], may
 * be NULL) feeds the backward. gamma bf16 [d], 16-byte aligned, or NULL.
 * eps finite and >= 0. Errors: TIM_ERR_SHAPE for T < 0, T > 65535 * 256 or a
 * bad d; TIM_ERR_VALUE for a bad eps or alignment; TIM_ERR_NULL for a NULL x
 * or h with T > 0. */
tim_status tim_rmsnorm(const void* x, const void* gamma, int64_t T, int32_t d, float eps,
                       void* h, float* rstd, hipStream_t stream);

/* Backward of tim_rmsnorm with the bf16 casts passed straight through, for
 * grad_h = dL/dh (fp32 [T, d], 16-byte aligned; tim_logprobs_backward's
 * grad_hidden) and rstd from the forward:
 *   grad_x[t,k]  = rstd g_k G_tk - (rstd^3 / d) x_tk sum_j G_tj g_j x_tj    (fp32 [T, d])
 *   grad_gamma[k] (+)= sum_t G_tk x_tk rstd_t                                (fp32 [d])
 * (g = gamma, or ones when NULL). grad_x's row sum runs in the forward's
 * fixed order (batch-invariant); grad_gamma sums blocks of 256 rows in row
 * order (for T >= 65536 and d = 2048 or 4096: blocks of 4 q rows, q = max(64,
 * ceil(T / (4 n))) with n = 512 at d = 4096 and 1024 at d = 2048, each q-row
 * quarter of a block in row order, the quarters as (q0 + q1) + (q2 + q3)),
 * then the blocks in order: deterministic, no atomics. Either output may
 * be NULL (not computed); with accumulate_grad_gamma = 1 the result is added
 * to grad_gamma's contents. The workspace holds
 * tim_rmsnorm_backward_workspace_size(T, d) = ceil(T / 256) * d * 4 bytes
 * (needed only for grad_gamma). Errors as tim_rmsnorm; TIM_ERR_WORKSPACE for a
 * missing or small workspace. */
size_t tim_rmsnorm_backward_workspace_size(int64_t T, int32_t d);
tim_status tim_rmsnorm_backward(const void* x, const void* gamma, const float* rstd, const float* grad_h,
                                int64_t T, int32_t d, float* grad_x, float* grad_gamma,
                                int32_t accumulate_grad_gamma, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* Test and debugging aid: writes the fp32 logits z[T, V] (row-major) exactly as
 * tim_logprobs forms them before the softmax (same kernel code, same
 * accumulation order, same temperature multiply), for checking the gather and
 * the contraction element by element. Same argument rules as tim_logprobs;
 * `order` selects the accumulation order. */
tim_status tim_logits(const void* hidden, const void* w_vocab, int64_t T, int32_t d, int32_t V,
                      float temperature, int32_t order, float* logits, hipStream_t stream);

/* Human-readable name of a status code (static string). */
const char* tim_status_string(tim_status s);

#ifdef __cplusplus
}
#endif

#endif /* TIM_H */
