// Host-side argument checks of the C ABI. Pure C++: no HIP calls, so every
// error path can be exercised without a GPU.
#pragma once

#include <cmath>
#include <cstddef>
#include <cstdint>

#include "tim.h"

namespace tim {

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline int n_tiles_of(int32_t V) { return (int)((V + TIM_VOCAB_TILE - 1) / TIM_VOCAB_TILE); }
inline int n_half_tiles_of(int32_t V) { return (int)((V + TIM_VOCAB_TILE / 2 - 1) / (TIM_VOCAB_TILE / 2)); }

// Shape/value checks shared by tim_logprobs, tim_logits and the workspace query.
inline tim_status check_shape(int64_t T, int32_t d, int32_t V, int32_t order) {
  if (T < 0) return TIM_ERR_SHAPE;
  if (d <= 0 || d % 128 != 0) return TIM_ERR_SHAPE;
  if (order == TIM_ORDER_SPLITK4 && d % 256 != 0) return TIM_ERR_SHAPE;
  if (V < 1 || V > TIM_MAX_VOCAB) return TIM_ERR_SHAPE;
  return TIM_OK;
}

inline bool valid_mode(int32_t mode) { return mode == TIM_MODE_ROLLOUT || mode == TIM_MODE_TRAINING; }
inline bool valid_order(int32_t order) { return order == TIM_ORDER_INVARIANT || order == TIM_ORDER_SPLITK4; }
inline bool positive_finite(float x) { return std::isfinite(x) && x > 0.f; }

// Training launches take at most training_launch_cap(d) rows: the largest
// multiple of 8192 (at least 8192) whose hidden block, beside the weight
// tiles the eight XCDs stream at once (a group of 4 vocabulary tiles of
// 256 x d bf16 each: 16384 d bytes), stays within 224 MiB of the 256 MB
// memory-side cache. 16384 rows at d = 4096, 8192 at d = 5120, 49152 at
// d = 2048. Rows are independent, so the split changes no result.
constexpr int64_t kLaunchRowUnit = 8192;
constexpr int64_t kLaunchCacheBudget = (int64_t)224 << 20;
inline int64_t training_launch_cap(int32_t d) {
  const int64_t fit = kLaunchCacheBudget / (2 * (int64_t)d) - kLaunchRowUnit;
  const int64_t cap = fit / kLaunchRowUnit * kLaunchRowUnit;
  return cap > kLaunchRowUnit ? cap : kLaunchRowUnit;
}

// Rows handed to one launch: T in rollout mode; in training mode the
// micro-batch (T when 0 or larger), at most training_launch_cap(d).
inline int64_t rows_per_launch(int64_t T, int32_t d, int32_t mode, int64_t micro_batch) {
  if (mode != TIM_MODE_TRAINING) return T;
  const int64_t rows = (micro_batch > 0 && micro_batch < T) ? micro_batch : T;
  const int64_t cap = training_launch_cap(d);
  return rows > cap ? cap : rows;
}

// Rollout launches of at most this many rows (decode batches) may form their
// partials over half vocabulary tiles; their workspace covers that case.
constexpr int64_t kHalfTileRows = 128;
inline bool uses_half_tiles(int64_t rows, int32_t mode) { return mode == TIM_MODE_ROLLOUT && rows <= kHalfTileRows; }

inline size_t workspace_bytes(int64_t T, int32_t d, int32_t V, int32_t mode, int64_t micro_batch) {
  const int64_t rows = rows_per_launch(T, d, mode, micro_batch);
  const int per_row = uses_half_tiles(rows, mode) ? n_half_tiles_of(V) : n_tiles_of(V);
  return (size_t)rows * (size_t)per_row * 16u;
}

// Every argument of tim_logprobs but the workspace.
inline tim_status validate_logprobs_args(const void* hidden, const void* w, const int32_t* tokens,
                                         int64_t T, int32_t d, int32_t V, float temperature,
                                         int32_t mode, int64_t micro_batch, int32_t order,
                                         const float* logp) {
  if (T < 0) return TIM_ERR_SHAPE;
  if (T == 0) return TIM_OK;
  if (!hidden || !w || !tokens || !logp) return TIM_ERR_NULL;
  const tim_status s = check_shape(T, d, V, order);
  if (s != TIM_OK) return s;
  if (!positive_finite(temperature)) return TIM_ERR_VALUE;
  if (!valid_mode(mode) || !valid_order(order) || micro_batch < 0) return TIM_ERR_VALUE;
  if (!aligned16(hidden) || !aligned16(w)) return TIM_ERR_VALUE;
  return TIM_OK;
}

inline tim_status validate_logprobs(const void* hidden, const void* w, const int32_t* tokens,
                                    int64_t T, int32_t d, int32_t V, float temperature,
                                    int32_t mode, int64_t micro_batch, int32_t order,
                                    const float* logp, const void* ws, size_t ws_bytes) {
  const tim_status s = validate_logprobs_args(hidden, w, tokens, T, d, V, temperature, mode, micro_batch, order, logp);
  if (s != TIM_OK || T == 0) return s;
  if (!ws || !aligned16(ws) || ws_bytes < workspace_bytes(T, d, V, mode, micro_batch))
    return TIM_ERR_WORKSPACE;
  return TIM_OK;
}

// tim_logprobs_noalloc: the arguments, then whether its partials fit the
// device scratch array (checked before the array's address is looked up).
inline tim_status validate_logprobs_noalloc(const void* hidden, const void* w, const int32_t* tokens,
                                            int64_t T, int32_t d, int32_t V, float temperature,
                                            int32_t mode, int64_t micro_batch, int32_t order,
                                            const float* logp) {
  const tim_status s = validate_logprobs_args(hidden, w, tokens, T, d, V, temperature, mode, micro_batch, order, logp);
  if (s != TIM_OK || T == 0) return s;
  if (workspace_bytes(T, d, V, mode, micro_batch) > TIM_NOALLOC_SCRATCH_BYTES) return TIM_ERR_WORKSPACE;
  return TIM_OK;
}

inline tim_status validate_mismatch(const float* a, const float* b, int64_t T, float C) {
  if (T < 0) return TIM_ERR_SHAPE;
  if (T == 0) return TIM_OK;
  if (!a || !b) return TIM_ERR_NULL;
  if (!positive_finite(C)) return TIM_ERR_VALUE;
  return TIM_OK;
}

inline bool valid_estimator(int32_t e) { return e == TIM_EST_K1 || e == TIM_EST_K3; }

inline tim_status validate_mismatch_seq(const float* a, const float* b, int64_t T, const int64_t* cu,
                                        int64_t n_seq, int32_t estimator, float C, double tau_seq) {
  if (T < 0 || n_seq < 0 || n_seq > INT32_MAX) return TIM_ERR_SHAPE;
  if (n_seq == 0) return TIM_OK;
  if (!cu) return TIM_ERR_NULL;
  if (T > 0 && (!a || !b)) return TIM_ERR_NULL;
  if (!valid_estimator(estimator) || !positive_finite(C) || std::isnan(tau_seq)) return TIM_ERR_VALUE;
  return TIM_OK;
}

inline tim_status validate_logits(const void* hidden, const void* w, int64_t T, int32_t d,
                                  int32_t V, float temperature, int32_t order, const float* out) {
  if (T < 0) return TIM_ERR_SHAPE;
  if (T == 0) return TIM_OK;
  if (!hidden || !w || !out) return TIM_ERR_NULL;
  const tim_status s = check_shape(T, d, V, order);
  if (s != TIM_OK) return s;
  if (!positive_finite(temperature) || !valid_order(order)) return TIM_ERR_VALUE;
  if (!aligned16(hidden) || !aligned16(w)) return TIM_ERR_VALUE;
  return TIM_OK;
}

// ------------------------------------------------------------ backward

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
inline size_t align256(size_t x) { return (x + 255u) & ~(size_t)255u; }

// micro_batch of the backward: 0 (all T in one pass) or a positive multiple
// of 128 tokens, so that micro-batches continue the weight-gradient chain on
// whole MFMA k-steps.
inline bool valid_backward_micro_batch(int64_t mb) { return mb == 0 || (mb > 0 && mb % 128 == 0); }

// Largest token count of one backward pass: the weight-gradient operands of a
// 256-row tile then stay within 32-bit buffer offsets.
constexpr int64_t kMaxBackwardStep = (int64_t)1 << 22;

// Workspace of tim_logprobs_backward, each part 256-byte aligned:
// row words [step] float4 | W^T bf16 [d_pad, V_pad] | dlogits bf16
// [step_pad, V_pad] | dlogits^T bf16 [V_pad, T_pad] | hidden^T bf16
// [d_pad, T_pad], the four bf16 operands in the products' packed layout of
// whole 256-row tiles (d_pad, step_pad: d, step rounded up to 256).
struct BackwardLayout {
  int64_t step, t_pad, v_pad, d_pad, step_pad;
  size_t coef, wt, dacc, dacct, ht, total;
};

inline BackwardLayout backward_layout(int64_t T, int32_t d, int32_t V, int64_t micro_batch) {
  BackwardLayout l;
  l.step = (micro_batch > 0 && micro_batch < T) ? micro_batch : T;
  l.t_pad = round_up(l.step, 128);
  l.v_pad = (int64_t)n_tiles_of(V) * TIM_VOCAB_TILE;
  l.d_pad = round_up(d, 256);
  l.step_pad = round_up(l.step, 256);
  size_t off = 0;
  l.coef = off;
  off += align256((size_t)l.step * 16u);
  l.wt = off;
  off += align256((size_t)l.d_pad * (size_t)l.v_pad * 2u);
  l.dacc = off;
  off += align256((size_t)l.step_pad * (size_t)l.v_pad * 2u);
  l.dacct = off;
  off += align256((size_t)l.v_pad * (size_t)l.t_pad * 2u);
  l.ht = off;
  off += align256((size_t)l.d_pad * (size_t)l.t_pad * 2u);
  l.total = off;
  return l;
}

// Arguments common to the logit-gradient pass and the full backward.
inline tim_status validate_grad_inputs(const void* hidden, const void* w, const int32_t* tokens, float temperature,
                                       const float* lse, const float* entropy, const float* grad_logp,
                                       const float* grad_entropy) {
  if (!hidden || !w || !tokens || !lse || !grad_logp) return TIM_ERR_NULL;
  if (grad_entropy && !entropy) return TIM_ERR_NULL;
  if (!positive_finite(temperature)) return TIM_ERR_VALUE;
  if (!aligned16(hidden) || !aligned16(w)) return TIM_ERR_VALUE;
  return TIM_OK;
}

inline tim_status validate_backward(const void* hidden, const void* w, const int32_t* tokens, int64_t T,
                                    int32_t d, int32_t V, float temperature, const float* lse,
                                    const float* entropy, const float* grad_logp, const float* grad_entropy,
                                    int64_t micro_batch, const float* grad_hidden, const float* grad_w,
                                    int32_t accumulate, const void* ws, size_t ws_bytes) {
  if (T < 0) return TIM_ERR_SHAPE;
  const tim_status s = check_shape(T, d, V, TIM_ORDER_INVARIANT);
  if (s != TIM_OK) return s;
  if (!positive_finite(temperature)) return TIM_ERR_VALUE;
  if (!valid_backward_micro_batch(micro_batch) || (accumulate != 0 && accumulate != 1)) return TIM_ERR_VALUE;
  if ((grad_hidden && !aligned16(grad_hidden)) || (grad_w && !aligned16(grad_w))) return TIM_ERR_VALUE;
  if (T == 0 || (!grad_hidden && !grad_w)) return TIM_OK;
  if (backward_layout(T, d, V, micro_batch).step > kMaxBackwardStep) return TIM_ERR_VALUE;
  const tim_status g = validate_grad_inputs(hidden, w, tokens, temperature, lse, entropy, grad_logp, grad_entropy);
  if (g != TIM_OK) return g;
  if (!ws || !aligned16(ws) || ws_bytes < backward_layout(T, d, V, micro_batch).total) return TIM_ERR_WORKSPACE;
  return TIM_OK;
}

inline tim_status validate_logit_grads(const void* hidden, const void* w, const int32_t* tokens, int64_t T,
                                       int32_t d, int32_t V, float temperature, const float* lse,
                                       const float* entropy, const float* grad_logp, const float* grad_entropy,
                                       const void* dlogits, const void* ws, size_t ws_bytes) {
  if (T < 0) return TIM_ERR_SHAPE;
  const tim_status s = check_shape(T, d, V, TIM_ORDER_INVARIANT);
  if (s != TIM_OK) return s;
  if (T == 0) return TIM_OK;
  if (!dlogits) return TIM_ERR_NULL;
  const tim_status g = validate_grad_inputs(hidden, w, tokens, temperature, lse, entropy, grad_logp, grad_entropy);
  if (g != TIM_OK) return g;
  if (!aligned16(dlogits)) return TIM_ERR_VALUE;
  if (!ws || !aligned16(ws) || ws_bytes < (size_t)T * 16u) return TIM_ERR_WORKSPACE;
  return TIM_OK;
}

// ------------------------------------------------------------ PPO / GRPO loss

inline tim_status validate_ppo(const float* logp, const float* logp_old, const float* adv, int64_t T,
                               const int64_t* cu, int64_t n_seq, float eps_low, float eps_high,
                               const double* seq_loss, const double* batch_loss) {
  if (T < 0 || n_seq < 0 || n_seq > INT32_MAX) return TIM_ERR_SHAPE;
  if (!std::isfinite(eps_low) || !std::isfinite(eps_high) || eps_low < 0.f || eps_low >= 1.f || eps_high < 0.f)
    return TIM_ERR_VALUE;
  if (n_seq == 0) return TIM_OK;
  if (!cu) return TIM_ERR_NULL;
  if (T > 0 && (!logp || !logp_old || !adv)) return TIM_ERR_NULL;
  if (batch_loss && !seq_loss) return TIM_ERR_NULL;
  return TIM_OK;
}

// ------------------------------------------------------------ final RMS norm

// Largest row count of the weight gradient (its column partial sums use one
// grid row per 256 rows).
constexpr int64_t kMaxNormRows = (int64_t)65535 * 256;

inline tim_status check_norm_shape(int64_t T, int32_t d) {
  if (T < 0 || T > kMaxNormRows) return TIM_ERR_SHAPE;
  if (d <= 0 || d % 8 != 0) return TIM_ERR_SHAPE;
  return TIM_OK;
}

inline size_t rmsnorm_backward_workspace(int64_t T, int32_t d) {
  return (size_t)((T + 255) / 256) * (size_t)d * 4u;
}

inline tim_status validate_rmsnorm(const void* x, const void* gamma, int64_t T, int32_t d, float eps,
                                   const void* h) {
  const tim_status s = check_norm_shape(T, d);
  if (s != TIM_OK) return s;
  if (!std::isfinite(eps) || eps < 0.f) return TIM_ERR_VALUE;
  if (T == 0) return TIM_OK;
  if (!x || !h) return TIM_ERR_NULL;
  if (!aligned16(x) || !aligned16(h) || (gamma && !aligned16(gamma))) return TIM_ERR_VALUE;
  return TIM_OK;
}

inline tim_status validate_rmsnorm_backward(const void* x, const void* gamma, const float* rstd, const float* grad_h,
                                            int64_t T, int32_t d, const float* grad_x, const float* grad_gamma,
                                            int32_t accumulate, const void* ws, size_t ws_bytes) {
  const tim_status s = check_norm_shape(T, d);
  if (s != TIM_OK) return s;
  if (accumulate != 0 && accumulate != 1) return TIM_ERR_VALUE;
  if (!grad_x && !grad_gamma) return TIM_OK;
  if (T > 0 && (!x || !rstd || !grad_h)) return TIM_ERR_NULL;
  if ((x && !aligned16(x)) || (gamma && !aligned16(gamma)) || (grad_h && !aligned16(grad_h)) ||
      (grad_x && !aligned16(grad_x)))
    return TIM_ERR_VALUE;
  if (grad_gamma && T > 0 && (!ws || !aligned16(ws) || ws_bytes < rmsnorm_backward_workspace(T, d)))
    return TIM_ERR_WORKSPACE;
  return TIM_OK;
}

}  // namespace tim
