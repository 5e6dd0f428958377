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

// Rows handed to one launch.
inline int64_t rows_per_launch(int64_t T, int32_t mode, int64_t micro_batch) {
  if (mode == TIM_MODE_TRAINING && micro_batch > 0 && micro_batch < T) return micro_batch;
  return T;
}

inline size_t workspace_bytes(int64_t T, int32_t V, int32_t mode, int64_t micro_batch) {
  return (size_t)rows_per_launch(T, mode, micro_batch) * (size_t)n_tiles_of(V) * 16u;
}

inline tim_status validate_logprobs(const void* hidden, const void* w, const int32_t* tokens,
                                    int64_t T, int32_t d, int32_t V, float temperature,
                                    int32_t mode, int64_t micro_batch, int32_t order,
                                    const float* logp, const void* ws, size_t ws_bytes) {
  if (T < 0) return TIM_ERR_SHAPE;
  if (T == 0) return TIM_OK;
  if (!hidden || !w || !tokens || !logp) return TIM_ERR_NULL;
  const tim_status s = check_shape(T, d, V, order);
  if (s != TIM_OK) return s;
  if (!positive_finite(temperature)) return TIM_ERR_VALUE;
  if (!valid_mode(mode) || !valid_order(order) || micro_batch < 0) return TIM_ERR_VALUE;
  if (!aligned16(hidden) || !aligned16(w)) return TIM_ERR_VALUE;
  if (!ws || !aligned16(ws) || ws_bytes < workspace_bytes(T, V, mode, micro_batch))
    return TIM_ERR_WORKSPACE;
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

}  // namespace tim
