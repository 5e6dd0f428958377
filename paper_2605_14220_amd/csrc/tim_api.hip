// C-ABI entry points: argument checks, launch planning, launches.
//
// The planner only chooses launch shapes. Rollout mode sends the whole ragged
// batch in one launch with a row tile sized to the batch (64, 128 or 256 rows
// per workgroup; a batch of at most 128 rows may take half vocabulary tiles,
// which run more workgroups per CU);
// training mode walks the packed stream in micro-batches with 256-row tiles.
// Every shape runs the same per-row instruction sequence.

#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>

#include "kernels.h"
#include "tim.h"
#include "validate.h"

namespace {

inline tim_status hip_status(hipError_t e) { return e == hipSuccess ? TIM_OK : TIM_ERR_HIP; }

inline float inv_temperature(float temperature) {
  return (float)(1.0 / (double)temperature);
}

// Rows per workgroup for a launch of `rows` rows.
inline int row_tile_for(int64_t rows, int32_t mode, bool splitk4) {
  int rt = 256;
  if (mode == TIM_MODE_ROLLOUT) rt = rows <= 64 ? 64 : (rows <= 128 ? 128 : 256);
  if (splitk4) rt = 64;  // the split-K engine keeps a second accumulator set
  return rt;
}

// Device scratch of tim_logprobs_noalloc (one copy per GPU, for the life of
// the process). Host code never passes this name to a kernel or a copy: on
// the host it is only a stand-in; its device address comes from
// hipGetSymbolAddress, once per device (scratch_on_current_device).
__device__ __align__(256) unsigned char scratch[TIM_NOALLOC_SCRATCH_BYTES];

// Address of `scratch` on the current device, looked up on the device's first
// call with that device current and kept per device (host threads may race on
// a first call; each looks up the same address). nullptr if the lookup fails.
void* scratch_on_current_device() {
  constexpr int kMaxDevices = 64;
  static std::atomic<void*> cache[kMaxDevices];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void* p = cache[dev].load(std::memory_order_acquire);
  if (p != nullptr) return p;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
  cache[dev].store(p, std::memory_order_release);
  return p;
}

// The launches of tim_logprobs over validated arguments, partials in `workspace`.
tim_status run_logprobs(const void* hidden, const void* w_vocab, const int32_t* tokens, int64_t T, int32_t d,
                        int32_t V, float temperature, int32_t mode, int64_t micro_batch, int32_t order, float* logp,
                        float* entropy, float* lse, void* workspace, hipStream_t stream) {
  tim_status st = TIM_OK;
  const bool splitk4 = order == TIM_ORDER_SPLITK4;
  const int64_t step = tim::rows_per_launch(T, d, mode, micro_batch);
  const int tb = row_tile_for(step, mode, splitk4);
  const bool halves = !splitk4 && tim::uses_half_tiles(step, mode) && tim::prefer_half_tiles(V, step);
  const float inv_tau = inv_temperature(temperature);
  const __bf16* h = (const __bf16*)hidden;
  tim::Partial* part = (tim::Partial*)workspace;

  for (int64_t t0 = 0; t0 < T; t0 += step) {
    const int64_t rows = (T - t0) < step ? (T - t0) : step;
    tim::LmHeadArgs a;
    a.hidden = h + t0 * d;
    a.w = w_vocab;
    a.tokens = tokens + t0;
    a.rows = rows;
    a.d = d;
    a.V = V;
    a.inv_tau = inv_tau;
    a.part = part;
    a.logits = nullptr;
    float* ent = entropy ? entropy + t0 : nullptr;
    float* ls = lse ? lse + t0 : nullptr;
    if (halves) {
      st = hip_status(tim::launch_partials_halves(a, stream));
      if (st != TIM_OK) return st;
      st = hip_status(tim::launch_merge_halves(part, tokens + t0, rows, V, logp + t0, ent, ls, stream));
    } else {
      st = hip_status(tim::launch_partials(a, tb, splitk4, stream));
      if (st != TIM_OK) return st;
      st = hip_status(tim::launch_merge(part, tokens + t0, rows, V, splitk4, logp + t0, ent, ls, stream));
    }
    if (st != TIM_OK) return st;
  }
  return TIM_OK;
}

}  // namespace

extern "C" {

int64_t tim_logprobs_rows_per_launch(int64_t T, int32_t d, int32_t mode, int64_t micro_batch) {
  if (T <= 0 || d <= 0 || d % 128 != 0 || !tim::valid_mode(mode) || micro_batch < 0) return 0;
  return tim::rows_per_launch(T, d, mode, micro_batch);
}

size_t tim_logprobs_workspace_size(int64_t T, int32_t d, int32_t V, int32_t mode, int64_t micro_batch) {
  if (T <= 0 || tim::check_shape(T, d, V, TIM_ORDER_INVARIANT) != TIM_OK) return 0;
  if (!tim::valid_mode(mode) || micro_batch < 0) return 0;
  return tim::workspace_bytes(T, d, V, mode, micro_batch);
}

tim_status tim_logprobs(const void* hidden, const void* w_vocab, const int32_t* tokens, int64_t T,
                        int32_t d, int32_t V, float temperature, int32_t mode, int64_t micro_batch,
                        int32_t order, float* logp, float* entropy, float* lse, void* workspace,
                        size_t workspace_bytes, hipStream_t stream) {
  const tim_status st = tim::validate_logprobs(hidden, w_vocab, tokens, T, d, V, temperature, mode,
                                               micro_batch, order, logp, workspace, workspace_bytes);
  if (st != TIM_OK || T == 0) return st;
  return run_logprobs(hidden, w_vocab, tokens, T, d, V, temperature, mode, micro_batch, order, logp, entropy, lse,
                      workspace, stream);
}

tim_status tim_logprobs_noalloc(const void* hidden, const void* w_vocab, const int32_t* tokens, int64_t T,
                                int32_t d, int32_t V, float temperature, int32_t mode, int64_t micro_batch,
                                int32_t order, float* logp, float* entropy, float* lse, hipStream_t stream) {
  const tim_status st = tim::validate_logprobs_noalloc(hidden, w_vocab, tokens, T, d, V, temperature, mode,
                                                       micro_batch, order, logp);
  if (st != TIM_OK || T == 0) return st;
  void* ws = scratch_on_current_device();
  if (ws == nullptr) return TIM_ERR_HIP;
  return run_logprobs(hidden, w_vocab, tokens, T, d, V, temperature, mode, micro_batch, order, logp, entropy, lse,
                      ws, stream);
}

tim_status tim_logprobs_partials(const void* hidden, const void* w_vocab, const int32_t* tokens,
                                 int64_t T, int32_t d, int32_t V, float temperature, int32_t mode,
                                 int32_t order, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream) {
  const tim_status st = tim::validate_logprobs(hidden, w_vocab, tokens, T, d, V, temperature, mode, 0,
                                               order, /*logp=*/(const float*)workspace, workspace,
                                               workspace_bytes);
  if (st != TIM_OK || T == 0) return st;
  const bool splitk4 = order == TIM_ORDER_SPLITK4;
  tim::LmHeadArgs a;
  a.hidden = hidden;
  a.w = w_vocab;
  a.tokens = tokens;
  a.rows = T;
  a.d = d;
  a.V = V;
  a.inv_tau = inv_temperature(temperature);
  a.part = (tim::Partial*)workspace;
  a.logits = nullptr;
  return hip_status(tim::launch_partials(a, row_tile_for(T, mode, splitk4), splitk4, stream));
}

tim_status tim_logprobs_merge(const void* workspace, const int32_t* tokens, int64_t T, int32_t V,
                              int32_t order, float* logp, float* entropy, float* lse,
                              hipStream_t stream) {
  if (T < 0) return TIM_ERR_SHAPE;
  if (T == 0) return TIM_OK;
  if (!workspace || !tokens || !logp) return TIM_ERR_NULL;
  if (V < 1 || V > TIM_MAX_VOCAB) return TIM_ERR_SHAPE;
  if (!tim::valid_order(order)) return TIM_ERR_VALUE;
  return hip_status(tim::launch_merge((const tim::Partial*)workspace, tokens, T, V,
                                      order == TIM_ORDER_SPLITK4, logp, entropy, lse, stream));
}

tim_status tim_mismatch(const float* logp_a, const float* logp_b, int64_t T, float C,
                        float* log_ratio, float* k3, float* is_weight, hipStream_t stream) {
  const tim_status st = tim::validate_mismatch(logp_a, logp_b, T, C);
  if (st != TIM_OK || T == 0) return st;
  if (!log_ratio && !k3 && !is_weight) return TIM_OK;
  return hip_status(tim::launch_mismatch(logp_a, logp_b, T, C, log_ratio, k3, is_weight, stream));
}

tim_status tim_mismatch_seq(const float* logp_a, const float* logp_b, int64_t T, const int64_t* cu_seqlens,
                            int64_t n_seq, int32_t estimator, float C, double tau_seq, double* score,
                            uint8_t* keep, float* weight, hipStream_t stream) {
  const tim_status st = tim::validate_mismatch_seq(logp_a, logp_b, T, cu_seqlens, n_seq, estimator, C, tau_seq);
  if (st != TIM_OK || n_seq == 0) return st;
  if (!score && !keep && !weight) return TIM_OK;
  return hip_status(tim::launch_mismatch_seq(logp_a, logp_b, T, cu_seqlens, n_seq, estimator == TIM_EST_K3, C,
                                             tau_seq, score, keep, weight, stream));
}

tim_status tim_logits(const void* hidden, const void* w_vocab, int64_t T, int32_t d, int32_t V,
                      float temperature, int32_t order, float* logits, hipStream_t stream) {
  const tim_status st = tim::validate_logits(hidden, w_vocab, T, d, V, temperature, order, logits);
  if (st != TIM_OK || T == 0) return st;
  const bool splitk4 = order == TIM_ORDER_SPLITK4;
  tim::LmHeadArgs a;
  a.hidden = hidden;
  a.w = w_vocab;
  a.tokens = nullptr;
  a.rows = T;
  a.d = d;
  a.V = V;
  a.inv_tau = inv_temperature(temperature);
  a.part = nullptr;
  a.logits = logits;
  return hip_status(tim::launch_partials(a, 128, splitk4, stream));
}

size_t tim_logprobs_backward_workspace_size(int64_t T, int32_t d, int32_t V, int64_t micro_batch) {
  if (T <= 0 || tim::check_shape(T, d, V, TIM_ORDER_INVARIANT) != TIM_OK) return 0;
  if (!tim::valid_backward_micro_batch(micro_batch)) return 0;
  const tim::BackwardLayout l = tim::backward_layout(T, d, V, micro_batch);
  return l.step > tim::kMaxBackwardStep ? 0 : l.total;
}

tim_status tim_logit_grads(const void* hidden, const void* w_vocab, const int32_t* tokens, int64_t T, int32_t d,
                           int32_t V, float temperature, const float* lse, const float* entropy,
                           const float* grad_logp, const float* grad_entropy, void* dlogits, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  const tim_status st = tim::validate_logit_grads(hidden, w_vocab, tokens, T, d, V, temperature, lse, entropy,
                                                  grad_logp, grad_entropy, dlogits, workspace, workspace_bytes);
  if (st != TIM_OK || T == 0) return st;
  tim_status r = hip_status(tim::launch_grad_coef(lse, entropy, grad_logp, grad_entropy, tokens, T, V, temperature,
                                                  workspace, stream));
  if (r != TIM_OK) return r;
  tim::DlogitsArgs a;
  a.hidden = hidden;
  a.w = w_vocab;
  a.tokens = tokens;
  a.coef = workspace;
  a.rows = T;
  a.d = d;
  a.V = V;
  a.inv_tau = inv_temperature(temperature);
  a.dacc = dlogits;
  a.ld = (int64_t)tim::n_tiles_of(V) * TIM_VOCAB_TILE;
  a.packed = 0;
  a.dacct = nullptr;
  a.t_pad = 0;
  return hip_status(tim::launch_dlogits(a, stream));
}

tim_status tim_logprobs_backward(const void* hidden, const void* w_vocab, const int32_t* tokens, int64_t T,
                                 int32_t d, int32_t V, float temperature, const float* lse, const float* entropy,
                                 const float* grad_logp, const float* grad_entropy, int64_t micro_batch,
                                 float* grad_hidden, float* grad_w, int32_t accumulate_grad_w, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  tim_status st = tim::validate_backward(hidden, w_vocab, tokens, T, d, V, temperature, lse, entropy, grad_logp,
                                         grad_entropy, micro_batch, grad_hidden, grad_w, accumulate_grad_w,
                                         workspace, workspace_bytes);
  if (st != TIM_OK) return st;
  if (!grad_hidden && !grad_w) return TIM_OK;
  if (T == 0) {  // no tokens: dW is zero unless it accumulates
    if (grad_w && !accumulate_grad_w) return hip_status(tim::launch_fill_zero(grad_w, (int64_t)V * d, stream));
    return TIM_OK;
  }
  const tim::BackwardLayout l = tim::backward_layout(T, d, V, micro_batch);
  unsigned char* ws = (unsigned char*)workspace;
  void* coef = ws + l.coef;
  void* wt = ws + l.wt;
  void* dacc = ws + l.dacc;
  void* dacct = ws + l.dacct;
  void* ht = ws + l.ht;
  const float inv_tau = inv_temperature(temperature);
  const __bf16* h = (const __bf16*)hidden;

  if (grad_hidden) {  // W^T [d_pad, V_pad] packed, zeros past V and d
    st = hip_status(tim::launch_transpose(w_vocab, false, V, d, d, wt, l.v_pad, l.d_pad, 64, stream));
    if (st != TIM_OK) return st;
  }
  for (int64_t t0 = 0; t0 < T; t0 += l.step) {
    const int64_t rows = (T - t0) < l.step ? (T - t0) : l.step;
    const int64_t t_pad = tim::round_up(rows, 128);
    st = hip_status(tim::launch_grad_coef(lse + t0, entropy ? entropy + t0 : nullptr, grad_logp + t0,
                                          grad_entropy ? grad_entropy + t0 : nullptr, tokens + t0, rows, V,
                                          temperature, coef, stream));
    if (st != TIM_OK) return st;
    // dlogits^T [V_pad, t_pad] and h^T [d_pad, t_pad] packed, zeros past the rows; in 32-deep stage blocks for
    // the deep pass (its five buffers hide the HBM latency of this short-K product) when the pass has at least
    // 8 of them, else in 64-deep ones. On the deep pass the logit-gradient epilogue writes dlogits^T itself.
    const bool deep = t_pad >= 256;
    const int ks = deep ? 32 : 64;
    tim::DlogitsArgs a;
    a.hidden = h + t0 * d;
    a.w = w_vocab;
    a.tokens = tokens + t0;
    a.coef = coef;
    a.rows = rows;
    a.d = d;
    a.V = V;
    a.inv_tau = inv_tau;
    a.dacc = (grad_hidden || !deep) ? dacc : nullptr;
    a.ld = l.v_pad;
    a.packed = 1;  // [step_pad, V_pad] packed: the products' operand
    a.dacct = (grad_w && deep) ? dacct : nullptr;
    a.t_pad = t_pad;
    st = hip_status(tim::launch_dlogits(a, stream));
    if (st != TIM_OK) return st;
    if (grad_hidden) {  // dh = dlogits . W over the padded vocabulary
      tim::GemmArgs g;
      g.a = wt;
      g.b = dacc;
      g.b_rows = rows;
      g.a_rows = d;
      g.K = (int32_t)l.v_pad;
      g.out = grad_hidden + t0 * d;
      g.ldo = d;
      g.accumulate = 0;
      g.deep = 0;
      st = hip_status(tim::launch_gemm(g, stream));
      if (st != TIM_OK) return st;
    }
    if (grad_w) {  // dW (+)= dlogits^T . h over this micro-batch's tokens
      if (!deep) {
        st = hip_status(tim::launch_transpose(dacc, true, rows, l.v_pad, l.v_pad, dacct, t_pad, l.v_pad, ks, stream));
        if (st != TIM_OK) return st;
      }
      st = hip_status(tim::launch_transpose(h + t0 * d, false, rows, d, d, ht, t_pad, l.d_pad, ks, stream));
      if (st != TIM_OK) return st;
      tim::GemmArgs g;
      g.a = ht;
      g.b = dacct;
      g.b_rows = V;
      g.a_rows = d;
      g.K = (int32_t)t_pad;
      g.out = grad_w;
      g.ldo = d;
      g.accumulate = (accumulate_grad_w || t0 > 0) ? 1 : 0;
      g.deep = deep ? 1 : 0;
      st = hip_status(tim::launch_gemm(g, stream));
      if (st != TIM_OK) return st;
    }
  }
  return TIM_OK;
}

tim_status tim_rmsnorm(const void* x, const void* gamma, int64_t T, int32_t d, float eps, void* h, float* rstd,
                       hipStream_t stream) {
  const tim_status st = tim::validate_rmsnorm(x, gamma, T, d, eps, h);
  if (st != TIM_OK || T == 0) return st;
  return hip_status(tim::launch_rmsnorm(x, gamma, T, d, eps, h, rstd, stream));
}

size_t tim_rmsnorm_backward_workspace_size(int64_t T, int32_t d) {
  if (T <= 0 || tim::check_norm_shape(T, d) != TIM_OK) return 0;
  return tim::rmsnorm_backward_workspace(T, d);
}

tim_status tim_rmsnorm_backward(const void* x, const void* gamma, const float* rstd, const float* grad_h, int64_t T,
                                int32_t d, float* grad_x, float* grad_gamma, int32_t accumulate_grad_gamma,
                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
  const tim_status st = tim::validate_rmsnorm_backward(x, gamma, rstd, grad_h, T, d, grad_x, grad_gamma,
                                                       accumulate_grad_gamma, workspace, workspace_bytes);
  if (st != TIM_OK || (!grad_x && !grad_gamma)) return st;
  if (T == 0 && (!grad_gamma || accumulate_grad_gamma)) return TIM_OK;
  return hip_status(tim::launch_rmsnorm_backward(x, gamma, rstd, grad_h, T, d, grad_x, grad_gamma,
                                                 accumulate_grad_gamma, (float*)workspace, stream));
}

tim_status tim_ppo_loss(const float* logp, const float* logp_old, const float* advantages, const float* weight,
                        int64_t T, const int64_t* cu_seqlens, int64_t n_seq, float eps_low, float eps_high,
                        double* seq_loss, double* batch_loss, float* token_loss, float* grad_logp,
                        float* contribution, uint8_t* clipped, hipStream_t stream) {
  const tim_status st = tim::validate_ppo(logp, logp_old, advantages, T, cu_seqlens, n_seq, eps_low, eps_high,
                                          seq_loss, batch_loss);
  if (st != TIM_OK || n_seq == 0) return st;
  if (!seq_loss && !batch_loss && !token_loss && !grad_logp && !contribution && !clipped) return TIM_OK;
  tim::PpoParams p;
  p.lo_threshold = std::log1p(-(double)eps_low);
  p.hi_threshold = std::log1p((double)eps_high);
  p.clip_lo = 1.0 - (double)eps_low;
  p.clip_hi = 1.0 + (double)eps_high;
  p.inv_n = 1.0 / (double)n_seq;
  return hip_status(tim::launch_ppo_loss(logp, logp_old, advantages, weight, T, cu_seqlens, n_seq, p, seq_loss,
                                         batch_loss, token_loss, grad_logp, contribution, clipped, stream));
}

const char* tim_status_string(tim_status s) {
  switch (s) {
    case TIM_OK: return "TIM_OK";
    case TIM_ERR_NULL: return "TIM_ERR_NULL: a required pointer is NULL";
    case TIM_ERR_SHAPE: return "TIM_ERR_SHAPE: T, d or V out of range";
    case TIM_ERR_VALUE: return "TIM_ERR_VALUE: bad temperature, C, mode, order, micro_batch or alignment";
    case TIM_ERR_WORKSPACE: return "TIM_ERR_WORKSPACE: workspace missing, misaligned or too small (or, without one, beyond the device scratch array)";
    case TIM_ERR_HIP: return "TIM_ERR_HIP: a HIP call or kernel launch failed";
  }
  return "unknown tim_status";
}

}  // extern "C"
