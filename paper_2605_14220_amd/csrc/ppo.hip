// Clipped PPO/GRPO token loss over a packed token stream (Section 4.1,
// Eqs. 2-5), weighted per token by the corrections of Section 4.2 (e.g. the
// truncated and rejected weights of tim_mismatch_seq), summed over each
// response and averaged over the responses, with its gradient with respect to
// the current log-probs and the zero-centred contribution C(r) = -(r - 1) A.
//
// One workgroup of 256 threads per response, as the sequence-level
// statistics: thread i takes the tokens i, i + 256, ... of the response in
// order, in fp64; the response's sum combines the 256 partial sums with a
// fixed tree. delta = logp - logp_old is exact in fp64, and the clip decision
// is taken on it exactly: with A > 0 the clipped term is the minimum iff
// r = e^delta > 1 + eps_high, i.e. delta > log1p(eps_high); with A < 0 iff
// delta < log1p(-eps_low); the thresholds are formed once in fp64 on the host.

#include <math.h>

#include "kernels.h"

namespace tim {
namespace {

constexpr int kPpoThreads = 256;

__device__ __forceinline__ double block_sum(double acc, double* wsum) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wsum[wave] = acc;
  __syncthreads();
  return (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
}

__global__ __launch_bounds__(kPpoThreads) void ppo_kernel(const float* __restrict__ lp, const float* __restrict__ lo,
                                                          const float* __restrict__ adv, const float* __restrict__ wt,
                                                          int64_t T, const int64_t* __restrict__ cu, PpoParams p,
                                                          double* seq_loss, float* token_loss, float* grad,
                                                          float* contrib, uint8_t* clipped) {
  const int64_t j = blockIdx.x;
  int64_t s0 = cu[j], s1 = cu[j + 1];
  s0 = s0 < 0 ? 0 : (s0 > T ? T : s0);
  s1 = s1 < s0 ? s0 : (s1 > T ? T : s1);
  double acc = 0.0;
  for (int64_t t = s0 + threadIdx.x; t < s1; t += kPpoThreads) {
    const double delta = (double)lp[t] - (double)lo[t];
    const double a = (double)adv[t];
    const double w = wt ? (double)wt[t] : 1.0;
    const double r = exp(delta);
    const bool clip = (a > 0.0 && delta > p.hi_threshold) || (a < 0.0 && delta < p.lo_threshold);
    const double L = clip ? -a * (a > 0.0 ? p.clip_hi : p.clip_lo) : -a * r;
    const double tl = w * L;
    if (token_loss) token_loss[t] = (float)tl;
    if (grad) grad[t] = clip ? 0.f : (float)(w * (-a * r) * p.inv_n);
    if (contrib) contrib[t] = (float)(-(r - 1.0) * a);
    if (clipped) clipped[t] = clip ? 1 : 0;
    acc += tl;
  }
  __shared__ double wsum[kPpoThreads / 64];
  const double S = block_sum(acc, wsum);
  if (threadIdx.x == 0 && seq_loss) seq_loss[j] = S;
}

// The batch loss: the response sums in a fixed order (thread i takes
// responses i, i + 256, ...), then the same tree, divided by n.
__global__ __launch_bounds__(kPpoThreads) void ppo_batch_kernel(const double* __restrict__ seq_loss, int64_t n,
                                                                double* batch_loss) {
  double acc = 0.0;
  for (int64_t j = threadIdx.x; j < n; j += kPpoThreads) acc += seq_loss[j];
  __shared__ double wsum[kPpoThreads / 64];
  const double S = block_sum(acc, wsum);
  if (threadIdx.x == 0) batch_loss[0] = S / (double)n;
}

}  // namespace

hipError_t launch_ppo_loss(const float* logp, const float* logp_old, const float* advantages, const float* weight,
                           int64_t T, const int64_t* cu_seqlens, int64_t n_seq, const PpoParams& p, double* seq_loss,
                           double* batch_loss, float* token_loss, float* grad, float* contrib, uint8_t* clipped,
                           hipStream_t s) {
  if (n_seq <= 0) return hipSuccess;
  if (n_seq > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ppo_kernel, dim3((unsigned)n_seq), dim3(kPpoThreads), 0, s, logp, logp_old, advantages, weight,
                     T, cu_seqlens, p, seq_loss, token_loss, grad, contrib, clipped);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !batch_loss) return e;
  hipLaunchKernelGGL(ppo_batch_kernel, dim3(1), dim3(kPpoThreads), 0, s, (const double*)seq_loss, n_seq, batch_loss);
  return hipGetLastError();
}

}  // namespace tim
