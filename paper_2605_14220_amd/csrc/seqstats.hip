// Sequence-level mismatch statistics over a packed token stream (Section 4.2:
// the sequence-level rejection 1[S_seq <= tau_seq] with S_seq the sum of a
// Section 4.1 KL estimator (K1 or K3) of the correction ratio over a response,
// combined with the token-level truncation min(r_corr, tau_tok) as in the
// appendix's tis-srs-k1/k3-corr objectives).
//
// One workgroup of 256 threads per response. Thread i sums, in fp64 and in
// ascending order, the tokens i, i + 256, ... of the response (counted from the
// response's first token); the 256 sums then combine with a fixed tree: the
// xor-shuffle tree of each wave, then the four waves as (w0 + w1) + (w2 + w3).
// The order depends only on the response's length, so a response's score is
// bitwise the same wherever it sits in the stream. The same workgroup then
// writes the response's token weights.

#include "kernels.h"

namespace tim {
namespace {

constexpr int kSeqThreads = 256;

__global__ __launch_bounds__(kSeqThreads) void seqstats_kernel(const float* __restrict__ a,
                                                               const float* __restrict__ b, int64_t T,
                                                               const int64_t* __restrict__ cu, int k3,
                                                               float C, double tau_seq, double* score,
                                                               uint8_t* keep, float* weight) {
  const int64_t j = blockIdx.x;
  // the response's tokens, clamped into [0, T]; reversed bounds give an empty response
  int64_t s0 = cu[j], s1 = cu[j + 1];
  s0 = s0 < 0 ? 0 : (s0 > T ? T : s0);
  s1 = s1 < s0 ? s0 : (s1 > T ? T : s1);
  double acc = 0.0;
  for (int64_t t = s0 + threadIdx.x; t < s1; t += kSeqThreads) {
    const double delta = (double)a[t] - (double)b[t];  // exact in fp64
    acc += k3 ? k3_of_delta(delta) : -delta;           // K3 = (r - 1) - log r, K1 = -log r; r = e^delta
  }
  // each xor step adds the same two values in every lane pair, so all lanes agree
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
  __shared__ double wsum[kSeqThreads / 64];
  __shared__ int keep_s;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wsum[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    const double S = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
    const int k = S <= tau_seq;  // a NaN score rejects
    if (score) score[j] = S;
    if (keep) keep[j] = (uint8_t)k;
    keep_s = k;
  }
  __syncthreads();
  if (weight) {
    const int k = keep_s;
    for (int64_t t = s0 + threadIdx.x; t < s1; t += kSeqThreads) {
      // tim_mismatch's correction ratio and truncation
      weight[t] = k ? tis_weight((double)a[t] - (double)b[t], C) : 0.f;
    }
  }
}

}  // namespace

hipError_t launch_mismatch_seq(const float* a, const float* b, int64_t T, const int64_t* cu_seqlens,
                               int64_t n_seq, bool k3, float C, double tau_seq, double* score,
                               uint8_t* keep, float* weight, hipStream_t s) {
  if (n_seq <= 0) return hipSuccess;
  if (n_seq > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(seqstats_kernel, dim3((unsigned)n_seq), dim3(kSeqThreads), 0, s, a, b, T, cu_seqlens,
                     k3 ? 1 : 0, C, tau_seq, score, keep, weight);
  return hipGetLastError();
}

}  // namespace tim
