// Token-level mismatch statistics (Section 2 Eq. 1; Section 4.1 K3; Section 4.2
// r_corr and the truncation of Eq. 6). Elementwise and HBM-bound: 8 bytes in,
// up to 12 bytes out per token, 4 tokens per thread with 16-byte accesses.
// Each statistic is formed in fp64 from the exact difference of the two fp32
// inputs and rounded once to fp32, so K3 keeps its relative accuracy however
// small the difference (an fp32 expm1(delta) - delta cancels to nothing near
// delta ~ 1e-7, the typical size of an engine-to-engine discrepancy).

#include "kernels.h"

namespace tim {
namespace {

struct Stats {
  float delta, k3, w;
};

__device__ __forceinline__ Stats stats_of(float a, float b, float C) {
  const double d = (double)a - (double)b;  // exact: two fp32 values differ by an fp64-representable amount
  Stats r;
  r.delta = (float)d;                      // log pi_a - log pi_b, rounded once
  r.k3 = (float)k3_of_delta(d);            // (ratio - 1) - log ratio, ratio = e^delta
  r.w = tis_weight(d, C);                  // ratio truncated above at C
  return r;
}

__global__ __launch_bounds__(256) void mismatch_kernel(const float* __restrict__ a,
                                                       const float* __restrict__ b, int64_t n,
                                                       float C, float* __restrict__ lr,
                                                       float* __restrict__ k3,
                                                       float* __restrict__ w) {
  const int64_t n4 = n >> 2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const bool vec = ((((uintptr_t)a | (uintptr_t)b | (uintptr_t)lr | (uintptr_t)k3 | (uintptr_t)w) & 15) == 0);
  int64_t tail0 = 0;
  if (vec) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
      const float4 av = ((const float4*)a)[i];
      const float4 bv = ((const float4*)b)[i];
      const Stats s0 = stats_of(av.x, bv.x, C), s1 = stats_of(av.y, bv.y, C);
      const Stats s2 = stats_of(av.z, bv.z, C), s3 = stats_of(av.w, bv.w, C);
      if (lr) ((float4*)lr)[i] = make_float4(s0.delta, s1.delta, s2.delta, s3.delta);
      if (k3) ((float4*)k3)[i] = make_float4(s0.k3, s1.k3, s2.k3, s3.k3);
      if (w) ((float4*)w)[i] = make_float4(s0.w, s1.w, s2.w, s3.w);
    }
    tail0 = n4 << 2;
  }
  for (int64_t i = tail0 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const Stats s = stats_of(a[i], b[i], C);
    if (lr) lr[i] = s.delta;
    if (k3) k3[i] = s.k3;
    if (w) w[i] = s.w;
  }
}

}  // namespace

hipError_t launch_mismatch(const float* a, const float* b, int64_t n, float C, float* log_ratio,
                           float* k3, float* w, hipStream_t s) {
  int64_t blocks = (n / 4 + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(mismatch_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a, b, n, C,
                     log_ratio, k3, w);
  return hipGetLastError();
}

}  // namespace tim
