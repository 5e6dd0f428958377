// Final RMS normalisation in front of the LM head, batch-invariant, and its
// backward (Section 3.1 lists RMSNorm among the batch-invariant kernels; the
// norm is Zhang and Sennrich's root-mean-square layer normalisation).
//
// Forward, one wavefront per row, d a multiple of 8:
//   r   = 1 / sqrt(mean_k x_k^2 + eps)                      fp32
//   h_k = bf16(g_k * bf16(x_k * r))  (bf16(x_k * r) without a weight)
// the arithmetic of the model implementation the engine follows: the row is
// widened to fp32, scaled, rounded to bf16, then multiplied by the bf16 weight
// and rounded again. Lane l takes the 8-element chunks l, l + 64, l + 128, ...
// and sums their squares in that order (one fma chain); the 64 lane sums
// combine in a fixed butterfly, so r depends only on the row and d.
//
// Backward, with G = dL/dh (fp32) and the casts passed straight through:
//   dx_k = r g_k G_k - (r^3 s / d) x_k,   s = sum_j G_j g_j x_j   (one wavefront per row)
//   dg_k = sum_t G_tk x_tk r_t   as fixed-order column sums over blocks of
//          rows, then over the blocks in order (no atomics). Blocks are 256
//          rows whose rows go in order, except in calls of at least 65536 rows
//          of width 2048 or 4096, whose grad_x pass also forms the block sums:
//          there a block is 4 rpw rows, rpw = max(64, ceil(T / (4 R))) with
//          R = 1024 at d = 2048 and 512 at d = 4096 (the blocks a 256-CU chip
//          holds at once), each quarter of rpw rows goes in order and the
//          quarters combine as (q0 + q1) + (q2 + q3). The order so depends on
//          (T, d) only.
// Each is one HBM pass over the rows; the norm costs ~0.2% of the LM head it
// feeds, so it runs as its own launch ahead of the head instead of inside the
// head's MFMA loop, which would repeat it once per vocabulary tile and add
// VALU work to the loop that bounds the head.

#include <hip/hip_runtime.h>
#include <algorithm>

#include "kernels.h"

namespace tim {
namespace {

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ uint16_t to_bf16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 1; off < 64; off *= 2) v = v + __shfl_xor(v, off);
  return v;
}

// The row's squares summed into `acc` in the fixed lane order (chunk by
// chunk, the 8 elements of a chunk in order).
__device__ __forceinline__ float sum_squares(uint4 v, float acc) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float a = bf16_lo(w[i]), b = bf16_hi(w[i]);
    acc = __builtin_fmaf(a, a, acc);
    acc = __builtin_fmaf(b, b, acc);
  }
  return acc;
}

// NCL > 0: d = 512 NCL, and a lane keeps its NCL chunks of the row in
// registers between the two passes (all loads issued up front); NCL = 0: any
// d, the row read again for the second pass. The arithmetic is the same.
template <int NCL>
__global__ __launch_bounds__(256) void rmsnorm_fwd(const uint4* __restrict__ x, const uint4* __restrict__ gamma,
                                                   int64_t T, int d, float eps, uint4* __restrict__ h,
                                                   float* __restrict__ rstd) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const int nc = NCL > 0 ? NCL * 64 : d / 8;
  const uint4* xr = x + t * nc;
  uint4 xv[NCL > 0 ? NCL : 1];
  float acc = 0.f;
  if constexpr (NCL > 0) {
#pragma unroll
    for (int i = 0; i < NCL; ++i) xv[i] = xr[lane + 64 * i];
#pragma unroll
    for (int i = 0; i < NCL; ++i) acc = sum_squares(xv[i], acc);
  } else {
    for (int c = lane; c < nc; c += 64) acc = sum_squares(xr[c], acc);
  }
  const float var = wave_sum(acc) / (float)d;
  const float r = 1.0f / __builtin_sqrtf(var + eps);
  if (rstd && lane == 0) rstd[t] = r;
  uint4* hr = h + t * nc;
  // h = bf16(g * bf16(x r)) for chunk c of the row
  auto out_chunk = [&](int c, uint4 v) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t g[4] = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
    if (gamma) {
      const uint4 gv = gamma[c];
      g[0] = gv.x, g[1] = gv.y, g[2] = gv.z, g[3] = gv.w;
    }
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float lo = bf16_lo((uint32_t)to_bf16(bf16_lo(w[i]) * r));
      float hi = bf16_lo((uint32_t)to_bf16(bf16_hi(w[i]) * r));
      if (gamma) {
        lo = lo * bf16_lo(g[i]);
        hi = hi * bf16_hi(g[i]);
      }
      o[i] = (uint32_t)to_bf16(lo) | ((uint32_t)to_bf16(hi) << 16);
    }
    hr[c] = uint4{o[0], o[1], o[2], o[3]};
  };
  if constexpr (NCL > 0) {
#pragma unroll
    for (int i = 0; i < NCL; ++i) out_chunk(lane + 64 * i, xv[i]);
  } else {
    for (int c = lane; c < nc; c += 64) out_chunk(c, xr[c]);
  }
}

// gamma's chunk c as 4 packed pairs (1.0 without a weight)
__device__ __forceinline__ uint4 gamma_chunk(const uint4* __restrict__ gamma, int c) {
  return gamma ? gamma[c] : uint4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
}

// s += G g x over one chunk, in element order
__device__ __forceinline__ float dot_chunk(uint4 v, float4 g0, float4 g1, uint4 gv, float acc) {
  const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  const uint32_t gm[4] = {gv.x, gv.y, gv.z, gv.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc = __builtin_fmaf(gg[2 * i] * bf16_lo(gm[i]), bf16_lo(w[i]), acc);
    acc = __builtin_fmaf(gg[2 * i + 1] * bf16_hi(gm[i]), bf16_hi(w[i]), acc);
  }
  return acc;
}

// dx = r g G - c2 x over chunk c of a row
__device__ __forceinline__ void out_chunk_dx(float4* __restrict__ out, int c, uint4 v, float4 g0, float4 g1, uint4 gv,
                                             float r, float c2) {
  const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  const uint32_t gm[4] = {gv.x, gv.y, gv.z, gv.w};
  float o[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = r * (bf16_lo(gm[i]) * gg[2 * i]) - c2 * bf16_lo(w[i]);
    o[2 * i + 1] = r * (bf16_hi(gm[i]) * gg[2 * i + 1]) - c2 * bf16_hi(w[i]);
  }
  out[2 * c] = float4{o[0], o[1], o[2], o[3]};
  out[2 * c + 1] = float4{o[4], o[5], o[6], o[7]};
}

// Same two-mode structure as the forward (NCL > 0: the row's x, G and gamma
// chunks kept in registers between the passes).
template <int NCL>
__global__ __launch_bounds__(256) void rmsnorm_bwd_x(const uint4* __restrict__ x, const uint4* __restrict__ gamma,
                                                     const float* __restrict__ rstd, const float4* __restrict__ G,
                                                     int64_t T, int d, float4* __restrict__ dx) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const int nc = NCL > 0 ? NCL * 64 : d / 8;
  const uint4* xr = x + t * nc;
  const float4* gr = G + t * (int64_t)(d / 4);
  uint4 xv[NCL > 0 ? NCL : 1], gmv[NCL > 0 ? NCL : 1];
  float4 g0v[NCL > 0 ? NCL : 1], g1v[NCL > 0 ? NCL : 1];
  float acc = 0.f;
  if constexpr (NCL > 0) {
#pragma unroll
    for (int i = 0; i < NCL; ++i) {
      const int c = lane + 64 * i;
      xv[i] = xr[c];
      g0v[i] = gr[2 * c];
      g1v[i] = gr[2 * c + 1];
      gmv[i] = gamma_chunk(gamma, c);
    }
#pragma unroll
    for (int i = 0; i < NCL; ++i) acc = dot_chunk(xv[i], g0v[i], g1v[i], gmv[i], acc);
  } else {
    for (int c = lane; c < nc; c += 64) acc = dot_chunk(xr[c], gr[2 * c], gr[2 * c + 1], gamma_chunk(gamma, c), acc);
  }
  const float s = wave_sum(acc);
  const float r = rstd[t];
  const float c2 = ((r * r) * r) * s / (float)d;
  float4* out = dx + t * (int64_t)(d / 4);
  if constexpr (NCL > 0) {
#pragma unroll
    for (int i = 0; i < NCL; ++i) out_chunk_dx(out, lane + 64 * i, xv[i], g0v[i], g1v[i], gmv[i], r, c2);
  } else {
    for (int c = lane; c < nc; c += 64)
      out_chunk_dx(out, c, xr[c], gr[2 * c], gr[2 * c + 1], gamma_chunk(gamma, c), r, c2);
  }
}

// Widths whose rows stay in registers: grad_x and the block's grad_gamma
// column sums in one pass over x and G. One workgroup per block of 4 rpw rows;
// wave w takes the block's rows rpw w .. rpw w + rpw - 1 in order, each as
// rmsnorm_bwd_x does (the same dx), and adds (G x) r of its columns to its own
// column sums in LDS in that row order; the four waves' sums then combine as
// (q0 + q1) + (q2 + q3) into the block's partial. The sums over the blocks in
// order follow in rmsnorm_dgamma_final.
template <int NCL, bool WANT_X>
__global__ __launch_bounds__(256) void rmsnorm_bwd_fused(const uint4* __restrict__ x, const uint4* __restrict__ gamma,
                                                         const float* __restrict__ rstd, const float4* __restrict__ G,
                                                         int64_t T, int rpw, float4* __restrict__ dx,
                                                         float* __restrict__ part) {
  constexpr int d = NCL * 512, nc = NCL * 64;
  __shared__ float4 red[4][nc][2];  // each wave's column sums, 8 per chunk
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t b0 = (int64_t)blockIdx.x * 4 * rpw;
#pragma unroll
  for (int i = 0; i < NCL; ++i) red[wave][lane + 64 * i][0] = red[wave][lane + 64 * i][1] = float4{0.f, 0.f, 0.f, 0.f};
  const int64_t r_end = (T - b0) < 4 * rpw ? T - b0 : 4 * rpw;
#pragma unroll 1
  for (int j = 0; j < rpw; ++j) {
    const int64_t rl = (int64_t)rpw * wave + j;
    if (rl >= r_end) break;  // uniform across the wave
    const int64_t t = b0 + rl;
    const uint4* xr = x + t * nc;
    const float4* gr = G + t * (int64_t)(d / 4);
    uint4 xv[NCL], gmv[NCL];
    float4 g0v[NCL], g1v[NCL];
#pragma unroll
    for (int i = 0; i < NCL; ++i) {
      const int c = lane + 64 * i;
      xv[i] = xr[c];
      g0v[i] = gr[2 * c];
      g1v[i] = gr[2 * c + 1];
      gmv[i] = gamma_chunk(gamma, c);
    }
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < NCL; ++i) acc = dot_chunk(xv[i], g0v[i], g1v[i], gmv[i], acc);
    const float sdot = wave_sum(acc);
    const float r = rstd[t];
    const float c2 = ((r * r) * r) * sdot / (float)d;
    float4* out = WANT_X ? dx + t * (int64_t)(d / 4) : nullptr;
    // per chunk: its dx (WANT_X), then its (G x) r added to the column sums
#pragma unroll
    for (int i = 0; i < NCL; ++i) {
      const int c = lane + 64 * i;
      if constexpr (WANT_X) out_chunk_dx(out, c, xv[i], g0v[i], g1v[i], gmv[i], r, c2);
      const uint32_t w[4] = {xv[i].x, xv[i].y, xv[i].z, xv[i].w};
      const float gg[8] = {g0v[i].x, g0v[i].y, g0v[i].z, g0v[i].w, g1v[i].x, g1v[i].y, g1v[i].z, g1v[i].w};
      float e[8];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        e[2 * k] = (gg[2 * k] * bf16_lo(w[k])) * r;
        e[2 * k + 1] = (gg[2 * k + 1] * bf16_hi(w[k])) * r;
      }
      const float4 p0 = red[wave][c][0], p1 = red[wave][c][1];
      red[wave][c][0] = float4{p0.x + e[0], p0.y + e[1], p0.z + e[2], p0.w + e[3]};
      red[wave][c][1] = float4{p1.x + e[4], p1.y + e[5], p1.z + e[6], p1.w + e[7]};
    }
  }
  __syncthreads();
  // (q0 + q1) + (q2 + q3), the block's 8 NCL columns per lane spread over the four waves
  auto add4 = [](float4 a, float4 b) { return float4{a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w}; };
  float4* po = (float4*)(part + (int64_t)blockIdx.x * d);
  for (int c = threadIdx.x; c < nc; c += 256) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
      po[2 * c + hh] = add4(add4(red[0][c][hh], red[1][c][hh]), add4(red[2][c][hh], red[3][c][hh]));
  }
}

// Column sums of G x r over one block of up to 256 rows, rows in order.
__global__ __launch_bounds__(256) void rmsnorm_dgamma_part(const uint16_t* __restrict__ x,
                                                           const float* __restrict__ rstd,
                                                           const float* __restrict__ G, int64_t T, int d,
                                                           float* __restrict__ part) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k >= d) return;
  const int64_t t0 = (int64_t)blockIdx.y * 256;
  const int64_t t1 = (T - t0) < 256 ? T : t0 + 256;
  float acc = 0.f;
  int64_t t = t0;
  // 8 rows' loads issued ahead of their terms (the adds stay in row order)
  for (; t + 8 <= t1; t += 8) {
    float xv[8], gv[8], rv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      xv[i] = __uint_as_float((uint32_t)x[(t + i) * d + k] << 16);
      gv[i] = G[(t + i) * d + k];
      rv[i] = rstd[t + i];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) acc = acc + (gv[i] * xv[i]) * rv[i];
  }
  for (; t < t1; ++t) {
    const float xv = __uint_as_float((uint32_t)x[t * d + k] << 16);
    acc = acc + (G[t * d + k] * xv) * rstd[t];
  }
  part[(int64_t)blockIdx.y * d + k] = acc;
}

// dg_k (+)= the blocks' sums in block order.
__global__ __launch_bounds__(256) void rmsnorm_dgamma_final(const float* __restrict__ part, int n_blocks, int d,
                                                            int accumulate, float* __restrict__ dg) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k >= d) return;
  float acc = accumulate ? dg[k] : 0.f;
  int b = 0;
  // 16 loads issued ahead of their adds (the adds stay in block order)
  for (; b + 16 <= n_blocks; b += 16) {
    float v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = part[(int64_t)(b + i) * d + k];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc = acc + v[i];
  }
  for (; b < n_blocks; ++b) acc = acc + part[(int64_t)b * d + k];
  dg[k] = acc;
}

}  // namespace

hipError_t launch_rmsnorm(const void* x, const void* gamma, int64_t T, int d, float eps, void* h, float* rstd,
                          hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const int64_t nb = (T + 3) / 4;
  if (nb > 0x7fffffff) return hipErrorInvalidValue;
  const dim3 g((unsigned)nb), b(256);
  const uint4* xp = (const uint4*)x;
  const uint4* gp = (const uint4*)gamma;
  switch (d) {  // widths whose rows stay in registers
    case 2048: hipLaunchKernelGGL(rmsnorm_fwd<4>, g, b, 0, s, xp, gp, T, d, eps, (uint4*)h, rstd); break;
    case 4096: hipLaunchKernelGGL(rmsnorm_fwd<8>, g, b, 0, s, xp, gp, T, d, eps, (uint4*)h, rstd); break;
    case 5120: hipLaunchKernelGGL(rmsnorm_fwd<10>, g, b, 0, s, xp, gp, T, d, eps, (uint4*)h, rstd); break;
    case 8192: hipLaunchKernelGGL(rmsnorm_fwd<16>, g, b, 0, s, xp, gp, T, d, eps, (uint4*)h, rstd); break;
    default: hipLaunchKernelGGL(rmsnorm_fwd<0>, g, b, 0, s, xp, gp, T, d, eps, (uint4*)h, rstd); break;
  }
  return hipGetLastError();
}

// Rows from which the norm backward takes grad_gamma in the grad_x pass.
constexpr int64_t kFusedNormRows = 65536;

template <int NCL>
static hipError_t launch_fused(const void* x, const void* gamma, const float* rstd, const float* grad_h, int64_t T,
                               int rpw, float* grad_x, float* part, hipStream_t s) {
  const dim3 g((unsigned)((T + 4 * rpw - 1) / (4 * rpw))), b(256);
  if (grad_x)
    hipLaunchKernelGGL((rmsnorm_bwd_fused<NCL, true>), g, b, 0, s, (const uint4*)x, (const uint4*)gamma, rstd,
                       (const float4*)grad_h, T, rpw, (float4*)grad_x, part);
  else
    hipLaunchKernelGGL((rmsnorm_bwd_fused<NCL, false>), g, b, 0, s, (const uint4*)x, (const uint4*)gamma, rstd,
                       (const float4*)grad_h, T, rpw, (float4*)nullptr, part);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_backward(const void* x, const void* gamma, const float* rstd, const float* grad_h,
                                   int64_t T, int d, float* grad_x, float* grad_gamma, int accumulate, float* part,
                                   hipStream_t s) {
  // Large calls at the widths whose rows stay in registers take grad_gamma's
  // block sums in the grad_x pass (with or without grad_x): one workgroup per
  // block of rows walks its rows in order, which pays once there are enough
  // blocks to fill the chip. The choice depends on (T, d) only.
  const bool fused = grad_gamma && (d == 2048 || d == 4096) && T >= kFusedNormRows;
  // Rows per wave: 64, or more where that many blocks would not all be
  // resident at once on a 256-CU MI355X (two workgroups per CU at d = 4096,
  // four at 2048), which would leave a second round of a few blocks walking
  // their rows alone. A constant, so the order depends on (T, d) only.
  const int64_t resident = d == 2048 ? 1024 : 512;
  const int rpw = (int)std::max<int64_t>(64, (T + 4 * resident - 1) / (4 * resident));
  if (fused && T > 0) {
    if ((T + 255) / 256 > 65535) return hipErrorInvalidValue;
    const hipError_t e = d == 2048 ? launch_fused<4>(x, gamma, rstd, grad_h, T, rpw, grad_x, part, s)
                                   : launch_fused<8>(x, gamma, rstd, grad_h, T, rpw, grad_x, part, s);
    if (e != hipSuccess) return e;
  }
  if (T > 0 && grad_x && !fused) {
    const int64_t nb = (T + 3) / 4;
    if (nb > 0x7fffffff) return hipErrorInvalidValue;
    const dim3 g((unsigned)nb), b(256);
    const uint4* xp = (const uint4*)x;
    const uint4* gp = (const uint4*)gamma;
    const float4* Gp = (const float4*)grad_h;
    switch (d) {  // widths whose rows stay in registers
      case 2048: hipLaunchKernelGGL(rmsnorm_bwd_x<4>, g, b, 0, s, xp, gp, rstd, Gp, T, d, (float4*)grad_x); break;
      case 4096: hipLaunchKernelGGL(rmsnorm_bwd_x<8>, g, b, 0, s, xp, gp, rstd, Gp, T, d, (float4*)grad_x); break;
      case 5120: hipLaunchKernelGGL(rmsnorm_bwd_x<10>, g, b, 0, s, xp, gp, rstd, Gp, T, d, (float4*)grad_x); break;
      default: hipLaunchKernelGGL(rmsnorm_bwd_x<0>, g, b, 0, s, xp, gp, rstd, Gp, T, d, (float4*)grad_x); break;
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (grad_gamma) {
    const int64_t n_blocks = fused ? (T + 4 * rpw - 1) / (4 * rpw) : (T + 255) / 256;
    if (n_blocks > 65535) return hipErrorInvalidValue;
    const unsigned gx = (unsigned)((d + 255) / 256);
    if (n_blocks > 0 && !fused) {
      hipLaunchKernelGGL(rmsnorm_dgamma_part, dim3(gx, (unsigned)n_blocks), dim3(256), 0, s, (const uint16_t*)x, rstd,
                         grad_h, T, d, part);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(rmsnorm_dgamma_final, dim3(gx), dim3(256), 0, s, part, (int)n_blocks, d, accumulate,
                       grad_gamma);
    return hipGetLastError();
  }
  return hipSuccess;
}

}  // namespace tim
