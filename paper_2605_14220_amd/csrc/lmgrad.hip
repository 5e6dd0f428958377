// Backward of the fused LM-head log-probability and entropy for gfx950.
//
// For a scalar loss L with upstream gradients g_t = dL/dlogp_t and
// e_t = dL/dH_t, and the forward's z = acc / tau, q_v = z_v - lse,
// p_v = e^{q_v}, the chain rule through the softmax gives per row
//   dacc_v = ( g_t ([v = a_t] - p_v) - e_t p_v (q_v + H_t) ) / tau
//          = gamma [v = a_t] - p_v (alpha + beta q_v)
// with gamma = g_t / tau, alpha = (g_t + e_t H_t) / tau, beta = e_t / tau, and
//   dh_t = sum_v dacc_{t,v} w_v,      dW_v = sum_t dacc_{t,v} h_t.
// These are the gradients the trainer takes of the same per-token log-probs
// whose forward values the rollout must match (Section 2, Eq. 1; the PPO and
// GRPO objectives of Section 4 differentiate log pi_train through the ratio).
//
// Three contractions, all on the tile pass (one fp32 chain per element, K
// ascending, no atomics):
//   1. lmhead_dlogits: z recomputed with the forward's own main loop (K = d),
//      so p is formed from exactly the logits whose lse the forward returned;
//      the epilogue writes dacc as bf16 [rows, V_pad] (the rounding a bf16
//      trainer applies to logit gradients before the weight products), in the
//      tile pass's packed layout when it feeds the products.
//   2. dh = dacc . W: A = W^T [d, V_pad], B = dacc, K = V_pad. A row's chain
//      runs over the whole padded vocabulary in one order whatever the batch,
//      so dh is batch-invariant like the forward.
//   3. dW = dacc^T . h: A = h^T [d, T_pad], B = dacc^T [V_pad, T_pad],
//      K = T_pad. The chain over tokens starts from the value already in dW
//      after the first micro-batch (or with accumulation), so micro-batches of
//      multiples of 128 tokens continue one chain: dW is bitwise the same for
//      every such micro-batch size.
// h^T and W^T are written by an LDS-tiled transpose; dacc^T by the
// logit-gradient epilogue itself when the weight pass is the deep one (each
// lane quad transposes its 4 x 4 blocks in registers), else by the transpose.
// Both products read packed operands (256-row tiles stored stage by stage as
// their LDS image, see tilepass.h), which their producers write at no extra
// cost: the transposes and the logit-gradient epilogue. The padding along K is
// zeros, which add exactly nothing; padding rows only reach outputs that are
// never written.

#include "tilepass.h"

namespace tim {
namespace {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// Two floats rounded to bf16 (round to nearest even), lo in the low half.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

// Logit gradients. A = W [V, d], B = hidden states, K = d: the forward's pass.
// For row block bj a lane holds row (l % 16) and, in register r of W block bi,
// the vocabulary entry v0 + wv * 128 + bi * 16 + 4 (l / 16) + r; the four
// registers go out as one 8-byte store to their row-major place or, packed,
// two lanes' halves of a 16-byte chunk (eight consecutive K of one row) as one
// 16-byte store. The transposed image (rows v, K = token rows) takes each
// quad's 4 x 4 blocks transposed across its lanes, one 8-byte store each. Per entry the epilogue spends five VALU operations and one
// exp: the tail mask only in the tail tile, the token's term only in the lane
// group that holds it.
struct EpiDlogits {
  using Args = DlogitsArgs;
  static constexpr bool kTokens = true;
  static constexpr bool kCoef = true;
  static constexpr bool kPacked = false;  // operands W and h as the caller holds them
  // stage loads one every 3 MFMAs from the k-step's start (2% faster here than
  // spread evenly, which stays faster for the forward)
  static constexpr int kLoadSpacing = 3;
  // vocab tiles per group of its tile order: 2 (1-2% faster here than the
  // forward's 4; 1 and 8 slower)
  static constexpr int kGroupA = 2;
  static constexpr int kNV = 2;  // vocab waves: whole 256-entry A tiles
  template <int BT>
  static constexpr int scratch_bytes() { return 0; }
  __device__ static TileOps ops(const Args& a) {
    return TileOps{a.w, a.hidden, a.tokens, a.coef, a.rows, a.V, a.d};
  }
  template <int NTB, int WT>
  __device__ static void init(const Args&, int64_t, int64_t, f32x4 (&acc)[8][2 * NTB], int, int) {
#pragma unroll
    for (int bi = 0; bi < 8; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2 * NTB; ++bj) acc[bi][bj] = f32x4{};
  }
  // One row block's gradients as bf16 pairs: every entry -p (alpha + beta q)
  // (FULL: no entry past V); in the lane group holding the row's token, its
  // entry then adds gamma, which is gamma - p (alpha + beta q) exactly.
  template <bool FULL>
  __device__ static void row_block(const f32x4 (&accj)[8], float inv_tau, float lse, float alpha, float beta,
                                   float gamma, int tl, int lim, uint2 (&pk)[8]) {
#pragma unroll
    for (int bi = 0; bi < 8; ++bi) {
      float o[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        // z * inv_tau: a multiply by exactly 1 returns z itself (fp32 denormals kept)
        const float q = accj[bi][r] * inv_tau - lse;
        const float p = exp2_hw(q * kLog2e);
        o[r] = -(p * __builtin_fmaf(beta, q, alpha));
        if (!FULL && bi * 16 + r >= lim) o[r] = 0.f;
      }
      if ((unsigned)(tl - bi * 16) < 4u) {
        // a real branch (taken by one lane group of one row), not selects on every entry
        asm volatile("" ::: "memory");
        const int rt = tl - bi * 16;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (r == rt) o[r] = gamma + o[r];
      }
      pk[bi] = uint2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
    }
  }
  // Lanes 4 m + j (j = 0..3) hold a 4 x 4 block as bf16 pairs: lane j the
  // entries r = 0..3 of token row j. Exchanged within the quad so that lane j
  // then holds token rows 0..3 of entry j, lo the rows 0 and 1: first the
  // 32-bit halves between lanes j and j ^ 2, then the 16-bit halves between
  // lanes j and j ^ 1 (byte selects from the partner's word).
  __device__ static uint2 quad_transpose(uint2 v, int j) {
    const bool upper = (j & 2) != 0;
    const int s = (int)(upper ? v.x : v.y);
    const uint32_t r = (uint32_t)__builtin_amdgcn_mov_dpp(s, 0x4e, 0xf, 0xf, true);  // quad_perm 2 3 0 1
    if (upper) v.x = r; else v.y = r;
    const uint32_t px = (uint32_t)__builtin_amdgcn_mov_dpp((int)v.x, 0xb1, 0xf, 0xf, true);  // quad_perm 1 0 3 2
    const uint32_t py = (uint32_t)__builtin_amdgcn_mov_dpp((int)v.y, 0xb1, 0xf, 0xf, true);
    // even j: own low half, then the partner's low half; odd j: the partner's high half, then own high half
    const uint32_t sel = (j & 1) ? 0x03020706u : 0x05040100u;
    return uint2{__builtin_amdgcn_perm(px, v.x, sel), __builtin_amdgcn_perm(py, v.y, sel)};
  }
  template <int NTB, int WT>
  __device__ static void epilogue(const Args& a, int, int, int64_t v0, int64_t t0, f32x4 (&acc)[8][2 * NTB], float*,
                                  const int* tok_lds, const f32x4* coef_lds, int wave, int lane) {
    constexpr int NJ = 2 * NTB;
    static_assert(WT * NTB * 32 == kPackRows, "a row tile is one 256-row tile of the packed output");
    const int wv = wave & 1, wt = wave >> 1;
    const int g = lane >> 4, c16 = lane & 15;
    const float inv_tau = a.inv_tau;
    const int64_t vlane = v0 + wv * 128 + 4 * g;
    const bool full = v0 + kVocabTile <= a.V;
    const int lim = a.V - (int)vlane;  // entries past V: bi * 16 + r >= lim (tail tile only)
    uint16_t* out = (uint16_t*)a.dacc;
    const int j4 = lane & 3, qd = c16 >> 2;
#pragma unroll
    for (int bj = 0; bj < NJ; ++bj) {
      const int t_loc = wt * NTB * 32 + bj * 16 + c16;
      const int64_t tg = t0 + t_loc;
      uint2 pk[8];
      if (tg < a.rows) {
        const f32x4 c = coef_lds[t_loc];
        // the token's offset from this lane's first entry (both below 2^31)
        const int tl = tok_lds[t_loc] - (int)vlane;
        f32x4 accj[8];
#pragma unroll
        for (int bi = 0; bi < 8; ++bi) accj[bi] = acc[bi][bj];
        if (full) row_block<true>(accj, inv_tau, c[0], c[1], c[2], c[3], tl, lim, pk);
        else row_block<false>(accj, inv_tau, c[0], c[1], c[2], c[3], tl, lim, pk);
        if (out && a.packed) {
          // Packed: tile t0 / 256, row t_loc of it; entry vlane + bi * 16 in stage vlane / 64 + bi / 4, chunk
          // 2 (bi % 4) + g / 2 before the swizzle, its half g % 2. Lanes l and l ^ 16 (lane groups g and g ^ 1,
          // the same row) hold the two halves of one chunk. Each swap exchanges the odd group's block 2m half
          // with the even group's block 2m + 1 half, so an even group then holds both halves of its block 2m
          // chunk and an odd group those of its block 2m + 1 chunk, each written as one 16-byte store. Both
          // lanes of a pair take the same branch above (same row).
          const bool odd = (g & 1) != 0;
          const int psw = swz(t_loc);
          uint16_t* pbase = out + (t0 >> 8) * (a.ld << 8) + (vlane >> 6) * (kPackRows * kKS) + t_loc * kKS;
#pragma unroll
          for (int m = 0; m < 4; ++m) {
            const auto x0 = __builtin_amdgcn_permlane16_swap(pk[2 * m].x, pk[2 * m + 1].x, false, false);
            const auto x1 = __builtin_amdgcn_permlane16_swap(pk[2 * m].y, pk[2 * m + 1].y, false, false);
            const int bi = 2 * m + (odd ? 1 : 0);
            uint16_t* dst = pbase + (bi >> 2) * (kPackRows * kKS) + (((2 * (bi & 3) + (g >> 1)) ^ psw) << 3);
            *(uint4*)dst = uint4{x0[0], x1[0], x0[1], x1[1]};
          }
        } else if (out) {
          uint16_t* row = out + tg * a.ld + vlane;
#pragma unroll
          for (int bi = 0; bi < 8; ++bi) *(uint2*)(row + bi * 16) = pk[bi];
        }
      } else {
#pragma unroll
        for (int bi = 0; bi < 8; ++bi) pk[bi] = uint2{0u, 0u};
      }
      if (a.dacct) {
        // Transposed image [ld, t_pad] in 32-deep blocks: after the quad transpose this lane holds entry row
        // vlane + bi * 16 + (l % 4) of the tile (row rr of its 256, whose chunk swizzle (rr / 4) % 4 is g) and
        // the four token rows tq .. tq + 3. Every lane of the quad takes part (rows past the end as zeros); the
        // quad's four rows lie together below t_pad or not at all (t_pad is a multiple of 128).
        const int tq = (int)t0 + wt * NTB * 32 + bj * 16 + 4 * qd;
        uint16_t* dst = (uint16_t*)a.dacct + (v0 >> 8) * (a.t_pad << 8) + (tq >> 5) * (kPackRows * 32) +
                        (wv * 128 + 4 * g + j4) * 32 + (((((bj * 16) & 31) >> 3) + (qd >> 1)) ^ g) * 8 + 4 * (qd & 1);
        // non-temporal: read back only by the weight pass, after grad_hidden (this pass measured 2.3% faster
        // than with plain stores; the packed stores above stay plain, 1.3% slower non-temporal)
#pragma unroll
        for (int bi = 0; bi < 8; ++bi) {
          const uint2 tv = quad_transpose(pk[bi], j4);
          if (tq < a.t_pad) __builtin_nontemporal_store(u32x2_t{tv.x, tv.y}, (u32x2_t*)(dst + bi * 16 * 32));
        }
      }
    }
  }
};

// fp32 stores of the tile (optionally continuing from the stored values):
// lane l holds B row j = t0 + wt * NTB * 32 + bj * 16 + l % 16 and the 4
// consecutive A rows i = v0 + wv * 128 + bi * 16 + 4 (l / 16) + r, one 16-byte
// access each. Both operands packed.
struct EpiStore {
  using Args = GemmArgs;
  static constexpr bool kTokens = false;
  static constexpr bool kCoef = false;
  static constexpr bool kPacked = true;
  static constexpr int kLoadSpacing = 3;  // stage loads one every 3 MFMAs (2% faster than spread evenly)
  static constexpr int kGroupA = kStoreGroup;
  static constexpr int kNV = 2;  // vocab waves: whole 256-entry A tiles
  template <int BT>
  static constexpr int scratch_bytes() { return 0; }
  __device__ static TileOps ops(const Args& a) {
    return TileOps{a.a, a.b, nullptr, nullptr, a.b_rows, a.a_rows, a.K};
  }
  template <int NTB, int WT>
  __device__ static void init(const Args& a, int64_t v0, int64_t t0, f32x4 (&acc)[8][2 * NTB], int wave, int lane) {
    const int wv = wave & 1, wt = wave >> 1;
    // A rows are int32 (a_rows < 2^31), so this lane's first row and the
    // distance to the end are formed in 32 bits
    const int i_lane = (int)v0 + wv * 128 + 4 * (lane >> 4);
    const int lim0 = a.a_rows - i_lane;  // A rows past the end: bi * 16 >= lim
    const int lim = lim0 > 256 ? 256 : lim0;
#pragma unroll
    for (int bj = 0; bj < 2 * NTB; ++bj) {
      const int64_t jr = t0 + wt * NTB * 32 + bj * 16 + (lane & 15);
#pragma unroll
      for (int bi = 0; bi < 8; ++bi) {
        const int i0 = i_lane + bi * 16;
        acc[bi][bj] = (a.accumulate && jr < a.b_rows && bi * 16 < lim) ? *(const f32x4*)(a.out + jr * a.ldo + i0)
                                                                     : f32x4{};
      }
    }
  }
  template <int NTB, int WT>
  __device__ static void epilogue(const Args& a, int, int, int64_t v0, int64_t t0, f32x4 (&acc)[8][2 * NTB], float*,
                                  const int*, const f32x4*, int wave, int lane) {
    const int wv = wave & 1, wt = wave >> 1;
    // A rows are int32 (a_rows < 2^31), so this lane's first row and the
    // distance to the end are formed in 32 bits
    const int i_lane = (int)v0 + wv * 128 + 4 * (lane >> 4);
    const int lim0 = a.a_rows - i_lane;  // A rows past the end: bi * 16 >= lim
    const int lim = lim0 > 256 ? 256 : lim0;
#pragma unroll
    for (int bj = 0; bj < 2 * NTB; ++bj) {
      const int64_t jr = t0 + wt * NTB * 32 + bj * 16 + (lane & 15);
      if (jr >= a.b_rows) continue;
#pragma unroll
      for (int bi = 0; bi < 8; ++bi) {
        const int i0 = i_lane + bi * 16;
        if (bi * 16 < lim) *(f32x4*)(a.out + jr * a.ldo + i0) = acc[bi][bj];
      }
    }
  }
};

template <int NTB, int WT>
__global__ __launch_bounds__(128 * WT, (Shape<NTB, WT, false>::PER_CU))
void lmhead_dlogits(DlogitsArgs a, int n_vt, int n_tt) {
  tile_pass<NTB, WT, false, EpiDlogits>(a, n_vt, n_tt);
}

template <int NTB, int WT>
__global__ __launch_bounds__(128 * WT, (Shape<NTB, WT, false>::PER_CU))
void gemm_nt_f32(GemmArgs a, int n_vt, int n_tt) {
  tile_pass<NTB, WT, false, EpiStore>(a, n_vt, n_tt);
}

// The same product on operands packed in 32-deep blocks, five stage buffers
// (one workgroup per CU): the weight gradient's short-K passes.
constexpr int kDeepBufs = 5;
template <int NTB, int WT>
__global__ __launch_bounds__(128 * WT, 1)
void gemm_nt_f32_deep(GemmArgs a, int n_vt, int n_tt) {
  tile_pass_deep<NTB, WT, kDeepBufs, EpiStore>(a, n_vt, n_tt);
}

// 64 x 64 bf16 tile per workgroup: 16-byte row loads into LDS, then each
// thread gathers 8 consecutive source rows of one column into one 16-byte
// store of the destination row, which is packed [C_pad, R_pad] (K = R_pad) in
// DST_KS-deep stage blocks. The source is row-major with row stride ld_src, or
// packed (64-deep blocks) with K = ld_src; entries past R or C read as zeros.
template <bool SRC_PACKED, int DST_KS>
__global__ __launch_bounds__(256) void transpose_bf16(const uint16_t* __restrict__ src, int64_t R, int64_t C,
                                                      int64_t ld_src, uint16_t* __restrict__ dst, int64_t R_pad) {
  __shared__ uint16_t t[64][66];
  const int64_t r0 = (int64_t)blockIdx.x * 64, c0 = (int64_t)blockIdx.y * 64;
  const int tid = threadIdx.x;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int idx = tid + 256 * s;
    const int rr = idx >> 3, cc = (idx & 7) * 8;
    uint4 v = uint4{0u, 0u, 0u, 0u};
    if (r0 + rr < R && c0 + cc < C)
      v = *(const uint4*)(src + (SRC_PACKED ? packed_index(r0 + rr, c0 + cc, ld_src) : (r0 + rr) * ld_src + c0 + cc));
    uint32_t* d = (uint32_t*)&t[rr][cc];
    d[0] = v.x;
    d[1] = v.y;
    d[2] = v.z;
    d[3] = v.w;
  }
  __syncthreads();
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int idx = tid + 256 * s;
    const int cc = idx >> 3, rr = (idx & 7) * 8;
    uint32_t w[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) w[k] = (uint32_t)t[rr + 2 * k][cc] | ((uint32_t)t[rr + 2 * k + 1][cc] << 16);
    *(uint4*)(dst + packed_index<DST_KS>(c0 + cc, r0 + rr, R_pad)) = uint4{w[0], w[1], w[2], w[3]};
  }
}

__global__ __launch_bounds__(256) void grad_coef_kernel(const float* __restrict__ lse, const float* __restrict__ ent,
                                                        const float* __restrict__ g, const float* __restrict__ e,
                                                        const int32_t* __restrict__ tok, int64_t rows, int V,
                                                        double tau, f32x4* __restrict__ coef) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= rows) return;
  const int a = tok[t];
  const double gl = (a >= 0 && a < V) ? (double)g[t] : 0.0;
  const double ev = e ? (double)e[t] : 0.0;
  const double eh = e ? ev * (double)ent[t] : 0.0;
  coef[t] = f32x4{lse[t], (float)((gl + eh) / tau), (float)(ev / tau), (float)(gl / tau)};
}

__global__ __launch_bounds__(256) void fill_zero_kernel(float* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0.f;
}

}  // namespace

template <class E, int NTB, int WT>
static hipError_t launch_pass(void (*kernel)(typename E::Args, int, int), const typename E::Args& a, int64_t a_rows,
                              int64_t b_rows, hipStream_t s) {
  constexpr int BT = Tile<NTB, WT>::BT;
  const int64_t n_vt = (a_rows + kVocabTile - 1) / kVocabTile;
  const int64_t n_tt = (b_rows + BT - 1) / BT;
  const int64_t nblk = n_vt * n_tt;
  if (nblk > 0x7fffffff) return hipErrorInvalidValue;
  int64_t grid = nblk;
  const int64_t resident = (int64_t)device_cu_count() * Shape<NTB, WT, false>::PER_CU;
  if (resident > 0 && resident < grid) grid = resident;
  hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(128 * WT), 0, s, a, (int)n_vt, (int)n_tt);
  return hipGetLastError();
}

hipError_t launch_dlogits(const DlogitsArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (!a.dacc && !a.dacct) return hipErrorInvalidValue;
  if (a.dacct && (a.t_pad % 128 != 0 || a.t_pad < a.rows || a.ld % kPackRows != 0)) return hipErrorInvalidValue;
  return launch_pass<EpiDlogits, 2, 4>(lmhead_dlogits<2, 4>, a, a.V, a.rows, s);
}

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s) {
  if (a.b_rows <= 0 || a.a_rows <= 0) return hipSuccess;
  if (a.deep) {  // 32-deep stages: a multiple of 4 of them, at least kDeepBufs + 1
    if (a.K % 128 != 0 || a.K / 32 < kDeepBufs + 1) return hipErrorInvalidValue;
    return launch_pass<EpiStore, 2, 4>(gemm_nt_f32_deep<2, 4>, a, a.a_rows, a.b_rows, s);
  }
  return launch_pass<EpiStore, 2, 4>(gemm_nt_f32<2, 4>, a, a.a_rows, a.b_rows, s);
}

hipError_t launch_transpose(const void* src, bool src_packed, int64_t R, int64_t C, int64_t ld_src, void* dst,
                            int64_t R_pad, int64_t C_pad, int dst_ks, hipStream_t s) {
  if (dst_ks != 64 && dst_ks != 32) return hipErrorInvalidValue;
  if (C_pad % kPackRows != 0 || R_pad % 64 != 0 || R > R_pad || C > C_pad || C % 8 != 0) return hipErrorInvalidValue;
  if (src_packed && (ld_src % kKS != 0 || C > ld_src)) return hipErrorInvalidValue;
  if (C_pad == 0 || R_pad == 0) return hipSuccess;
  if (R_pad / 64 > 0x7fffffff || C_pad / 64 > 65535) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(R_pad / 64), (unsigned)(C_pad / 64));
  auto kernel = src_packed ? (dst_ks == 64 ? transpose_bf16<true, 64> : transpose_bf16<true, 32>)
                           : (dst_ks == 64 ? transpose_bf16<false, 64> : transpose_bf16<false, 32>);
  hipLaunchKernelGGL(kernel, grid, dim3(256), 0, s, (const uint16_t*)src, R, C, ld_src, (uint16_t*)dst, R_pad);
  return hipGetLastError();
}

hipError_t launch_grad_coef(const float* lse, const float* entropy, const float* grad_logp,
                            const float* grad_entropy, const int32_t* tokens, int64_t rows, int V,
                            float temperature, void* coef, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int64_t nb = (rows + 255) / 256;
  if (nb > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(grad_coef_kernel, dim3((unsigned)nb), dim3(256), 0, s, lse, entropy, grad_logp, grad_entropy,
                     tokens, rows, V, (double)temperature, (f32x4*)coef);
  return hipGetLastError();
}

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t nb = (n + 255) / 256;
  if (nb > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)nb), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace tim
