// Fused LM-head log-softmax kernels for gfx950 (CDNA4).
//
// The per-row quantity is the token log-probability of Section 2 of the paper
// (the terms of Eq. 1) plus the entropy of the same distribution. Every row is
// computed with one fixed sequence of floating-point operations that depends
// only on d and V, never on how many rows share a launch, on a row's position
// among them, or on the launch grid: the batch-invariance principle of
// Section 3.1 (fixed tiling and reduction order, no atomics).
//
// Kernel 1, lmhead_partials: one workgroup per (vocab tile of 256, row tile).
//   z^T = W_tile . h_tile^T on MFMA (v_mfma_f32_32x32x16_bf16, fp32 accumulate,
//   hidden dimension in ascending 16-element steps, one accumulation chain per
//   logit). W is the A operand and the hidden states the B operand, so each
//   lane's 16 accumulator registers of a 32x32 block hold 16 vocabulary entries
//   of ONE row: most of the softmax reduction happens inside a lane.
//   Operands are staged HBM -> LDS with direct global->LDS DMA loads
//   (global_load_lds_dwordx4), double buffered, XOR-swizzled against LDS bank
//   conflicts. The epilogue turns the 256 logits of each row into one partial
//   (m, s, u) = (max z, sum e^(z-m), sum e^(z-m) (z-m)) and captures the
//   sampled token's logit from the same register value. Logits never reach HBM.
//
// Kernel 2, lmhead_merge: one wavefront per row merges that row's partials with
//   a fixed balanced binary tree over the tile index, then
//   logp = z_tok - (M + log S) and H = log S - U / S.
//
// Reduction structure inside one vocab tile, for one row (fixed):
//   lane-local: 64 values in (block b = 0..3, register r = 0..15) order;
//   then the two lane halves (lane, lane ^ 32); then the two vocab waves.
// The tile's max is found first (max is exact in any order), so the sums are
// taken against the tile max directly, with no rescaling inside a tile.

#include "kernels.h"

namespace tim {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;
// Buffer resources exist only in the device pass; the host pass compiles the
// kernels as launch stubs and never runs their bodies.
#if defined(__HIP_DEVICE_COMPILE__)
typedef __amdgpu_buffer_rsrc_t rsrc_t;
#else
struct rsrc_t {
  int w[4];
};
#endif

constexpr int kRowBytes = kKStage * 2;   // bytes of one row in one stage (128)
constexpr int kWBytes = kVocabTile * kRowBytes;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

template <int NTB>
struct Tile {
  static constexpr int BT = 2 * NTB * 32;               // rows per workgroup
  static constexpr int kHBytes = BT * kRowBytes;
  static constexpr int kStageBytes = kWBytes + kHBytes;
};

// 16-byte chunk c of row r sits at physical chunk c ^ swz(r) of that row.
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

__device__ __forceinline__ void wait_vmem() {
  // s_waitcnt vmcnt(0): every outstanding global->LDS load of this wave landed.
  __builtin_amdgcn_s_waitcnt(0x0F70);
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// Bijective blockIdx -> (vocab tile, row tile). Consecutive workgroups are
// dealt round-robin to the 8 XCDs, so first undo that deal (each XCD gets a
// contiguous run of logical ids), then walk logical ids in groups of 8 vocab
// tiles: rows outer, vocab inner, so the workgroups resident on one XCD share
// W tiles and hidden-state tiles through that XCD's L2.
__device__ __forceinline__ void tile_of(int bid, int nblk, int n_vt, int& vt, int& tt) {
  const int q = nblk >> 3, rem = nblk & 7;
  const int x = bid & 7, i = bid >> 3;
  const int lid = x * q + (x < rem ? x : rem) + i;
  constexpr int GV = 8;
  const int n_tt = nblk / n_vt;
  const int group = lid / (GV * n_tt);
  const int first = group * GV;
  const int gv = (n_vt - first) < GV ? (n_vt - first) : GV;
  const int local = lid - group * GV * n_tt;
  vt = first + local % gv;
  tt = local / gv;
}

// Per-lane byte offsets of this workgroup's DMA loads, relative to the tile's
// first row at hidden index 0. They do not change along the hidden dimension:
// each stage only moves the scalar offset.
template <int NTB>
struct LoadPlan {
  static constexpr int HB = Tile<NTB>::BT / 32;  // hidden-state blocks per wave
  uint32_t w_off[8];
  uint32_t h_off[HB];
};

template <int NTB>
__device__ __forceinline__ LoadPlan<NTB> make_load_plan(int w_rows, int h_rows, int d, int wave,
                                                        int lane) {
  LoadPlan<NTB> pl;
  // W tile: 256 rows x 8 chunks = 32 blocks of 1 KB (64 lanes x 16 B); 8 per wave.
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int p = (wave * 8 + q) * 64 + lane;
    int r = p >> 3;
    const int c = (p & 7) ^ swz(r);
    if (r >= w_rows) r = w_rows - 1;  // rows past V: a valid row, masked in the epilogue
    pl.w_off[q] = (uint32_t)(r * d + c * 8) * 2u;
  }
  // Hidden-state tile: BT rows x 8 chunks = BT / 8 blocks.
#pragma unroll
  for (int q = 0; q < LoadPlan<NTB>::HB; ++q) {
    const int p = (wave * LoadPlan<NTB>::HB + q) * 64 + lane;
    int r = p >> 3;
    const int c = (p & 7) ^ swz(r);
    if (r >= h_rows) r = h_rows - 1;  // rows past the batch: never written out
    pl.h_off[q] = (uint32_t)(r * d + c * 8) * 2u;
  }
  return pl;
}

// Buffer resource over [base, base + bytes): loads outside it return zeros.
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint64_t bytes) {
#if defined(__HIP_DEVICE_COMPILE__)
  const uint32_t n = bytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
  // dword 3 = 0x00020000: raw (unswizzled) 32-bit-format buffer, the gfx9 encoding.
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
#else
  return rsrc_t{};
#endif
}

template <int NTB>
__device__ __forceinline__ void load_stage(unsigned char* lds, rsrc_t wr, rsrc_t hr,
                                           const LoadPlan<NTB>& pl, int wave, int soff) {
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
  for (int q = 0; q < 8; ++q)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void*)(lds + (wave * 8 + q) * 1024), 16,
                                             pl.w_off[q], soff, 0, 0);
#pragma unroll
  for (int q = 0; q < LoadPlan<NTB>::HB; ++q)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        hr, (lds_void*)(lds + kWBytes + (wave * LoadPlan<NTB>::HB + q) * 1024), 16, pl.h_off[q],
        soff, 0, 0);
#endif
}

template <int NTB>
__device__ __forceinline__ void compute_stage(const unsigned char* lds, f32x16 (&acc)[4][NTB],
                                              int wv, int wt, int lane) {
  const int r32 = lane & 31, hi = lane >> 5;
  const int sw = swz(r32);  // every operand row is (multiple of 32) + r32
#pragma unroll
  for (int s = 0; s < kKStage / 16; ++s) {
    const int c = ((2 * s + hi) ^ sw) * 16;
    bf16x8 a[4], b[NTB];
#pragma unroll
    for (int bb = 0; bb < 4; ++bb)
      a[bb] = *(const bf16x8*)(lds + (wv * 128 + bb * 32 + r32) * kRowBytes + c);
#pragma unroll
    for (int j = 0; j < NTB; ++j)
      b[j] = *(const bf16x8*)(lds + kWBytes + (wt * NTB * 32 + j * 32 + r32) * kRowBytes + c);
#pragma unroll
    for (int bb = 0; bb < 4; ++bb)
#pragma unroll
      for (int j = 0; j < NTB; ++j)
        acc[bb][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[bb], b[j], acc[bb][j], 0, 0, 0);
  }
}

// SPLITK4: after each quarter of the hidden dimension, fold the quarter's
// accumulator into the running sum: ((q0 + q1) + q2) + q3.
template <int NTB>
__device__ __forceinline__ void quarter_fold(f32x16 (&acc)[4][NTB], f32x16 (&sum)[4][NTB], int q) {
#pragma unroll
  for (int bb = 0; bb < 4; ++bb)
#pragma unroll
    for (int j = 0; j < NTB; ++j) {
      if (q == 0) sum[bb][j] = acc[bb][j];
      else sum[bb][j] = sum[bb][j] + acc[bb][j];
      acc[bb][j] = f32x16{};
    }
}

template <int NTB, bool SPLITK4, bool DUMP>
__global__ __launch_bounds__(256, 1) void lmhead_partials(LmHeadArgs a, int n_vt) {
  using TL = Tile<NTB>;
  constexpr int BT = TL::BT;
  __shared__ __attribute__((aligned(1024))) unsigned char lds0[TL::kStageBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char lds1[TL::kStageBytes];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wv = wave & 1, wt = wave >> 1;
  int vt, tt;
  tile_of(blockIdx.x, gridDim.x, n_vt, vt, tt);
  const int64_t v0 = (int64_t)vt * kVocabTile;
  const int64_t t0 = (int64_t)tt * BT;
  const __bf16* __restrict__ w = (const __bf16*)a.w;
  const __bf16* __restrict__ h = (const __bf16*)a.hidden;
  const int d = a.d, V = a.V;
  const int64_t rows = a.rows;

  f32x16 acc[4][NTB];
#pragma unroll
  for (int bb = 0; bb < 4; ++bb)
#pragma unroll
    for (int j = 0; j < NTB; ++j) acc[bb][j] = f32x16{};
  f32x16 sum[4][SPLITK4 ? NTB : 1];

  const int nk = d / kKStage;
  const int nk_q = nk / 4;

  const int w_rows = (V - v0) < kVocabTile ? (int)(V - v0) : kVocabTile;
  const int h_rows = (rows - t0) < BT ? (int)(rows - t0) : BT;
  const LoadPlan<NTB> pl = make_load_plan<NTB>(w_rows, h_rows, d, wave, lane);
  const rsrc_t wr = make_rsrc(w + v0 * d, (uint64_t)w_rows * d * 2);
  const rsrc_t hr = make_rsrc(h + t0 * d, (uint64_t)h_rows * d * 2);
  constexpr int kStep = kKStage * 2;  // bytes per stage along a row

  // nk is even: each iteration consumes stage kt from lds0 and kt + 1 from lds1.
  load_stage<NTB>(lds0, wr, hr, pl, wave, 0);
  for (int kt = 0; kt < nk; kt += 2) {
    wait_vmem();
    __syncthreads();
    load_stage<NTB>(lds1, wr, hr, pl, wave, (kt + 1) * kStep);
    compute_stage<NTB>(lds0, acc, wv, wt, lane);
    if constexpr (SPLITK4) {
      if ((kt + 1) % nk_q == 0) quarter_fold<NTB>(acc, sum, (kt + 1) / nk_q - 1);
    }
    wait_vmem();
    __syncthreads();
    if (kt + 2 < nk) load_stage<NTB>(lds0, wr, hr, pl, wave, (kt + 2) * kStep);
    compute_stage<NTB>(lds1, acc, wv, wt, lane);
    if constexpr (SPLITK4) {
      if ((kt + 2) % nk_q == 0) quarter_fold<NTB>(acc, sum, (kt + 2) / nk_q - 1);
    }
  }
  if constexpr (SPLITK4) {
#pragma unroll
    for (int bb = 0; bb < 4; ++bb)
#pragma unroll
      for (int j = 0; j < NTB; ++j) acc[bb][j] = sum[bb][j];
  }
  __syncthreads();  // LDS stages are free; the epilogue reuses lds0

  // ---------------------------------------------------------------- epilogue
  const int hi = lane >> 5, r32 = lane & 31;
  const float inv_tau = a.inv_tau;
  // lane's vocab offset inside the tile for (block bb, register r):
  //   wv*128 + bb*32 + 8*(r>>2) + 4*hi + (r&3)
  const int64_t vlane = v0 + wv * 128 + 4 * hi;
  float* red_m = (float*)lds0;           // [2][BT]
  float* red_s = red_m + 2 * BT;         // [2][BT]
  float* red_u = red_s + 2 * BT;         // [2][BT]
  float* zt_l = red_u + 2 * BT;          // [BT]

  int tok_loc[NTB];  // token - (vlane), meaningful only when the row is valid
  bool row_ok[NTB];
#pragma unroll
  for (int j = 0; j < NTB; ++j) {
    const int t_loc = wt * NTB * 32 + j * 32 + r32;
    const int64_t tg = t0 + t_loc;
    row_ok[j] = tg < rows;
    const int tok = (row_ok[j] && !DUMP) ? a.tokens[tg] : -1;
    tok_loc[j] = (tok >= 0) ? (int)((int64_t)tok - vlane) : -1000000;
  }

  // Phase A: temperature, vocab mask, tile max. z is formed from the
  // accumulator by the same single multiply wherever it is needed, so the
  // accumulators stay in their registers and every use sees the same bits.
#pragma unroll
  for (int j = 0; j < NTB; ++j) {
    float mx = kNegInf;
#pragma unroll
    for (int bb = 0; bb < 4; ++bb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int off = bb * 32 + 8 * (r >> 2) + (r & 3);
        const float z = (vlane + off < V) ? acc[bb][j][r] * inv_tau : kNegInf;
        mx = fmaxf(mx, z);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    if (hi == 0) red_m[wv * BT + wt * NTB * 32 + j * 32 + r32] = mx;
    if constexpr (DUMP) {
      const int64_t tg = t0 + wt * NTB * 32 + j * 32 + r32;
      if (row_ok[j]) {
#pragma unroll
        for (int bb = 0; bb < 4; ++bb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int64_t v = vlane + bb * 32 + 8 * (r >> 2) + (r & 3);
            if (v < V) a.logits[tg * (int64_t)V + v] = acc[bb][j][r] * inv_tau;
          }
      }
    }
  }
  if constexpr (DUMP) return;
  __syncthreads();

  // Phase B: sums against the tile max, in fixed (bb, r) order; token gather.
#pragma unroll
  for (int j = 0; j < NTB; ++j) {
    const int t_loc = wt * NTB * 32 + j * 32 + r32;
    const float M = fmaxf(red_m[t_loc], red_m[BT + t_loc]);
    float s = 0.f, u = 0.f;
    float zfound = 0.f;
    bool found = false;
#pragma unroll
    for (int bb = 0; bb < 4; ++bb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int off = bb * 32 + 8 * (r >> 2) + (r & 3);
        const float z = (vlane + off < V) ? acc[bb][j][r] * inv_tau : kNegInf;
        float x = z - M;
        float e = exp2_hw(x * kLog2e);
        if (z == kNegInf) { x = 0.f; e = 0.f; }
        s = s + e;
        u = __builtin_fmaf(e, x, u);
        if (tok_loc[j] == off) { zfound = z; found = true; }
      }
    if (found) zt_l[t_loc] = zfound;
    s = s + __shfl_xor(s, 32);
    u = u + __shfl_xor(u, 32);
    if (hi == 0) {
      red_s[wv * BT + t_loc] = s;
      red_u[wv * BT + t_loc] = u;
    }
  }
  __syncthreads();

  // Phase C: combine the two vocab waves and store one partial per row.
  if (wv == 0 && hi == 0) {
#pragma unroll
    for (int j = 0; j < NTB; ++j) {
      const int t_loc = wt * NTB * 32 + j * 32 + r32;
      const int64_t tg = t0 + t_loc;
      if (!row_ok[j]) continue;
      Partial p;
      p.m = fmaxf(red_m[t_loc], red_m[BT + t_loc]);
      p.s = red_s[t_loc] + red_s[BT + t_loc];
      p.u = red_u[t_loc] + red_u[BT + t_loc];
      const int tv = tok_loc[j] + wv * 128 + 4 * hi;  // token - v0
      p.ztok = (tv >= 0 && tv < kVocabTile) ? zt_l[t_loc] : 0.f;
      a.part[tg * n_vt + vt] = p;
    }
  }
}

// ---------------------------------------------------------------- merge

struct MSU {
  float m, s, u;
};

// (m, s, u) of the union of two disjoint vocab sets; `a` is the lower-index set.
__device__ __forceinline__ MSU merge2(MSU a, MSU b) {
  if (b.m == kNegInf) return a;  // empty set: exact identity
  if (a.m == kNegInf) return b;
  const float M = fmaxf(a.m, b.m);
  const float da = a.m - M, db = b.m - M;
  const float ea = exp2_hw(da * kLog2e), eb = exp2_hw(db * kLog2e);
  MSU r;
  r.m = M;
  r.s = a.s * ea + b.s * eb;
  r.u = (a.u + da * a.s) * ea + (b.u + db * b.s) * eb;
  return r;
}

__device__ __forceinline__ void finish_row(MSU v, const Partial* p, int tok, int V, int64_t row,
                                           float* logp, float* ent, float* lse) {
  const float logS = logf(v.s);
  const float L = v.m + logS;
  const bool ok = tok >= 0 && tok < V;
  logp[row] = ok ? p[tok / kVocabTile].ztok - L : __builtin_nanf("");
  if (ent) ent[row] = logS - v.u / v.s;
  if (lse) lse[row] = L;
}

// One wavefront per row. Lane l owns leaves [l*L, l*L + L); missing leaves are
// the identity, so the result is the balanced pairwise tree over the tile
// index whatever L is.
template <int L>
__global__ __launch_bounds__(256) void lmhead_merge_tree(const Partial* __restrict__ part,
                                                         const int32_t* __restrict__ tokens,
                                                         int64_t rows, int n_vt, int V, float* logp,
                                                         float* ent, float* lse) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const Partial* p = part + row * n_vt;
  MSU leaf[L];
#pragma unroll
  for (int i = 0; i < L; ++i) {
    const int jt = lane * L + i;
    if (jt < n_vt) {
      const Partial q = p[jt];
      leaf[i] = MSU{q.m, q.s, q.u};
    } else {
      leaf[i] = MSU{kNegInf, 0.f, 0.f};
    }
  }
#pragma unroll
  for (int wdt = 1; wdt < L; wdt *= 2)
#pragma unroll
    for (int i = 0; i < L; i += 2 * wdt) leaf[i] = merge2(leaf[i], leaf[i + wdt]);
  MSU v = leaf[0];
#pragma unroll
  for (int off = 1; off < 64; off *= 2) {
    MSU o;
    o.m = __shfl_xor(v.m, off);
    o.s = __shfl_xor(v.s, off);
    o.u = __shfl_xor(v.u, off);
    v = (lane & off) ? merge2(o, v) : merge2(v, o);
  }
  if (lane == 0) finish_row(v, p, tokens[row], V, row, logp, ent, lse);
}

// SPLITK4 engine: one thread per row, partials folded left to right.
__global__ __launch_bounds__(256) void lmhead_merge_fold(const Partial* __restrict__ part,
                                                         const int32_t* __restrict__ tokens,
                                                         int64_t rows, int n_vt, int V, float* logp,
                                                         float* ent, float* lse) {
  const int64_t row = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (row >= rows) return;
  const Partial* p = part + row * n_vt;
  MSU v = MSU{p[0].m, p[0].s, p[0].u};
  for (int jt = 1; jt < n_vt; ++jt) v = merge2(v, MSU{p[jt].m, p[jt].s, p[jt].u});
  finish_row(v, p, tokens[row], V, row, logp, ent, lse);
}

}  // namespace

int n_vocab_tiles(int V) { return (V + kVocabTile - 1) / kVocabTile; }

template <int NTB, bool SPLITK4, bool DUMP>
static hipError_t launch_partials_t(const LmHeadArgs& a, hipStream_t s) {
  const int n_vt = n_vocab_tiles(a.V);
  const int64_t n_tt = (a.rows + Tile<NTB>::BT - 1) / Tile<NTB>::BT;
  const int64_t nblk = n_tt * n_vt;
  if (nblk > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((lmhead_partials<NTB, SPLITK4, DUMP>), dim3((unsigned)nblk), dim3(256), 0, s,
                     a, n_vt);
  return hipGetLastError();
}

hipError_t launch_partials(const LmHeadArgs& a, int token_blocks, bool splitk4, hipStream_t s) {
  const bool dump = a.logits != nullptr;
  if (splitk4) {
    if (token_blocks >= 2)
      return dump ? launch_partials_t<2, true, true>(a, s) : launch_partials_t<2, true, false>(a, s);
    return dump ? launch_partials_t<1, true, true>(a, s) : launch_partials_t<1, true, false>(a, s);
  }
  switch (token_blocks) {
    case 1: return dump ? launch_partials_t<1, false, true>(a, s) : launch_partials_t<1, false, false>(a, s);
    case 2: return dump ? launch_partials_t<2, false, true>(a, s) : launch_partials_t<2, false, false>(a, s);
    default: return dump ? launch_partials_t<4, false, true>(a, s) : launch_partials_t<4, false, false>(a, s);
  }
}

hipError_t launch_merge(const Partial* part, const int32_t* tokens, int64_t rows, int V,
                        bool left_fold, float* logp, float* entropy, float* lse, hipStream_t s) {
  const int n_vt = n_vocab_tiles(V);
  if (left_fold) {
    const int64_t nb = (rows + 255) / 256;
    hipLaunchKernelGGL(lmhead_merge_fold, dim3((unsigned)nb), dim3(256), 0, s, part, tokens, rows,
                       n_vt, V, logp, entropy, lse);
    return hipGetLastError();
  }
  const int64_t nb = (rows + 3) / 4;
  if (nb > 0x7fffffff) return hipErrorInvalidValue;
  const dim3 g((unsigned)nb), b(256);
  if (n_vt <= 64) hipLaunchKernelGGL(lmhead_merge_tree<1>, g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else if (n_vt <= 128) hipLaunchKernelGGL(lmhead_merge_tree<2>, g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else if (n_vt <= 256) hipLaunchKernelGGL(lmhead_merge_tree<4>, g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else if (n_vt <= 512) hipLaunchKernelGGL(lmhead_merge_tree<8>, g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else if (n_vt <= 1024) hipLaunchKernelGGL(lmhead_merge_tree<16>, g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else if (n_vt <= kMaxTiles) hipLaunchKernelGGL(lmhead_merge_tree<32>, g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tim
