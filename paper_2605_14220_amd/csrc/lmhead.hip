// Fused LM-head log-softmax kernels for gfx950 (CDNA4).
//
// The per-row quantity is the token log-probability of Section 2 of the paper
// (the terms of Eq. 1) plus the entropy of the same distribution. Every row is
// computed with one fixed sequence of floating-point operations that depends
// only on d and V, never on how many rows share a launch, on a row's position
// among them, or on the launch grid: the batch-invariance principle of
// Section 3.1 (fixed tiling and reduction order, no atomics).
//
// Kernel 1, lmhead_partials: (vocab tile of 256, row tile) output tiles.
//   z^T = W_tile . h_tile^T on MFMA (v_mfma_f32_16x16x32_bf16, fp32
//   accumulate, hidden dimension in ascending 32-element steps, one
//   accumulation chain per logit). W is the A operand and the hidden states
//   the B operand: a lane's 4 accumulator registers of a 16x16 block hold 4
//   consecutive vocabulary entries of ONE row. Of the two MFMA shapes with
//   the full bf16 rate, this one moves fewer accumulator bytes per flop and
//   sustains a higher clock under the card's power limit.
//   Operands are staged HBM -> LDS with direct global->LDS DMA loads
//   (buffer_load_dwordx4 into LDS), double buffered, XOR-swizzled against LDS
//   bank conflicts. The epilogue turns the 256 logits of each row into one
//   partial (m, s, u) = (max z, sum e^(z-m), sum e^(z-m) (z-m)) and captures
//   the sampled token's logit from the same register value. Logits never
//   reach HBM.
//
// Kernel 2, lmhead_merge: one wavefront per row merges that row's partials with
//   a fixed balanced binary tree over the tile index, then
//   logp = z_tok - (M + log S) and H = log S - U / S.
//
// Reduction structure inside one vocab tile, for one row (fixed): each of the
// two vocab waves holds 128 entries of the row, 32 per lane in 4 lanes; per
// wave, the max and then the sums against it go lane-local in (block, register)
// order, then over the lane groups (lane ^ 16, then lane ^ 32); the two waves'
// partials are then merged, lower vocabulary half first.

#include "kernels.h"

namespace tim {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
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

// Compile-time launch and pipeline shape. None of these changes the
// arithmetic: the hidden dimension is accumulated in the same ascending
// 32-element MFMA steps whatever the buffer count, LDS swizzle or tile order.
#ifndef TIM_NBUF
#define TIM_NBUF 2         // LDS stage buffers: a power of two >= 2 (as many as fit, up to this)
#endif
#ifndef TIM_GROUP_V
#define TIM_GROUP_V 4      // vocab tiles per group in the workgroup -> tile order
#endif
#ifndef TIM_LOAD_AUX
#define TIM_LOAD_AUX 0     // cache-policy bits of the global->LDS loads (gfx950 sc0=1, nt=2, sc1=16)
#endif
#ifndef TIM_PERSISTENT
#define TIM_PERSISTENT 1   // full-size launches: one workgroup per CU looping over tiles
#endif
#ifndef TIM_WIDE_WAVES
#define TIM_WIDE_WAVES 1   // 256-row tiles: 8 waves of 128x64 (2 per SIMD); 0 = 4 waves of 128x128
#endif

constexpr int kKS = 64;                  // hidden-dimension elements per LDS stage
constexpr int kRowBytes = kKS * 2;       // bytes of one row in one stage
constexpr int kChunks = kRowBytes / 16;  // 16-byte chunks per row per stage
constexpr int kKM = 32;                  // hidden-dimension elements per MFMA
constexpr int kSteps = kKS / kKM;        // MFMA k-steps per stage
constexpr int kWBytes = kVocabTile * kRowBytes;
static_assert(kSteps == 2, "the operand double buffer alternates once per k-step");
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

// Workgroup shape: 2 waves along the vocab tile (128 entries, 8 blocks of 16,
// each) times WT waves along the rows, each wave holding NTB * 32 rows (2 * NTB
// blocks of 16).
template <int NTB, int WT>
struct Tile {
  static constexpr int NW = 2 * WT;            // waves per workgroup
  static constexpr int NJ = 2 * NTB;           // row blocks of 16 per wave
  static constexpr int BT = WT * NTB * 32;     // rows per workgroup
  static constexpr int kHBytes = BT * kRowBytes;
  static constexpr int kStageBytes = kWBytes + kHBytes;
};

// Residency and pipeline depth of one kernel shape. Shapes whose wave holds
// at most 128 x 64 accumulators (and no second accumulator set) run two
// workgroups per CU when two stage buffers fit in half of the 160 KB LDS.
template <int NTB, int WT, bool SPLITK4>
struct Shape {
  using TL = Tile<NTB, WT>;
  static constexpr int PER_CU =
      (WT == 2 && NTB <= 2 && !SPLITK4 && (80 * 1024) / TL::kStageBytes >= 2) ? 2 : 1;
  static constexpr int FIT = (160 * 1024 / PER_CU) / TL::kStageBytes;
  static constexpr int CAP = FIT < TIM_NBUF ? FIT : TIM_NBUF;
  // a power of two, so that it divides the stage count
  static constexpr int NBUF = CAP >= 8 ? 8 : CAP >= 4 ? 4 : 2;
  static_assert(FIT >= 2, "double buffering at least");
};

// 16-byte chunk c of row r sits at physical chunk c ^ swz(r) of that row. A
// ds_read_b128 serves 16 lanes per cycle; its 16 lanes read 16 consecutive
// rows at one logical chunk, and with 128-byte rows this swizzle puts them in
// 16 distinct 16-byte bank groups of the 64 banks.
__device__ __forceinline__ int swz(int r) { return (r >> 1) & (kChunks - 1); }

// s_waitcnt vmcnt(N) (expcnt and lgkmcnt left at their maxima): at most N of
// this wave's vector-memory loads (here: global->LDS DMA) are still in flight.
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// s_waitcnt vmcnt(N) lgkmcnt(0): additionally every LDS access of this wave done.
template <int N>
__device__ __forceinline__ void wait_lgkm0_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0070);
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// Combine a value over the four lane groups (lanes l, l ^ 16, l ^ 32, l ^ 48)
// as (g0 op g1) op (g2 op g3). v_permlane16_swap / v_permlane32_swap of a
// register with itself return, in every lane, the two halves' values in the
// same order, so every lane computes the same operation on the same operands.
__device__ __forceinline__ float group_sum(float x) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}
__device__ __forceinline__ float group_max(float x) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}

// Workgroup barrier between pipeline stages. Each wave has already waited
// for what the barrier must order (its own DMA of the next stage, and its own
// reads of the buffer about to be refilled), so no memory fence is needed;
// the empty asm statements keep the compiler from moving memory operations
// across it, and the scheduling fences keep every other instruction on its
// side too.
__device__ __forceinline__ void stage_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  // the k-step after a boundary runs at raised priority (see region_a_prio)
  __builtin_amdgcn_s_setprio(1);
}

// Wave priority of the k-step before a boundary. The two waves sharing a SIMD
// drift apart (the older one issues first); a wave that is already into the
// next stage's first k-step yields to its sibling still finishing the k-step
// after the last boundary, so the two reach the next barrier closer together
// and the time one of them idles there -- with the other issuing MFMAs alone,
// which does not fill the pipe -- shrinks.
__device__ __forceinline__ void region_a_prio() { __builtin_amdgcn_s_setprio(0); }

// Tile order: logical id -> (vocab tile, row tile), walking groups of
// TIM_GROUP_V vocab tiles with the row tiles outer and the vocab tiles inner,
// so that the workgroups resident on one XCD at a time (consecutive logical
// ids, see lmhead_partials) share W tiles and hidden-state tiles through that
// XCD's L2.
__device__ __forceinline__ void tile_of_lid(int lid, int n_vt, int n_tt, int& vt, int& tt) {
  constexpr int GV = TIM_GROUP_V;
  const int group = lid / (GV * n_tt);
  const int first = group * GV;
  const int gv = (n_vt - first) < GV ? (n_vt - first) : GV;
  const int local = lid - group * GV * n_tt;
  vt = first + local % gv;
  tt = local / gv;
}

// Per-lane byte offsets of this wave's DMA loads, relative to the tile's
// first row at hidden index 0. They do not change along the hidden dimension:
// each stage only moves the scalar offset.
template <int NTB, int WT>
struct LoadPlan {
  static constexpr int NW = Tile<NTB, WT>::NW;
  static constexpr int WB = 4 * kChunks / NW;                         // W blocks of 1 KB per wave
  static constexpr int HB = Tile<NTB, WT>::BT * kChunks / (64 * NW);  // hidden-state blocks per wave
  static constexpr int L = WB + HB;                                   // DMA loads per wave per stage
  uint32_t w_off[WB];
  uint32_t h_off[HB];
};

template <int NTB, int WT>
__device__ __forceinline__ LoadPlan<NTB, WT> make_load_plan(int w_rows, int h_rows, int d, int wave, int lane) {
  LoadPlan<NTB, WT> pl;
#pragma unroll
  for (int q = 0; q < LoadPlan<NTB, WT>::WB; ++q) {
    const int p = (wave * LoadPlan<NTB, WT>::WB + q) * 64 + lane;
    int r = p / kChunks;
    const int c = (p % kChunks) ^ swz(r);
    if (r >= w_rows) r = w_rows - 1;  // rows past V: a valid row, masked in the epilogue
    pl.w_off[q] = (uint32_t)(r * d + c * 8) * 2u;
  }
#pragma unroll
  for (int q = 0; q < LoadPlan<NTB, WT>::HB; ++q) {
    const int p = (wave * LoadPlan<NTB, WT>::HB + q) * 64 + lane;
    int r = p / kChunks;
    const int c = (p % kChunks) ^ swz(r);
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

// Load q of a stage request: the wave's L DMA loads of a stage, W blocks first.
template <int NTB, int WT>
__device__ __forceinline__ void request_load(unsigned char* buf, rsrc_t wr, rsrc_t hr, const LoadPlan<NTB, WT>& pl,
                                             int wave, int soff, int q) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int WB = LoadPlan<NTB, WT>::WB;
  constexpr int L = LoadPlan<NTB, WT>::L;
  if (q < WB)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void*)(buf + (wave * WB + q) * 1024), 16, pl.w_off[q], soff, 0,
                                             TIM_LOAD_AUX);
  else
    __builtin_amdgcn_raw_ptr_buffer_load_lds(hr, (lds_void*)(buf + kWBytes + (wave * (L - WB) + (q - WB)) * 1024), 16,
                                             pl.h_off[q - WB], soff, 0, TIM_LOAD_AUX);
#endif
}

// The tile's BT tokens into LDS, 64 per wave from the first BT / 64 waves
// (rows past the batch read as 0 and are never used).
template <int BT>
__device__ __forceinline__ void request_tokens(int* dst, rsrc_t tr, int wave, int lane) {
#if defined(__HIP_DEVICE_COMPILE__)
  if (wave < BT / 64)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(tr, (lds_void*)(dst + wave * 64), 4, (uint32_t)(wave * 64 + lane) * 4u, 0,
                                             0, 0);
#endif
}

// MFMA operands of k-step s of a stage buffer, 8 bf16 per lane: lane l reads
// row (l % 16) of a 16-row block at hidden offset 32 s + 8 (l / 16).
__device__ __forceinline__ bf16x8 read_operand(const unsigned char* base, int row, int s, int lane) {
  const int c = (4 * s + (lane >> 4)) ^ swz(row);
  return *(const bf16x8*)(base + row * kRowBytes + c * 16);
}
// W block bi (16 vocabulary rows) of vocab wave wv
__device__ __forceinline__ bf16x8 read_a(const unsigned char* buf, int s, int bi, int wv, int lane) {
  return read_operand(buf, wv * 128 + bi * 16 + (lane & 15), s, lane);
}
// hidden-state block bj (16 rows) of row wave wt
template <int NTB>
__device__ __forceinline__ bf16x8 read_b(const unsigned char* buf, int s, int bj, int wt, int lane) {
  return read_operand(buf + kWBytes, wt * NTB * 32 + bj * 16 + (lane & 15), s, lane);
}

// One k-step as 8 * NJ scheduling units, each pinned on its own: unit i
// issues the MFMA of W block bi = i / NJ and row block bj = i % NJ (the
// accumulation order of every logit is the k-step order; the order of the
// units only interleaves independent chains), then, with LOAD, its share of
// the DMA loads of a stage request into `lb`, and, with READ, the reads of
// k-step `rs` of buffer `rb`. Operands alternate between two register sets by
// k-step parity P: the row-block operands always, read from the first units
// on; the W operands too with AD (then read right after the row blocks, so
// every read lands early), else the single W set is refilled block by block
// right after each block's last use here.
template <int NTB, int WT, int P, bool AD, bool LOAD, bool READ = true>
__device__ __forceinline__ void kstep(bf16x8 (&fa)[2][8], bf16x8 (&fb)[2][2 * NTB], f32x4 (&acc)[8][2 * NTB],
                                      unsigned char* lb, rsrc_t wr, rsrc_t hr, const LoadPlan<NTB, WT>& pl, int soff,
                                      const unsigned char* rb, int rs, int wave, int wv, int wt, int lane) {
  constexpr int NJ = 2 * NTB;
  constexpr int NM = 8 * NJ;
  constexpr int L = LoadPlan<NTB, WT>::L;
  constexpr int PA = AD ? P : 0, PN = AD ? (P ^ 1) : 0;
  static_assert(L <= NM, "at most one DMA load per unit");
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    const int bi = i / NJ, bj = i % NJ;
    acc[bi][bj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[PA][bi], fb[P][bj], acc[bi][bj], 0, 0, 0);
    if (LOAD) {  // load q goes with unit q * NM / L
      const int q = (i * L + NM - 1) / NM;
      if (q < L && q * NM / L == i) request_load<NTB, WT>(lb, wr, hr, pl, wave, soff, q);
    }
    if (READ) {
      if (!AD && i < NJ) fb[P ^ 1][i] = read_b<NTB>(rb, rs, i, wt, lane);
      if (AD) {
        // NJ + 8 reads spread evenly over the units, in the order the next
        // k-step consumes them: a0, b0 .. b[NJ-1], a1 .. a7
        constexpr int NR = NJ + 8;
        const int r = (i * NR + NM - 1) / NM;
        if (r < NR && r * NM / NR == i) {
          if (r == 0) fa[PN][0] = read_a(rb, rs, 0, wv, lane);
          else if (r <= NJ) fb[P ^ 1][r - 1] = read_b<NTB>(rb, rs, r - 1, wt, lane);
          else fa[PN][r - NJ] = read_a(rb, rs, r - NJ, wv, lane);
        }
      } else {
        if (bj == NJ - 1) fa[PN][bi] = read_a(rb, rs, bi, wv, lane);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// SPLITK4: after each quarter of the hidden dimension, fold the quarter's
// accumulator into the running sum: ((q0 + q1) + q2) + q3.
template <int NTB>
__device__ __forceinline__ void quarter_fold(f32x4 (&acc)[8][2 * NTB], f32x4 (&sum)[8][2 * NTB], int q) {
#pragma unroll
  for (int bi = 0; bi < 8; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2 * NTB; ++bj) {
      if (q == 0) sum[bi][bj] = acc[bi][bj];
      else sum[bi][bj] = sum[bi][bj] + acc[bi][bj];
      acc[bi][bj] = f32x4{};
    }
}

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

// One tile's per-row results from its accumulators. Each wave holds 128 of
// the tile's 256 vocabulary entries of its rows: for row block bj, lane l holds
// row (l % 16) and, in register r of W block bi, the entry
// wv * 128 + bi * 16 + 4 (l / 16) + r. Per row block the wave takes the logits
// z = acc * inv_tau (a multiply by exactly 1 is skipped, which changes
// nothing), masks entries past V to -inf (tail tile only), forms its half's
// partial (m, s, u) -- max first, then the sums against that max, lane-local
// in (bi, r) order, then over lane ^ 16 and lane ^ 32 -- and captures the
// sampled token's logit from the same register value. The two vocab halves
// are merged in a fixed order (lower half first) into the tile's Partial.
// `scratch` holds 7 * BT floats of LDS; with `tok_lds` the tile's tokens come
// from LDS.
template <int NTB, int WT, bool DUMP>
__device__ __forceinline__ void tile_epilogue(const LmHeadArgs& a, int n_vt, int vt, int64_t v0, int64_t t0,
                                              f32x4 (&acc)[8][2 * NTB], float* scratch, const int* tok_lds, int wave,
                                              int lane) {
  constexpr int BT = Tile<NTB, WT>::BT;
  constexpr int NJ = 2 * NTB;
  const int wv = wave & 1, wt = wave >> 1;
  const int V = a.V;
  const int64_t rows = a.rows;
  const int g = lane >> 4, c16 = lane & 15;
  const float inv_tau = a.inv_tau;
  const int64_t vlane = v0 + wv * 128 + 4 * g;  // + bi * 16 + r
  float* red_m = scratch;                // [2][BT]
  float* red_s = red_m + 2 * BT;         // [2][BT]
  float* red_u = red_s + 2 * BT;         // [2][BT]
  float* zt_l = red_u + 2 * BT;          // [BT]
  // Whether a tile is the tail depends only on (v0, V), so a tile takes the
  // same path in every launch shape.
  const bool full = v0 + kVocabTile <= V;

#pragma unroll
  for (int bj = 0; bj < NJ; ++bj) {
    const int t_loc = wt * NTB * 32 + bj * 16 + c16;
    const int64_t tg = t0 + t_loc;
    const bool row_ok = tg < rows;
    float z[32];  // z[4 bi + r]: entry vlane + 16 bi + r
#pragma unroll
    for (int bi = 0; bi < 8; ++bi)
#pragma unroll
      for (int r = 0; r < 4; ++r) z[bi * 4 + r] = acc[bi][bj][r];
    if (inv_tau != 1.0f) {
#pragma unroll
      for (int i = 0; i < 32; ++i) z[i] = z[i] * inv_tau;
    }
    if (!full) {
#pragma unroll
      for (int i = 0; i < 32; ++i)
        if (vlane + (i >> 2) * 16 + (i & 3) >= V) z[i] = kNegInf;
    }
    if constexpr (DUMP) {
      if (row_ok) {
#pragma unroll
        for (int i = 0; i < 32; ++i) {
          const int64_t v = vlane + (i >> 2) * 16 + (i & 3);
          if (v < V) a.logits[tg * (int64_t)V + v] = z[i];
        }
      }
      continue;
    }
    // the half's max, then e^(z - m) and e^(z - m) (z - m) summed against it
    // (z - m is exact 0 at the max, which so adds exactly 1 and 0); masked
    // entries add exactly zero to both. Lane groups combine as
    // (g0 + g1) + (g2 + g3): each permlane swap leaves one operand pair in the
    // same order in all four lanes, so they agree bit for bit.
    float m = kNegInf;
#pragma unroll
    for (int i = 0; i < 32; ++i) m = fmaxf(m, z[i]);
    m = group_max(m);
    float sv = 0.f, uv = 0.f;
    if (full) {
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        const float x = z[i] - m;
        const float e = exp2_hw(x * kLog2e);
        sv = sv + e;
        uv = __builtin_fmaf(e, x, uv);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        float x = z[i] - m;
        float e = exp2_hw(x * kLog2e);
        if (z[i] == kNegInf) { x = 0.f; e = 0.f; }
        sv = sv + e;
        uv = __builtin_fmaf(e, x, uv);
      }
    }
    sv = group_sum(sv);
    uv = group_sum(uv);
    if (g == 0) {
      red_m[wv * BT + t_loc] = m;
      red_s[wv * BT + t_loc] = sv;
      red_u[wv * BT + t_loc] = uv;
    }
    // Token gather: the lane holding the row's token has tl = token - vlane
    // in [0, 128) with tl % 16 < 4 (entry z[4 (tl / 16) + tl % 16]). Rare, so
    // the 32-way select runs under a divergent branch.
    const int tok = row_ok ? (tok_lds != nullptr ? tok_lds[t_loc] : a.tokens[tg]) : -1;
    const int tl = (tok >= 0) ? (int)((int64_t)tok - vlane) : -1000000;
    if (tl >= 0 && tl < 128 && (tl & 15) < 4) {
      float zf = 0.f;
#pragma unroll
      for (int i = 0; i < 32; ++i)
        if ((i >> 2) * 16 + (i & 3) == tl) zf = z[i];
      zt_l[t_loc] = zf;
    }
  }
  if constexpr (DUMP) return;
  __syncthreads();

  // the tile's Partial: lower vocab half merged with the upper one
  if (wv == 0 && g == 0) {
#pragma unroll
    for (int bj = 0; bj < NJ; ++bj) {
      const int t_loc = wt * NTB * 32 + bj * 16 + c16;
      const int64_t tg = t0 + t_loc;
      if (tg >= rows) continue;
      const MSU h = merge2(MSU{red_m[t_loc], red_s[t_loc], red_u[t_loc]},
                           MSU{red_m[BT + t_loc], red_s[BT + t_loc], red_u[BT + t_loc]});
      const int tok = tok_lds != nullptr ? tok_lds[t_loc] : a.tokens[tg];
      const int64_t tv = (int64_t)tok - v0;
      Partial p;
      p.m = h.m;
      p.s = h.s;
      p.u = h.u;
      p.ztok = (tv >= 0 && tv < kVocabTile) ? zt_l[t_loc] : 0.f;
      a.part[tg * n_vt + vt] = p;
    }
  }
}

template <int NTB, int WT>
struct TileCtx {
  int vt;
  int64_t v0, t0;
  LoadPlan<NTB, WT> pl;
  rsrc_t wr, hr, tr;
};

template <int NTB, int WT>
__device__ __forceinline__ TileCtx<NTB, WT> make_tile(const LmHeadArgs& a, int lid, int n_vt, int n_tt, int wave,
                                                      int lane) {
  constexpr int BT = Tile<NTB, WT>::BT;
  // Opaque copies: every call recomputes its context instead of the compiler
  // reusing (and keeping live) the result of an earlier call.
  asm volatile("" : "+s"(lid));
  asm volatile("" : "+v"(lane));
  TileCtx<NTB, WT> c;
  int tt;
  tile_of_lid(lid, n_vt, n_tt, c.vt, tt);
  c.v0 = (int64_t)c.vt * kVocabTile;
  c.t0 = (int64_t)tt * BT;
  const int w_rows = (a.V - c.v0) < kVocabTile ? (int)(a.V - c.v0) : kVocabTile;
  const int h_rows = (a.rows - c.t0) < BT ? (int)(a.rows - c.t0) : BT;
  c.pl = make_load_plan<NTB, WT>(w_rows, h_rows, a.d, wave, lane);
  c.wr = make_rsrc((const __bf16*)a.w + c.v0 * a.d, (uint64_t)w_rows * a.d * 2);
  c.hr = make_rsrc((const __bf16*)a.hidden + c.t0 * a.d, (uint64_t)h_rows * a.d * 2);
  c.tr = make_rsrc(a.tokens + c.t0, (uint64_t)h_rows * 4);
  return c;
}

// Partials of a sequence of (vocab tile, row tile) output tiles. The logical
// tile ids are dealt to the 8 XCDs in contiguous chunks, and within an XCD
// round-robin to its workgroups, so at any time the workgroups of one XCD work
// on consecutive ids. With one workgroup per tile this is a plain launch; with
// a grid of one workgroup per CU it is persistent, and the stage pipeline then
// runs on across tiles: the last stages of a tile already request the next
// tile's first stages, which land while this tile's epilogue runs.
//
// Pipeline. Stage s of a tile (kKS hidden-dimension elements of its W and
// hidden-state rows) lives in LDS buffer s % kNBuf. Each stage has a boundary
// before its last k-step: every wave waits for its own reads of the stage and
// for its own DMA of stage s + 1, then the workgroup barrier makes stage s + 1
// visible and frees buffer s % kNBuf, which takes stage s + kNBuf, its loads
// spread over that last k-step. MFMA operands are read one k-step ahead,
// across the boundary too. Requests past the tile go to the next tile's
// stages, or, with none, re-read the tile's own stages into the freed buffer,
// so every boundary's wait counts stay the same.
template <int NTB, int WT, bool SPLITK4, bool DUMP>
__global__ __launch_bounds__(128 * WT, (Shape<NTB, WT, SPLITK4>::PER_CU))
void lmhead_partials(LmHeadArgs a, int n_vt, int n_tt) {
  using TL = Tile<NTB, WT>;
  using LP = LoadPlan<NTB, WT>;
  using TC = TileCtx<NTB, WT>;
  constexpr int kNBuf = Shape<NTB, WT, SPLITK4>::NBUF;
  static_assert((128 / kKS) % kNBuf == 0, "the stage count (a multiple of 128 / kKS) must be a multiple of kNBuf");
  constexpr int NJ = TL::NJ;
  constexpr int BT = TL::BT;
  constexpr int SB = TL::kStageBytes;
  constexpr int EPI = 7 * BT * 4;
  constexpr int L = LP::L;
  // Epilogue scratch of its own when it fits, so the next tile's stages can
  // land during the epilogue; otherwise it reuses the first stage buffer.
  constexpr bool kSep = kNBuf * SB + EPI + (DUMP ? 0 : 2 * BT * 4) <= (160 * 1024) / Shape<NTB, WT, SPLITK4>::PER_CU;
  // With its own scratch, the epilogue also finds the tile's tokens staged
  // in LDS (two slots, alternating per tile), requested with the tile's first
  // stage, so it never waits on a global load behind the next tile's stages.
  constexpr bool kTokLds = kSep && !DUMP;
  constexpr int TOKB = kTokLds ? 2 * BT * 4 : 0;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kNBuf * SB + (kSep ? EPI : 0) + TOKB];
  float* scratch = (float*)(kSep ? lds + kNBuf * SB : lds);
  int* tok_slot = (int*)(lds + kNBuf * SB + (kSep ? EPI : 0));  // [2][BT] when kTokLds
  int par = 0;

  const int lane0 = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wv = wave & 1, wt = wave >> 1;

  // this workgroup's tiles: start + wi, start + wi + w_x, ... below start + t_x
  const int n_tiles = n_vt * n_tt;
  const int x = blockIdx.x & 7, wi = blockIdx.x >> 3;
  const int w_x = (int)(gridDim.x >> 3) + (x < (int)(gridDim.x & 7) ? 1 : 0);
  const int tq = n_tiles >> 3, trm = n_tiles & 7;
  const int t_x = tq + (x < trm ? 1 : 0);
  const int start = x * tq + (x < trm ? x : trm);
  int j = wi;
  if (j >= t_x) return;

  const int nk = a.d / kKS;  // stages per tile; a multiple of kNBuf
  const int nk_q = nk / 4;   // stages per quarter (SPLITK4)
  constexpr int kStep = kKS * 2;

  TC cur = make_tile<NTB, WT>(a, start + j, n_vt, n_tt, wave, lane0);

  // prologue: the tile's tokens and stages 0 .. kNBuf - 1
  auto prologue = [&]() {
    if constexpr (kTokLds) request_tokens<BT>(tok_slot + par * BT, cur.tr, wave, lane0);
#pragma unroll
    for (int s = 0; s < kNBuf; ++s)
#pragma unroll
      for (int q = 0; q < L; ++q)
        request_load<NTB, WT>(lds + s * SB, cur.wr, cur.hr, cur.pl, wave, (s < nk ? s : nk - 1) * kStep, q);
    wait_vmem<(kNBuf - 1) * L>();  // stage 0 landed
    __syncthreads();
  };
  prologue();

  f32x4 acc[8][NJ];
  f32x4 sum[8][SPLITK4 ? NJ : 1];
  // One wave per SIMD (four waves) leaves registers for a second W operand set.
  constexpr bool kAD = TL::NW == 4 && Shape<NTB, WT, SPLITK4>::PER_CU == 1;
  bf16x8 fa[2][8];   // W operands by k-step parity (with kAD), else fa[0] refilled in place
  bf16x8 fb[2][NJ];  // hidden-state operands, double buffered by k-step parity
  while (true) {
    // Per-tile lane arithmetic is recomputed inside the loop rather than
    // hoisted out of it (which would keep it live across the whole loop and
    // push the epilogue into spills): the empty asm hides that the lane index
    // is loop-invariant.
    int lane = lane0;
    asm volatile("" : "+v"(lane));
    // The next tile's context is rebuilt where it is needed (cheap integer
    // work) rather than kept live across the loop.
    const bool has_next = j + w_x < t_x;
    const int next_lid = start + j + w_x;
#pragma unroll
    for (int bi = 0; bi < 8; ++bi)
#pragma unroll
      for (int bj = 0; bj < NJ; ++bj) acc[bi][bj] = f32x4{};

    // stage 0 has landed and is visible: after the prologue, or, when the
    // pipeline runs on from the previous tile, since its last boundary
#pragma unroll
    for (int bj = 0; bj < NJ; ++bj) fb[0][bj] = read_b<NTB>(lds, 0, bj, wt, lane);
#pragma unroll
    for (int bi = 0; bi < 8; ++bi) fa[0][bi] = read_a(lds, 0, bi, wv, lane);
    int k = 0;
    // steady state: every request is a stage of this tile
    for (; k + kNBuf < nk; ++k) {
      unsigned char* cb = lds + (k % kNBuf) * SB;
      region_a_prio();
      kstep<NTB, WT, 0, kAD, false>(fa, fb, acc, cb, cur.wr, cur.hr, cur.pl, 0, cb, 1, wave, wv, wt, lane);
      wait_lgkm0_vmem<(kNBuf - 2) * L>();
      stage_barrier();
      kstep<NTB, WT, 1, kAD, true>(fa, fb, acc, cb, cur.wr, cur.hr, cur.pl, (k + kNBuf) * kStep,
                                   lds + ((k + 1) % kNBuf) * SB, 0, wave, wv, wt, lane);
      if constexpr (SPLITK4) {
        if ((k + 1) % nk_q == 0) quarter_fold<NTB>(acc, sum, (k + 1) / nk_q - 1);
      }
    }
    // tail: the last kNBuf stages, whose requests reach past the tile: to the
    // next tile's first stages or, with no next tile (or no LDS to keep them
    // through the epilogue), to this tile's own stages again. Stage k sits in
    // buffer k % kNBuf = t, as the stage count is a multiple of kNBuf.
    {
      const TC nx = make_tile<NTB, WT>(a, (kSep && has_next) ? next_lid : start + j, n_vt, n_tt, wave, lane);
#pragma unroll
      for (int t = 0; t < kNBuf; ++t) {
        k = nk - kNBuf + t;
        unsigned char* cb = lds + t * SB;
        region_a_prio();
        kstep<NTB, WT, 0, kAD, false>(fa, fb, acc, cb, nx.wr, nx.hr, nx.pl, 0, cb, 1, wave, wv, wt, lane);
        wait_lgkm0_vmem<(kNBuf - 2) * L>();
        stage_barrier();
        // request k + kNBuf: stage t of the next tile (with its tokens)
        if constexpr (kTokLds) {
          if (t == 0) request_tokens<BT>(tok_slot + (par ^ 1) * BT, nx.tr, wave, lane);
        }
        if (t + 1 < kNBuf)
          kstep<NTB, WT, 1, kAD, true>(fa, fb, acc, cb, nx.wr, nx.hr, nx.pl, t * kStep, lds + (t + 1) * SB, 0,
                                       wave, wv, wt, lane);
        else
          kstep<NTB, WT, 1, kAD, true, false>(fa, fb, acc, cb, nx.wr, nx.hr, nx.pl, t * kStep, lds, 0, wave, wv,
                                              wt, lane);
        if constexpr (SPLITK4) {
          if ((k + 1) % nk_q == 0) quarter_fold<NTB>(acc, sum, (k + 1) / nk_q - 1);
        }
      }
    }
    if constexpr (SPLITK4) {
#pragma unroll
      for (int bi = 0; bi < 8; ++bi)
#pragma unroll
        for (int bj = 0; bj < NJ; ++bj) acc[bi][bj] = sum[bi][bj];
    }
    if constexpr (!kSep) {
      wait_vmem<0>();  // every request landed: the epilogue reuses the first buffer
      __syncthreads();
    }
    tile_epilogue<NTB, WT, DUMP>(a, n_vt, cur.vt, cur.v0, cur.t0, acc, scratch,
                                 kTokLds ? tok_slot + par * BT : nullptr, wave, lane);
    par ^= 1;
    if (!has_next) break;
    j += w_x;
    cur = make_tile<NTB, WT>(a, next_lid, n_vt, n_tt, wave, lane);
    if constexpr (!kSep) {
      __syncthreads();  // the epilogue's reads of the first buffer are done
      prologue();
    }
  }
  wait_vmem<0>();  // no global->LDS request may outlive the workgroup
}

// ---------------------------------------------------------------- merge

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

// Compute units of the current device (cached per device).
static int device_cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
  static int cache[64] = {0};
  if (dev < 64 && cache[dev] > 0) return cache[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (dev < 64) cache[dev] = n;
  return n;
}

template <int NTB, int WT, bool SPLITK4, bool DUMP>
static hipError_t launch_partials_t(const LmHeadArgs& a, bool persistent, hipStream_t s) {
  const int n_vt = n_vocab_tiles(a.V);
  constexpr int BT = Tile<NTB, WT>::BT;
  const int64_t n_tt = (a.rows + BT - 1) / BT;
  const int64_t nblk = n_tt * n_vt;
  if (nblk > 0x7fffffff) return hipErrorInvalidValue;
  int64_t grid = nblk;
  if (persistent) {
    const int64_t resident = (int64_t)device_cu_count() * Shape<NTB, WT, SPLITK4>::PER_CU;
    if (resident > 0 && resident < grid) grid = resident;
  }
  hipLaunchKernelGGL((lmhead_partials<NTB, WT, SPLITK4, DUMP>), dim3((unsigned)grid), dim3(128 * WT), 0,
                     s, a, n_vt, (int)n_tt);
  return hipGetLastError();
}

hipError_t launch_partials(const LmHeadArgs& a, int rows_per_wg, bool splitk4, hipStream_t s) {
  const bool dump = a.logits != nullptr;
  if (splitk4)  // a second accumulator set: 64-row tiles of 4 waves
    return dump ? launch_partials_t<1, 2, true, true>(a, false, s) : launch_partials_t<1, 2, true, false>(a, false, s);
  switch (rows_per_wg) {
    case 64: return dump ? launch_partials_t<1, 2, false, true>(a, false, s) : launch_partials_t<1, 2, false, false>(a, false, s);
    case 128: return dump ? launch_partials_t<2, 2, false, true>(a, false, s) : launch_partials_t<2, 2, false, false>(a, false, s);
    default: {
      const bool pers = TIM_PERSISTENT != 0;
#if TIM_WIDE_WAVES
      return dump ? launch_partials_t<2, 4, false, true>(a, pers, s) : launch_partials_t<2, 4, false, false>(a, pers, s);
#else
      return dump ? launch_partials_t<4, 2, false, true>(a, pers, s) : launch_partials_t<4, 2, false, false>(a, pers, s);
#endif
    }
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
