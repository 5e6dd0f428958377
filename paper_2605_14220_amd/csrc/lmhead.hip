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

// Compile-time pipeline shape. None of these changes the arithmetic: the
// hidden dimension is accumulated in the same ascending 16-element MFMA steps
// whatever the stage depth, buffer count, LDS swizzle or tile order.
#ifndef TIM_KSTAGE
#define TIM_KSTAGE 64      // hidden-dimension elements per LDS stage (32 or 64)
#endif
#ifndef TIM_NBUF
#define TIM_NBUF 2         // LDS stage buffers (>= 2)
#endif
#ifndef TIM_SWZ_SHIFT     // LDS XOR swizzle: chunk ^= (row >> shift) & (chunks - 1); these
#if TIM_KSTAGE == 64       // shifts make the 16 lanes of each ds_read_b128 phase hit 16
#define TIM_SWZ_SHIFT 1    // distinct 16-byte bank groups of the 64 banks
#else
#define TIM_SWZ_SHIFT 2
#endif
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
#ifndef TIM_TRAIN_ROWS
#define TIM_TRAIN_ROWS 256 // row tile of full-size launches: 256 (one workgroup per CU) or 128 (two)
#endif
#ifndef TIM_WIDE_WAVES
#define TIM_WIDE_WAVES 1   // 256-row tiles: 8 waves of 128x64 (2 per SIMD); 0 = 4 waves of 128x128
#endif

constexpr int kKS = TIM_KSTAGE;
constexpr int kRowBytes = kKS * 2;       // bytes of one row in one stage
constexpr int kChunks = kRowBytes / 16;  // 16-byte chunks per row per stage
constexpr int kSteps = kKS / 16;         // MFMA k-steps per stage
constexpr int kWBytes = kVocabTile * kRowBytes;
static_assert(kKS == 32 || kKS == 64, "stage depth");
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

// Workgroup shape: 2 waves along the vocab tile (128 entries each) times WT
// waves along the rows, each wave holding NTB blocks of 32 rows.
template <int NTB, int WT>
struct Tile {
  static constexpr int NW = 2 * WT;            // waves per workgroup
  static constexpr int BT = WT * NTB * 32;     // rows per workgroup
  static constexpr int kHBytes = BT * kRowBytes;
  static constexpr int kStageBytes = kWBytes + kHBytes;
};

// Residency and pipeline depth of one kernel shape. Shapes whose wave holds
// at most 128 x 64 accumulators (and no second accumulator set) are built to
// run two workgroups per CU -- two waves per SIMD from independent
// workgroups, so one workgroup's barrier stalls and epilogue overlap the
// other's MFMA stream -- and then get as many LDS stage buffers as fit in
// half of the 160 KB LDS.
template <int NTB, int WT, bool SPLITK4>
struct Shape {
  using TL = Tile<NTB, WT>;
  static constexpr int PER_CU =
      (WT == 2 && NTB <= 2 && !SPLITK4 && (80 * 1024) / TL::kStageBytes >= 2) ? 2 : 1;
  static constexpr int FIT = (160 * 1024 / PER_CU) / TL::kStageBytes;
  static constexpr int NBUF = FIT < TIM_NBUF ? FIT : TIM_NBUF;
  static_assert(NBUF >= 2, "double buffering at least");
};

// 16-byte chunk c of row r sits at physical chunk c ^ swz(r) of that row.
__device__ __forceinline__ int swz(int r) { return (r >> TIM_SWZ_SHIFT) & (kChunks - 1); }

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

// Workgroup barrier between pipeline stages. Each wave has already waited
// for what the barrier must order (its own DMA of the next stage, and its own
// reads of the buffer about to be refilled), so no memory fence is needed;
// the empty asm statements keep the compiler from moving memory operations
// across it.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

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

// Per-lane byte offsets of this workgroup's DMA loads, relative to the tile's
// first row at hidden index 0. They do not change along the hidden dimension:
// each stage only moves the scalar offset.
template <int NTB, int WT>
struct LoadPlan {
  static constexpr int NW = Tile<NTB, WT>::NW;
  static constexpr int WB = 4 * kChunks / NW;                       // W blocks of 1 KB per wave
  static constexpr int HB = Tile<NTB, WT>::BT * kChunks / (64 * NW);  // hidden-state blocks per wave
  static constexpr int L = WB + HB;                          // DMA loads per wave per stage
  uint32_t w_off[WB];
  uint32_t h_off[HB];
};

template <int NTB, int WT>
__device__ __forceinline__ LoadPlan<NTB, WT> make_load_plan(int w_rows, int h_rows, int d, int wave,
                                                        int lane) {
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

template <int NTB, int WT>
__device__ __forceinline__ void load_stage(unsigned char* buf, rsrc_t wr, rsrc_t hr,
                                           const LoadPlan<NTB, WT>& pl, int wave, int soff) {
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
  for (int q = 0; q < LoadPlan<NTB, WT>::WB; ++q)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        wr, (lds_void*)(buf + (wave * LoadPlan<NTB, WT>::WB + q) * 1024), 16, pl.w_off[q], soff, 0,
        TIM_LOAD_AUX);
#pragma unroll
  for (int q = 0; q < LoadPlan<NTB, WT>::HB; ++q)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        hr, (lds_void*)(buf + kWBytes + (wave * LoadPlan<NTB, WT>::HB + q) * 1024), 16, pl.h_off[q],
        soff, 0, TIM_LOAD_AUX);
#endif
}

// MFMA operands of one k-step: 4 W fragments (128 vocab rows) and NTB
// hidden-state fragments (NTB * 32 rows), 8 bf16 per lane each.
template <int NTB>
struct Frags {
  bf16x8 a[4];
  bf16x8 b[NTB];
};

template <int NTB>
__device__ __forceinline__ void load_frags(const unsigned char* buf, int s, Frags<NTB>& f,
                                           int wv, int wt, int lane) {
  const int r32 = lane & 31, hi = lane >> 5;
  const int c = ((2 * s + hi) ^ swz(r32)) * 16;  // every operand row is (multiple of 32) + r32
#pragma unroll
  for (int bb = 0; bb < 4; ++bb)
    f.a[bb] = *(const bf16x8*)(buf + (wv * 128 + bb * 32 + r32) * kRowBytes + c);
#pragma unroll
  for (int j = 0; j < NTB; ++j)
    f.b[j] = *(const bf16x8*)(buf + kWBytes + (wt * NTB * 32 + j * 32 + r32) * kRowBytes + c);
}

// Scheduling hints for one region of the main loop: spread NV vector-memory
// loads and ND LDS reads among the NM MFMAs (one load and one read after each
// MFMA while they last), so that no burst of loads backs up the vector-memory
// queue behind which a wave's next MFMA would wait.
template <int NM, int NV, int ND>
__device__ __forceinline__ void interleave() {
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // 1 MFMA
    if (i < NV) __builtin_amdgcn_sched_group_barrier(0x010, 1, 0);  // 1 VMEM
    if (i < ND) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // 1 DS read
  }
}

template <int NTB>
__device__ __forceinline__ void mma(const Frags<NTB>& f, f32x16 (&acc)[4][NTB]) {
#pragma unroll
  for (int bb = 0; bb < 4; ++bb)
#pragma unroll
    for (int j = 0; j < NTB; ++j)
      acc[bb][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[bb], f.b[j], acc[bb][j], 0, 0, 0);
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

// One tile's per-row results from its accumulators (see the file comment):
// phase A scales, masks and finds each row's tile max and gathers the token's
// logit, phase B sums against that max, phase C combines the two vocab waves
// and stores one Partial per row. `scratch` holds 7 * BT floats of LDS.
template <int NTB, int WT, bool DUMP>
__device__ __forceinline__ void tile_epilogue(const LmHeadArgs& a, int n_vt, int vt, int64_t v0, int64_t t0,
                                              f32x16 (&acc)[4][NTB], float* scratch, int wave, int lane) {
  constexpr int BT = Tile<NTB, WT>::BT;
  const int wv = wave & 1, wt = wave >> 1;
  const int V = a.V;
  const int64_t rows = a.rows;
  const int hi = lane >> 5, r32 = lane & 31;
  const float inv_tau = a.inv_tau;
  // lane's vocab offset inside the tile for (block bb, register r):
  //   wv*128 + bb*32 + 8*(r>>2) + 4*hi + (r&3)
  const int64_t vlane = v0 + wv * 128 + 4 * hi;
  float* red_m = scratch;                // [2][BT]
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

  // Phase A: temperature (z = acc * inv_tau, written back in place so every
  // later use reads the same bits; a multiply by exactly 1 is skipped, which
  // changes nothing), vocabulary mask (tail tile only: entries past V become
  // -inf) and the row's max over the tile. Whether a tile is the tail depends
  // only on (v0, V), so a tile takes the same path in every launch shape.
  const bool full = v0 + kVocabTile <= V;
  if (inv_tau != 1.0f) {
#pragma unroll
    for (int j = 0; j < NTB; ++j)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[bb][j][r] = acc[bb][j][r] * inv_tau;
  }
  if (!full) {
#pragma unroll
    for (int j = 0; j < NTB; ++j)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (vlane + (bb * 32 + 8 * (r >> 2) + (r & 3)) >= V) acc[bb][j][r] = kNegInf;
  }
#pragma unroll
  for (int j = 0; j < NTB; ++j) {
    float mx = kNegInf;
#pragma unroll
    for (int bb = 0; bb < 4; ++bb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, acc[bb][j][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const int t_loc = wt * NTB * 32 + j * 32 + r32;
    if (hi == 0) red_m[wv * BT + t_loc] = mx;
    // Token gather: the row's token lies in this lane's 64 entries only for
    // offsets tl in [0, 128) with bit 2 clear (the other lane half holds the
    // rest). Rare, so the 64-way select runs under a divergent branch.
    const int tl = tok_loc[j];
    if (tl >= 0 && tl < 128 && ((tl >> 2) & 1) == 0) {
      float zf = 0.f;
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (bb * 32 + 8 * (r >> 2) + (r & 3) == tl) zf = acc[bb][j][r];
      zt_l[t_loc] = zf;
    }
    if constexpr (DUMP) {
      const int64_t tg = t0 + t_loc;
      if (row_ok[j]) {
#pragma unroll
        for (int bb = 0; bb < 4; ++bb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int64_t v = vlane + bb * 32 + 8 * (r >> 2) + (r & 3);
            if (v < V) a.logits[tg * (int64_t)V + v] = acc[bb][j][r];
          }
      }
    }
  }
  if constexpr (DUMP) return;
  __syncthreads();

  // Phase B: s = sum e^(z - M) and u = sum e^(z - M) (z - M) against the
  // tile max M, in fixed (bb, r) order. In the tail tile the masked entries
  // add exactly zero to both, so valid entries see the same arithmetic as in
  // a full tile.
#pragma unroll
  for (int j = 0; j < NTB; ++j) {
    const int t_loc = wt * NTB * 32 + j * 32 + r32;
    const float M = fmaxf(red_m[t_loc], red_m[BT + t_loc]);
    float s = 0.f, u = 0.f;
    if (full) {
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float x = acc[bb][j][r] - M;
          const float e = exp2_hw(x * kLog2e);
          s = s + e;
          u = __builtin_fmaf(e, x, u);
        }
    } else {
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float z = acc[bb][j][r];
          float x = z - M;
          float e = exp2_hw(x * kLog2e);
          if (z == kNegInf) { x = 0.f; e = 0.f; }
          s = s + e;
          u = __builtin_fmaf(e, x, u);
        }
    }
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

template <int NTB, int WT>
struct TileCtx {
  int vt;
  int64_t v0, t0;
  LoadPlan<NTB, WT> pl;
  rsrc_t wr, hr;
};

template <int NTB, int WT>
__device__ __forceinline__ TileCtx<NTB, WT> make_tile(const LmHeadArgs& a, int lid, int n_vt, int n_tt,
                                                      int wave, int lane) {
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
  return c;
}

// Partials of a sequence of (vocab tile, row tile) output tiles. The logical
// tile ids are dealt to the 8 XCDs in contiguous chunks, and within an XCD
// round-robin to its workgroups, so at any time the workgroups of one XCD work
// on consecutive ids. With one workgroup per tile this is a plain launch; with
// a grid of one workgroup per CU it is persistent, and the stage pipeline then
// runs on across tiles: the last stage boundaries of a tile already request
// the next tile's first stages, which land while this tile's epilogue runs.
template <int NTB, int WT, bool SPLITK4, bool DUMP>
__global__ __launch_bounds__(128 * WT, (Shape<NTB, WT, SPLITK4>::PER_CU))
void lmhead_partials(LmHeadArgs a, int n_vt, int n_tt) {
  using TL = Tile<NTB, WT>;
  using LP = LoadPlan<NTB, WT>;
  using TC = TileCtx<NTB, WT>;
  constexpr int kNBuf = Shape<NTB, WT, SPLITK4>::NBUF;
  constexpr int BT = TL::BT;
  constexpr int SB = TL::kStageBytes;
  constexpr int EPI = 7 * BT * 4;
  // Epilogue scratch of its own when it fits, so the next tile's stages can
  // land during the epilogue; otherwise it reuses the first stage buffer.
  constexpr bool kSep = kNBuf * SB + EPI <= (160 * 1024) / Shape<NTB, WT, SPLITK4>::PER_CU;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kNBuf * SB + (kSep ? EPI : 0)];
  float* scratch = (float*)(kSep ? lds + kNBuf * SB : lds);

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

#pragma unroll
  for (int s = 0; s < kNBuf; ++s)
    load_stage<NTB, WT>(lds + s * SB, cur.wr, cur.hr, cur.pl, wave, (s < nk ? s : nk - 1) * kStep);

  f32x16 acc[4][NTB];
  f32x16 sum[4][SPLITK4 ? NTB : 1];
  Frags<NTB> f[2];
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
    for (int bb = 0; bb < 4; ++bb)
#pragma unroll
      for (int jj = 0; jj < NTB; ++jj) acc[bb][jj] = f32x16{};

    // Stage s of a tile lives in buffer s % kNBuf. Stage k + kNBuf is
    // requested at the boundary of stage k, right after the barrier that shows
    // every wave done with stage k's buffer and stage k + 1 landed. Requests
    // past the tile's end go to the next tile, else re-read the last stage
    // (a buffer nobody reads again), so every boundary issues the same loads
    // and the wait counts stay uniform. MFMA operands are read one k-step
    // ahead, across the stage boundary too.
    wait_vmem<(kNBuf - 1) * LP::L>();
    __syncthreads();
    load_frags<NTB>(lds, 0, f[0], wv, wt, lane);
    int k = 0;
    // steady state: every request is a stage of this tile
    for (; k + kNBuf < nk; ++k) {
      unsigned char* cb = lds + (k % kNBuf) * SB;
#pragma unroll
      for (int s = 0; s + 1 < kSteps; ++s) {
        load_frags<NTB>(cb, s + 1, f[(s + 1) & 1], wv, wt, lane);
        mma<NTB>(f[s & 1], acc);
      }
      interleave<4 * NTB * (kSteps - 1), 0, (4 + NTB) * (kSteps - 1)>();
      wait_lgkm0_vmem<(kNBuf - 2) * LP::L>();
      stage_barrier();
      load_stage<NTB, WT>(cb, cur.wr, cur.hr, cur.pl, wave, (k + kNBuf) * kStep);
      load_frags<NTB>(lds + ((k + 1) % kNBuf) * SB, 0, f[kSteps & 1], wv, wt, lane);
      mma<NTB>(f[(kSteps - 1) & 1], acc);
      interleave<4 * NTB, LP::L, 4 + NTB>();
      if constexpr (SPLITK4) {
        if ((k + 1) % nk_q == 0) quarter_fold<NTB>(acc, sum, (k + 1) / nk_q - 1);
      }
    }
    // tail (at most kNBuf - 1 boundaries): requests go to the next tile's
    // first stages, or re-read this tile's last stage when there is none
    for (; k + 1 < nk; ++k) {
      unsigned char* cb = lds + (k % kNBuf) * SB;
#pragma unroll
      for (int s = 0; s + 1 < kSteps; ++s) {
        load_frags<NTB>(cb, s + 1, f[(s + 1) & 1], wv, wt, lane);
        mma<NTB>(f[s & 1], acc);
      }
      wait_lgkm0_vmem<(kNBuf - 2) * LP::L>();
      stage_barrier();
      if (kSep && has_next) {
        const TC nx = make_tile<NTB, WT>(a, next_lid, n_vt, n_tt, wave, lane);
        load_stage<NTB, WT>(cb, nx.wr, nx.hr, nx.pl, wave, (k + kNBuf - nk) * kStep);
      } else {
        load_stage<NTB, WT>(cb, cur.wr, cur.hr, cur.pl, wave, (nk - 1) * kStep);
      }
      load_frags<NTB>(lds + ((k + 1) % kNBuf) * SB, 0, f[kSteps & 1], wv, wt, lane);
      mma<NTB>(f[(kSteps - 1) & 1], acc);
      if constexpr (SPLITK4) {
        if ((k + 1) % nk_q == 0) quarter_fold<NTB>(acc, sum, (k + 1) / nk_q - 1);
      }
    }
    {  // last stage: no boundary
      const unsigned char* cb = lds + (k % kNBuf) * SB;
#pragma unroll
      for (int s = 0; s + 1 < kSteps; ++s) {
        load_frags<NTB>(cb, s + 1, f[(s + 1) & 1], wv, wt, lane);
        mma<NTB>(f[s & 1], acc);
      }
      mma<NTB>(f[(kSteps - 1) & 1], acc);
    }
    if constexpr (SPLITK4) {
      quarter_fold<NTB>(acc, sum, 3);
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
#pragma unroll
        for (int jj = 0; jj < NTB; ++jj) acc[bb][jj] = sum[bb][jj];
    }
    if constexpr (kSep) {
      // the last stage's buffer takes the next tile's stage kNBuf - 1
      wait_lgkm0_vmem<63>();
      stage_barrier();
      if (has_next) {
        const TC nx = make_tile<NTB, WT>(a, next_lid, n_vt, n_tt, wave, lane);
        load_stage<NTB, WT>(lds + ((nk - 1) % kNBuf) * SB, nx.wr, nx.hr, nx.pl, wave, (kNBuf - 1) * kStep);
      }
    } else {
      wait_vmem<0>();   // every request landed: the epilogue reuses the first buffer
      __syncthreads();
    }
    tile_epilogue<NTB, WT, DUMP>(a, n_vt, cur.vt, cur.v0, cur.t0, acc, scratch, wave, lane);
    if (!has_next) break;
    j += w_x;
    cur = make_tile<NTB, WT>(a, next_lid, n_vt, n_tt, wave, lane);
    if constexpr (!kSep) {
      __syncthreads();  // the epilogue's reads of the first buffer are done
#pragma unroll
      for (int s = 0; s < kNBuf; ++s)
        load_stage<NTB, WT>(lds + s * SB, cur.wr, cur.hr, cur.pl, wave, (s < nk ? s : nk - 1) * kStep);
    }
  }
  wait_vmem<0>();  // no global->LDS request may outlive the workgroup
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
  if (splitk4) {  // a second accumulator set: at most 128 rows, 4 waves
    if (rows_per_wg >= 128)
      return dump ? launch_partials_t<2, 2, true, true>(a, false, s) : launch_partials_t<2, 2, true, false>(a, false, s);
    return dump ? launch_partials_t<1, 2, true, true>(a, false, s) : launch_partials_t<1, 2, true, false>(a, false, s);
  }
  switch (rows_per_wg) {
    case 64: return dump ? launch_partials_t<1, 2, false, true>(a, false, s) : launch_partials_t<1, 2, false, false>(a, false, s);
    case 128: return dump ? launch_partials_t<2, 2, false, true>(a, false, s) : launch_partials_t<2, 2, false, false>(a, false, s);
    default: {
      const bool pers = TIM_PERSISTENT != 0;
#if TIM_TRAIN_ROWS == 128
      return dump ? launch_partials_t<2, 2, false, true>(a, pers, s) : launch_partials_t<2, 2, false, false>(a, pers, s);
#elif TIM_WIDE_WAVES
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
