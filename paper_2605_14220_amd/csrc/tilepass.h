// Tile pass on gfx950 (CDNA4) MFMA: the contraction engine shared by the LM
// head forward and its backward.
//
// A pass computes output tiles C[i][j] = sum_k A[i][k] B[j][k] over two
// bf16 row-major operands with K contiguous (A [a_rows, K] in tiles of 256
// rows, or 128 for the half-tile shape of decode batches, B [b_rows, K] in
// tiles of the workgroup's row tile) on
// v_mfma_f32_16x16x32_bf16 with fp32 accumulation, K in ascending 32-element
// steps and one accumulation chain per output element: an element's value
// depends only on its own A row, B row and K, never on how many rows share a
// launch, on their position or on the launch grid. A is the MFMA's first
// operand: a lane's 4 accumulator registers of a 16x16 block hold 4
// consecutive A rows of ONE B row. Of the two MFMA shapes with the full bf16
// rate, this one moves fewer accumulator bytes per flop and sustains a higher
// clock under the card's power limit.
//
// Operands are staged HBM -> LDS with direct global->LDS DMA loads
// (buffer_load_dwordx4 into LDS), double buffered, XOR-swizzled against LDS
// bank conflicts; the epilogue policy of the pass decides what becomes of each
// finished tile (softmax partials, logit gradients, plain fp32 stores).
#pragma once

#include <atomic>

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

// Launch and pipeline shape. None of these changes the arithmetic: the
// hidden dimension is accumulated in the same ascending 32-element MFMA steps
// whatever the buffer count, LDS swizzle or tile order.
constexpr int kMaxNBuf = 2;     // LDS stage buffers per workgroup (a power of two, as many as fit up to this)
constexpr int kGroupV = 4;      // vocab tiles per group in the LM head's workgroup -> tile order
constexpr int kStoreGroup = 8;  // A tiles per group in the tile order of the plain products

constexpr int kKS = 64;                  // hidden-dimension elements per LDS stage
constexpr int kRowBytes = kKS * 2;       // bytes of one row in one stage
constexpr int kChunks = kRowBytes / 16;  // 16-byte chunks per row per stage
constexpr int kKM = 32;                  // hidden-dimension elements per MFMA
constexpr int kSteps = kKS / kKM;        // MFMA k-steps per stage
static_assert(kSteps == 2, "the operand double buffer alternates once per k-step");
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

// Workgroup shape: NV waves along the A tile (128 entries, 8 blocks of 16,
// each; NV = 2 covers a vocabulary tile, NV = 1 one half of it) times WT waves
// along the rows, each wave holding NTB * 32 rows (2 * NTB blocks of 16).
template <int NTB, int WT, int NV = 2>
struct Tile {
  static constexpr int NW = NV * WT;           // waves per workgroup
  static constexpr int NJ = 2 * NTB;           // row blocks of 16 per wave
  static constexpr int BT = WT * NTB * 32;     // rows per workgroup
  static constexpr int TA = 128 * NV;          // A-tile rows per workgroup
  static constexpr int kWB = TA * kRowBytes;
  static constexpr int kHBytes = BT * kRowBytes;
  static constexpr int kStageBytes = kWB + kHBytes;
};

// Residency and pipeline depth of one kernel shape. Shapes whose wave holds
// at most 128 x 64 accumulators (and no second accumulator set) run two
// workgroups per CU when two stage buffers fit in half of the 160 KB LDS;
// half-tile shapes (NV = 1) as many as fit with two buffers each, up to 3.
template <int NTB, int WT, bool SPLITK4, int NV = 2>
struct Shape {
  using TL = Tile<NTB, WT, NV>;
  static constexpr int FIT2 = (160 * 1024) / (2 * TL::kStageBytes);
  static constexpr int PER_CU =
      NV == 1 ? (FIT2 >= 3 ? 3 : FIT2)
              : ((WT == 2 && NTB <= 2 && !SPLITK4 && (80 * 1024) / TL::kStageBytes >= 2) ? 2 : 1);
  static constexpr int FIT = (160 * 1024 / PER_CU) / TL::kStageBytes;
  static constexpr int CAP = FIT < kMaxNBuf ? FIT : kMaxNBuf;
  // a power of two, so that it divides the stage count
  static constexpr int NBUF = CAP >= 8 ? 8 : CAP >= 4 ? 4 : 2;
  static_assert(FIT >= 2, "double buffering at least");
};

// 16-byte chunk c of row r sits at physical chunk c ^ swz(r) of that row. A
// ds_read_b128 serves 16 lanes per cycle; its 16 lanes read 16 consecutive
// rows at one logical chunk, and with 128-byte rows this swizzle puts them in
// 16 distinct 16-byte bank groups of the 64 banks.
__device__ __forceinline__ int swz(int r) { return (r >> 1) & (kChunks - 1); }

// Packed operand layout, for operands the library writes itself (the
// backward's transposed copies and its logit gradients): an operand [R, K]
// (R a multiple of 256, K of KS) is stored tile by tile of 256 rows and, in a
// tile, stage by stage, each 256 x KS block exactly as a stage's DMA lays it
// out in LDS (row r at r * 2 KS bytes, its logical 16-byte chunk c at physical
// chunk c ^ swz_ks<KS>(r)). Block (tile i, stage s) starts at element
// (i * K / KS + s) * 256 KS, so a stage of a tile is 512 KS bytes of
// consecutive memory and every DMA load of it reads 1 KB of consecutive bytes;
// the row-major layout's stage reads 2 KS bytes from each of 256 rows far
// apart. KS = 64 for the two-buffer tile pass, 32 for the deep pass below.
constexpr int kPackRows = 256;
// With 2 KS-byte rows, a ds_read_b128's 16 consecutive rows at one logical
// chunk land in 16 distinct 16-byte bank groups: rows 2 apart (KS = 64) or 4
// apart (KS = 32) share a bank line and take different chunks.
template <int KS>
__device__ __forceinline__ int swz_ks(int r) {
  return KS == 64 ? swz(r) : (r >> 2) & 3;
}
template <int KS = kKS>
__device__ __forceinline__ int64_t packed_index(int64_t r, int64_t k, int64_t K) {
  const int rr = (int)(r & (kPackRows - 1));
  const int kk = (int)(k & (KS - 1));
  const int64_t block = (r / kPackRows) * (K / KS) + k / KS;
  return block * (kPackRows * KS) + rr * KS + ((((kk >> 3) ^ swz_ks<KS>(rr)) << 3) | (kk & 7));
}

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

// Tile order: logical id -> (A tile, B tile), walking groups of GV A tiles
// with the B tiles outer and the A tiles inner, so that the workgroups
// resident on one XCD at a time (consecutive logical ids, see tile_pass) share
// A tiles and B tiles through that XCD's L2.
template <int GV>
__device__ __forceinline__ void tile_of_lid(int lid, int n_vt, int n_tt, int& vt, int& tt) {
  const int group = lid / (GV * n_tt);
  const int first = group * GV;
  const int gv = (n_vt - first) < GV ? (n_vt - first) : GV;
  const int local = lid - group * GV * n_tt;
  vt = first + local % gv;
  tt = local / gv;
}

// Operands of one tile pass, C[i][j] = sum_k A[i][k] B[j][k] over A [a_rows, K]
// and B [b_rows, K], bf16, row-major with row stride K. The A tile is 128 NV
// rows (256: the vocabulary tile of the LM head) and the B tile the
// workgroup's row tile.
struct TileOps {
  const void* a;
  const void* b;
  const int32_t* tokens;  // [b_rows], staged in LDS per tile when the epilogue takes them
  const void* coef;       // [b_rows] 16-byte words, staged likewise
  int64_t b_rows;
  int32_t a_rows;
  int32_t K;
};

// Per-lane byte offsets of this wave's DMA loads, relative to the tile's
// first row at hidden index 0. They do not change along the hidden dimension
// (each stage only moves the scalar offset) nor from tile to tile (the tile is
// the buffer resource's base), so one plan serves the whole pass. Row-major
// operands: rows past an operand's end (a tail tile) lie outside its
// resource's range, checked on these per-lane offsets, so their loads return
// zeros: entries the epilogue masks (past V) or rows it never writes (past the
// batch). Packed operands (PK): the offset is the lane's place in the stage
// block, which is its place in LDS.
template <int NTB, int WT, int NV = 2>
struct LoadPlan {
  static constexpr int NW = Tile<NTB, WT, NV>::NW;
  static constexpr int WB = Tile<NTB, WT, NV>::TA * kChunks / (64 * NW);  // W blocks of 1 KB per wave
  static constexpr int HB = Tile<NTB, WT, NV>::BT * kChunks / (64 * NW);  // hidden-state blocks per wave
  static constexpr int L = WB + HB;                                   // DMA loads per wave per stage
  uint32_t w_off[WB];
  uint32_t h_off[HB];
};

template <int NTB, int WT, int NV = 2, bool PK = false>
__device__ __forceinline__ LoadPlan<NTB, WT, NV> make_load_plan(int d, int wave, int lane) {
  LoadPlan<NTB, WT, NV> pl;
#pragma unroll
  for (int q = 0; q < LoadPlan<NTB, WT, NV>::WB; ++q) {
    const int p = (wave * LoadPlan<NTB, WT, NV>::WB + q) * 64 + lane;
    const int r = p / kChunks;
    const int c = (p % kChunks) ^ swz(r);
    pl.w_off[q] = PK ? (uint32_t)p * 16u : (uint32_t)(r * d + c * 8) * 2u;
  }
#pragma unroll
  for (int q = 0; q < LoadPlan<NTB, WT, NV>::HB; ++q) {
    const int p = (wave * LoadPlan<NTB, WT, NV>::HB + q) * 64 + lane;
    const int r = p / kChunks;
    const int c = (p % kChunks) ^ swz(r);
    pl.h_off[q] = PK ? (uint32_t)p * 16u : (uint32_t)(r * d + c * 8) * 2u;
  }
  return pl;
}

// This lane's index in its wave, counted afresh at each use rather than kept
// live across the pass (where register pressure would spill it, and a spill's
// reload waits for every DMA load in flight): the mask goes through an empty
// asm, so the count cannot be hoisted out of a loop.
__device__ __forceinline__ int lane_index() {
  unsigned m = ~0u;
  asm volatile("" : "+s"(m));
  return (int)__builtin_amdgcn_mbcnt_hi(m, __builtin_amdgcn_mbcnt_lo(m, 0u));
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
template <int NTB, int WT, int NV = 2>
__device__ __forceinline__ void request_load(unsigned char* buf, rsrc_t wr, rsrc_t hr,
                                             const LoadPlan<NTB, WT, NV>& pl, int wave, int soff, int q) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int WB = LoadPlan<NTB, WT, NV>::WB;
  constexpr int L = LoadPlan<NTB, WT, NV>::L;
  constexpr int kWB = Tile<NTB, WT, NV>::kWB;
  if (q < WB)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void*)(buf + (wave * WB + q) * 1024), 16, pl.w_off[q], soff, 0,
                                             0);
  else
    __builtin_amdgcn_raw_ptr_buffer_load_lds(hr, (lds_void*)(buf + kWB + (wave * (L - WB) + (q - WB)) * 1024), 16,
                                             pl.h_off[q - WB], soff, 0, 0);
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

// The tile's BT 16-byte row words into LDS, 1 KB per wave from the first
// BT / 64 waves (rows past the batch read as 0 and are never used).
template <int BT>
__device__ __forceinline__ void request_coef(f32x4* dst, rsrc_t cr, int wave, int lane) {
#if defined(__HIP_DEVICE_COMPILE__)
  if (wave < BT / 64)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(cr, (lds_void*)(dst + wave * 64), 16, (uint32_t)(wave * 64 + lane) * 16u,
                                             0, 0, 0);
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
template <int NTB, int NV = 2>
__device__ __forceinline__ bf16x8 read_b(const unsigned char* buf, int s, int bj, int wt, int lane) {
  return read_operand(buf + 128 * NV * kRowBytes, wt * NTB * 32 + bj * 16 + (lane & 15), s, lane);
}

// One k-step as 8 * NJ scheduling units, each pinned on its own: unit i
// issues the MFMA of W block bi = i / NJ and row block bj = i % NJ (the
// accumulation order of every logit is the k-step order; the order of the
// units only interleaves independent chains), then, with LOAD, its share of
// the DMA loads of a stage request into `lb` (spread evenly over the units,
// or with SP > 0 one every SP units from the first), and, with READ, the
// reads of k-step `rs` of buffer `rb`. Operands alternate between two register sets by
// k-step parity P: the row-block operands always, read from the first units
// on; the W operands too with AD (then read right after the row blocks, so
// every read lands early), else the single W set is refilled block by block
// right after each block's last use here.
template <int NTB, int WT, int P, bool AD, bool LOAD, bool READ = true, int NV = 2, int SP = 0>
__device__ __forceinline__ void kstep(bf16x8 (&fa)[2][8], bf16x8 (&fb)[2][2 * NTB], f32x4 (&acc)[8][2 * NTB],
                                      unsigned char* lb, rsrc_t wr, rsrc_t hr, const LoadPlan<NTB, WT, NV>& pl,
                                      int soff, const unsigned char* rb, int rs, int wave, int wv, int wt, int lane) {
  constexpr int NJ = 2 * NTB;
  constexpr int NM = 8 * NJ;
  constexpr int L = LoadPlan<NTB, WT, NV>::L;
  constexpr int PA = AD ? P : 0, PN = AD ? (P ^ 1) : 0;
  static_assert(L <= NM, "at most one DMA load per unit");
  static_assert(SP == 0 || SP * (L - 1) < NM, "the spaced loads fit in the k-step");
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    const int bi = i / NJ, bj = i % NJ;
    acc[bi][bj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[PA][bi], fb[P][bj], acc[bi][bj], 0, 0, 0);
    if (LOAD) {  // load q goes with unit q * NM / L, or q * SP
      if constexpr (SP > 0) {
        if (i % SP == 0 && i / SP < L) request_load<NTB, WT, NV>(lb, wr, hr, pl, wave, soff, i / SP);
      } else {
        const int q = (i * L + NM - 1) / NM;
        if (q < L && q * NM / L == i) request_load<NTB, WT, NV>(lb, wr, hr, pl, wave, soff, q);
      }
    }
    if (READ) {
      if (!AD && i < NJ) fb[P ^ 1][i] = read_b<NTB, NV>(rb, rs, i, wt, lane);
      if (AD) {
        // NJ + 8 reads spread evenly over the units, in the order the next
        // k-step consumes them: a0, b0 .. b[NJ-1], a1 .. a7
        constexpr int NR = NJ + 8;
        const int r = (i * NR + NM - 1) / NM;
        if (r < NR && r * NM / NR == i) {
          if (r == 0) fa[PN][0] = read_a(rb, rs, 0, wv, lane);
          else if (r <= NJ) fb[P ^ 1][r - 1] = read_b<NTB, NV>(rb, rs, r - 1, wt, lane);
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
template <int NTB, int WT, int NV = 2>
struct TileCtx {
  int vt;
  int64_t v0, t0;
  rsrc_t wr, hr, tr, cr;
};

// PK: packed operands (whole padded tile blocks, all in range).
template <int NTB, int WT, int GV, int NV = 2, bool PK = false>
__device__ __forceinline__ TileCtx<NTB, WT, NV> make_tile(const TileOps& o, int lid, int n_vt, int n_tt) {
  constexpr int BT = Tile<NTB, WT, NV>::BT;
  constexpr int TA = Tile<NTB, WT, NV>::TA;
  // Opaque copy: every call recomputes its context instead of the compiler
  // reusing (and keeping live) the result of an earlier call.
  asm volatile("" : "+s"(lid));
  TileCtx<NTB, WT, NV> c;
  int tt;
  tile_of_lid<GV>(lid, n_vt, n_tt, c.vt, tt);
  c.v0 = (int64_t)c.vt * TA;
  c.t0 = (int64_t)tt * BT;
  const int w_rows = (o.a_rows - c.v0) < TA ? (int)(o.a_rows - c.v0) : TA;
  const int h_rows = (o.b_rows - c.t0) < BT ? (int)(o.b_rows - c.t0) : BT;
  c.wr = make_rsrc((const __bf16*)o.a + c.v0 * o.K, (uint64_t)(PK ? TA : w_rows) * o.K * 2);
  c.hr = make_rsrc((const __bf16*)o.b + c.t0 * o.K, (uint64_t)(PK ? BT : h_rows) * o.K * 2);
  c.tr = make_rsrc(o.tokens + c.t0, (uint64_t)h_rows * 4);
  c.cr = make_rsrc((const unsigned char*)o.coef + c.t0 * 16, (uint64_t)h_rows * 16);
  return c;
}

// Tile passes over a sequence of (A tile, B tile) output tiles. The logical
// tile ids are dealt to the 8 XCDs in contiguous chunks, and within an XCD
// round-robin to its workgroups, so at any time the workgroups of one XCD work
// on consecutive ids. With one workgroup per tile this is a plain launch; with
// a grid of one workgroup per CU it is persistent, and the stage pipeline then
// runs on across tiles: the last stages of a tile already request the next
// tile's first stages, which land while this tile's epilogue runs.
//
// Pipeline. Stage s of a tile (kKS elements along K of its A and B rows)
// lives in LDS buffer s % kNBuf. Each stage has a boundary before its last
// k-step: every wave waits for its own reads of the stage and for its own DMA
// of stage s + 1, then the workgroup barrier makes stage s + 1 visible and
// frees buffer s % kNBuf, which takes stage s + kNBuf, its loads spread over
// that last k-step. MFMA operands are read one k-step ahead, across the
// boundary too. Requests past the tile go to the next tile's stages, or, with
// none, re-read the tile's own stages into the freed buffer, so every
// boundary's wait counts stay the same. (Row-data requests add loads between
// the stage requests; that only makes the later waits stricter.)
template <int NTB, int WT, bool SPLITK4, class E>
__device__ __forceinline__ void tile_pass(const typename E::Args& a, int n_vt, int n_tt) {
  constexpr int NV = E::kNV;
  using TL = Tile<NTB, WT, NV>;
  using LP = LoadPlan<NTB, WT, NV>;
  using TC = TileCtx<NTB, WT, NV>;
  using SH = Shape<NTB, WT, SPLITK4, NV>;
  constexpr int kNBuf = SH::NBUF;
  static_assert((128 / kKS) % kNBuf == 0, "the stage count (a multiple of 128 / kKS) must be a multiple of kNBuf");
  constexpr int NJ = TL::NJ;
  constexpr int BT = TL::BT;
  constexpr int SB = TL::kStageBytes;
  constexpr int EPI = E::template scratch_bytes<BT>();
  constexpr int L = LP::L;
  constexpr int ROWB = (E::kTokens ? 2 * BT * 4 : 0) + (E::kCoef ? 2 * BT * 16 : 0);
  // Epilogue scratch of its own when it fits, so the next tile's stages can
  // land during the epilogue; otherwise it reuses the first stage buffer.
  constexpr bool kSep = kNBuf * SB + EPI + ROWB <= (160 * 1024) / SH::PER_CU;
  // With its own scratch, the epilogue also finds the tile's per-row data
  // staged in LDS (two slots, alternating per tile), requested with the
  // tile's first stage, so it never waits on a global load behind the next
  // tile's stages.
  constexpr bool kTokLds = kSep && E::kTokens;
  constexpr bool kCoefLds = kSep && E::kCoef;
  static_assert(!E::kCoef || kCoefLds, "staged row words need LDS of their own");
  constexpr int TOKB = kTokLds ? 2 * BT * 4 : 0;
  constexpr int COEFB = kCoefLds ? 2 * BT * 16 : 0;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kNBuf * SB + (kSep ? EPI : 0) + COEFB + TOKB];
  float* scratch = (float*)(kSep ? lds + kNBuf * SB : lds);
  f32x4* coef_slot = (f32x4*)(lds + kNBuf * SB + (kSep ? EPI : 0));       // [2][BT] when kCoefLds
  int* tok_slot = (int*)(lds + kNBuf * SB + (kSep ? EPI : 0) + COEFB);  // [2][BT] when kTokLds
  int par = 0;
  const TileOps ops = E::ops(a);

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wv = NV == 2 ? (wave & 1) : 0, wt = wave / NV;

  // this workgroup's tiles: start + wi, start + wi + w_x, ... below start + t_x
  const int n_tiles = n_vt * n_tt;
  const int x = blockIdx.x & 7, wi = blockIdx.x >> 3;
  const int w_x = (int)(gridDim.x >> 3) + (x < (int)(gridDim.x & 7) ? 1 : 0);
  const int tq = n_tiles >> 3, trm = n_tiles & 7;
  const int t_x = tq + (x < trm ? 1 : 0);
  const int start = x * tq + (x < trm ? x : trm);
  int j = wi;
  if (j >= t_x) return;

  const int nk = ops.K / kKS;  // stages per tile; a multiple of kNBuf
  const int nk_q = nk / 4;     // stages per quarter (SPLITK4)
  // scalar offset from one stage to the next: along a row, or to the next
  // packed block (A and B tiles alike)
  constexpr bool kPK = E::kPacked;
  static_assert(!kPK || (TL::TA == kPackRows && BT == kPackRows), "packed operands come in 256-row tiles");
  constexpr int kStep = kPK ? kPackRows * kRowBytes : kRowBytes;

  TC cur = make_tile<NTB, WT, E::kGroupA, NV, kPK>(ops, start + j, n_vt, n_tt);
  const LP pl = make_load_plan<NTB, WT, NV, kPK>(ops.K, wave, lane_index());

  // prologue: the tile's row data and stages 0 .. kNBuf - 1
  auto prologue = [&]() {
    const int lane_p = lane_index();
    if constexpr (kCoefLds) request_coef<BT>(coef_slot + par * BT, cur.cr, wave, lane_p);
    if constexpr (kTokLds) request_tokens<BT>(tok_slot + par * BT, cur.tr, wave, lane_p);
#pragma unroll
    for (int s = 0; s < kNBuf; ++s)
#pragma unroll
      for (int q = 0; q < L; ++q)
        request_load<NTB, WT, NV>(lds + s * SB, cur.wr, cur.hr, pl, wave, (s < nk ? s : nk - 1) * kStep, q);
    wait_vmem<(kNBuf - 1) * L>();  // stage 0 (and the row data) landed
    __syncthreads();
  };
  prologue();

  f32x4 acc[8][NJ];
  f32x4 sum[8][SPLITK4 ? NJ : 1];
  // One wave per SIMD (four waves) leaves registers for a second A operand set.
  constexpr bool kAD = TL::NW == 4 && SH::PER_CU == 1;
  bf16x8 fa[2][8];   // A operands by k-step parity (with kAD), else fa[0] refilled in place
  bf16x8 fb[2][NJ];  // B operands, double buffered by k-step parity
  while (true) {
    // Per-tile lane arithmetic is recomputed inside the loop rather than
    // hoisted out of it (which would keep it live across the whole loop and
    // push the epilogue into spills).
    const int lane = lane_index();
    // The next tile's context is rebuilt where it is needed (cheap integer
    // work) rather than kept live across the loop.
    const bool has_next = j + w_x < t_x;
    const int next_lid = start + j + w_x;
    E::template init<NTB, WT>(a, cur.v0, cur.t0, acc, wave, lane);

    // stage 0 has landed and is visible: after the prologue, or, when the
    // pipeline runs on from the previous tile, since its last boundary
#pragma unroll
    for (int bj = 0; bj < NJ; ++bj) fb[0][bj] = read_b<NTB, NV>(lds, 0, bj, wt, lane);
#pragma unroll
    for (int bi = 0; bi < 8; ++bi) fa[0][bi] = read_a(lds, 0, bi, wv, lane);
    int k = 0;
    // steady state: every request is a stage of this tile
    for (; k + kNBuf < nk; ++k) {
      unsigned char* cb = lds + (k % kNBuf) * SB;
      region_a_prio();
      kstep<NTB, WT, 0, kAD, false, true, NV>(fa, fb, acc, cb, cur.wr, cur.hr, pl, 0, cb, 1, wave, wv, wt, lane);
      wait_lgkm0_vmem<(kNBuf - 2) * L>();
      stage_barrier();
      kstep<NTB, WT, 1, kAD, true, true, NV, E::kLoadSpacing>(fa, fb, acc, cb, cur.wr, cur.hr, pl, (k + kNBuf) * kStep,
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
      const TC nx = make_tile<NTB, WT, E::kGroupA, NV, kPK>(ops, (kSep && has_next) ? next_lid : start + j, n_vt,
                                                            n_tt);
#pragma unroll
      for (int t = 0; t < kNBuf; ++t) {
        k = nk - kNBuf + t;
        unsigned char* cb = lds + t * SB;
        region_a_prio();
        kstep<NTB, WT, 0, kAD, false, true, NV>(fa, fb, acc, cb, nx.wr, nx.hr, pl, 0, cb, 1, wave, wv, wt, lane);
        wait_lgkm0_vmem<(kNBuf - 2) * L>();
        stage_barrier();
        // request k + kNBuf: stage t of the next tile (with its row data)
        if (t == 0) {
          if constexpr (kCoefLds) request_coef<BT>(coef_slot + (par ^ 1) * BT, nx.cr, wave, lane);
          if constexpr (kTokLds) request_tokens<BT>(tok_slot + (par ^ 1) * BT, nx.tr, wave, lane);
        }
        if (t + 1 < kNBuf)
          kstep<NTB, WT, 1, kAD, true, true, NV, E::kLoadSpacing>(fa, fb, acc, cb, nx.wr, nx.hr, pl, t * kStep,
                                                                  lds + (t + 1) * SB, 0,
                                       wave, wv, wt, lane);
        else
          kstep<NTB, WT, 1, kAD, true, false, NV, E::kLoadSpacing>(fa, fb, acc, cb, nx.wr, nx.hr, pl, t * kStep, lds,
                                                                   0, wave, wv,
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
    E::template epilogue<NTB, WT>(a, n_vt, cur.vt, cur.v0, cur.t0, acc, scratch,
                                  kTokLds ? tok_slot + par * BT : nullptr,
                                  kCoefLds ? coef_slot + par * BT : nullptr, wave, lane);
    par ^= 1;
    if (!has_next) break;
    j += w_x;
    cur = make_tile<NTB, WT, E::kGroupA, NV, kPK>(ops, next_lid, n_vt, n_tt);
    if constexpr (!kSep) {
      __syncthreads();  // the epilogue's reads of the first buffer are done
      prologue();
    }
  }
  wait_vmem<0>();  // no global->LDS request may outlive the workgroup
}

// Deep pipeline for packed operands in 32-deep stages (packed_index<32>).
// The arithmetic is tile_pass's -- the same MFMA, the same operands per lane,
// K in the same ascending 32-element k-steps, so the same bits -- staged
// differently: a stage is one k-step (16 KB per 256-row operand tile) and NB
// buffers keep up to NB - 1 stages in flight, a prefetch lead of about NB - 1.5
// k-steps against about 1.5 for tile_pass's two 64-deep buffers, at the cost
// of a barrier per k-step instead of per two. Each stage boundary: every wave
// waits for its own reads of stage k (issued during k-step k - 1) and its own
// DMA of stage k + 1, the barrier makes stage k + 1 visible and frees stage
// k's buffer, which the k-step then refills with stage k + NB while it reads
// stage k + 1's operands. Used for 256 x 256 tiles of eight waves.
template <int NTB, int WT>
struct DeepTile {
  static constexpr int NW = 2 * WT;
  static constexpr int NJ = 2 * NTB;
  static constexpr int BT = WT * NTB * 32;
  static constexpr int kRow = 64;                     // bytes of a row in a stage
  static constexpr int kWB = kPackRows * kRow;        // A block of a stage
  static constexpr int SB = (kPackRows + BT) * kRow;  // stage bytes
  static constexpr int WB = kWB / (1024 * NW);        // 1 KB DMA loads per wave per stage, A
  static constexpr int HB = BT * kRow / (1024 * NW);  // and B
  static constexpr int L = WB + HB;
};

// Load q of a wave's stage request: the lane's 16 bytes at its place in the
// stage block (which is its place in LDS), A blocks first.
template <int NTB, int WT>
__device__ __forceinline__ void deep_load(unsigned char* buf, rsrc_t wr, rsrc_t hr, int wave, int lane, int soff, int q) {
#if defined(__HIP_DEVICE_COMPILE__)
  using DT = DeepTile<NTB, WT>;
  if (q < DT::WB) {
    const int blk = wave * DT::WB + q;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void*)(buf + blk * 1024), 16, (uint32_t)(blk * 64 + lane) * 16u,
                                             soff, 0, 0);
  } else {
    const int blk = wave * DT::HB + (q - DT::WB);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(hr, (lds_void*)(buf + DT::kWB + blk * 1024), 16,
                                             (uint32_t)(blk * 64 + lane) * 16u, soff, 0, 0);
  }
#endif
}

// MFMA operand of a 16-row block from a 32-deep stage: lane l reads row
// (l % 16) at hidden offset 8 (l / 16) of the stage.
__device__ __forceinline__ bf16x8 deep_read(const unsigned char* base, int row, int lane) {
  const int c = (lane >> 4) ^ swz_ks<32>(row);
  return *(const bf16x8*)(base + row * 64 + c * 16);
}

// One k-step: MFMA unit i (A block i / NJ, B block i % NJ) with the operands
// of parity P, its share of the stage request into `lb` (LOAD), and (READ)
// the next stage's operands from `rb`: the B blocks into the other parity
// set, each A block into its own register right after its last use here.
template <int NTB, int WT, int P, bool READ>
__device__ __forceinline__ void deep_kstep(bf16x8 (&fa)[8], bf16x8 (&fb)[2][2 * NTB], f32x4 (&acc)[8][2 * NTB],
                                           unsigned char* lb, rsrc_t wr, rsrc_t hr, int soff, const unsigned char* rb,
                                           int wave, int wv, int wt, int lane) {
  using DT = DeepTile<NTB, WT>;
  constexpr int NJ = DT::NJ;
  constexpr int NM = 8 * NJ;
  constexpr int L = DT::L;
  static_assert(L <= NM, "at most one DMA load per unit");
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    const int bi = i / NJ, bj = i % NJ;
    acc[bi][bj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[bi], fb[P][bj], acc[bi][bj], 0, 0, 0);
    const int q = (i * L + NM - 1) / NM;  // load q goes with unit q * NM / L
    if (q < L && q * NM / L == i) deep_load<NTB, WT>(lb, wr, hr, wave, lane, soff, q);
    if (READ) {
      if (i < NJ) fb[P ^ 1][i] = deep_read(rb + DT::kWB, wt * NTB * 32 + i * 16 + (lane & 15), lane);
      if (bj == NJ - 1) fa[bi] = deep_read(rb, wv * 128 + bi * 16 + (lane & 15), lane);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// The boundary before k-step k and the k-step: refill buffer bk (stage k's)
// with the request (wr, hr, soff) and read stage k + 1 from the next buffer.
template <int NTB, int WT, int NB, int P, bool READ>
__device__ __forceinline__ void deep_step(bf16x8 (&fa)[8], bf16x8 (&fb)[2][2 * NTB], f32x4 (&acc)[8][2 * NTB],
                                          unsigned char* lds, int& bk, rsrc_t wr, rsrc_t hr, int soff, int wave,
                                          int wv, int wt, int lane) {
  using DT = DeepTile<NTB, WT>;
  wait_lgkm0_vmem<(NB - 2) * DT::L>();
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  int bn = bk + 1;
  if (bn == NB) bn = 0;
  deep_kstep<NTB, WT, P, READ>(fa, fb, acc, lds + bk * DT::SB, wr, hr, soff, lds + bn * DT::SB, wave, wv, wt, lane);
  bk = bn;
}

// Tile pass over packed operands in 32-deep stages, NB stage buffers (global
// stage g in buffer g % NB); the tile walk and epilogue policy as in
// tile_pass (the policy's operands packed, no per-row data, no LDS scratch).
// The stage count ops.K / 32 must be a multiple of 4 and at least NB + 1.
template <int NTB, int WT, int NB, class E>
__device__ __forceinline__ void tile_pass_deep(const typename E::Args& a, int n_vt, int n_tt) {
  using DT = DeepTile<NTB, WT>;
  using TC = TileCtx<NTB, WT, 2>;
  constexpr int NJ = DT::NJ;
  constexpr int SB = DT::SB;
  constexpr int L = DT::L;
  constexpr int kStep = kPackRows * DT::kRow;  // from one packed block to the next
  static_assert(E::kPacked && !E::kTokens && !E::kCoef && E::template scratch_bytes<DT::BT>() == 0,
                "packed operands, no per-row data, no epilogue scratch");
  static_assert(DT::BT == kPackRows, "256-row tiles");
  static_assert(NB * SB <= 160 * 1024, "stage buffers within the LDS");
  __shared__ __attribute__((aligned(1024))) unsigned char lds[NB * SB];
  const TileOps ops = E::ops(a);
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
  const int nk = ops.K / 32;

  TC cur = make_tile<NTB, WT, E::kGroupA, 2, true>(ops, start + j, n_vt, n_tt);
  {  // prologue: stages 0 .. NB - 1
    const int lane_p = lane_index();
#pragma unroll
    for (int st = 0; st < NB; ++st)
#pragma unroll
      for (int q = 0; q < L; ++q) deep_load<NTB, WT>(lds + st * SB, cur.wr, cur.hr, wave, lane_p, st * kStep, q);
    wait_vmem<(NB - 1) * L>();  // stage 0 landed
    __syncthreads();
  }
  int bk = 0;  // buffer of the current stage
  f32x4 acc[8][NJ];
  bf16x8 fa[8];
  bf16x8 fb[2][NJ];
  // the last TL stages (TL even, at least NB: their requests may reach the
  // next tile) run unrolled with the operand parity known
  constexpr int TL = (NB + 1) & ~1;
  while (true) {
    const int lane = lane_index();
    const bool has_next = j + w_x < t_x;
    const int next_lid = start + j + w_x;
    E::template init<NTB, WT>(a, cur.v0, cur.t0, acc, wave, lane);
    {  // stage 0 has landed and is visible
      const unsigned char* b0 = lds + bk * SB;
#pragma unroll
      for (int bj = 0; bj < NJ; ++bj) fb[0][bj] = deep_read(b0 + DT::kWB, wt * NTB * 32 + bj * 16 + (lane & 15), lane);
#pragma unroll
      for (int bi = 0; bi < 8; ++bi) fa[bi] = deep_read(b0, wv * 128 + bi * 16 + (lane & 15), lane);
    }
    int k = 0;
    for (; k + TL < nk; k += 2) {  // every request is a stage of this tile
      deep_step<NTB, WT, NB, 0, true>(fa, fb, acc, lds, bk, cur.wr, cur.hr, (k + NB) * kStep, wave, wv, wt, lane);
      deep_step<NTB, WT, NB, 1, true>(fa, fb, acc, lds, bk, cur.wr, cur.hr, (k + 1 + NB) * kStep, wave, wv, wt,
                                      lane);
    }
    {  // requests past the tile go to the next tile's first stages, or, with
       // none, re-read this tile's
      const TC nx = make_tile<NTB, WT, E::kGroupA, 2, true>(ops, has_next ? next_lid : start + j, n_vt, n_tt);
#pragma unroll
      for (int t = 0; t < TL; ++t) {
        const int kn = k + t + NB;
        const bool in_tile = kn < nk;
        const int soff = (in_tile ? kn : kn - nk) * kStep;
        const rsrc_t wr = in_tile ? cur.wr : nx.wr;
        const rsrc_t hr = in_tile ? cur.hr : nx.hr;
        if (t + 1 < TL) {
          if (t & 1) deep_step<NTB, WT, NB, 1, true>(fa, fb, acc, lds, bk, wr, hr, soff, wave, wv, wt, lane);
          else deep_step<NTB, WT, NB, 0, true>(fa, fb, acc, lds, bk, wr, hr, soff, wave, wv, wt, lane);
        } else {
          deep_step<NTB, WT, NB, 1, false>(fa, fb, acc, lds, bk, wr, hr, soff, wave, wv, wt, lane);
        }
      }
    }
    E::template epilogue<NTB, WT>(a, n_vt, cur.vt, cur.v0, cur.t0, acc, nullptr, nullptr, nullptr, wave,
                                  lane_index());
    if (!has_next) break;
    j += w_x;
    cur = make_tile<NTB, WT, E::kGroupA, 2, true>(ops, next_lid, n_vt, n_tt);
  }
  wait_vmem<0>();  // no global->LDS request may outlive the workgroup
}

}  // namespace

// Compute units of the current device (cached per device).
static int device_cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
  // atomic: host threads may launch on one device at once (a racing first
  // call only queries the same attribute twice)
  static std::atomic<int> cache[64];
  if (dev < 64) {
    const int c = cache[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (dev < 64) cache[dev].store(n, std::memory_order_relaxed);
  return n;
}

}  // namespace tim
