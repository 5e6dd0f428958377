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
// Decode batches may run lmhead_half_partials instead: the same pass over
//   128-entry halves of the vocab tiles, writing each half's partial where
//   the whole-tile epilogue merges the two; the merge pairs them up again.
//
// Kernel 2, lmhead_merge: one wavefront per row (four for launches of at most
//   512 rows) merges that row's partials with a fixed balanced binary tree
//   over the tile index, then logp = z_tok - (M + log S) and H = log S - U / S.
//
// Reduction structure inside one vocab tile, for one row (fixed): each of the
// two vocab waves holds 128 entries of the row, 32 per lane in 4 lanes; per
// wave, the max and then the sums against it go lane-local in (block, register)
// order, then over the lane groups (lane ^ 16, then lane ^ 32); the two waves'
// partials are then merged, lower vocabulary half first.


#include "tilepass.h"

namespace tim {
namespace {

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

// z[i] for the i with 16 (i / 4) + i % 4 == tl (there is one: tl < 128,
// tl % 16 < 4), as a chain of compare-selects. Each compare takes its own
// opaque copy of tl, so none is hoisted ahead of the chain (which would hold
// all 32 conditions in scalar registers at once).
__device__ __forceinline__ float select_entry(const float (&z)[32], int tl) {
  float zf = 0.f;
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    int t = tl;
    asm volatile("" : "+v"(t));
    if ((i >> 2) * 16 + (i & 3) == t) zf = z[i];
  }
  return zf;
}

// One tile's per-row results from its accumulators. Each wave holds 128 of
// the tile's 256 vocabulary entries of its rows: for row block bj, lane l holds
// row (l % 16) and, in register r of W block bi, the entry
// wv * 128 + bi * 16 + 4 (l / 16) + r. With NV = 1 the workgroup covers one
// 128-entry half of a vocabulary tile (v0 its first entry, vt its index among
// the halves) and writes that half's partial as it is. Per row block the wave takes the logits
// z = acc * inv_tau (a multiply by exactly 1 is skipped, which changes
// nothing), masks entries past V to -inf (tail tile only), forms its half's
// partial (m, s, u) -- max first, then the sums against that max, lane-local
// in (bi, r) order, then over lane ^ 16 and lane ^ 32 -- and captures the
// sampled token's logit from the same register value. The two vocab halves
// are merged in a fixed order (lower half first) into the tile's Partial.
// `scratch` holds 7 * BT floats of LDS; with `tok_lds` the tile's tokens come
// from LDS.
template <int NTB, int WT, bool DUMP, int NV = 2>
__device__ __forceinline__ void tile_epilogue(const LmHeadArgs& a, int n_vt, int vt, int64_t v0, int64_t t0,
                                              f32x4 (&acc)[8][2 * NTB], float* scratch, const int* tok_lds, int wave,
                                              int lane) {
  constexpr int BT = Tile<NTB, WT, NV>::BT;
  constexpr int NJ = 2 * NTB;
  static_assert(NV == 2 || (NV == 1 && !DUMP), "half tiles form partials only");
  const int wv = NV == 2 ? (wave & 1) : 0, wt = NV == 2 ? (wave >> 1) : wave;
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
  // same path in every launch shape; a half takes its vocabulary tile's path.
  const bool full = (NV == 2 ? v0 : v0 - v0 % kVocabTile) + kVocabTile <= V;

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
      const int lim = (int)(V - vlane);  // entries past V: (i / 4) 16 + i % 4 >= lim (32-bit: V < 2^31)
#pragma unroll
      for (int i = 0; i < 32; ++i)
        if ((i >> 2) * 16 + (i & 3) >= lim) z[i] = kNegInf;
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
    if constexpr (NV == 2) {
      if (g == 0) {
        red_m[wv * BT + t_loc] = m;
        red_s[wv * BT + t_loc] = sv;
        red_u[wv * BT + t_loc] = uv;
      }
    }
    // Token gather: the lane holding the row's token has tl = token - vlane
    // in [0, 128) with tl % 16 < 4 (entry z[4 (tl / 16) + tl % 16]). Rare, so
    // the 32-way select runs under a divergent branch.
    const int tok = row_ok ? (tok_lds != nullptr ? tok_lds[t_loc] : a.tokens[tg]) : -1;
    const int tl = (tok >= 0) ? (int)((int64_t)tok - vlane) : -1000000;
    if constexpr (NV == 2) {
      if (tl >= 0 && tl < 128 && (tl & 15) < 4) zt_l[t_loc] = select_entry(z, tl);
    } else {
      float zf = 0.f;
      if (tl >= 0 && tl < 128 && (tl & 15) < 4) zf = select_entry(z, tl);
      // the half's Partial, with the token's logit from the lane holding it
      // (lane group ((token - v0) % 16) / 4 of the row's four)
      const int64_t th = (int64_t)tok - v0;
      const bool mine = tok >= 0 && th >= 0 && th < 128;
      const float zt = __shfl(zf, c16 + (mine ? 16 * (int)((th & 15) >> 2) : 0));
      if (g == 0 && row_ok) {
        Partial p;
        p.m = m;
        p.s = sv;
        p.u = uv;
        p.ztok = mine ? zt : 0.f;
        a.part[tg * n_vt + vt] = p;
      }
    }
  }
  if constexpr (DUMP || NV == 1) return;
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

// Epilogue policies of a tile pass. Each one names the pass's operands (and
// whether they are in the packed layout), how the stage loads are placed in a
// k-step, the LDS it needs beside the stage buffers, the per-row data it wants
// staged in LDS with each tile, how the accumulators start, and what it does
// with them.
//
// EpiPartials: the LM head forward. A = W [V, d], B = hidden states, K = d;
// the epilogue forms the tile's softmax partials (or, DUMP, writes logits);
// with NV = 1, those of half tiles.
template <bool DUMP, int NV = 2>
struct EpiPartials {
  using Args = LmHeadArgs;
  static constexpr bool kTokens = !DUMP;
  static constexpr bool kCoef = false;
  static constexpr bool kPacked = false;  // W and h as the caller holds them
  static constexpr int kLoadSpacing = 0;  // stage loads spread evenly over a k-step's MFMAs
  static constexpr int kGroupA = kGroupV;
  static constexpr int kNV = NV;
  template <int BT>
  static constexpr int scratch_bytes() { return NV == 2 ? 7 * BT * 4 : 0; }
  __device__ static TileOps ops(const Args& a) {
    return TileOps{a.w, a.hidden, a.tokens, nullptr, a.rows, a.V, a.d};
  }
  template <int NTB, int WT>
  __device__ static void init(const Args&, int64_t, int64_t, f32x4 (&acc)[8][2 * NTB], int, int) {
#pragma unroll
    for (int bi = 0; bi < 8; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2 * NTB; ++bj) acc[bi][bj] = f32x4{};
  }
  template <int NTB, int WT>
  __device__ static void epilogue(const Args& a, int n_vt, int vt, int64_t v0, int64_t t0, f32x4 (&acc)[8][2 * NTB],
                                  float* scratch, const int* tok_lds, const f32x4*, int wave, int lane) {
    tile_epilogue<NTB, WT, DUMP, NV>(a, n_vt, vt, v0, t0, acc, scratch, tok_lds, wave, lane);
  }
};

// Softmax partials (or, DUMP, logits) of every (vocab tile, row tile).
template <int NTB, int WT, bool SPLITK4, bool DUMP>
__global__ __launch_bounds__(128 * WT, (Shape<NTB, WT, SPLITK4>::PER_CU))
void lmhead_partials(LmHeadArgs a, int n_vt, int n_tt) {
  tile_pass<NTB, WT, SPLITK4, EpiPartials<DUMP>>(a, n_vt, n_tt);
}

// Softmax partials of every (half vocabulary tile, row tile), for decode
// batches: one vocab wave per workgroup along the vocabulary (WT waves along
// the rows), a third or half of the LDS of a CU each, so that several
// workgroups share a CU and the vocabulary's 2 * ceil(V / 256) halves fill the
// chip more evenly than its ceil(V / 256) tiles. A half's partial is the one
// the whole-tile epilogue forms for that half before merging the two.
// (PER_CU workgroups of WT waves put up to ceil(PER_CU * WT / 4) waves on
// one SIMD, which bounds each wave's registers.)
template <int NTB, int WT>
__global__ __launch_bounds__(64 * WT)
__attribute__((amdgpu_waves_per_eu((Shape<NTB, WT, false, 1>::PER_CU * WT + 3) / 4)))
void lmhead_half_partials(LmHeadArgs a, int n_ht, int n_tt) {
  tile_pass<NTB, WT, false, EpiPartials<false, 1>>(a, n_ht, n_tt);
}

// ---------------------------------------------------------------- merge

// TW: vocabulary entries per partial (whole or half tiles)
template <int TW>
__device__ __forceinline__ void finish_row(MSU v, const Partial* p, int tok, int V, int64_t row,
                                           float* logp, float* ent, float* lse) {
  const float logS = logf(v.s);
  const float L = v.m + logS;
  const bool ok = tok >= 0 && tok < V;
  logp[row] = ok ? p[tok / TW].ztok - L : __builtin_nanf("");
  if (ent) ent[row] = logS - v.u / v.s;
  if (lse) lse[row] = L;
}

// The balanced pairwise tree over 64 L consecutive leaves of a row, from
// leaf `first`: lane l owns leaves [first + l L, first + l L + L), merged in a
// tree within the lane, then across lanes by index (lane ^ 1, ^ 2, ... ^ 32),
// lower index first at every node. Leaves at or past n_vt are the identity, so
// the tree is the same whatever L is. With HALVES the row holds the partials of
// half tiles, and leaf jt is merge2(half 2 jt, half 2 jt + 1), as the
// whole-tile epilogue forms tile jt's partial (a missing upper half is the
// identity there too). Every lane returns the subtree's value.
template <int L, bool HALVES>
__device__ __forceinline__ MSU wave_subtree(const Partial* p, int n_vt, int n_ht, int first, int lane) {
  MSU leaf[L];
#pragma unroll
  for (int i = 0; i < L; ++i) {
    const int jt = first + lane * L + i;
    if (jt < n_vt) {
      if constexpr (HALVES) {
        const Partial q0 = p[2 * jt];
        leaf[i] = MSU{q0.m, q0.s, q0.u};
        if (2 * jt + 1 < n_ht) {
          const Partial q1 = p[2 * jt + 1];
          leaf[i] = merge2(leaf[i], MSU{q1.m, q1.s, q1.u});
        }
      } else {
        const Partial q = p[jt];
        leaf[i] = MSU{q.m, q.s, q.u};
      }
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
  return v;
}

// One wavefront per row: the balanced pairwise tree over the tile index.
template <int L, bool HALVES = false>
__global__ __launch_bounds__(256) void lmhead_merge_tree(const Partial* __restrict__ part,
                                                         const int32_t* __restrict__ tokens,
                                                         int64_t rows, int n_vt, int V, float* logp,
                                                         float* ent, float* lse) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int n_ht = (V + kHalfTile - 1) / kHalfTile;
  const Partial* p = part + row * (HALVES ? n_ht : n_vt);
  const MSU v = wave_subtree<L, HALVES>(p, n_vt, n_ht, 0, lane);
  if (lane == 0) finish_row<HALVES ? kHalfTile : kVocabTile>(v, p, tokens[row], V, row, logp, ent, lse);
}

// Few rows (decode batches): four wavefronts per row, wave w reducing the
// quarter [w 64 LQ, (w + 1) 64 LQ) of the leaves as above, the quarters then
// merged as (q0 + q1) + (q2 + q3): the top two levels of the same balanced
// tree over 256 LQ leaves, so the same bits as lmhead_merge_tree<4 LQ> with a
// quarter of the serial work per lane.
template <int LQ, bool HALVES>
__global__ __launch_bounds__(256) void lmhead_merge_quad(const Partial* __restrict__ part,
                                                         const int32_t* __restrict__ tokens,
                                                         int64_t rows, int n_vt, int V, float* logp,
                                                         float* ent, float* lse) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = blockIdx.x;
  const int n_ht = (V + kHalfTile - 1) / kHalfTile;
  const Partial* p = part + row * (HALVES ? n_ht : n_vt);
  const MSU v = wave_subtree<LQ, HALVES>(p, n_vt, n_ht, wave * 64 * LQ, lane);
  __shared__ MSU q[4];
  if (lane == 0) q[wave] = v;
  __syncthreads();
  if (threadIdx.x == 0)
    finish_row<HALVES ? kHalfTile : kVocabTile>(merge2(merge2(q[0], q[1]), merge2(q[2], q[3])), p, tokens[row], V,
                                                row, logp, ent, lse);
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
  finish_row<kVocabTile>(v, p, tokens[row], V, row, logp, ent, lse);
}

}  // namespace

int n_vocab_tiles(int V) { return (V + kVocabTile - 1) / kVocabTile; }
int n_half_tiles(int V) { return (V + kHalfTile - 1) / kHalfTile; }

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
    default:  // 256-row tiles, 8 waves; full-size launches persistent
      return dump ? launch_partials_t<2, 4, false, true>(a, true, s) : launch_partials_t<2, 4, false, false>(a, true, s);
  }
}

// Share of the slots of the last round that hold a unit, for `units` units
// dealt to `slots` resident workgroups.
static double round_fill(int64_t units, int64_t slots) {
  const int64_t rounds = (units + slots - 1) / slots;
  return (double)units / (double)(rounds * slots);
}

bool prefer_half_tiles(int V, int64_t rows) {
  // 65..128 rows: whole tiles of this row tile run one workgroup per CU,
  // halves two (four waves each), which measured faster at every vocabulary
  // size tried
  if (rows > 64) return true;
  const int cus = device_cu_count();
  if (cus <= 0) return false;
  const int64_t whole_slots = (int64_t)cus * Shape<1, 2, false>::PER_CU;
  const int64_t half_slots = (int64_t)cus * Shape<1, 2, false, 1>::PER_CU;
  return round_fill(n_half_tiles(V), half_slots) > round_fill(n_vocab_tiles(V), whole_slots);
}

template <int NTB, int WT>
static hipError_t launch_halves_t(const LmHeadArgs& a, hipStream_t s) {
  const int n_ht = n_half_tiles(a.V);
  constexpr int BT = Tile<NTB, WT, 1>::BT;
  const int64_t n_tt = (a.rows + BT - 1) / BT;
  const int64_t nblk = n_tt * n_ht;
  if (nblk > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((lmhead_half_partials<NTB, WT>), dim3((unsigned)nblk), dim3(64 * WT), 0, s, a, n_ht, (int)n_tt);
  return hipGetLastError();
}

// 64-row tiles (three workgroups of 2 waves of 128 x 32 per CU) up to 64
// rows, 128-row tiles (two workgroups of 4 waves of 128 x 32 per CU: two waves
// per SIMD) above.
hipError_t launch_partials_halves(const LmHeadArgs& a, hipStream_t s) {
  return a.rows <= 64 ? launch_halves_t<1, 2>(a, s) : launch_halves_t<1, 4>(a, s);
}

// Launches of at most this many rows merge with four waves per row.
constexpr int64_t kQuadMergeRows = 512;

template <bool HALVES>
static hipError_t launch_merge_tree(const Partial* part, const int32_t* tokens, int64_t rows, int V, float* logp,
                                    float* entropy, float* lse, hipStream_t s) {
  const int n_vt = n_vocab_tiles(V);
  const dim3 b(256);
  if (rows <= kQuadMergeRows && n_vt > 128) {
    const dim3 g((unsigned)rows);
    if (n_vt <= 256) hipLaunchKernelGGL((lmhead_merge_quad<1, HALVES>), g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
    else if (n_vt <= 512) hipLaunchKernelGGL((lmhead_merge_quad<2, HALVES>), g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
    else if (n_vt <= 1024) hipLaunchKernelGGL((lmhead_merge_quad<4, HALVES>), g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
    else if (n_vt <= kMaxTiles) hipLaunchKernelGGL((lmhead_merge_quad<8, HALVES>), g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
    else return hipErrorInvalidValue;
    return hipGetLastError();
  }
  const int64_t nb = (rows + 3) / 4;
  if (nb > 0x7fffffff) return hipErrorInvalidValue;
  const dim3 g((unsigned)nb);
  if (n_vt <= 64) hipLaunchKernelGGL((lmhead_merge_tree<1, HALVES>), g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else if (n_vt <= 128) hipLaunchKernelGGL((lmhead_merge_tree<2, HALVES>), g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else if (n_vt <= 256) hipLaunchKernelGGL((lmhead_merge_tree<4, HALVES>), g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else if (n_vt <= 512) hipLaunchKernelGGL((lmhead_merge_tree<8, HALVES>), g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else if (n_vt <= 1024) hipLaunchKernelGGL((lmhead_merge_tree<16, HALVES>), g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else if (n_vt <= kMaxTiles) hipLaunchKernelGGL((lmhead_merge_tree<32, HALVES>), g, b, 0, s, part, tokens, rows, n_vt, V, logp, entropy, lse);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_merge(const Partial* part, const int32_t* tokens, int64_t rows, int V,
                        bool left_fold, float* logp, float* entropy, float* lse, hipStream_t s) {
  if (left_fold) {
    const int64_t nb = (rows + 255) / 256;
    hipLaunchKernelGGL(lmhead_merge_fold, dim3((unsigned)nb), dim3(256), 0, s, part, tokens, rows,
                       n_vocab_tiles(V), V, logp, entropy, lse);
    return hipGetLastError();
  }
  return launch_merge_tree<false>(part, tokens, rows, V, logp, entropy, lse, s);
}

hipError_t launch_merge_halves(const Partial* part, const int32_t* tokens, int64_t rows, int V, float* logp,
                               float* entropy, float* lse, hipStream_t s) {
  return launch_merge_tree<true>(part, tokens, rows, V, logp, entropy, lse, s);
}

}  // namespace tim
