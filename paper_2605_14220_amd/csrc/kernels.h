// Internal launch interface between the C-ABI entry points and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tim {

constexpr int kVocabTile = 256;   // vocabulary entries per softmax partial
constexpr int kHalfTile = 128;    // entries per partial of the decode-batch shape
constexpr int kMaxTiles = 2048;   // merge supports up to 64 lanes x 32 leaves

// One partial per (row, vocab tile): running max, sum of exp(z - m),
// sum of exp(z - m) * (z - m), and the gathered logit of the row's token
// (valid only in the tile that holds the token).
struct alignas(16) Partial {
  float m, s, u, ztok;
};

struct LmHeadArgs {
  const void* hidden;     // bf16 [rows, d]
  const void* w;          // bf16 [V, d]
  const int32_t* tokens;  // [rows]
  int64_t rows;
  int32_t d;
  int32_t V;
  float inv_tau;
  Partial* part;          // [rows, n_tiles]
  float* logits;          // [rows, V] for the logits dump, else null
};

// Backward of the fused log-prob, logit-gradient pass: the LM-head
// contraction recomputed exactly as the forward forms it, then per entry
// dacc = gamma [v == token] - p (alpha + beta q), q = z - lse, p = e^q, from
// the row's words coef = (lse, alpha, beta, gamma); written as bf16.
struct DlogitsArgs {
  const void* hidden;     // bf16 [rows, d]
  const void* w;          // bf16 [V, d]
  const int32_t* tokens;  // [rows]
  const void* coef;       // float4 [rows]
  int64_t rows;
  int32_t d;
  int32_t V;
  float inv_tau;
  void* dacc;             // bf16 [rows, ld]; entries V .. ld - 1 of a row are written as 0
  int64_t ld;             // a multiple of 256 covering V
  int32_t packed;         // dacc row-major, or packed (K = ld) over ceil(rows / 256) whole tiles
  // Optional (null: none): the same gradients transposed, bf16 [ld, t_pad] packed in 32-deep stage blocks
  // (K = t_pad), the weight gradient's operand; token rows rows .. t_pad - 1 are written as 0. With it, dacc may
  // be null (no [rows, ld] image written).
  void* dacct;
  int64_t t_pad;          // rows rounded up to a multiple of 128, at least 256 (used with dacct)
};

// Plain tile pass: out[j * ldo + i] = (accumulate ? out[j * ldo + i] : 0)
// + sum_k A[i][k] B[j][k] in one fp32 accumulation chain per element, K
// ascending; A bf16 [a_rows, K] and B bf16 [b_rows, K] in the packed layout
// (tilepass.h) over whole 256-row tiles (rows padded up to a multiple of 256,
// the padding's outputs never written), in 64-deep stage blocks or, with
// deep, 32-deep ones (then K >= 256); K a multiple of 128, a_rows a multiple
// of 4. Both forms give the same bits.
struct GemmArgs {
  const void* a;
  const void* b;
  int64_t b_rows;
  int32_t a_rows;
  int32_t K;
  float* out;
  int64_t ldo;
  int32_t accumulate;
  int32_t deep;
};

// K3 estimator of the correction ratio r = e^delta (Section 4.1), e^delta - 1
// - delta, from the exact fp64 difference of two fp32 log-probabilities. In
// fp64 the form expm1(delta) - delta loses about 2^-52 / |delta| of relative
// accuracy to expm1's rounding (the subtraction itself is exact), which for
// |delta| below 2^-5 a Taylor polynomial avoids: delta^2 (1/2 + delta/6 + ...
// + delta^6/8!), whose first omitted term is below 2^-50 of the sum there.
// Either way the fp64 value is within 2^-46 of K3 relative, so its one
// rounding to fp32 is correct to within that of a correctly rounded K3.
__device__ __forceinline__ double k3_of_delta(double d) {
  if (__builtin_fabs(d) < 0.03125) {
    double p = 1.0 / 40320.0;
    p = __builtin_fma(p, d, 1.0 / 5040.0);
    p = __builtin_fma(p, d, 1.0 / 720.0);
    p = __builtin_fma(p, d, 1.0 / 120.0);
    p = __builtin_fma(p, d, 1.0 / 24.0);
    p = __builtin_fma(p, d, 1.0 / 6.0);
    p = __builtin_fma(p, d, 0.5);
    return (d * d) * p;
  }
  return expm1(d) - d;  // NaN stays NaN; delta = -inf gives +inf
}

// Truncated importance weight min(e^delta, C) (Section 4.2, Eq. 6) from the
// exact fp64 difference, rounded once to fp32; a NaN ratio stays NaN.
__device__ __forceinline__ float tis_weight(double d, float C) {
  const double r = exp(d);
  return (r > (double)C) ? C : (float)r;
}

int n_vocab_tiles(int V);
int n_half_tiles(int V);

// Partials of every (row, vocab tile). rows_per_wg in {64, 128, 256} is the
// row tile of one workgroup; it changes the launch shape only.
hipError_t launch_partials(const LmHeadArgs& a, int rows_per_wg, bool splitk4, hipStream_t s);
// Partials of every (row, half vocabulary tile), 64 or 128 rows per row tile
// (by the launch's row count; 2 or 4 waves of 128 x 32): part is
// [rows, n_half_tiles]; each half's
// partial equals the one the whole-tile epilogue merges, so
// launch_merge_halves gives the outputs of launch_partials + launch_merge bit
// for bit.
hipError_t launch_partials_halves(const LmHeadArgs& a, hipStream_t s);
// Whether a decode batch of `rows` rows on the current device takes half
// tiles. Up to 64 rows: the shape (whole tiles two per CU, or half tiles
// three per CU) whose last round of workgroups leaves fewer slots idle; the
// half shape re-reads the row tile once per 128 vocabulary entries instead of
// 256, so it only pays where it evens out the rounds. 65..128 rows: always
// (whole tiles one workgroup per CU against halves two, each of four waves).
// Either gives the same bits.
bool prefer_half_tiles(int V, int64_t rows);
hipError_t launch_merge_halves(const Partial* part, const int32_t* tokens, int64_t rows, int V, float* logp,
                               float* entropy, float* lse, hipStream_t s);
// Fixed-order merge of each row's partials into logp / entropy / lse.
hipError_t launch_merge(const Partial* part, const int32_t* tokens, int64_t rows, int V,
                        bool left_fold, float* logp, float* entropy, float* lse, hipStream_t s);
hipError_t launch_dlogits(const DlogitsArgs& a, hipStream_t s);
hipError_t launch_gemm(const GemmArgs& a, hipStream_t s);
// dst[c][r] = src[r][c] for r < R, c < C, and 0 for the rest of r < R_pad,
// c < C_pad (bf16), dst in the packed layout [C_pad, R_pad] (K = R_pad) in
// dst_ks-deep stage blocks (64 or 32); src row-major with row stride ld_src,
// or (src_packed) packed in 64-deep blocks with K = ld_src. C_pad a multiple
// of 256, R_pad of 64, C of 8; 16-byte aligned rows.
hipError_t launch_transpose(const void* src, bool src_packed, int64_t R, int64_t C, int64_t ld_src, void* dst,
                            int64_t R_pad, int64_t C_pad, int dst_ks, hipStream_t s);
// Per-row words (lse, alpha, beta, gamma) of the logit gradient for upstream
// gradients g (of logp) and e (of the entropy; may be null): with g' = g for
// a token in [0, V) else 0, alpha = (g' + e H) / tau, beta = e / tau,
// gamma = g' / tau, each formed in fp64 and rounded once.
hipError_t launch_grad_coef(const float* lse, const float* entropy, const float* grad_logp,
                            const float* grad_entropy, const int32_t* tokens, int64_t rows, int V,
                            float temperature, void* coef, hipStream_t s);
hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s);
// Final RMS norm, one wavefront per row: h (bf16 [T, d]) and rstd (fp32 [T], may be null).
hipError_t launch_rmsnorm(const void* x, const void* gamma, int64_t T, int d, float eps, void* h, float* rstd,
                          hipStream_t s);
// Its backward: grad_x (fp32 [T, d]) and/or grad_gamma (fp32 [d]) from grad_h
// (fp32 [T, d]); `part` holds ceil(T / 256) * d floats of column partial sums.
hipError_t launch_rmsnorm_backward(const void* x, const void* gamma, const float* rstd, const float* grad_h,
                                   int64_t T, int d, float* grad_x, float* grad_gamma, int accumulate, float* part,
                                   hipStream_t s);
// Clipped PPO/GRPO loss constants, formed on the host in fp64.
struct PpoParams {
  double lo_threshold;  // log1p(-eps_low): A < 0 clips below it
  double hi_threshold;  // log1p(eps_high): A > 0 clips above it
  double clip_lo;       // 1 - eps_low
  double clip_hi;       // 1 + eps_high
  double inv_n;         // 1 / number of responses (the batch mean)
};
hipError_t launch_ppo_loss(const float* logp, const float* logp_old, const float* advantages, const float* weight,
                           int64_t T, const int64_t* cu_seqlens, int64_t n_seq, const PpoParams& p, double* seq_loss,
                           double* batch_loss, float* token_loss, float* grad, float* contrib, uint8_t* clipped,
                           hipStream_t s);
hipError_t launch_mismatch(const float* a, const float* b, int64_t n, float C,
                           float* log_ratio, float* k3, float* w, hipStream_t s);
// Per-response score / keep and per-token weights of a packed stream (one
// workgroup per response, fixed-order fp64 sum).
hipError_t launch_mismatch_seq(const float* a, const float* b, int64_t T, const int64_t* cu_seqlens,
                               int64_t n_seq, bool k3, float C, double tau_seq, double* score,
                               uint8_t* keep, float* weight, hipStream_t s);

}  // namespace tim
