// Internal launch interface between the C-ABI entry points and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tim {

constexpr int kVocabTile = 256;   // vocabulary entries per softmax partial
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

int n_vocab_tiles(int V);

// Partials of every (row, vocab tile). rows_per_wg in {64, 128, 256} is the
// row tile of one workgroup; it changes the launch shape only.
hipError_t launch_partials(const LmHeadArgs& a, int rows_per_wg, bool splitk4, hipStream_t s);
// Fixed-order merge of each row's partials into logp / entropy / lse.
hipError_t launch_merge(const Partial* part, const int32_t* tokens, int64_t rows, int V,
                        bool left_fold, float* logp, float* entropy, float* lse, hipStream_t s);
hipError_t launch_mismatch(const float* a, const float* b, int64_t n, float C,
                           float* log_ratio, float* k3, float* w, hipStream_t s);
// Per-response score / keep and per-token weights of a packed stream (one
// workgroup per response, fixed-order fp64 sum).
hipError_t launch_mismatch_seq(const float* a, const float* b, int64_t T, const int64_t* cu_seqlens,
                               int64_t n_seq, bool k3, float C, double tau_seq, double* score,
                               uint8_t* keep, float* weight, hipStream_t s);

}  // namespace tim
