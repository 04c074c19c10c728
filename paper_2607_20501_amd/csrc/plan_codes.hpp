// Codes shared by the plan and the kernels: element-wise chain steps and
// terminal reductions.
#pragma once

#include <stdint.h>

namespace mk {

enum EpiCode : int32_t {
  EPI_BIAS_COL = 1,   // + b[col]
  EPI_BIAS_CH = 2,    // + b[channel]
  EPI_RELU = 3,
  EPI_GELU_ERF = 4,
  EPI_GELU_TANH = 5,
  EPI_SCALE = 6,      // * s
  EPI_ADD = 7,        // + r[same flat index as the output]
  EPI_CAUSAL = 8,     // col > row -> -inf  (row/col inside an S x S score matrix)
  // Test-only codes, used by mutant implementations (injected bugs).
  EPI_GELU_SIGMOID = 100,   // x * sigmoid(1.702 x)
  EPI_CAUSAL_STRICT = 101   // col >= row -> -inf (diagonal masked too)
};
constexpr int kMaxEpi = 8;

// Terminal reductions that need a whole row (or image) and are split at the
// GEMM's column tile: per-tile partials, then a finisher.  TERM_LAYERNORM is
// the post-LN "residual + LayerNorm" ending of a CvT-style block.
enum Terminal : int32_t {
  TERM_NONE = 0,
  TERM_ROWSUM = 1,
  TERM_SOFTMAX = 2,
  TERM_GAP = 3,
  TERM_LAYERNORM = 4
};

}  // namespace mk
