// Launch interfaces of the HIP kernels.  Plain pointers and sizes; every
// launcher enqueues on `stream` and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/mk.h"

namespace mk {

// Element-wise chain as the kernels see it (codes from plan.hpp's EpiCode).
struct EpiDev {
  int32_t n;
  int32_t code[8];
  const void* ptr[8];
  float s[8];
};

struct EwArgs {
  const void* x;
  void* y;
  int64_t numel, last, C, HW, S;
  EpiDev epi;
};

// One row op per row of a [rows, len] view (GAP: rows = N*C, len = H*W).
struct RowArgs {
  const void* x;
  void* y;
  int64_t rows, len;
  int32_t op;              // MK_OP_ROWSUM / SOFTMAX / LAYERNORM / GAP
  const void* gamma;
  const void* beta;
  float eps;
  EwArgs pre;              // element-wise prologue (pre.epi.n == 0: none)
  // Test-only variants (simple kernel): 1 softmax without the max
  // subtracted, 2 softmax over dim -2 (n2 rows of each group of rows),
  // 3 LayerNorm without the mean subtracted before scaling.
  int32_t variant;
  int64_t n2;
  float p;                 // LPPOOL exponent
};

struct GemmArgs {
  const void* A;
  const void* B;
  void* C;
  int64_t M, N, K, lda, ldb, ldc;
  int64_t a_off, a_sb, a_sh, b_off, b_sb, b_sh, c_off, c_sb, c_sh;
  int32_t batch, heads, layout, terminal;
  float alpha;
  int32_t acc_bf16;        // test-only: round the accumulator to bf16 after every step
  const float* ln_stats;   // [M][2] (mean, rstd) of A's rows, or null
  const void* ln_g;
  const void* ln_b;
  EpiDev epi;
  float* partial;          // row partials of the terminal reduction
  int64_t n_tiles;         // column tiles per row in `partial`
  // Implicit-GEMM convolution (conv != 0): rows of A are output channels
  // (weights repacked as [K][R][S][C]), columns are output positions
  // m = (n, p, q) whose B rows are gathered from a zero-padded NHWC copy of the
  // input; C is written NCHW, or reduced to per-tile GAP partials
  // (terminal == TERM_GAP: partial[(tile * 2 + slot) * M + k]).
  int32_t conv;
  int64_t cv_C, cv_Hp, cv_Wp, cv_P, cv_Q, cv_S, cv_stride;
  int32_t pool;            // kind of the global pool of TERM_GAP (GAP, GMP, LPPOOL)
  float pool_p;
};

struct ConvArgs {
  const void* x;
  const void* w;
  void* y;
  int64_t N, C, H, W, K, R, S, P, Q, stride, pad;
  EpiDev epi;              // channel-indexed chain
  int32_t gap;             // ends in a global pool of kind pool (GAP, GMP, LPPOOL)
  int32_t pool;
  float pool_p;
  float* partial;          // GAP partial sums [N][K][n_pos_tiles]
  int64_t n_pos_tiles;
  void* scratch;           // tuned conv: repacked operands
};

struct AttnArgs {
  const void* qkv;
  void* o;
  int64_t B, H, dh, S;
  float scale;
  int32_t causal;
  int64_t kdim;            // dims of q.k summed (dh; test-only: fewer)
};

// dtype: 0 float32, 1 bfloat16 (mk_dtype).
hipError_t launch_ew(int dtype, const EwArgs& a, hipStream_t st, int impl);
hipError_t launch_row(int dtype, const RowArgs& a, hipStream_t st, int impl);
// Tuned row kernel: one wave per row, the row in registers (len a multiple of
// 8 bf16 / 4 fp32 elements, at most 4096 / 2048, 16-byte aligned buffers).
bool row_wave_supported(int dtype, const RowArgs& a);
hipError_t launch_row_wave(int dtype, const RowArgs& a, hipStream_t st);
// unsafe (test-only): the mean is reported as 0, so rows are not centred.
hipError_t launch_ln_stats(int dtype, const void* x, int64_t rows, int64_t len, float eps,
                           float* stats, hipStream_t st, int unsafe);
hipError_t launch_gemm_simple(int dtype, const GemmArgs& a, hipStream_t st);
hipError_t launch_rowsum_finish(int dtype, const float* partial, int64_t rows, int64_t n_tiles,
                                void* out, hipStream_t st);
hipError_t launch_softmax_finish(int dtype, const float* partial, int64_t rows, int64_t n_tiles,
                                 int64_t N, void* out, hipStream_t st);
hipError_t launch_conv_simple(int dtype, const ConvArgs& a, hipStream_t st);
hipError_t launch_attn_simple(int dtype, const AttnArgs& a, hipStream_t st);

// Tuned kernels.
// Tuned element-wise kernel (k_ew.hip): 16-byte groups, 32-bit index
// arithmetic; ew_fast_supported() states when it applies.
bool ew_fast_supported(const EwArgs& a);
bool softmax_finish_wave_supported(int dtype, int64_t N, const void* out);
// Post-LN finisher for TERM_LAYERNORM (per-tile moments of `tile` columns).
hipError_t launch_ln_finish(int dtype, const float* partial, int64_t rows, int64_t nt, int64_t N,
                            int64_t tile, const void* gamma, const void* beta, float eps,
                            void* out, hipStream_t st);
hipError_t launch_softmax_finish_wave(int dtype, const float* partial, int64_t rows, int64_t nt,
                                      int64_t N, void* out, hipStream_t st);
hipError_t launch_ew_fast(int dtype, const EwArgs& a, hipStream_t st);
// Column tiles of the bf16 MFMA GEMM for plain GEMMs and for conv GEMMs; the
// per-tile partial layouts of the terminal finishers follow them.
constexpr int kGemmTileN = 256;
constexpr int kConvTileN = 128;
// A bf16 conv GEMM whose chain is exactly (channel bias, ReLU) ending in an
// average pool, with C a multiple of 64 and at least 256 positions per image,
// runs on the persistent 256 x 256 kernel (column tiles of 256 positions);
// other conv GEMMs on the 256 x kConvTileN one.
bool conv_bias_relu_gap_wide(int dtype, int64_t C, int64_t PQ, const EpiDev& epi, bool gap,
                             int pool);
int64_t conv_gemm_tile_n(int dtype, int64_t C, int64_t PQ, const EpiDev& epi, bool gap,
                         int pool);
// mk_tuned_limit code: why these arguments cannot run on the MFMA kernel
// (MK_LIMIT_NONE when they can).
int gemm_mfma_limit(int dtype, const GemmArgs& a);
bool gemm_mfma_supported(int dtype, const GemmArgs& a);   // bf16 or fp32
// The MFMA kernel takes B as [N, K]; a [K, N] operand (layout 1) is first
// transposed into scratch of gemm_mfma_bt_bytes() bytes, and gemm_with_bt()
// gives the arguments that read it there.
int64_t gemm_mfma_bt_bytes(int dtype, const GemmArgs& a);
hipError_t launch_transpose_b(int dtype, const GemmArgs& a, void* dst, hipStream_t st);
GemmArgs gemm_with_bt(const GemmArgs& a, const void* bt);
hipError_t launch_gemm_mfma(int dtype, const GemmArgs& a, hipStream_t st);
// Column-tile width of the MFMA GEMM on these arguments: kGemmTileN, or 64
// when the 256 x 256 grid would have fewer than kSmallGemmTiles tiles (then a
// 64 x 64-tile kernel runs, k_gemm_small.hip); the per-tile partials of the
// terminal finishers follow it.
constexpr int kSmallGemmTiles = 64;
int64_t gemm_mfma_tile_n(int dtype, const GemmArgs& a);
// True when a [K, N] weight (layout 1) is read in place, with no transpose.
bool gemm_mfma_native_kn(int dtype, const GemmArgs& a);
hipError_t launch_gemm_small(int dtype, const GemmArgs& a, hipStream_t st);
// Implicit-GEMM conv: one packing launch (x -> zero-padded NHWC, w ->
// [K][R][S][C]), the GEMM kernel in conv mode, and for a fused GAP the
// finisher over per-tile partials.
struct ConvScratch {
  int64_t xp_bytes, wp_bytes, partial_bytes;
};
int conv_mfma_limit(int dtype, const ConvArgs& a);
bool conv_mfma_supported(int dtype, const ConvArgs& a);
ConvScratch conv_mfma_scratch(int dtype, const ConvArgs& a);
hipError_t launch_conv_pack(int dtype, const ConvArgs& a, void* xp, void* wp, hipStream_t st);
GemmArgs conv_gemm_args(const ConvArgs& a, const void* xp, const void* wp, float* partial);
hipError_t launch_gap_finish(int dtype, const ConvArgs& a, const float* partial, hipStream_t st);
int attn_fused_limit(int dtype, const AttnArgs& a);
bool attn_fused_supported(int dtype, const AttnArgs& a);
hipError_t launch_attn_fused(int dtype, const AttnArgs& a, hipStream_t st);

}  // namespace mk
