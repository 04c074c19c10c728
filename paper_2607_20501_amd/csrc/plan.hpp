// Host-side plan of a composed module: shape inference, grouping validation,
// family matching and workspace layout.  The structs here are what the
// executor hands to the kernel launchers; no device code.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/mk.h"
#include "plan_codes.hpp"

namespace mk {

// Last-error text (thread-local), set by every failing ABI call.
void set_error(const std::string& msg);
mk_status fail(mk_status s, const std::string& msg);

struct EpiStep {
  int32_t code;
  int32_t value;   // value id of the bias / residual operand, -1 if none
  float s;         // scale
};

struct EpiChain {
  int32_t n = 0;
  EpiStep step[kMaxEpi];
};

enum GemmKind : int32_t { GK_PLAIN = 0, GK_QK = 1, GK_PV = 2 };

// C[z][m, n] = chain(alpha * sum_k A[z][m, k] * B[z](k, n)) for z = b * heads + h.
// Element offsets: A[z] starts at a_off + b * a_sb + h * a_sh with row stride lda;
// B(k, n) is at b_off + b * b_sb + h * b_sh + (layout 0: n * ldb + k, 1: k * ldb + n);
// C[z] at c_off + b * c_sb + h * c_sh with row stride ldc.
struct GemmSpec {
  int32_t kind = GK_PLAIN;
  bool ln = false;                 // LayerNorm prologue applied to A rows
  int32_t ln_g = -1, ln_b = -1;    // gamma / beta value ids
  float eps = 0.f;
  int32_t a_value = -1, b_value = -1;
  int32_t layout = 0;
  int64_t M = 0, N = 0, K = 0;
  int64_t batch = 1, heads = 1;
  int64_t lda = 0, ldb = 0, ldc = 0;
  int64_t a_off = 0, a_sb = 0, a_sh = 0;
  int64_t b_off = 0, b_sb = 0, b_sh = 0;
  int64_t c_off = 0, c_sb = 0, c_sh = 0;
  float alpha = 1.f;
  EpiChain epi;
  int32_t terminal = TERM_NONE;
  int32_t post_g = -1, post_b = -1;   // TERM_LAYERNORM gamma / beta value ids
  float post_eps = 0.f;
};

struct ConvSpec {
  int32_t x_value = -1, w_value = -1;
  int64_t N = 0, C = 0, H = 0, W = 0, K = 0, R = 0, S = 0, P = 0, Q = 0, stride = 1, pad = 0;
  EpiChain epi;          // channel-indexed chain
  bool gap = false;      // ends in a global pool
  int32_t pool = MK_OP_GAP;   // GAP, GMP or LPPOOL
  float pool_p = 1.f;         // LPPOOL exponent
};

struct EwSpec {
  int32_t x_value = -1;
  int64_t numel = 0;
  int64_t last = 1;      // last dimension (BIAS_COL index = flat % last)
  int64_t C = 1, HW = 1; // BIAS_CH index = (flat / HW) % C
  int64_t S = 1;         // CAUSAL: row = (flat / S) % S, col = flat % S
  EpiChain epi;
};

struct RowSpec {
  int32_t x_value = -1;
  int32_t op = MK_OP_ROWSUM;   // ROWSUM, SOFTMAX, LAYERNORM or GAP
  int64_t rows = 0, len = 0;
  EwSpec pre;                  // element-wise prologue on the input (indexing as EwSpec)
  int32_t g_value = -1, b_value = -1;
  float eps = 0.f;
  int64_t n2 = 1;              // size of the input's dim -2 (1 for a vector)
  float p = 1.f;               // LPPOOL exponent
};

struct AttnSpec {
  int32_t qkv_value = -1;
  int64_t B = 0, H = 0, dh = 0, S = 0;
  float scale = 1.f;
  bool causal = false;
};

struct Subkernel {
  int32_t op_begin = 0, op_end = 0, out_value = -1;
  int32_t family = MK_FAM_EW, impl = MK_IMPL_TUNED;
  int64_t ws_offset = -1, out_bytes = 0, flops = 0, alg_bytes = 0;
  GemmSpec gemm;
  ConvSpec conv;
  EwSpec ew;
  RowSpec row;
  AttnSpec attn;
};

struct Plan {
  int32_t dtype = MK_F32;
  int32_t n_inputs = 0;
  std::vector<mk_op> ops;
  std::vector<mk_shape> vshape;   // [n_inputs + n_ops]
  std::vector<int32_t> group;
  std::vector<Subkernel> subs;
  int64_t ws_intermediate = 0;
  int64_t scratch_off = 0;
  int64_t scratch_bytes = 0;
  int64_t flops = 0, alg_bytes = 0;
};

int64_t numel(const mk_shape& s);
int64_t elem_size(int32_t dtype);

// Shape inference for every value; MK_OK or MK_E_* with the error text set.
mk_status infer(const mk_module_desc* d, std::vector<mk_shape>& vshape);
// Does the op range [b, e) match a family?  Fills sk's family and spec.
bool match_group(const Plan& p, int32_t b, int32_t e, Subkernel& sk, std::string* why);
// Are the values produced inside [b, e) other than its last read only inside it?
bool group_closed(const Plan& p, int32_t b, int32_t e);
mk_status build_plan(const mk_module_desc* d, const int32_t* group_of_op, Plan& p);
mk_status preset(const mk_module_desc* d, int32_t which, int32_t* group_of_op);

}  // namespace mk
