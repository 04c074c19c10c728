// Implementation table and subkernel dispatch.
//
// Every family has a tuned implementation (MK_IMPL_TUNED) and a simple one
// (MK_IMPL_SIMPLE); a subkernel's implementation can be swapped without
// touching the others (MKEvolve Sec. 3, "Swap").  Ids >= 100 are test-only
// mutants reproducing the eleven injected bugs of App. D (five attention,
// six FFN; the tile-boundary and accumulator bugs serve both blocks), used to
// show that per-stage verification catches them, plus one that leaves an
// output row unwritten (the verifier must not pass on stale output bytes).
// Mutants run on the simple kernels, except the epilogue-chain ones, which
// rewrite the chain.
#include "impls.hpp"

#include <algorithm>
#include <string>

#include "kernels.hpp"

namespace mk {

enum Mutant : int32_t {
  MUT_UNSAFE_SOFTMAX = 101,     // exp(x) without the row max subtracted
  MUT_MASK_OFF_BY_ONE = 102,    // the diagonal is masked too
  MUT_TILE_BOUNDARY = 103,      // the last partial (or last 16-deep) K tile is not loaded
  MUT_BF16_ACCUM = 104,         // the contraction accumulates in bf16
  MUT_SOFTMAX_WRONG_DIM = 105,  // softmax over dim -2 instead of -1
  MUT_UNSAFE_LAYERNORM = 106,   // rows scaled by 1/sigma without subtracting the mean
  MUT_GELU_SIGMOID = 107,       // x * sigmoid(1.702 x) instead of exact GELU
  MUT_NO_RESIDUAL = 108,        // residual add dropped
  MUT_RELU_FOR_GELU = 109,      // ReLU instead of GELU
  MUT_SKIP_LAST_ROW = 110       // a row kernel that leaves its last output row unwritten
};

static bool chain_has(const EpiChain& c, int code) {
  for (int i = 0; i < c.n; ++i)
    if (c.step[i].code == code) return true;
  return false;
}

static bool chain_has_gelu(const EpiChain& c) {
  return chain_has(c, EPI_GELU_ERF) || chain_has(c, EPI_GELU_TANH);
}

static const EpiChain* chain_of(const Subkernel& sk) {
  switch (sk.family) {
    case MK_FAM_GEMM: return &sk.gemm.epi;
    case MK_FAM_CONV: return &sk.conv.epi;
    case MK_FAM_EW: return &sk.ew.epi;
    case MK_FAM_ROW: return &sk.row.pre.epi;
    default: return nullptr;
  }
}

bool impl_exists(const Plan& p, const Subkernel& sk, int impl) {
  (void)p;
  if (impl == MK_IMPL_TUNED) return true;
  if (impl == MK_IMPL_SIMPLE) {
    if (sk.family == MK_FAM_ATTN) return sk.attn.S * 4 <= 65536;
    return true;
  }
  const EpiChain* c = chain_of(sk);
  switch (impl) {
    case MUT_MASK_OFF_BY_ONE:
      return (c && chain_has(*c, EPI_CAUSAL)) || (sk.family == MK_FAM_ATTN && sk.attn.causal);
    case MUT_TILE_BOUNDARY:
      return (sk.family == MK_FAM_GEMM && sk.gemm.K > 16) ||
             (sk.family == MK_FAM_ATTN && sk.attn.dh > 16 && sk.attn.S * 4 <= 65536);
    case MUT_UNSAFE_SOFTMAX:
      return sk.family == MK_FAM_ROW && sk.row.op == MK_OP_SOFTMAX;
    case MUT_SOFTMAX_WRONG_DIM:
      return sk.family == MK_FAM_ROW && sk.row.op == MK_OP_SOFTMAX && sk.row.n2 > 1;
    case MUT_BF16_ACCUM:
      return sk.family == MK_FAM_GEMM;
    case MUT_UNSAFE_LAYERNORM:
      return (sk.family == MK_FAM_ROW && sk.row.op == MK_OP_LAYERNORM) ||
             (sk.family == MK_FAM_GEMM && sk.gemm.ln);
    case MUT_GELU_SIGMOID: case MUT_RELU_FOR_GELU:
      return c && chain_has_gelu(*c);
    case MUT_NO_RESIDUAL:
      return c && chain_has(*c, EPI_ADD);
    case MUT_SKIP_LAST_ROW:
      return sk.family == MK_FAM_ROW && sk.row.rows > 1;
    default:
      return false;
  }
}

// The GEMM arguments of a subkernel as far as the host decides on them
// (operands unbound).
static GemmArgs gemm_probe(const Subkernel& sk) {
  GemmArgs probe{};
  probe.M = sk.gemm.M;
  probe.N = sk.gemm.N;
  probe.K = sk.gemm.K;
  probe.lda = sk.gemm.lda;
  probe.ldb = sk.gemm.ldb;
  probe.ldc = sk.gemm.ldc;
  probe.layout = sk.gemm.layout;
  probe.batch = (int32_t)sk.gemm.batch;
  probe.heads = (int32_t)sk.gemm.heads;
  probe.terminal = sk.gemm.terminal;
  probe.a_off = sk.gemm.a_off; probe.a_sb = sk.gemm.a_sb; probe.a_sh = sk.gemm.a_sh;
  probe.b_off = sk.gemm.b_off; probe.b_sb = sk.gemm.b_sb; probe.b_sh = sk.gemm.b_sh;
  probe.c_off = sk.gemm.c_off; probe.c_sb = sk.gemm.c_sb; probe.c_sh = sk.gemm.c_sh;
  return probe;
}

static bool use_mfma(const Plan& p, const Subkernel& sk, int impl) {
  if (impl != MK_IMPL_TUNED || sk.family != MK_FAM_GEMM) return false;
  return gemm_mfma_supported(p.dtype, gemm_probe(sk));
}

static EpiDev resolve(const EpiChain& c, const std::vector<void*>& vals, int impl);

// A softmax terminal over rows one wave holds: the MFMA GEMM writes the
// chain's values and a one-wave-per-row softmax runs after it in place.
static bool row_softmax_after(const Plan& p, const GemmSpec& g, bool mfma, const void* out,
                              RowArgs* rs_out) {
  if (!(mfma && g.terminal == TERM_SOFTMAX && g.batch * g.heads == 1 && g.ldc == g.N)) return false;
  RowArgs rs{};
  char* c0 = (char*)out + g.c_off * elem_size(p.dtype);
  rs.x = c0;
  rs.y = c0;
  rs.rows = g.M;
  rs.len = g.N;
  rs.op = MK_OP_SOFTMAX;
  rs.pre.last = rs.pre.S = rs.pre.C = rs.pre.HW = 1;
  rs.n2 = 1;
  if (rs_out) *rs_out = rs;
  return row_wave_supported(p.dtype, rs);
}

// A [K, N] weight the MFMA GEMM reads in place (no transpose launch); decided
// from the spec (the chain's steps, a 16-byte aligned bias assumed: the
// launch rejects an unaligned one).
static bool gemm_native_kn(const Plan& p, const Subkernel& sk, int impl) {
  const GemmSpec& g = sk.gemm;
  if (!use_mfma(p, sk, impl) || g.layout != 1) return false;
  GemmArgs a = gemm_probe(sk);
  int nv = 1;
  for (int i = 0; i < g.epi.n; ++i) nv = std::max(nv, g.epi.step[i].value + 1);
  std::vector<void*> dummy((size_t)nv, (void*)256);
  a.epi = resolve(g.epi, dummy, impl);
  a.alpha = g.alpha;
  if (row_softmax_after(p, g, true, nullptr, nullptr)) a.terminal = TERM_NONE;
  return gemm_mfma_native_kn(p.dtype, a);
}

static int64_t align256(int64_t b) { return (b + 255) / 256 * 256; }

// Scratch layout of a GEMM subkernel: [LayerNorm region][row partials].
// The MFMA path applies a LayerNorm prologue as a pre-pass that writes the
// normalised rows (storage dtype) to scratch; the simple path keeps per-row
// (mean, rstd) and normalises while loading A.
struct GemmScratch {
  bool mfma;
  int64_t tile_n, n_tiles, ln_bytes, bt_bytes, partial_bytes;
};

static GemmScratch gemm_scratch(const Plan& p, const Subkernel& sk, int impl) {
  const GemmSpec& g = sk.gemm;
  GemmScratch s{};
  s.mfma = use_mfma(p, sk, impl);
  s.tile_n = s.mfma ? gemm_mfma_tile_n(p.dtype, gemm_probe(sk)) : 64;
  s.n_tiles = (g.N + s.tile_n - 1) / s.tile_n;
  if (g.ln) s.ln_bytes = align256(s.mfma ? g.M * g.K * elem_size(p.dtype) : 2 * g.M * 4);
  if (s.mfma && g.layout == 1 && !gemm_native_kn(p, sk, impl))
    s.bt_bytes = align256(g.batch * g.heads * g.N * g.K * elem_size(p.dtype));
  if (g.terminal == TERM_ROWSUM) s.partial_bytes = align256(g.M * s.n_tiles * 4);
  if (g.terminal == TERM_SOFTMAX || g.terminal == TERM_LAYERNORM)
    s.partial_bytes = align256(g.M * s.n_tiles * 8);
  return s;
}

static ConvArgs conv_args(const ConvSpec& c) {
  ConvArgs a{};
  a.N = c.N; a.C = c.C; a.H = c.H; a.W = c.W; a.K = c.K; a.R = c.R; a.S = c.S;
  a.P = c.P; a.Q = c.Q; a.stride = c.stride; a.pad = c.pad;
  a.gap = c.gap ? 1 : 0;
  a.pool = c.pool;
  a.pool_p = c.pool_p;
  return a;
}

static bool use_conv_mfma(const Plan& p, const Subkernel& sk, int impl) {
  return impl != MK_IMPL_SIMPLE && sk.family == MK_FAM_CONV &&
         conv_mfma_supported(p.dtype, conv_args(sk.conv));
}

int64_t impl_scratch(const Plan& p, const Subkernel& sk, int impl) {
  if (sk.family == MK_FAM_CONV) {
    if (!use_conv_mfma(p, sk, impl)) return 0;
    const ConvScratch c = conv_mfma_scratch(p.dtype, conv_args(sk.conv));
    return c.xp_bytes + c.wp_bytes + c.partial_bytes;
  }
  if (sk.family != MK_FAM_GEMM) return 0;
  const GemmScratch s = gemm_scratch(p, sk, impl);
  return s.ln_bytes + s.bt_bytes + s.partial_bytes;
}

int64_t max_scratch_bytes(const Plan& p, const Subkernel& sk) {
  return std::max(impl_scratch(p, sk, MK_IMPL_TUNED), impl_scratch(p, sk, MK_IMPL_SIMPLE));
}

bool impl_uses_mfma(const Plan& p, const Subkernel& sk, int impl) {
  if (sk.family == MK_FAM_GEMM) return use_mfma(p, sk, impl);
  if (sk.family == MK_FAM_CONV) return use_conv_mfma(p, sk, impl);
  if (sk.family == MK_FAM_ATTN && impl != MK_IMPL_SIMPLE) {
    AttnArgs a{};
    a.B = sk.attn.B; a.H = sk.attn.H; a.dh = sk.attn.dh; a.S = sk.attn.S;
    a.causal = sk.attn.causal ? 1 : 0;
    return attn_fused_supported(p.dtype, a);
  }
  return false;
}

int tuned_limit(const Plan& p, const Subkernel& sk) {
  if (sk.family == MK_FAM_GEMM) return gemm_mfma_limit(p.dtype, gemm_probe(sk));
  if (sk.family == MK_FAM_CONV) return conv_mfma_limit(p.dtype, conv_args(sk.conv));
  if (sk.family == MK_FAM_ATTN) {
    AttnArgs a{};
    a.B = sk.attn.B; a.H = sk.attn.H; a.dh = sk.attn.dh; a.S = sk.attn.S;
    a.causal = sk.attn.causal ? 1 : 0;
    return attn_fused_limit(p.dtype, a);
  }
  return MK_LIMIT_NONE;
}

int impl_launches(const Plan& p, const Subkernel& sk, int impl) {
  if (sk.family == MK_FAM_GEMM) {
    const bool transpose = use_mfma(p, sk, impl) && sk.gemm.layout == 1 && !gemm_native_kn(p, sk, impl);
    return 1 + (sk.gemm.ln ? 1 : 0) + (transpose ? 1 : 0) +
           (sk.gemm.terminal != TERM_NONE ? 1 : 0);
  }
  if (sk.family == MK_FAM_CONV && use_conv_mfma(p, sk, impl)) return sk.conv.gap ? 3 : 2;
  return 1;
}

static EpiDev resolve(const EpiChain& c, const std::vector<void*>& vals, int impl) {
  EpiDev d{};
  for (int i = 0; i < c.n; ++i) {
    int code = c.step[i].code;
    if (impl == MUT_NO_RESIDUAL && code == EPI_ADD) continue;
    if (impl == MUT_RELU_FOR_GELU && (code == EPI_GELU_ERF || code == EPI_GELU_TANH))
      code = EPI_RELU;
    if (impl == MUT_GELU_SIGMOID && (code == EPI_GELU_ERF || code == EPI_GELU_TANH))
      code = EPI_GELU_SIGMOID;
    if (impl == MUT_MASK_OFF_BY_ONE && code == EPI_CAUSAL) code = EPI_CAUSAL_STRICT;
    d.code[d.n] = code;
    d.ptr[d.n] = c.step[i].value >= 0 ? vals[c.step[i].value] : nullptr;
    d.s[d.n] = c.step[i].s;
    ++d.n;
  }
  return d;
}

static EwArgs ew_args(const EwSpec& e, const std::vector<void*>& vals, void* out, int impl) {
  EwArgs a{};
  a.x = vals[e.x_value];
  a.y = out;
  a.numel = e.numel;
  a.last = e.last;
  a.C = e.C;
  a.HW = e.HW;
  a.S = e.S;
  a.epi = resolve(e.epi, vals, impl);
  return a;
}

static mk_status hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return MK_OK;
  return fail(MK_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

mk_status run_subkernel(const Plan& p, const Subkernel& sk, const std::vector<void*>& vals,
                        void* out, void* scratch, hipStream_t st, LaunchTimer* tm) {
  // Each launch is bracketed by tm->begin() / tm->end() when launch timing
  // is active.
  auto timed = [tm](auto&& launch) {
    if (tm) tm->begin();
    hipError_t e = launch();
    if (tm) tm->end();
    return e;
  };
  const int impl = sk.impl;
  const int dt = p.dtype;
  switch (sk.family) {
    case MK_FAM_EW:
      return hip_check(timed([&] { return launch_ew(dt, ew_args(sk.ew, vals, out, impl), st, impl); }),
                       "element-wise");
    case MK_FAM_ROW: {
      const RowSpec& r = sk.row;
      RowArgs a{};
      a.x = vals[r.x_value];
      a.y = out;
      a.rows = impl == MUT_SKIP_LAST_ROW ? r.rows - 1 : r.rows;
      a.len = r.len;
      a.op = r.op;
      a.gamma = r.g_value >= 0 ? vals[r.g_value] : nullptr;
      a.beta = r.b_value >= 0 ? vals[r.b_value] : nullptr;
      a.eps = r.eps;
      a.pre = ew_args(r.pre, vals, nullptr, impl);
      a.n2 = r.n2;
      a.p = r.p;
      a.variant = impl == MUT_UNSAFE_SOFTMAX      ? 1
                  : impl == MUT_SOFTMAX_WRONG_DIM ? 2
                  : impl == MUT_UNSAFE_LAYERNORM  ? 3
                                                  : 0;
      return hip_check(timed([&] { return launch_row(dt, a, st, impl); }), "row");
    }
    case MK_FAM_GEMM: {
      const GemmSpec& g = sk.gemm;
      GemmArgs a{};
      a.A = vals[g.a_value];
      a.B = vals[g.b_value];
      a.C = out;
      a.M = g.M; a.N = g.N; a.K = g.K;
      a.lda = g.lda; a.ldb = g.ldb; a.ldc = g.ldc;
      a.a_off = g.a_off; a.a_sb = g.a_sb; a.a_sh = g.a_sh;
      a.b_off = g.b_off; a.b_sb = g.b_sb; a.b_sh = g.b_sh;
      a.c_off = g.c_off; a.c_sb = g.c_sb; a.c_sh = g.c_sh;
      a.batch = (int32_t)g.batch;
      a.heads = (int32_t)g.heads;
      a.layout = g.layout;
      a.terminal = g.terminal;
      a.alpha = g.alpha;
      a.acc_bf16 = impl == MUT_BF16_ACCUM ? 1 : 0;
      a.epi = resolve(g.epi, vals, impl);
      if (impl == MUT_TILE_BOUNDARY) a.K = g.K - ((g.K % 16) ? (g.K % 16) : 16);
      const GemmScratch gs = gemm_scratch(p, sk, impl);
      const bool aligned = ((uintptr_t)a.B % 16 == 0) && ((uintptr_t)vals[g.a_value] % 16 == 0);
      if (gs.mfma && !aligned) return fail(MK_E_INVALID_ARG, "GEMM operands must be 16-byte aligned");
      char* sc = (char*)scratch;
      if (g.ln) {
        if (gs.mfma) {
          RowArgs r{};
          r.x = vals[g.a_value];
          r.y = sc;
          r.rows = g.M;
          r.len = g.K;
          r.op = MK_OP_LAYERNORM;
          r.gamma = vals[g.ln_g];
          r.beta = vals[g.ln_b];
          r.eps = g.eps;
          r.pre.last = r.pre.S = r.pre.C = r.pre.HW = 1;
          mk_status s = hip_check(timed([&] { return launch_row(dt, r, st, MK_IMPL_TUNED); }),
                                  "layernorm prologue");
          if (s != MK_OK) return s;
          a.A = sc;
        } else {
          float* stats = (float*)sc;
          mk_status s = hip_check(timed([&] {
                                    return launch_ln_stats(dt, vals[g.a_value], g.M, g.K, g.eps,
                                                           stats, st,
                                                           impl == MUT_UNSAFE_LAYERNORM);
                                  }),
                                  "layernorm stats");
          if (s != MK_OK) return s;
          a.ln_stats = stats;
          a.ln_g = vals[g.ln_g];
          a.ln_b = vals[g.ln_b];
        }
        sc += gs.ln_bytes;
      }
      if (gs.bt_bytes) {
        void* bt = sc;
        mk_status s = hip_check(timed([&] { return launch_transpose_b(dt, a, bt, st); }),
                                "transpose B");
        if (s != MK_OK) return s;
        a = gemm_with_bt(a, bt);
        sc += gs.bt_bytes;
      }
      a.partial = (float*)sc;
      a.n_tiles = gs.n_tiles;
      // A softmax over rows one wave can hold: the GEMM writes the chain's
      // values (as stored, i.e. rounded) and a one-wave-per-row softmax reads
      // them back in place (max, exp, sum, normalise; the same HBM traffic as
      // the partials' finisher, and no softmax work in the GEMM epilogue).
      // Otherwise the epilogue emits per-tile partials for the finisher.
      RowArgs rs{};
      const bool row_softmax = row_softmax_after(p, g, gs.mfma, out, &rs);
      if (row_softmax) a.terminal = TERM_NONE;
      if (gs.mfma && a.layout == 1 && !gs.bt_bytes && !gemm_mfma_native_kn(dt, a))
        return fail(MK_E_INVALID_ARG, "GEMM chain operands must be 16-byte aligned");
      mk_status s = hip_check(timed([&] {
                                return gs.mfma ? launch_gemm_mfma(dt, a, st)
                                               : launch_gemm_simple(dt, a, st);
                              }),
                              "gemm");
      if (s != MK_OK) return s;
      if (row_softmax)
        return hip_check(timed([&] { return launch_row(dt, rs, st, MK_IMPL_TUNED); }),
                         "softmax rows");
      if (g.terminal == TERM_ROWSUM)
        return hip_check(timed([&] {
                           return launch_rowsum_finish(dt, a.partial, g.M, a.n_tiles, out, st);
                         }),
                         "row-sum finish");
      if (g.terminal == TERM_LAYERNORM)
        return hip_check(timed([&] {
                           return launch_ln_finish(dt, a.partial, g.M, a.n_tiles, g.N,
                                                   gs.tile_n, vals[g.post_g],
                                                   vals[g.post_b], g.post_eps, out, st);
                         }),
                         "layernorm finish");
      if (g.terminal == TERM_SOFTMAX)
        return hip_check(timed([&] {
                           return launch_softmax_finish(dt, a.partial, g.M, a.n_tiles, g.N, out,
                                                        st);
                         }),
                         "softmax finish");
      return MK_OK;
    }
    case MK_FAM_CONV: {
      const ConvSpec& c = sk.conv;
      ConvArgs a = conv_args(c);
      a.x = vals[c.x_value];
      a.w = vals[c.w_value];
      a.y = out;
      a.epi = resolve(c.epi, vals, impl);
      if (!use_conv_mfma(p, sk, impl))
        return hip_check(timed([&] { return launch_conv_simple(dt, a, st); }), "conv");
      // Implicit GEMM: repack input and weights into scratch, run the MFMA
      // GEMM in conv mode, then (GAP) combine the per-tile partials.
      const ConvScratch cs = conv_mfma_scratch(dt, a);
      char* xp = (char*)scratch;
      char* wp = xp + cs.xp_bytes;
      float* part = (float*)(wp + cs.wp_bytes);
      mk_status s =
          hip_check(timed([&] { return launch_conv_pack(dt, a, xp, wp, st); }), "conv pack");
      if (s != MK_OK) return s;
      const GemmArgs g = conv_gemm_args(a, xp, wp, part);
      s = hip_check(timed([&] { return launch_gemm_mfma(dt, g, st); }), "conv gemm");
      if (s != MK_OK || !a.gap) return s;
      return hip_check(timed([&] { return launch_gap_finish(dt, a, part, st); }), "gap finish");
    }
    case MK_FAM_ATTN: {
      const AttnSpec& t = sk.attn;
      AttnArgs a{};
      a.qkv = vals[t.qkv_value];
      a.o = out;
      a.B = t.B; a.H = t.H; a.dh = t.dh; a.S = t.S;
      a.scale = t.scale;
      a.causal = t.causal ? (impl == MUT_MASK_OFF_BY_ONE ? 2 : 1) : 0;
      a.kdim = impl == MUT_TILE_BOUNDARY ? t.dh - ((t.dh % 16) ? (t.dh % 16) : 16) : t.dh;
      const bool fused = impl != MK_IMPL_SIMPLE && impl != MUT_TILE_BOUNDARY &&
                         attn_fused_supported(dt, a) &&
                         (uintptr_t)a.qkv % 16 == 0 && (uintptr_t)a.o % 16 == 0;
      return hip_check(timed([&] {
                         return fused ? launch_attn_fused(dt, a, st)
                                      : launch_attn_simple(dt, a, st);
                       }),
                       "attention");
    }
    default:
      return fail(MK_E_INTERNAL, "unknown family");
  }
}

}  // namespace mk
