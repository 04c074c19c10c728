// Shape inference, grouping validation, family matching, presets and the
// workspace layout of a composed module.
//
// A module is an operator sequence; a decomposition partitions it into
// contiguous subproblems that a top-level module chains (MKEvolve Sec. 3,
// "LLMDecompose agent": every value the chain needs must be covered by the
// subproblems, checked programmatically).  Which groups may become one
// subkernel follows the paper's fusion guidance (App. I.1, "fusion-friendly
// groupings"): a GEMM with bias, element-wise activations, scaling and the
// residual add; chains of element-wise ops; attention as QK^T, scale, mask,
// softmax and PV in one kernel when online softmax is possible; splits at
// global reductions otherwise.
#include "plan.hpp"

#include <algorithm>
#include <cmath>

#include "impls.hpp"

namespace mk {

static thread_local std::string g_err;

void set_error(const std::string& msg) { g_err = msg; }
const char* last_error() { return g_err.c_str(); }

mk_status fail(mk_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

int64_t numel(const mk_shape& s) {
  int64_t n = 1;
  for (int i = 0; i < s.ndim; ++i) n *= s.dims[i];
  return n;
}

int64_t elem_size(int32_t dtype) { return dtype == MK_BF16 ? 2 : 4; }

static int n_operands(int32_t kind) {
  switch (kind) {
    case MK_OP_GEMM: case MK_OP_BIAS: case MK_OP_BIAS_CHANNEL: case MK_OP_ADD:
    case MK_OP_CONV2D: case MK_OP_PV:
      return 2;
    case MK_OP_LAYERNORM:
      return 3;
    default:
      return 1;
  }
}

static bool same_shape(const mk_shape& a, const mk_shape& b) {
  if (a.ndim != b.ndim) return false;
  for (int i = 0; i < a.ndim; ++i)
    if (a.dims[i] != b.dims[i]) return false;
  return true;
}

static mk_shape make_shape(std::initializer_list<int64_t> d) {
  mk_shape s{};
  s.ndim = (int32_t)d.size();
  int i = 0;
  for (int64_t v : d) s.dims[i++] = v;
  return s;
}

mk_status infer(const mk_module_desc* d, std::vector<mk_shape>& vs) {
  if (!d || !d->ops || d->n_ops < 1 || d->n_ops > 64 || d->n_inputs < 0 || d->n_inputs > 64 ||
      (d->n_inputs > 0 && !d->input_shapes))
    return fail(MK_E_INVALID_ARG, "module descriptor: null pointer or op/input count out of range");
  if (d->dtype != MK_F32 && d->dtype != MK_BF16) return fail(MK_E_DTYPE, "unknown dtype");
  vs.assign(d->n_inputs + d->n_ops, mk_shape{});
  for (int i = 0; i < d->n_inputs; ++i) {
    const mk_shape& s = d->input_shapes[i];
    if (s.ndim < 1 || s.ndim > 4) return fail(MK_E_SHAPE, "input " + std::to_string(i) + ": ndim");
    for (int k = 0; k < s.ndim; ++k)
      if (s.dims[k] < 1) return fail(MK_E_SHAPE, "input " + std::to_string(i) + ": empty dim");
    vs[i] = s;
    for (int k = s.ndim; k < 4; ++k) vs[i].dims[k] = 0;
  }
  for (int i = 0; i < d->n_ops; ++i) {
    const mk_op& o = d->ops[i];
    std::string where = "op " + std::to_string(i) + ": ";
    if (o.kind < 0 || o.kind >= MK_OP_COUNT) return fail(MK_E_INVALID_ARG, where + "unknown kind");
    for (int k = 0; k < n_operands(o.kind); ++k)
      if (o.in[k] < 0 || o.in[k] >= d->n_inputs + i)
        return fail(MK_E_INVALID_ARG, where + "operand is not an earlier value");
    const mk_shape x = vs[o.in[0]];
    const int64_t last = x.dims[x.ndim - 1];
    mk_shape y = x;
    switch (o.kind) {
      case MK_OP_GEMM: {
        const mk_shape& w = vs[o.in[1]];
        if (w.ndim != 2 || (o.ip[0] != 0 && o.ip[0] != 1))
          return fail(MK_E_SHAPE, where + "GEMM weight must be 2-D with layout 0 or 1");
        int64_t K = o.ip[0] == 0 ? w.dims[1] : w.dims[0];
        int64_t N = o.ip[0] == 0 ? w.dims[0] : w.dims[1];
        if (last != K) return fail(MK_E_SHAPE, where + "GEMM inner dimensions differ");
        y.dims[y.ndim - 1] = N;
        break;
      }
      case MK_OP_BIAS: {
        const mk_shape& b = vs[o.in[1]];
        if (b.ndim != 1 || b.dims[0] != last) return fail(MK_E_SHAPE, where + "bias length");
        break;
      }
      case MK_OP_BIAS_CHANNEL: {
        const mk_shape& b = vs[o.in[1]];
        if (x.ndim != 4 || b.ndim != 1 || b.dims[0] != x.dims[1])
          return fail(MK_E_SHAPE, where + "channel bias needs x[N,C,H,W] and b[C]");
        break;
      }
      case MK_OP_RELU: case MK_OP_GELU_ERF: case MK_OP_GELU_TANH: case MK_OP_SCALE:
      case MK_OP_SOFTMAX:
        break;
      case MK_OP_ADD:
        if (!same_shape(x, vs[o.in[1]])) return fail(MK_E_SHAPE, where + "ADD operand shapes");
        break;
      case MK_OP_ROWSUM:
        if (x.ndim < 2) return fail(MK_E_SHAPE, where + "ROWSUM needs ndim >= 2");
        y.ndim = x.ndim - 1;
        break;
      case MK_OP_LAYERNORM: {
        const mk_shape& g = vs[o.in[1]];
        const mk_shape& b = vs[o.in[2]];
        if (g.ndim != 1 || b.ndim != 1 || g.dims[0] != last || b.dims[0] != last)
          return fail(MK_E_SHAPE, where + "LayerNorm gamma/beta length");
        if (!(o.fp[0] >= 0.0)) return fail(MK_E_SHAPE, where + "LayerNorm eps < 0");
        break;
      }
      case MK_OP_CONV2D: {
        const mk_shape& w = vs[o.in[1]];
        const int64_t st = o.ip[0], pd = o.ip[1];
        if (x.ndim != 4 || w.ndim != 4 || w.dims[1] != x.dims[1] || st < 1 || pd < 0)
          return fail(MK_E_SHAPE, where + "conv needs x[N,C,H,W], w[K,C,R,S], stride >= 1");
        const int64_t hp = x.dims[2] + 2 * pd - w.dims[2], wp = x.dims[3] + 2 * pd - w.dims[3];
        if (hp < 0 || wp < 0) return fail(MK_E_SHAPE, where + "conv window larger than input");
        y = make_shape({x.dims[0], w.dims[0], hp / st + 1, wp / st + 1});
        break;
      }
      case MK_OP_GAP: case MK_OP_GMP: case MK_OP_LPPOOL:
        if (x.ndim != 4) return fail(MK_E_SHAPE, where + "global pool needs [N,C,H,W]");
        if (o.kind == MK_OP_LPPOOL && !(o.fp[0] > 0.0))
          return fail(MK_E_SHAPE, where + "LPPOOL needs p > 0");
        y = make_shape({x.dims[0], x.dims[1]});
        break;
      case MK_OP_QK: case MK_OP_PV: {
        const int64_t B = o.ip[0], H = o.ip[1], dh = o.ip[2], S = o.ip[3];
        if (B < 1 || H < 1 || dh < 1 || S < 1) return fail(MK_E_SHAPE, where + "B, H, dh, S >= 1");
        const mk_shape& q = vs[o.in[o.kind == MK_OP_QK ? 0 : 1]];
        if (numel(q) != B * S * 3 * H * dh || q.dims[q.ndim - 1] != 3 * H * dh)
          return fail(MK_E_SHAPE, where + "qkv must hold B*S rows of 3*H*dh");
        if (o.kind == MK_OP_QK) {
          y = make_shape({B, H, S, S});
        } else {
          if (!same_shape(x, make_shape({B, H, S, S})))
            return fail(MK_E_SHAPE, where + "PV probabilities must be [B,H,S,S]");
          y = make_shape({B, S, H * dh});
        }
        break;
      }
      case MK_OP_CAUSAL_MASK:
        if (x.ndim < 2 || x.dims[x.ndim - 1] != x.dims[x.ndim - 2])
          return fail(MK_E_SHAPE, where + "causal mask needs square trailing dims");
        break;
      default:
        return fail(MK_E_INVALID_ARG, where + "unknown kind");
    }
    for (int k = y.ndim; k < 4; ++k) y.dims[k] = 0;
    vs[d->n_inputs + i] = y;
  }
  return MK_OK;
}

// ---------------------------------------------------------------- flops/bytes

static bool qk_masked(const Plan& p, int i) {
  const int v = p.n_inputs + i;
  for (size_t j = i + 1; j < p.ops.size(); ++j)
    if (p.ops[j].kind == MK_OP_CAUSAL_MASK && p.ops[j].in[0] == v) return true;
  return false;
}

static bool pv_masked(const Plan& p, int i) {
  const int sm = p.ops[i].in[0] - p.n_inputs;
  if (sm < 0 || p.ops[sm].kind != MK_OP_SOFTMAX) return false;
  const int mk = p.ops[sm].in[0] - p.n_inputs;
  return mk >= 0 && p.ops[mk].kind == MK_OP_CAUSAL_MASK;
}

// Algorithmic flops: contractions only; causal attention counts the kept
// (j <= i) score entries.
static int64_t flops_of(const Plan& p, int i) {
  const mk_op& o = p.ops[i];
  const mk_shape& y = p.vshape[p.n_inputs + i];
  switch (o.kind) {
    case MK_OP_GEMM: {
      const mk_shape& a = p.vshape[o.in[0]];
      const int64_t K = a.dims[a.ndim - 1];
      return 2 * (numel(a) / K) * y.dims[y.ndim - 1] * K;
    }
    case MK_OP_CONV2D: {
      const mk_shape& w = p.vshape[o.in[1]];
      return 2 * y.dims[0] * y.dims[2] * y.dims[3] * w.dims[0] * w.dims[1] * w.dims[2] * w.dims[3];
    }
    case MK_OP_QK: case MK_OP_PV: {
      const int64_t S = o.ip[3];
      const bool causal = o.kind == MK_OP_QK ? qk_masked(p, i) : pv_masked(p, i);
      return 2 * o.ip[0] * o.ip[1] * o.ip[2] * (causal ? S * (S + 1) / 2 : S * S);
    }
    default:
      return 0;
  }
}

// ---------------------------------------------------------------- matching

static bool is_ew(int32_t kind) {
  switch (kind) {
    case MK_OP_BIAS: case MK_OP_BIAS_CHANNEL: case MK_OP_RELU: case MK_OP_GELU_ERF:
    case MK_OP_GELU_TANH: case MK_OP_SCALE: case MK_OP_ADD: case MK_OP_CAUSAL_MASK:
      return true;
    default:
      return false;
  }
}

static bool inside(int32_t v, int32_t vb, int32_t ve) { return v >= vb && v < ve; }

// Append op i as a chain step; `ctx` restricts which steps are legal:
// 0 element-wise pass, 1 GEMM epilogue, 2 QK epilogue, 3 conv epilogue.
static bool push_step(const Plan& p, int i, int32_t vb, int32_t ve, int ctx, EpiChain& c,
                      std::string* why) {
  const mk_op& o = p.ops[i];
  if (c.n >= kMaxEpi) {
    if (why) *why = "element-wise chain longer than 8";
    return false;
  }
  EpiStep s{0, -1, 1.f};
  switch (o.kind) {
    case MK_OP_BIAS:
      if (ctx == 3 || ctx == 2) return false;
      s.code = EPI_BIAS_COL;
      s.value = o.in[1];
      break;
    case MK_OP_BIAS_CHANNEL:
      if (ctx == 1 || ctx == 2) return false;
      s.code = EPI_BIAS_CH;
      s.value = o.in[1];
      break;
    case MK_OP_RELU: s.code = EPI_RELU; break;
    case MK_OP_GELU_ERF: s.code = EPI_GELU_ERF; break;
    case MK_OP_GELU_TANH: s.code = EPI_GELU_TANH; break;
    case MK_OP_SCALE: s.code = EPI_SCALE; s.s = (float)o.fp[0]; break;
    case MK_OP_ADD: s.code = EPI_ADD; s.value = o.in[1]; break;
    case MK_OP_CAUSAL_MASK:
      if (ctx == 1 || ctx == 3) return false;
      s.code = EPI_CAUSAL;
      break;
    default:
      return false;
  }
  if (s.value >= 0 && inside(s.value, vb, ve)) {
    if (why) *why = "second operand produced inside the group";
    return false;
  }
  c.step[c.n++] = s;
  return true;
}

static void ew_indexing(const mk_shape& s, EwSpec& e) {
  e.numel = numel(s);
  e.last = s.dims[s.ndim - 1];
  e.C = s.ndim == 4 ? s.dims[1] : 1;
  e.HW = s.ndim == 4 ? s.dims[2] * s.dims[3] : 1;
  e.S = s.dims[s.ndim - 1];
}

bool match_group(const Plan& p, int32_t b, int32_t e, Subkernel& sk, std::string* why) {
  const int32_t vb = p.n_inputs + b, ve = p.n_inputs + e;
  auto val = [&](int i) { return p.n_inputs + i; };
  auto chained = [&](int i) { return i == b || p.ops[i].in[0] == val(i - 1); };
  for (int i = b; i < e; ++i)
    if (!chained(i)) {
      if (why) *why = "op " + std::to_string(i) + " does not consume the previous op's output";
      return false;
    }
  const mk_op& first = p.ops[b];
  const int n = e - b;

  // Attention: QK [CAUSAL_MASK] SOFTMAX PV, with PV reading the same qkv.
  if (first.kind == MK_OP_QK && (n == 3 || n == 4)) {
    const bool masked = n == 4;
    if ((!masked || p.ops[b + 1].kind == MK_OP_CAUSAL_MASK) &&
        p.ops[e - 2].kind == MK_OP_SOFTMAX && p.ops[e - 1].kind == MK_OP_PV &&
        p.ops[e - 1].in[1] == first.in[0]) {
      bool same = true;
      for (int k = 0; k < 4; ++k) same = same && p.ops[e - 1].ip[k] == first.ip[k];
      if (same) {
        sk.family = MK_FAM_ATTN;
        AttnSpec& a = sk.attn;
        a.qkv_value = first.in[0];
        a.B = first.ip[0];
        a.H = first.ip[1];
        a.dh = first.ip[2];
        a.S = first.ip[3];
        a.scale = (float)first.fp[0];
        a.causal = masked;
        return true;
      }
    }
  }

  // GEMM family: [LAYERNORM] GEMM|QK|PV, epilogue, [ROWSUM|SOFTMAX|LAYERNORM].
  {
    int i = b;
    GemmSpec g;
    if (p.ops[i].kind == MK_OP_LAYERNORM && i + 1 < e && p.ops[i + 1].kind == MK_OP_GEMM) {
      g.ln = true;
      g.ln_g = p.ops[i].in[1];
      g.ln_b = p.ops[i].in[2];
      g.eps = (float)p.ops[i].fp[0];
      g.a_value = p.ops[i].in[0];
      ++i;
    }
    const mk_op& c = p.ops[i];
    if (c.kind == MK_OP_GEMM || c.kind == MK_OP_QK || c.kind == MK_OP_PV) {
      const mk_shape& y = p.vshape[val(i)];
      if (c.kind == MK_OP_GEMM) {
        if (!g.ln) g.a_value = c.in[0];
        g.b_value = c.in[1];
        g.layout = (int32_t)c.ip[0];
        const mk_shape& a = p.vshape[g.a_value];
        g.K = a.dims[a.ndim - 1];
        g.M = numel(a) / g.K;
        g.N = y.dims[y.ndim - 1];
        g.lda = g.K;
        g.ldb = g.layout == 0 ? g.K : g.N;
        g.ldc = g.N;
      } else {
        const int64_t B = c.ip[0], H = c.ip[1], dh = c.ip[2], S = c.ip[3];
        const int64_t ld3 = 3 * H * dh;
        g.batch = B;
        g.heads = H;
        if (c.kind == MK_OP_QK) {
          g.kind = GK_QK;
          g.a_value = g.b_value = c.in[0];
          g.M = S; g.N = S; g.K = dh;
          g.lda = ld3; g.a_off = 0; g.a_sb = S * ld3; g.a_sh = dh;
          g.layout = 0; g.ldb = ld3; g.b_off = H * dh; g.b_sb = S * ld3; g.b_sh = dh;
          g.ldc = S; g.c_off = 0; g.c_sb = H * S * S; g.c_sh = S * S;
          g.alpha = (float)c.fp[0];
        } else {
          g.kind = GK_PV;
          g.a_value = c.in[0];
          g.b_value = c.in[1];
          g.M = S; g.N = dh; g.K = S;
          g.lda = S; g.a_off = 0; g.a_sb = H * S * S; g.a_sh = S * S;
          g.layout = 1; g.ldb = ld3; g.b_off = 2 * H * dh; g.b_sb = S * ld3; g.b_sh = dh;
          g.ldc = H * dh; g.c_off = 0; g.c_sb = S * H * dh; g.c_sh = dh;
        }
      }
      ++i;
      const int ctx = c.kind == MK_OP_QK ? 2 : 1;
      bool ok = true;
      for (; i < e && ok; ++i) {
        const int32_t k = p.ops[i].kind;
        if ((k == MK_OP_ROWSUM || k == MK_OP_SOFTMAX || k == MK_OP_LAYERNORM) && i == e - 1 &&
            c.kind == MK_OP_GEMM) {
          g.terminal = k == MK_OP_ROWSUM    ? TERM_ROWSUM
                       : k == MK_OP_SOFTMAX ? TERM_SOFTMAX
                                            : TERM_LAYERNORM;
          if (k == MK_OP_LAYERNORM) {
            g.post_g = p.ops[i].in[1];
            g.post_b = p.ops[i].in[2];
            g.post_eps = (float)p.ops[i].fp[0];
          }
          continue;
        }
        ok = push_step(p, i, vb, ve, ctx, g.epi, why);
      }
      if (ok) {
        sk.family = MK_FAM_GEMM;
        sk.gemm = g;
        return true;
      }
      return false;
    }
  }

  // Conv family: CONV2D, channel epilogue, [GAP].
  if (first.kind == MK_OP_CONV2D) {
    ConvSpec cs;
    const mk_shape& x = p.vshape[first.in[0]];
    const mk_shape& w = p.vshape[first.in[1]];
    const mk_shape& y = p.vshape[vb];
    cs.x_value = first.in[0];
    cs.w_value = first.in[1];
    cs.N = x.dims[0]; cs.C = x.dims[1]; cs.H = x.dims[2]; cs.W = x.dims[3];
    cs.K = w.dims[0]; cs.R = w.dims[2]; cs.S = w.dims[3];
    cs.P = y.dims[2]; cs.Q = y.dims[3];
    cs.stride = first.ip[0];
    cs.pad = first.ip[1];
    for (int i = b + 1; i < e; ++i) {
      const int32_t k = p.ops[i].kind;
      if ((k == MK_OP_GAP || k == MK_OP_GMP || k == MK_OP_LPPOOL) && i == e - 1) {
        cs.gap = true;
        cs.pool = k;
        cs.pool_p = k == MK_OP_LPPOOL ? (float)p.ops[i].fp[0] : 1.f;
        continue;
      }
      if (!push_step(p, i, vb, ve, 3, cs.epi, why)) return false;
    }
    sk.family = MK_FAM_CONV;
    sk.conv = cs;
    return true;
  }

  // Row family: element-wise prologue, then one row op.
  {
    const mk_op& last = p.ops[e - 1];
    const bool pool = last.kind == MK_OP_GAP || last.kind == MK_OP_GMP ||
                      last.kind == MK_OP_LPPOOL;
    if (last.kind == MK_OP_ROWSUM || last.kind == MK_OP_SOFTMAX || last.kind == MK_OP_LAYERNORM ||
        pool) {
      RowSpec r;
      r.x_value = first.in[0];
      const mk_shape& x = p.vshape[r.x_value];
      ew_indexing(x, r.pre);
      r.pre.x_value = r.x_value;
      for (int i = b; i < e - 1; ++i)
        if (!push_step(p, i, vb, ve, 0, r.pre.epi, why)) return false;
      r.op = last.kind;
      const mk_shape& xin = p.vshape[last.in[0]];
      if (pool) {
        r.len = xin.dims[2] * xin.dims[3];
        r.rows = xin.dims[0] * xin.dims[1];
        r.p = last.kind == MK_OP_LPPOOL ? (float)last.fp[0] : 1.f;
      } else {
        r.len = xin.dims[xin.ndim - 1];
        r.rows = numel(xin) / r.len;
        r.n2 = xin.ndim >= 2 ? xin.dims[xin.ndim - 2] : 1;
      }
      if (last.kind == MK_OP_LAYERNORM) {
        r.g_value = last.in[1];
        r.b_value = last.in[2];
        r.eps = (float)last.fp[0];
      }
      sk.family = MK_FAM_ROW;
      sk.row = r;
      return true;
    }
  }

  // Element-wise chain.
  if (is_ew(first.kind)) {
    EwSpec ew;
    ew.x_value = first.in[0];
    ew_indexing(p.vshape[ew.x_value], ew);
    for (int i = b; i < e; ++i)
      if (!push_step(p, i, vb, ve, 0, ew.epi, why)) return false;
    sk.family = MK_FAM_EW;
    sk.ew = ew;
    return true;
  }
  if (why) *why = "no subkernel family accepts this group";
  return false;
}

bool group_closed(const Plan& p, int32_t b, int32_t e) {
  const int nops = (int)p.ops.size();
  for (int j = 0; j < nops; ++j) {
    if (j >= b && j < e) continue;
    for (int k = 0; k < n_operands(p.ops[j].kind); ++k) {
      const int prod = p.ops[j].in[k] - p.n_inputs;
      if (prod >= b && prod < e - 1) return false;
    }
  }
  return true;
}

static mk_status base_plan(const mk_module_desc* d, Plan& p) {
  mk_status s = infer(d, p.vshape);
  if (s != MK_OK) return s;
  p.dtype = d->dtype;
  p.n_inputs = d->n_inputs;
  p.ops.assign(d->ops, d->ops + d->n_ops);
  return MK_OK;
}

mk_status build_plan(const mk_module_desc* d, const int32_t* g, Plan& p) {
  mk_status s = base_plan(d, p);
  if (s != MK_OK) return s;
  if (!g) return fail(MK_E_INVALID_ARG, "group_of_op is null");
  const int nops = d->n_ops;
  if (g[0] != 0) return fail(MK_E_DECOMP, "groups must start at 0");
  for (int i = 1; i < nops; ++i)
    if (g[i] != g[i - 1] && g[i] != g[i - 1] + 1)
      return fail(MK_E_DECOMP, "groups must be contiguous and numbered in op order");
  p.group.assign(g, g + nops);
  const int ng = g[nops - 1] + 1;
  const int64_t es = elem_size(p.dtype);
  int64_t off = 0;
  int b = 0;
  for (int gi = 0; gi < ng; ++gi) {
    int e = b;
    while (e < nops && g[e] == gi) ++e;
    if (!group_closed(p, b, e))
      return fail(MK_E_DECOMP, "group " + std::to_string(gi) +
                                   " hides a value that another group reads");
    Subkernel sk;
    std::string why;
    if (!match_group(p, b, e, sk, &why))
      return fail(MK_E_DECOMP, "group " + std::to_string(gi) + ": " + why);
    sk.op_begin = b;
    sk.op_end = e;
    sk.out_value = p.n_inputs + e - 1;
    sk.out_bytes = numel(p.vshape[sk.out_value]) * es;
    if (gi == ng - 1) {
      sk.ws_offset = -1;
    } else {
      sk.ws_offset = off;
      off += (sk.out_bytes + 255) / 256 * 256;
    }
    sk.flops = 0;
    int64_t by = sk.out_bytes;
    std::vector<char> seen(p.vshape.size(), 0);
    for (int i = b; i < e; ++i) {
      sk.flops += flops_of(p, i);
      for (int k = 0; k < n_operands(p.ops[i].kind); ++k) {
        const int v = p.ops[i].in[k];
        if (inside(v, p.n_inputs + b, p.n_inputs + e) || seen[v]) continue;
        seen[v] = 1;
        by += numel(p.vshape[v]) * es;
      }
    }
    sk.alg_bytes = by;
    sk.impl = MK_IMPL_TUNED;
    p.flops += sk.flops;
    p.subs.push_back(sk);
    b = e;
  }
  p.ws_intermediate = off;
  p.scratch_off = (off + 255) / 256 * 256;
  int64_t scratch = 0;
  for (const Subkernel& sk : p.subs) scratch = std::max(scratch, max_scratch_bytes(p, sk));
  p.scratch_bytes = (scratch + 255) / 256 * 256;
  int64_t mb = numel(p.vshape[p.n_inputs + nops - 1]) * es;
  for (int i = 0; i < p.n_inputs; ++i) mb += numel(p.vshape[i]) * es;
  p.alg_bytes = mb;
  return MK_OK;
}

mk_status preset(const mk_module_desc* d, int32_t which, int32_t* out) {
  if (!out) return fail(MK_E_INVALID_ARG, "group_of_op is null");
  if (which != 0 && which != 1) return fail(MK_E_INVALID_ARG, "preset must be 0 or 1");
  Plan p;
  mk_status s = base_plan(d, p);
  if (s != MK_OK) return s;
  const int nops = d->n_ops;
  std::vector<int32_t> g(nops);
  if (which == 0) {
    // A bias or residual add joins the contraction that produces its input,
    // directly or through bias / add steps that already joined it.
    int gi = 0;
    std::vector<char> joined(nops, 0);
    for (int i = 0; i < nops; ++i) {
      const int32_t k = p.ops[i].kind;
      const bool after_contraction =
          i > 0 && (p.ops[i - 1].kind == MK_OP_GEMM || p.ops[i - 1].kind == MK_OP_CONV2D ||
                    joined[i - 1]);
      joined[i] = i > 0 && (k == MK_OP_BIAS || k == MK_OP_BIAS_CHANNEL || k == MK_OP_ADD) &&
                  after_contraction && p.ops[i].in[0] == p.n_inputs + i - 1 && g[i - 1] == gi;
      if (i > 0 && !joined[i]) ++gi;
      g[i] = gi;
    }
  } else {
    int gi = 0, b = 0;
    while (b < nops) {
      int best = -1;
      for (int e = nops; e > b; --e) {
        Subkernel sk;
        if (group_closed(p, b, e) && match_group(p, b, e, sk, nullptr)) {
          best = e;
          break;
        }
      }
      if (best < 0) return fail(MK_E_DECOMP, "op " + std::to_string(b) + " matches no family");
      for (int i = b; i < best; ++i) g[i] = gi;
      ++gi;
      b = best;
    }
  }
  // The result must be a valid plan.
  Plan check;
  s = build_plan(d, g.data(), check);
  if (s != MK_OK) return s;
  std::copy(g.begin(), g.end(), out);
  return MK_OK;
}

}  // namespace mk
