/*
 * mko.c -- the oracle (test infrastructure only; see mko.h).
 *
 * Plain C99 + OpenMP over independent output rows.  Every operator is its
 * textbook definition evaluated in fp64; no blocking, fusion or reordering
 * beyond what the definition states.  Citations name the MKEvolve paper
 * (arXiv 2607.20501) section, appendix or table that fixes each meaning.
 */
#include "mko.h"

#include <float.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------ */
/* Rounding model.                                                     */
/* ------------------------------------------------------------------ */

/* Nearest bfloat16 to v, ties to even.  bfloat16 keeps 8 significant bits
   and the float32 exponent range (normal exponent >= -126, subnormal quantum
   2^-133, largest finite (2 - 2^-7) * 2^127).  The value is rounded directly
   from fp64, so there is no double rounding. */
double mko_round_bf16(double v) {
  if (v != v || v == 0.0 || isinf(v)) return v;
  double a = fabs(v);
  int e;
  (void)frexp(a, &e);          /* a = m * 2^e, m in [0.5, 1) */
  int q = e - 8;               /* weight of the last kept bit */
  if (q < -133) q = -133;      /* subnormal range */
  double r = nearbyint(ldexp(a, -q));  /* current mode: to nearest, ties even */
  r = ldexp(r, q);
  if (r > 0x1.fep127) r = INFINITY;
  return v < 0 ? -r : r;
}

double mko_round_f32(double v) { return (double)(float)v; }

double mko_decode_bf16(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* GELU: the exact form x * Phi(x) (App. D lists the sigmoid approximation as
   a bug; the exact GELU is the reference), and the tanh approximation. */
double mko_gelu_erf(double x) { return 0.5 * x * (1.0 + erf(x / sqrt(2.0))); }

double mko_gelu_tanh(double x) {
  const double c = sqrt(2.0 / 3.14159265358979323846);
  return 0.5 * x * (1.0 + tanh(c * (x + 0.044715 * x * x * x)));
}

/* ------------------------------------------------------------------ */
/* Shape inference and bookkeeping.                                    */
/* ------------------------------------------------------------------ */

static int64_t numel(const mko_shape* s) {
  int64_t n = 1;
  for (int i = 0; i < s->ndim; ++i) n *= s->dims[i];
  return n;
}

static int64_t esize(int dtype) { return dtype == MKO_BF16 ? 2 : 4; }

static int shape_eq(const mko_shape* a, const mko_shape* b) {
  if (a->ndim != b->ndim) return 0;
  for (int i = 0; i < a->ndim; ++i)
    if (a->dims[i] != b->dims[i]) return 0;
  return 1;
}

static int n_in_of(int kind) {
  switch (kind) {
    case MKO_GEMM: case MKO_BIAS: case MKO_BIAS_CHANNEL: case MKO_ADD: case MKO_CONV2D:
    case MKO_PV:
      return 2;
    case MKO_LAYERNORM:
      return 3;
    default:
      return 1;
  }
}

/* Fill vs[0 .. n_inputs+n_ops-1]; returns 0, -1 (argument) or -2 (shape). */
static int infer_shapes(const mko_desc* d, mko_shape* vs) {
  if (!d || d->n_inputs < 0 || d->n_ops < 1 || d->n_ops > MKO_MAX_OPS ||
      d->n_inputs > MKO_MAX_OPS)
    return -1;
  if (d->dtype != MKO_F32 && d->dtype != MKO_BF16) return -1;
  for (int i = 0; i < d->n_inputs; ++i) {
    const mko_shape* s = &d->input_shapes[i];
    if (s->ndim < 1 || s->ndim > 4) return -2;
    for (int k = 0; k < s->ndim; ++k)
      if (s->dims[k] < 1) return -2;
    vs[i] = *s;
  }
  for (int i = 0; i < d->n_ops; ++i) {
    const mko_op* o = &d->ops[i];
    if (o->kind < 0 || o->kind >= MKO_N_KINDS) return -1;
    int nin = n_in_of(o->kind);
    int lim = d->n_inputs + i;
    for (int k = 0; k < nin; ++k)
      if (o->in[k] < 0 || o->in[k] >= lim) return -1;
    const mko_shape* x = &vs[o->in[0]];
    mko_shape y = *x;
    switch (o->kind) {
      case MKO_GEMM: {
        const mko_shape* w = &vs[o->in[1]];
        if (w->ndim != 2 || (o->ip[0] != 0 && o->ip[0] != 1)) return -2;
        int64_t K = o->ip[0] == 0 ? w->dims[1] : w->dims[0];
        int64_t N = o->ip[0] == 0 ? w->dims[0] : w->dims[1];
        if (x->dims[x->ndim - 1] != K) return -2;
        y.dims[y.ndim - 1] = N;
        break;
      }
      case MKO_BIAS: {
        const mko_shape* b = &vs[o->in[1]];
        if (b->ndim != 1 || b->dims[0] != x->dims[x->ndim - 1]) return -2;
        break;
      }
      case MKO_BIAS_CHANNEL: {
        const mko_shape* b = &vs[o->in[1]];
        if (x->ndim != 4 || b->ndim != 1 || b->dims[0] != x->dims[1]) return -2;
        break;
      }
      case MKO_RELU: case MKO_GELU_ERF: case MKO_GELU_TANH: case MKO_SCALE: case MKO_SOFTMAX:
        break;
      case MKO_ADD:
        if (!shape_eq(x, &vs[o->in[1]])) return -2;
        break;
      case MKO_ROWSUM:
        if (x->ndim < 2) return -2;
        y.ndim = x->ndim - 1;
        break;
      case MKO_LAYERNORM: {
        const mko_shape* g = &vs[o->in[1]];
        const mko_shape* b = &vs[o->in[2]];
        int64_t D = x->dims[x->ndim - 1];
        if (g->ndim != 1 || b->ndim != 1 || g->dims[0] != D || b->dims[0] != D) return -2;
        if (!(o->fp[0] >= 0.0)) return -2;
        break;
      }
      case MKO_CONV2D: {
        const mko_shape* w = &vs[o->in[1]];
        int64_t st = o->ip[0], pd = o->ip[1];
        if (x->ndim != 4 || w->ndim != 4 || w->dims[1] != x->dims[1]) return -2;
        if (st < 1 || pd < 0) return -2;
        int64_t hp = x->dims[2] + 2 * pd - w->dims[2];
        int64_t wp = x->dims[3] + 2 * pd - w->dims[3];
        if (hp < 0 || wp < 0) return -2;
        y.ndim = 4;
        y.dims[0] = x->dims[0];
        y.dims[1] = w->dims[0];
        y.dims[2] = hp / st + 1;
        y.dims[3] = wp / st + 1;
        break;
      }
      case MKO_GAP: case MKO_GMP: case MKO_LPPOOL:
        if (x->ndim != 4) return -2;
        if (o->kind == MKO_LPPOOL && !(o->fp[0] > 0.0)) return -2;
        y.ndim = 2;
        break;
      case MKO_QK: case MKO_PV: {
        int64_t B = o->ip[0], H = o->ip[1], dh = o->ip[2], S = o->ip[3];
        if (B < 1 || H < 1 || dh < 1 || S < 1) return -2;
        const mko_shape* qkv = &vs[o->in[o->kind == MKO_QK ? 0 : 1]];
        if (numel(qkv) != B * S * 3 * H * dh || qkv->dims[qkv->ndim - 1] != 3 * H * dh) return -2;
        if (o->kind == MKO_QK) {
          y.ndim = 4;
          y.dims[0] = B; y.dims[1] = H; y.dims[2] = S; y.dims[3] = S;
        } else {
          mko_shape ps = {4, {B, H, S, S}};
          if (!shape_eq(x, &ps)) return -2;
          y.ndim = 3;
          y.dims[0] = B; y.dims[1] = S; y.dims[2] = H * dh;
          y.dims[3] = 0;
        }
        break;
      }
      case MKO_CAUSAL_MASK:
        if (x->ndim < 2 || x->dims[x->ndim - 1] != x->dims[x->ndim - 2]) return -2;
        break;
      default:
        return -1;
    }
    for (int k = y.ndim; k < 4; ++k) y.dims[k] = 0;
    vs[d->n_inputs + i] = y;
  }
  return 0;
}

/* Is the score matrix produced by QK op i causally masked by a later op? */
static int qk_is_causal(const mko_desc* d, int i) {
  int v = d->n_inputs + i;
  for (int j = i + 1; j < d->n_ops; ++j)
    if (d->ops[j].kind == MKO_CAUSAL_MASK && d->ops[j].in[0] == v) return 1;
  return 0;
}

/* Does PV op i consume softmax(causal_mask(.))? */
static int pv_is_causal(const mko_desc* d, int i) {
  int p = d->ops[i].in[0] - d->n_inputs;
  if (p < 0 || d->ops[p].kind != MKO_SOFTMAX) return 0;
  int m = d->ops[p].in[0] - d->n_inputs;
  return m >= 0 && d->ops[m].kind == MKO_CAUSAL_MASK;
}

/* Algorithmic flops of op i: 2*M*N*K for a GEMM, 2*N*P*Q*K*C*R*S for a conv,
   and for the attention contractions only the score entries a causal mask
   keeps when the module masks them.  Element-wise and row ops count 0. */
static int64_t op_flops(const mko_desc* d, const mko_shape* vs, int i) {
  const mko_op* o = &d->ops[i];
  switch (o->kind) {
    case MKO_GEMM: {
      const mko_shape* a = &vs[o->in[0]];
      int64_t K = a->dims[a->ndim - 1];
      int64_t M = numel(a) / K;
      const mko_shape* y = &vs[d->n_inputs + i];
      int64_t N = y->dims[y->ndim - 1];
      return 2 * M * N * K;
    }
    case MKO_CONV2D: {
      const mko_shape* w = &vs[o->in[1]];
      const mko_shape* y = &vs[d->n_inputs + i];
      return 2 * y->dims[0] * y->dims[2] * y->dims[3] * w->dims[0] * w->dims[1] * w->dims[2] *
             w->dims[3];
    }
    case MKO_QK: case MKO_PV: {
      int64_t B = o->ip[0], H = o->ip[1], dh = o->ip[2], S = o->ip[3];
      int causal = o->kind == MKO_QK ? qk_is_causal(d, i) : pv_is_causal(d, i);
      int64_t pairs = causal ? S * (S + 1) / 2 : S * S;
      return 2 * B * H * dh * pairs;
    }
    default:
      return 0;
  }
}

static int check_groups(const mko_desc* d, const int32_t* g) {
  if (!g) return -1;
  if (g[0] != 0) return -3;
  for (int i = 1; i < d->n_ops; ++i)
    if (g[i] != g[i - 1] && g[i] != g[i - 1] + 1) return -3;
  /* A value produced inside a group and used by another group must be the
     producing group's last op (only that one is materialised). */
  for (int j = 0; j < d->n_ops; ++j) {
    int nin = n_in_of(d->ops[j].kind);
    for (int k = 0; k < nin; ++k) {
      int p = d->ops[j].in[k] - d->n_inputs;
      if (p < 0) continue;
      if (g[p] != g[j]) {
        int last = (p == d->n_ops - 1) || (g[p + 1] != g[p]);
        if (!last) return -3;
      }
    }
  }
  return 0;
}

int mko_plan(const mko_desc* d, const int32_t* group_of_op, mko_plan_info* out) {
  if (!d || !out) return -1;
  memset(out, 0, sizeof(*out));
  int rc = infer_shapes(d, out->value_shapes);
  if (rc) return rc;
  rc = check_groups(d, group_of_op);
  if (rc) return rc;
  const mko_shape* vs = out->value_shapes;
  int64_t es = esize(d->dtype);
  int ng = group_of_op[d->n_ops - 1] + 1;
  out->n_groups = ng;
  int64_t off = 0;
  for (int gi = 0; gi < ng; ++gi) {
    mko_group_info* G = &out->g[gi];
    int b = -1, e = -1;
    for (int i = 0; i < d->n_ops; ++i)
      if (group_of_op[i] == gi) {
        if (b < 0) b = i;
        e = i + 1;
      }
    G->op_begin = b;
    G->op_end = e;
    G->out_value = d->n_inputs + e - 1;
    G->out_shape = vs[G->out_value];
    G->out_bytes = numel(&G->out_shape) * es;
    if (gi == ng - 1) {
      G->ws_offset = -1;
    } else {
      G->ws_offset = off;
      off += (G->out_bytes + 255) / 256 * 256;
    }
    int64_t fl = 0, by = G->out_bytes;
    int seen[2 * MKO_MAX_OPS];
    memset(seen, 0, sizeof(seen));
    for (int i = b; i < e; ++i) {
      fl += op_flops(d, vs, i);
      int nin = n_in_of(d->ops[i].kind);
      for (int k = 0; k < nin; ++k) {
        int v = d->ops[i].in[k];
        int internal = v >= d->n_inputs + b && v < d->n_inputs + e;
        if (internal || seen[v]) continue;
        seen[v] = 1;
        by += numel(&vs[v]) * es;
      }
    }
    G->flops = fl;
    G->alg_bytes = by;
    out->flops += fl;
  }
  out->ws_intermediate_bytes = off;
  int64_t mb = numel(&vs[d->n_inputs + d->n_ops - 1]) * es;
  for (int i = 0; i < d->n_inputs; ++i) mb += numel(&vs[i]) * es;
  out->alg_bytes = mb;
  return 0;
}

/* ------------------------------------------------------------------ */
/* Operators, fp64.                                                    */
/* ------------------------------------------------------------------ */

/* y[m, n] = sum_k A[m, k] * B(k, n), the sum taken in k order, where
   B(k, n) = W[n, k] (nn.Linear layout, App. H.2 linear kernels) or W[k, n]. */
static void op_gemm(const double* A, const double* W, double* y, int64_t M, int64_t N,
                    int64_t K, int layout) {
  double* B = (double*)malloc(sizeof(double) * (size_t)(K * N));
  for (int64_t k = 0; k < K; ++k)
    for (int64_t n = 0; n < N; ++n) B[k * N + n] = layout == 0 ? W[n * K + k] : W[k * N + n];
#pragma omp parallel for schedule(static)
  for (int64_t m = 0; m < M; ++m) {
    double* yr = y + m * N;
    for (int64_t n = 0; n < N; ++n) yr[n] = 0.0;
    for (int64_t k = 0; k < K; ++k) {
      double a = A[m * K + k];
      const double* br = B + k * N;
      for (int64_t n = 0; n < N; ++n) yr[n] += a * br[n];
    }
  }
  free(B);
}

/* y[n, k, p, q] = sum_{c, r, s} x[n, c, p*st + r - pad, q*st + s - pad] * w[k, c, r, s]
   with zeros outside the image (cross-correlation, as torch's conv2d).  For
   each output element the terms are added in (c, r, s) order. */
static void op_conv(const double* x, const double* w, double* y, int64_t N, int64_t C,
                    int64_t H, int64_t Wd, int64_t K, int64_t R, int64_t S, int64_t P,
                    int64_t Q, int64_t st, int64_t pd) {
#pragma omp parallel for schedule(static)
  for (int64_t nk = 0; nk < N * K; ++nk) {
    int64_t n = nk / K, k = nk % K;
    double* yp = y + nk * P * Q;
    for (int64_t i = 0; i < P * Q; ++i) yp[i] = 0.0;
    for (int64_t c = 0; c < C; ++c)
      for (int64_t r = 0; r < R; ++r)
        for (int64_t s = 0; s < S; ++s) {
          double wv = w[((k * C + c) * R + r) * S + s];
          const double* xc = x + (n * C + c) * H * Wd;
          for (int64_t p = 0; p < P; ++p) {
            int64_t h = p * st + r - pd;
            if (h < 0 || h >= H) continue;
            for (int64_t q = 0; q < Q; ++q) {
              int64_t ww = q * st + s - pd;
              if (ww < 0 || ww >= Wd) continue;
              yp[p * Q + q] += wv * xc[h * Wd + ww];
            }
          }
        }
  }
}

/* Softmax over the last dimension with the row maximum subtracted first
   (App. D: "unsafe softmax" without it is one of the injected bugs). */
static void op_softmax(const double* x, double* y, int64_t rows, int64_t n) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    const double* xr = x + r * n;
    double* yr = y + r * n;
    double m = -INFINITY;
    for (int64_t i = 0; i < n; ++i) m = xr[i] > m ? xr[i] : m;
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i) {
      yr[i] = exp(xr[i] - m);
      s += yr[i];
    }
    for (int64_t i = 0; i < n; ++i) yr[i] /= s;
  }
}

/* LayerNorm over the last dimension: mean, then the biased variance of the
   centred values (divide by D), then (x - mean) / sqrt(var + eps) * g + b
   (App. H.2 LN kernels; App. I.2 LayerNorm guidance). */
static void op_layernorm(const double* x, const double* g, const double* b, double* y,
                         int64_t rows, int64_t D, double eps) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    const double* xr = x + r * D;
    double mu = 0.0;
    for (int64_t i = 0; i < D; ++i) mu += xr[i];
    mu /= (double)D;
    double var = 0.0;
    for (int64_t i = 0; i < D; ++i) var += (xr[i] - mu) * (xr[i] - mu);
    var /= (double)D;
    double rs = 1.0 / sqrt(var + eps);
    for (int64_t i = 0; i < D; ++i) y[r * D + i] = (xr[i] - mu) * rs * g[i] + b[i];
  }
}

/* Scores s[b, h, i, j] = (q_i . k_j) * scale, with q, k, v packed per token as
   [Q | K | V] blocks of H*dh columns and head h at columns h*dh .. h*dh+dh-1
   (App. H.2, attention kernel's packed-QKV convention). */
static void op_qk(const double* qkv, double* s, int64_t B, int64_t H, int64_t dh, int64_t S,
                  double scale) {
  int64_t ld = 3 * H * dh;
#pragma omp parallel for schedule(static)
  for (int64_t bhi = 0; bhi < B * H * S; ++bhi) {
    int64_t i = bhi % S, bh = bhi / S, h = bh % H, b = bh / H;
    const double* q = qkv + (b * S + i) * ld + h * dh;
    for (int64_t j = 0; j < S; ++j) {
      const double* k = qkv + (b * S + j) * ld + H * dh + h * dh;
      double acc = 0.0;
      for (int64_t e = 0; e < dh; ++e) acc += q[e] * k[e];
      s[bhi * S + j] = acc * scale;
    }
  }
}

/* o[b, i, h*dh + e] = sum_j p[b, h, i, j] * v[b, j, h, e] (heads merged). */
static void op_pv(const double* p, const double* qkv, double* o, int64_t B, int64_t H,
                  int64_t dh, int64_t S) {
  int64_t ld = 3 * H * dh;
#pragma omp parallel for schedule(static)
  for (int64_t bhi = 0; bhi < B * H * S; ++bhi) {
    int64_t i = bhi % S, bh = bhi / S, h = bh % H, b = bh / H;
    double* out = o + (b * S + i) * H * dh + h * dh;
    for (int64_t e = 0; e < dh; ++e) out[e] = 0.0;
    const double* pr = p + bhi * S;
    for (int64_t j = 0; j < S; ++j) {
      const double* v = qkv + (b * S + j) * ld + 2 * H * dh + h * dh;
      double pj = pr[j];
      for (int64_t e = 0; e < dh; ++e) out[e] += pj * v[e];
    }
  }
}

/* ------------------------------------------------------------------ */
/* Module evaluation with the rounding model.                          */
/* ------------------------------------------------------------------ */

static void round_to(double* v, int64_t n, int dtype) {
  if (dtype == MKO_BF16) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) v[i] = mko_round_bf16(v[i]);
  } else {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) v[i] = mko_round_f32(v[i]);
  }
}

int mko_run(const mko_desc* d, const int32_t* group_of_op, const void* const* host_inputs,
            double* const* values, int ideal, int nthreads) {
  if (!d || !host_inputs) return -1;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
  mko_plan_info* pl = (mko_plan_info*)malloc(sizeof(mko_plan_info));
  int rc = mko_plan(d, group_of_op, pl);
  if (rc) {
    free(pl);
    return rc;
  }
  int nv = d->n_inputs + d->n_ops;
  double** val = (double**)calloc((size_t)nv, sizeof(double*));
  int* owned = (int*)calloc((size_t)nv, sizeof(int));
  for (int i = 0; i < d->n_inputs; ++i) {
    int64_t n = numel(&pl->value_shapes[i]);
    val[i] = (double*)malloc(sizeof(double) * (size_t)n);
    owned[i] = 1;
    if (d->dtype == MKO_BF16) {
      const uint16_t* src = (const uint16_t*)host_inputs[i];
      for (int64_t k = 0; k < n; ++k) val[i][k] = mko_decode_bf16(src[k]);
    } else {
      const float* src = (const float*)host_inputs[i];
      for (int64_t k = 0; k < n; ++k) val[i][k] = (double)src[k];
    }
  }
  for (int i = 0; i < d->n_ops; ++i) {
    const mko_op* o = &d->ops[i];
    int v = d->n_inputs + i;
    const mko_shape* ys = &pl->value_shapes[v];
    const mko_shape* xs = &pl->value_shapes[o->in[0]];
    int64_t n = numel(ys);
    if (values && values[i]) {
      val[v] = values[i];
    } else {
      val[v] = (double*)malloc(sizeof(double) * (size_t)n);
      owned[v] = 1;
    }
    double* y = val[v];
    const double* x = val[o->in[0]];
    int64_t last = xs->dims[xs->ndim - 1];
    switch (o->kind) {
      case MKO_GEMM: {
        int64_t K = last, N = ys->dims[ys->ndim - 1];
        op_gemm(x, val[o->in[1]], y, numel(xs) / K, N, K, (int)o->ip[0]);
        break;
      }
      case MKO_BIAS: {
        const double* b = val[o->in[1]];
        for (int64_t k = 0; k < n; ++k) y[k] = x[k] + b[k % last];
        break;
      }
      case MKO_BIAS_CHANNEL: {
        const double* b = val[o->in[1]];
        int64_t C = xs->dims[1], hw = xs->dims[2] * xs->dims[3];
        for (int64_t k = 0; k < n; ++k) y[k] = x[k] + b[(k / hw) % C];
        break;
      }
      case MKO_RELU:
        for (int64_t k = 0; k < n; ++k) y[k] = x[k] > 0.0 ? x[k] : 0.0;
        break;
      case MKO_GELU_ERF:
        for (int64_t k = 0; k < n; ++k) y[k] = mko_gelu_erf(x[k]);
        break;
      case MKO_GELU_TANH:
        for (int64_t k = 0; k < n; ++k) y[k] = mko_gelu_tanh(x[k]);
        break;
      case MKO_SCALE:
        for (int64_t k = 0; k < n; ++k) y[k] = x[k] * o->fp[0];
        break;
      case MKO_ADD: {
        const double* r = val[o->in[1]];
        for (int64_t k = 0; k < n; ++k) y[k] = x[k] + r[k];
        break;
      }
      case MKO_ROWSUM:
        for (int64_t r = 0; r < n; ++r) {
          double s = 0.0;
          for (int64_t k = 0; k < last; ++k) s += x[r * last + k];
          y[r] = s;
        }
        break;
      case MKO_SOFTMAX:
        op_softmax(x, y, n / last, last);
        break;
      case MKO_LAYERNORM:
        op_layernorm(x, val[o->in[1]], val[o->in[2]], y, n / last, last, o->fp[0]);
        break;
      case MKO_CONV2D: {
        const mko_shape* ws = &pl->value_shapes[o->in[1]];
        op_conv(x, val[o->in[1]], y, xs->dims[0], xs->dims[1], xs->dims[2], xs->dims[3],
                ws->dims[0], ws->dims[2], ws->dims[3], ys->dims[2], ys->dims[3], o->ip[0],
                o->ip[1]);
        break;
      }
      case MKO_GAP: {
        int64_t hw = xs->dims[2] * xs->dims[3];
        for (int64_t r = 0; r < n; ++r) {
          double s = 0.0;
          for (int64_t k = 0; k < hw; ++k) s += x[r * hw + k];
          y[r] = s / (double)hw;
        }
        break;
      }
      case MKO_GMP: {   /* global max pool (a MobileNet-style pooling variant, Sec. 4) */
        int64_t hw = xs->dims[2] * xs->dims[3];
        for (int64_t r = 0; r < n; ++r) {
          double m = -INFINITY;
          for (int64_t k = 0; k < hw; ++k) m = x[r * hw + k] > m ? x[r * hw + k] : m;
          y[r] = m;
        }
        break;
      }
      case MKO_LPPOOL: {   /* global LP pool: (sum x^p)^(1/p), sign kept */
        int64_t hw = xs->dims[2] * xs->dims[3];
        double p = o->fp[0];
        for (int64_t r = 0; r < n; ++r) {
          double s = 0.0;
          for (int64_t k = 0; k < hw; ++k) s += pow(x[r * hw + k], p);
          y[r] = copysign(pow(fabs(s), 1.0 / p), s);
        }
        break;
      }
      case MKO_QK:
        op_qk(x, y, o->ip[0], o->ip[1], o->ip[2], o->ip[3], o->fp[0]);
        break;
      case MKO_CAUSAL_MASK: {
        int64_t S = last;
        for (int64_t k = 0; k < n; ++k) {
          int64_t j = k % S, r = (k / S) % S;
          y[k] = j > r ? -INFINITY : x[k];
        }
        break;
      }
      case MKO_PV:
        op_pv(x, val[o->in[1]], y, o->ip[0], o->ip[1], o->ip[2], o->ip[3]);
        break;
      default:
        break;
    }
    if (!ideal) {
      int g = group_of_op[i];
      int is_last = (i == d->n_ops - 1) || group_of_op[i + 1] != g;
      /* A LayerNorm applied inside a group as the prologue of a GEMM is handed
         to the contraction in the storage dtype (its operand type). */
      int ln_prologue = o->kind == MKO_LAYERNORM && !is_last &&
                        d->ops[i + 1].kind == MKO_GEMM && d->ops[i + 1].in[0] == v;
      if (is_last || ln_prologue) round_to(y, n, d->dtype);
    }
  }
  for (int v = 0; v < nv; ++v)
    if (owned[v]) free(val[v]);
  free(val);
  free(owned);
  free(pl);
  return 0;
}
