/*
 * mko.h -- the oracle: a plain, slow, fp64 CPU evaluation of composed
 * modules.  TEST INFRASTRUCTURE ONLY: it is called by the test-suite, by the
 * package's smoke check and by the CPU-baseline leg of the benchmark, never by
 * the product library.  It shares no code, header, helper or table with the
 * HIP path; its enums and structs are declared here on their own.
 *
 * What it computes follows MKEvolve (arXiv 2607.20501): a PyTorch-style module
 * given as an operator sequence with shapes (Sec. 3, "LLMDecompose agent"),
 * partitioned into contiguous subproblems that a top-level module chains
 * (Sec. 3 and App. H.1).  Every operator is evaluated from its textbook
 * definition in fp64.  Values are rounded to the module storage dtype exactly
 * where a subkernel boundary materialises them (the rounding model), so split
 * and fused decompositions have different, individually exact, references.
 */
#ifndef MKO_H
#define MKO_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum mko_dtype { MKO_F32 = 0, MKO_BF16 = 1 };

enum mko_kind {
  MKO_GEMM = 0,      /* in {A[..,K], W}; ip[0]=0: W[N,K] (y = A W^T), 1: W[K,N] (y = A W) */
  MKO_BIAS,          /* in {x[..,N], b[N]} */
  MKO_BIAS_CHANNEL,  /* in {x[N,C,H,W], b[C]} */
  MKO_RELU,
  MKO_GELU_ERF,      /* 0.5 x (1 + erf(x / sqrt 2)) */
  MKO_GELU_TANH,     /* 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3))) */
  MKO_SCALE,         /* fp[0] = s */
  MKO_ADD,           /* in {x, r}, same shape */
  MKO_ROWSUM,        /* [.., N] -> [..] */
  MKO_SOFTMAX,       /* over the last dimension, max subtracted */
  MKO_LAYERNORM,     /* in {x[..,D], gamma[D], beta[D]}; fp[0] = eps; biased variance */
  MKO_CONV2D,        /* in {x[N,C,H,W], w[K,C,R,S]}; ip[0]=stride, ip[1]=pad; cross-correlation */
  MKO_GAP,           /* [N,C,H,W] -> [N,C], mean over H*W */
  MKO_QK,            /* in {qkv[B*S, 3*H*dh]}; ip={B,H,dh,S}; fp[0]=scale -> [B,H,S,S] */
  MKO_CAUSAL_MASK,   /* [.., S, S]: j > i -> -inf, diagonal kept */
  MKO_PV,            /* in {p[B,H,S,S], qkv}; ip={B,H,dh,S} -> [B,S,H*dh] */
  MKO_GMP,           /* [N,C,H,W] -> [N,C], max over H*W */
  MKO_LPPOOL,        /* [N,C,H,W] -> [N,C], fp[0] = p: S = sum x^p over H*W,
                        y = sign(S) |S|^(1/p) */
  MKO_N_KINDS
};

typedef struct { int32_t ndim; int64_t dims[4]; } mko_shape;

typedef struct {
  int32_t kind;
  int32_t in[3];     /* value ids, -1 unused; ids 0..n_inputs-1 are module inputs,
                        n_inputs+i is the output of op i */
  int64_t ip[4];
  double  fp[2];
} mko_op;

typedef struct {
  int32_t dtype;
  int32_t n_inputs;
  const mko_shape* input_shapes;
  int32_t n_ops;
  const mko_op* ops;
} mko_desc;

enum { MKO_MAX_OPS = 64 };

/* Bookkeeping of one subproblem (a contiguous group of ops). */
typedef struct {
  int32_t op_begin, op_end;   /* [begin, end) */
  int32_t out_value;          /* value id of the group's materialised output */
  mko_shape out_shape;
  int64_t out_bytes;          /* numel * dtype size */
  int64_t ws_offset;          /* byte offset of the materialised intermediate, -1 = module output */
  int64_t flops;              /* algorithmic flops of the group's ops */
  int64_t alg_bytes;          /* distinct external inputs read once + output written once */
} mko_group_info;

typedef struct {
  int32_t n_groups;
  mko_group_info g[MKO_MAX_OPS];
  mko_shape value_shapes[MKO_MAX_OPS * 2];
  int64_t ws_intermediate_bytes; /* sum of round_up(out_bytes, 256) over non-output groups */
  int64_t flops;                 /* module flops */
  int64_t alg_bytes;             /* module inputs read once + output written once */
} mko_plan_info;

/* Shape inference plus grouping bookkeeping.  Returns 0 on success, a
   negative code on a malformed module (-1 argument, -2 shape, -3 grouping). */
int mko_plan(const mko_desc* d, const int32_t* group_of_op, mko_plan_info* out);

/* Evaluate the module.  host_inputs[i] holds the raw storage bytes of module
   input i (float32, or bfloat16 bit patterns).  values[i], if non-NULL, receives
   the fp64 value of op i's output (numel doubles, row-major).  With
   ideal != 0 nothing is rounded after the inputs (the "ideal" reference).
   nthreads <= 0 uses the OpenMP default.  Returns 0 or a negative code. */
int mko_run(const mko_desc* d, const int32_t* group_of_op,
            const void* const* host_inputs, double* const* values,
            int ideal, int nthreads);

/* Rounding helpers, exported so that their pins can be tested directly. */
double mko_round_bf16(double v);    /* nearest bfloat16, ties to even */
double mko_round_f32(double v);     /* nearest float32, ties to even */
double mko_decode_bf16(uint16_t bits);
/* Scalar definitions of the activations (pinned against closed forms). */
double mko_gelu_erf(double x);
double mko_gelu_tanh(double x);

#ifdef __cplusplus
}
#endif
#endif
