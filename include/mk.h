/*
 * mk.h -- C ABI of libmk: composed multi-operator modules on MI355X (gfx950).
 *
 * MKEvolve (arXiv 2607.20501) states the problem as a PyTorch module M,
 * decomposed into subproblems that a top-level module S chains; each
 * subproblem has its own, independently verified and swappable, kernel
 * (Sec. 3, Alg. 1 and "LLMDecompose agent"; App. H.1 shows such an S).  This
 * library is that hot path: a module is an operator sequence with shapes
 * (mk_module_desc), a decomposition is a contiguous grouping of its ops
 * (group_of_op), every group runs as one subkernel made of hand-written HIP
 * kernels, and each subkernel's implementation can be swapped on its own
 * (Sec. 3, "Swap").  mk_run executes the composition; mk_verify checks each
 * materialised stage and the output against caller-given reference values
 * (Sec. 3 "Evaluate"; App. D, decomposed per-stage checking).
 *
 * Conventions
 *  - Every function returns mk_status; nothing throws across the ABI.  On an
 *    error, mk_last_error() gives a thread-local message.
 *  - Tensors are dense and row-major.  Every module input, materialised
 *    intermediate and the output are stored in the module dtype (float32, or
 *    bfloat16 as raw 16-bit patterns); arithmetic inside kernels is fp32.
 *  - Value ids: 0..n_inputs-1 are the module inputs (activations and weights
 *    alike); n_inputs+i is the output of op i; the module output is the
 *    output of the last op.
 *  - Device buffers (inputs, output, workspace) are allocated and owned by the
 *    caller.  A module owns host-side plan state only; mk_run never allocates
 *    device memory.  Two concurrent runs of one module need distinct
 *    workspaces.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 */
#ifndef MK_H
#define MK_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MK_OK = 0,
  MK_E_INVALID_ARG = 1,  /* null pointer, bad id, bad enum value */
  MK_E_SHAPE = 2,        /* shapes of an op's operands do not agree */
  MK_E_DTYPE = 3,        /* unknown dtype */
  MK_E_DECOMP = 4,       /* grouping not contiguous, hides a value another
                            group reads, or matches no subkernel family */
  MK_E_UNSUPPORTED = 5,  /* valid request with no implementation (impl id) */
  MK_E_WORKSPACE = 6,    /* workspace smaller than mk_workspace_size */
  MK_E_HIP = 7,          /* a HIP runtime call failed; see mk_last_error */
  MK_E_INTERNAL = 8
} mk_status;

typedef enum { MK_F32 = 0, MK_BF16 = 1 } mk_dtype;

/* Operators.  Semantics (all over the last dimension unless stated):
 *  GEMM         in {A[..,K], W}; ip[0] = 0: W is [N,K] and y = A W^T (nn.Linear
 *               layout), 1: W is [K,N] and y = A W.  y[..,N].
 *  BIAS         in {x[..,N], b[N]}: x + b.
 *  BIAS_CHANNEL in {x[N,C,H,W], b[C]}: x + b[c].
 *  RELU, GELU_ERF (0.5x(1+erf(x/sqrt2))), GELU_TANH
 *               (0.5x(1+tanh(sqrt(2/pi)(x+0.044715x^3)))), SCALE (x*fp[0]).
 *  ADD          in {x, r} of equal shape: x + r (residual).
 *  ROWSUM       [..,N] -> [..]: sum over the last dimension.
 *  SOFTMAX      exp(x - max) / sum over the last dimension.
 *  LAYERNORM    in {x[..,D], gamma[D], beta[D]}, fp[0] = eps:
 *               (x - mean) / sqrt(biased var + eps) * gamma + beta.
 *  CONV2D       in {x[N,C,H,W], w[K,C,R,S]}, ip = {stride, pad}:
 *               cross-correlation with zero padding -> [N,K,P,Q].
 *  GAP          [N,C,H,W] -> [N,C]: mean over H*W.
 *  QK           in {qkv[B*S, 3*H*dh]} packed per token as [Q | K | V], head h
 *               at columns h*dh..h*dh+dh-1 of each block; ip = {B, H, dh, S};
 *               fp[0] = scale: s[b,h,i,j] = (q_i . k_j) * scale -> [B,H,S,S].
 *  CAUSAL_MASK  [..,S,S]: entries with j > i become -inf (diagonal kept).
 *  PV           in {p[B,H,S,S], qkv}, ip = {B, H, dh, S}:
 *               o[b,i,h*dh+e] = sum_j p[b,h,i,j] v[b,j,h,e] -> [B,S,H*dh].
 *  GMP          [N,C,H,W] -> [N,C]: max over H*W (global max pool).
 *  LPPOOL       [N,C,H,W] -> [N,C], fp[0] = p > 0: S = sum over H*W of x^p,
 *               y = sign(S) |S|^(1/p) (global LP pool; the pooling variants
 *               that replace GAP in Sec. 4's MobileNet adaptation). */
typedef enum {
  MK_OP_GEMM = 0, MK_OP_BIAS, MK_OP_BIAS_CHANNEL, MK_OP_RELU, MK_OP_GELU_ERF,
  MK_OP_GELU_TANH, MK_OP_SCALE, MK_OP_ADD, MK_OP_ROWSUM, MK_OP_SOFTMAX,
  MK_OP_LAYERNORM, MK_OP_CONV2D, MK_OP_GAP, MK_OP_QK, MK_OP_CAUSAL_MASK, MK_OP_PV,
  MK_OP_GMP, MK_OP_LPPOOL,
  MK_OP_COUNT
} mk_op_kind;

typedef struct { int32_t ndim; int64_t dims[4]; } mk_shape;

typedef struct {
  int32_t kind;     /* mk_op_kind */
  int32_t in[3];    /* value ids; -1 where unused */
  int64_t ip[4];    /* integer parameters, see mk_op_kind */
  double fp[2];     /* real parameters, see mk_op_kind */
} mk_op;

typedef struct {
  int32_t dtype;                 /* mk_dtype */
  int32_t n_inputs;
  const mk_shape* input_shapes;  /* [n_inputs] */
  int32_t n_ops;                 /* 1..64 */
  const mk_op* ops;              /* [n_ops] */
} mk_module_desc;

typedef struct mk_module mk_module;

/* Subkernel families (what a group of ops is run as). */
typedef enum {
  MK_FAM_GEMM = 0,   /* [LAYERNORM] GEMM|QK|PV, element-wise epilogue, [ROWSUM|SOFTMAX] */
  MK_FAM_CONV = 1,   /* CONV2D, element-wise epilogue, [GAP] */
  MK_FAM_EW = 2,     /* chain of element-wise ops */
  MK_FAM_ROW = 3,    /* element-wise prologue, then ROWSUM|SOFTMAX|LAYERNORM|GAP */
  MK_FAM_ATTN = 4    /* QK [CAUSAL_MASK] SOFTMAX PV */
} mk_family;

/* Implementation ids accepted by mk_subkernel_select. */
enum { MK_IMPL_TUNED = 0, MK_IMPL_SIMPLE = 1, MK_IMPL_MUTANT_BASE = 100 };

/* Why MK_IMPL_TUNED of a GEMM, CONV or ATTN subkernel runs the simple kernels
 * (the ones MK_IMPL_SIMPLE selects) instead of the matrix-core kernels.  The
 * results stay correct either way; mk_subkernel_info reports the code so a
 * caller can tell, and the Python binding warns (or raises, strict=True). */
typedef enum {
  MK_LIMIT_NONE = 0,   /* the tuned kernels run (always for EW and ROW subkernels) */
  MK_LIMIT_DTYPE = 1,  /* no matrix-core form for the dtype (fused attention: bf16 only) */
  MK_LIMIT_ALIGN = 2,  /* K, a [K,N] weight's N, a leading dimension or a batch offset
                          is not a multiple of 16 bytes (8 bf16 / 4 fp32 elements) */
  MK_LIMIT_SHAPE = 3,  /* conv: C not a multiple of 32 (bf16) / 16 (fp32) channels,
                          P*Q not a multiple of 8, or a pooled image smaller than a
                          column tile; attention: head dim not 64 or 128; a row
                          terminal (ROWSUM / SOFTMAX / LAYERNORM) after a batched GEMM */
  MK_LIMIT_RANGE = 4   /* an operand slice of 2 GiB or more, or a grid past the launch
                          limits */
} mk_tuned_limit;

typedef struct {
  int32_t n_subkernels;
  int32_t n_ops;
  mk_shape out_shape;
  int64_t ws_bytes;               /* workspace mk_run needs (intermediates + scratch) */
  int64_t ws_intermediate_bytes;  /* sum of round_up(bytes, 256) of materialised intermediates */
  int64_t flops;                  /* algorithmic flops of the module */
  int64_t alg_bytes;              /* module inputs read once + output written once */
} mk_module_info_t;

typedef struct {
  int32_t op_begin, op_end;       /* ops [begin, end) */
  int32_t out_value;              /* value id of the materialised output */
  mk_shape out_shape;
  int64_t out_bytes;
  int64_t ws_offset;              /* byte offset in the workspace; -1 = module output buffer */
  int64_t flops;                  /* algorithmic flops of the group's ops */
  int64_t alg_bytes;              /* distinct external inputs read once + output written once */
  int32_t family;                 /* mk_family */
  int32_t impl;                   /* selected implementation id */
  int32_t n_launches;             /* kernel launches of the selected implementation */
  int64_t scratch_bytes;          /* scratch the selected implementation uses */
  int32_t uses_mfma;              /* 1: the contraction runs on the matrix cores */
  int32_t tuned_limit;            /* mk_tuned_limit of MK_IMPL_TUNED on this subkernel,
                                     whichever impl is selected */
} mk_subkernel_info_t;

/* Fill group_of_op[n_ops] with a preset decomposition.  The groupings follow
 * the fusion guidance of the decomposition prompt (App. I.1, "FUSION-FRIENDLY
 * GROUPINGS" and "FUSION EXAMPLES"): a contraction keeps its bias, element-wise
 * activations, scaling and residual add; a reduction that needs a whole row
 * (softmax) is its own subproblem unless an online form exists (attention).
 * preset 0 = split (one subkernel per op, except that a BIAS, BIAS_CHANNEL or
 * ADD joins the GEMM or CONV2D that produces its input, directly or through
 * bias / add steps that joined it); preset 1 = fused (from each op, the
 * longest group a family accepts).  Host only.  MK_E_INVALID_ARG on a null
 * argument or an unknown preset; shape errors as for mk_module_create. */
mk_status mk_decomposition_preset(const mk_module_desc* desc, int32_t preset,
                                  int32_t* group_of_op);

/* Validate the module (shape inference) and the grouping, match every group to
 * a family and lay out the workspace.  This is the programmatic check of a
 * decomposition (Sec. 3, "LLMDecompose agent": subproblems with shapes, whose
 * coverage and interfaces are checked before any kernel runs; App. I.1,
 * "VERIFICATION CRITERIA").  Host only: no device is touched.
 * group_of_op[i] is op i's group; groups are numbered 0,1,.. in op order.
 * On success *out owns a new module (free with mk_module_destroy); on an
 * error *out is NULL and the status says why (MK_E_SHAPE, MK_E_DTYPE,
 * MK_E_DECOMP, MK_E_INVALID_ARG). */
mk_status mk_module_create(const mk_module_desc* desc, const int32_t* group_of_op,
                           mk_module** out);
void mk_module_destroy(mk_module* m);

/* Introspection of the plan: the module's and each subkernel's shapes,
 * workspace placement, algorithmic flops / bytes and launches, so that run
 * time and speedups can be attributed to subkernels (Sec. 3,
 * "AllocateLLMBudget" and "Swap" act per subkernel; Sec. 1 states speedups
 * as traceable to specific subkernels).  Host only; MK_E_INVALID_ARG on a
 * null argument or a subkernel index out of range. */
mk_status mk_module_info(const mk_module* m, mk_module_info_t* info);
mk_status mk_subkernel_info(const mk_module* m, int32_t i, mk_subkernel_info_t* info);

/* Swap subkernel i's implementation (MK_IMPL_TUNED, MK_IMPL_SIMPLE or a
 * test-only mutant id).  MK_E_UNSUPPORTED if the family has no such impl. */
mk_status mk_subkernel_select(mk_module* m, int32_t i, int32_t impl_id);

/* Bytes of device workspace mk_run needs for this module under any of its
 * subkernels' implementations: the materialised intermediates of the chosen
 * decomposition (the tensors the top-level module passes between subproblems,
 * Sec. 3 and App. H.1) followed by the largest scratch of any subkernel.
 * The caller allocates it (the top-level wrapper allocates and launches,
 * App. I.2).  Host only. */
mk_status mk_workspace_size(const mk_module* m, int64_t* bytes);

/* Enqueue the composition on `stream`: the top-level module S calling its
 * subproblem kernels in order (Sec. 3; App. H.1 shows such an S for a CvT
 * block).  dev_inputs[n_inputs] are device
 * pointers to the module inputs, dev_out receives the module output, dev_ws is
 * a device workspace of ws_bytes >= mk_workspace_size.  Returns after
 * enqueueing, unless per_subkernel_ms is non-NULL: then each subkernel is
 * bracketed by HIP events, the stream is synchronised and per_subkernel_ms[i]
 * receives subkernel i's elapsed milliseconds. */
mk_status mk_run(mk_module* m, const void* const* dev_inputs, void* dev_out, void* dev_ws,
                 int64_t ws_bytes, void* stream, float* per_subkernel_ms);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): mk_run with
 * no workspace argument.  The workspace is a static device array of
 * MK_NOALLOC_WS_BYTES owned by the library; each device the library runs on
 * holds its own copy until the process ends (its address is looked up on the
 * first call on that device).  The caller still passes the inputs and the
 * output; the call only enqueues, allocates no device memory and creates no
 * events.  Every call on one device shares that device's array, which keeps
 * the last call's contents: calls that overlap on one device (two streams, two
 * threads) race and must be serialised by the caller.  MK_E_WORKSPACE if
 * mk_workspace_size exceeds MK_NOALLOC_WS_BYTES; other errors as for mk_run. */
#define MK_NOALLOC_WS_BYTES (64ll << 20)
mk_status mk_run_noalloc(mk_module* m, const void* const* dev_inputs, void* dev_out,
                         void* stream);

/* Launch-level profiling (timing of each kernel launch, for roofline
 * figures; Sec. 4 times kernels with HIP / CUDA events over repeated runs
 * after warm-up).  While a profile is open, every mk_run of the module also
 * brackets its kernel launches with timing-only HIP events (no system-scope
 * fence at each record), without synchronising, until max_launches launches
 * are recorded (later launches are not recorded).  only_launch = -1 records
 * every launch: a run contributes sum(mk_subkernel_info.n_launches)
 * consecutive entries.  only_launch = k >= 0 records only the run's k-th
 * launch (0-based, in launch order): one entry per run, the other launches
 * run back to back without events, as in an unprofiled run (each event pair
 * adds a few microseconds of dispatch time to the figure and an idle gap in
 * the stream; a chip that runs at its power limit clocks higher after gaps).
 * mk_profile_end synchronises on the last recorded launch, writes the elapsed
 * milliseconds of the recorded launches in launch order to launch_ms (at most
 * capacity entries), sets *n_recorded and closes the profile.
 * MK_E_INVALID_ARG if a profile is already open / not open, or only_launch is
 * outside [-1, launches per run). */
mk_status mk_profile_begin(mk_module* m, int32_t max_launches, int32_t only_launch);
mk_status mk_profile_end(mk_module* m, float* launch_ms, int32_t capacity, int32_t* n_recorded);

/* One reference check: stage s is subkernel s's materialised output (the last
 * subkernel's is the module output).  Element index[k] (flat, row-major; NULL
 * means index k) of that tensor must satisfy
 *   |got - expect[k]| <= atol + rtol * |expect[k]|
 * (the torch.allclose criterion, App. D); an infinite expect must be matched
 * exactly and a non-finite got against a finite expect always fails. */
typedef struct {
  int32_t stage;
  int64_t n;
  const int64_t* index;   /* host, [n] or NULL */
  const double* expect;   /* host, [n] */
  double rtol, atol;
} mk_check;

typedef struct {
  int32_t stage;
  int32_t pass;
  int64_t n_checked, n_violations, n_nonfinite;
  double max_abs_err, max_rel_err;
  double worst_ratio;     /* max |err| / (atol + rtol |expect|) */
  int64_t worst_index;    /* flat index at worst_ratio */
  double got_at_worst, expect_at_worst;
} mk_check_result;

enum { MK_MAX_CHECKS = 64 };

typedef struct {
  int32_t pass;                  /* every check passed */
  int32_t first_failing_stage;   /* lowest failing stage, -1 if none */
  int32_t n_results;
  mk_check_result results[MK_MAX_CHECKS];
} mk_verify_report;

/* The verifier (Sec. 3, "Evaluate"; per stage as in App. D's decomposed
 * checking).  Poison the workspace and the output buffer with NaN bytes (0xFF), run the
 * module once (as mk_run), synchronise, copy each checked stage to the host
 * and compare: an element that no kernel wrote reads back as NaN and fails.
 * Returns MK_OK when the checks ran; pass/fail is in *report.
 * n_checks <= MK_MAX_CHECKS. */
mk_status mk_verify(mk_module* m, const void* const* dev_inputs, void* dev_out, void* dev_ws,
                    int64_t ws_bytes, void* stream, int32_t n_checks, const mk_check* checks,
                    mk_verify_report* report);

/* Swap policy (Sec. 3, "Swap"; Alg. 1): subkernel i's speedup is
 * ms_reference[i] / ms_selected[i], the time of the reference implementation
 * over the time of the selected one.  When there are at least two subkernels
 * and at least one of them is not slower than its reference (speedup >= 1),
 * every subkernel with speedup < tau is marked for replacement by the
 * reference (swap[i] = 1); otherwise nothing is (*triggered = 0).  A
 * subkernel with no reference time (ms_reference[i] < 0) is never swapped.
 * Pure host function: arrays are host memory of length n, swap is written,
 * triggered may be NULL.  MK_E_INVALID_ARG on a null array or n < 0. */
mk_status mk_swap_decide(int32_t n, const float* ms_selected, const float* ms_reference,
                         float tau, int32_t* swap, int32_t* triggered);

/* The swap policy applied to a module: every subkernel is timed with its
 * selected implementation and with reference_impl (usually MK_IMPL_SIMPLE),
 * n_runs runs each after one warm-up run (mean of the HIP-event times of
 * mk_run, which synchronises), then mk_swap_decide runs and the marked
 * subkernels are switched to reference_impl.  Subkernels without
 * reference_impl keep their implementation.  Buffers as for mk_run; the
 * output buffer holds the last run's result.  The optional host arrays
 * [n_subkernels] receive the times and the decision. */
mk_status mk_swap(mk_module* m, const void* const* dev_inputs, void* dev_out, void* dev_ws,
                  int64_t ws_bytes, void* stream, int32_t reference_impl, float tau,
                  int32_t n_runs, float* ms_selected, float* ms_reference, int32_t* swapped,
                  int32_t* triggered);

/* Budget allocation over subkernels (the AllocateLLMBudget rule of Sec. 3):
 * if any subkernel has needs_work[i] != 0 (new or failing verification), the
 * budget is shared evenly among those; otherwise in proportion to ms[i] (the
 * last end-to-end run's per-subkernel time).  shares[n] sums to 1 (all 0 if
 * every ms is 0).  Pure host function; needs_work may be NULL. */
mk_status mk_budget_shares(int32_t n, const float* ms, const int32_t* needs_work,
                           float* shares);

/* Seeded synthetic inputs: fill host_dst with elements 0 .. n-1 of input
 * tensor `tensor_id` under `seed`, drawn from N(p0, p1) (dist 0; p1 is the
 * standard deviation) or U(p0, p1) (dist 1), rounded to float32 and, for
 * MK_BF16, to bfloat16 (raw 16-bit patterns), both to nearest even.  The
 * generator is counter based (SplitMix64 mixing, Steele, Lea and Flood,
 * OOPSLA 2014; Box-Muller cosine branch), so element i does not depend on n
 * or on the thread count.  It replaces the fixed-seed input rule of the
 * kernel-generation prompt (App. I.1, "SUBKERNEL INPUT FUNCTION
 * REQUIREMENTS") with per-tensor streams, and its bytes are exactly those of
 * the stand-alone generator the tests feed to the reference evaluation.
 * host_dst is caller-owned host memory of n floats or n uint16.
 * MK_E_INVALID_ARG on a null host_dst with n > 0, n < 0 or an unknown dist;
 * MK_E_DTYPE on an unknown dtype. */
mk_status mk_gen_fill(uint64_t seed, int32_t tensor_id, int32_t dist, double p0, double p1,
                      int32_t dtype, void* host_dst, int64_t n);

/* Status names and the calling thread's last error message (a static or
 * thread-local string; never NULL). */
const char* mk_status_str(mk_status s);
const char* mk_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
