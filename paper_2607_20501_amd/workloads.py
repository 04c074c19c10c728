"""Synthetic composed modules shaped like the paper's workloads.

MKEvolve (arXiv 2607.20501) evaluates on KernelBench L2 operator sequences
(e.g. convolution, ReLU and bias) and L3 full models (e.g. MiniGPT), and
studies a MinGPT causal-attention block and a Transformer FFN block in App. D.
Those suites are not available here; these seeded modules of the same
structure stand in for them.  A module is a plain dict:

    {"name", "dtype": "f32"|"bf16", "inputs": [shape, ...],
     "recipes": [(dist, p0, p1), ...], "ops": [{"kind", "in", "ip", "fp"}, ...]}

Value ids 0..n_inputs-1 are the module inputs; n_inputs+i is op i's output;
the last op's output is the module output.  Nothing here computes anything.
"""
import math

from .inputs import NORMAL, UNIFORM


def _op(kind, ins, ip=(), fp=()):
    return {"kind": kind, "in": list(ins), "ip": list(ip), "fp": list(fp)}


def linear_relu_rowsum(M=128, K=256, N=256, dtype="f32", std=0.05):
    """Linear(K->N) + bias + ReLU + row-sum; x, W, b ~ N(0, 1) * std."""
    return {
        "name": f"linear_relu_rowsum_{M}x{K}x{N}_{dtype}",
        "dtype": dtype,
        "inputs": [[M, K], [N, K], [N]],
        "recipes": [(NORMAL, 0.0, std)] * 3,
        "ops": [_op("GEMM", [0, 1], [0]), _op("BIAS", [3, 2]), _op("RELU", [4]),
                _op("ROWSUM", [5])],
    }


def gemm_gelu_softmax(M=8192, K=4096, N=4096, dtype="bf16", scale=0.5):
    """x[M,K] @ W[K,N] + b, tanh-GELU, scale, row softmax;
    x, W ~ N(0, 0.02), b ~ U(-0.1, 0.1)."""
    return {
        "name": f"gemm_gelu_softmax_{M}x{K}x{N}_{dtype}",
        "dtype": dtype,
        "inputs": [[M, K], [K, N], [N]],
        "recipes": [(NORMAL, 0.0, 0.02), (NORMAL, 0.0, 0.02), (UNIFORM, -0.1, 0.1)],
        "ops": [_op("GEMM", [0, 1], [1]), _op("BIAS", [3, 2]), _op("GELU_TANH", [4]),
                _op("SCALE", [5], fp=[scale]), _op("SOFTMAX", [6])],
    }


def conv_relu_gap(N=64, C=128, H=56, W=56, K=256, R=3, stride=1, pad=1, dtype="bf16",
                  pool="GAP", p=2.0):
    """3x3 conv (NCHW, KCRS) + per-channel bias + ReLU + global pool: average
    (GAP), or the variants of Sec. 4's MobileNet adaptation, max (GMP) and
    LP with exponent p (LPPOOL); x ~ N(0, 1), w ~ N(0, 0.02), b ~ U(-0.1, 0.1)."""
    tag = {"GAP": "gap", "GMP": "gmp", "LPPOOL": f"lp{p:g}"}[pool]
    return {
        "name": f"conv_relu_{tag}_{N}x{C}x{H}x{W}_k{K}_{dtype}",
        "dtype": dtype,
        "inputs": [[N, C, H, W], [K, C, R, R], [K]],
        "recipes": [(NORMAL, 0.0, 1.0), (NORMAL, 0.0, 0.02), (UNIFORM, -0.1, 0.1)],
        "ops": [_op("CONV2D", [0, 1], [stride, pad]), _op("BIAS_CHANNEL", [3, 2]),
                _op("RELU", [4]), _op(pool, [5], fp=[p] if pool == "LPPOOL" else [])],
    }


def mlp_block(M=16384, D=4096, F=14336, dtype="bf16", eps=1e-5, affine=None):
    """x -> LayerNorm -> Linear(D->F) -> exact GELU -> Linear(F->D) -> + x.
    x ~ N(0, 1); W ~ N(0, 0.02); gamma = 1, beta = 0 unless `affine` gives
    recipes for them (used by tests to exercise a general affine)."""
    g, b = affine if affine else ((UNIFORM, 1.0, 1.0), (UNIFORM, 0.0, 0.0))
    return {
        "name": f"mlp_block_{M}x{D}x{F}_{dtype}",
        "dtype": dtype,
        "inputs": [[M, D], [D], [D], [F, D], [D, F]],
        "recipes": [(NORMAL, 0.0, 1.0), g, b, (NORMAL, 0.0, 0.02), (NORMAL, 0.0, 0.02)],
        "ops": [_op("LAYERNORM", [0, 1, 2], fp=[eps]), _op("GEMM", [5, 3], [0]),
                _op("GELU_ERF", [6]), _op("GEMM", [7, 4], [0]), _op("ADD", [8, 0])],
    }


def transformer_layer(B=8, S=2048, D=2048, H=16, F=8192, dtype="bf16", eps=1e-5,
                      affine=None):
    """Pre-LN layer: h = x + W_o Attn(LN1(x)) with causal attention over packed
    [Q|K|V], then out = h + MLP(LN2(h)) with exact GELU; no biases.
    x ~ N(0, 1); W ~ N(0, 0.02); LN gamma = 1, beta = 0 unless `affine`."""
    dh = D // H
    g, b = affine if affine else ((UNIFORM, 1.0, 1.0), (UNIFORM, 0.0, 0.0))
    w = (NORMAL, 0.0, 0.02)
    n = 9
    return {
        "name": f"transformer_layer_b{B}_s{S}_d{D}_h{H}_f{F}_{dtype}",
        "dtype": dtype,
        "inputs": [[B, S, D], [D], [D], [3 * D, D], [D, D], [D], [D], [F, D], [D, F]],
        "recipes": [(NORMAL, 0.0, 1.0), g, b, w, w, g, b, w, w],
        "ops": [
            _op("LAYERNORM", [0, 1, 2], fp=[eps]),          # 0 -> n+0
            _op("GEMM", [n + 0, 3], [0]),                    # 1 qkv
            _op("QK", [n + 1], [B, H, dh, S], [1.0 / math.sqrt(dh)]),  # 2
            _op("CAUSAL_MASK", [n + 2]),                     # 3
            _op("SOFTMAX", [n + 3]),                         # 4
            _op("PV", [n + 4, n + 1], [B, H, dh, S]),        # 5
            _op("GEMM", [n + 5, 4], [0]),                    # 6 out-proj
            _op("ADD", [n + 6, 0]),                          # 7 h
            _op("LAYERNORM", [n + 7, 5, 6], fp=[eps]),       # 8
            _op("GEMM", [n + 8, 7], [0]),                    # 9
            _op("GELU_ERF", [n + 9]),                        # 10
            _op("GEMM", [n + 10, 8], [0]),                   # 11
            _op("ADD", [n + 11, n + 7]),                     # 12
        ],
    }


def cvt_ffn_block(M=4096, D=768, F=3072, dtype="bf16", eps=1e-5):
    """Post-LN ReLU FFN of a CvT block (App. H.2): out = LN(x + W2 relu(W1 x +
    b1) + b2).  x ~ N(0, 1); W ~ N(0, 0.02); b ~ U(-0.1, 0.1); gamma ~
    U(0.5, 1.5), beta ~ U(-0.5, 0.5)."""
    w, bias = (NORMAL, 0.0, 0.02), (UNIFORM, -0.1, 0.1)
    n = 7
    return {
        "name": f"cvt_ffn_{M}x{D}x{F}_{dtype}",
        "dtype": dtype,
        "inputs": [[M, D], [F, D], [F], [D, F], [D], [D], [D]],
        "recipes": [(NORMAL, 0.0, 1.0), w, bias, w, bias, (UNIFORM, 0.5, 1.5),
                    (UNIFORM, -0.5, 0.5)],
        "ops": [_op("GEMM", [0, 1], [0]),                      # 0
                _op("BIAS", [n + 0, 2]),                        # 1
                _op("RELU", [n + 1]),                           # 2
                _op("GEMM", [n + 2, 3], [0]),                   # 3
                _op("BIAS", [n + 3, 4]),                        # 4
                _op("ADD", [n + 4, 0]),                         # 5 residual
                _op("LAYERNORM", [n + 5, 5, 6], fp=[eps])],     # 6 post-LN
    }


def causal_attention_block(B=2, S=256, D=512, H=4, dtype="bf16", x_std=1.0):
    """MinGPT-style causal self-attention without residual (App. D case 1):
    QKV projection -> scaled q.k -> causal mask -> softmax -> PV -> output
    projection.  x ~ N(0, x_std); W ~ N(0, 0.02)."""
    dh = D // H
    w = (NORMAL, 0.0, 0.02)
    n = 3
    return {
        "name": f"causal_attention_b{B}_s{S}_d{D}_h{H}" + (f"_x{x_std:g}" if x_std != 1.0 else "")
                + f"_{dtype}",
        "dtype": dtype,
        "inputs": [[B, S, D], [3 * D, D], [D, D]],
        "recipes": [(NORMAL, 0.0, x_std), w, w],
        "ops": [
            _op("GEMM", [0, 1], [0]),                                  # 0 qkv
            _op("QK", [n + 0], [B, H, dh, S], [1.0 / math.sqrt(dh)]),  # 1
            _op("CAUSAL_MASK", [n + 1]),                               # 2
            _op("SOFTMAX", [n + 2]),                                   # 3
            _op("PV", [n + 3, n + 0], [B, H, dh, S]),                  # 4
            _op("GEMM", [n + 4, 2], [0]),                              # 5 out-proj
        ],
    }


def full_size(k):
    """The five full-size workloads, numbered as in the benchmark's config list
    (1-based): 1 linear+ReLU+row-sum fp32, 2 GEMM+GELU+softmax bf16,
    3 conv+ReLU+GAP (bf16; fp32 via dtype), 4 MLP block bf16, 5 transformer
    layer bf16."""
    return {1: linear_relu_rowsum, 2: gemm_gelu_softmax, 3: conv_relu_gap, 4: mlp_block,
            5: transformer_layer}[k]()
