"""GPU parity of the GEMM family at shapes that exercise the tuned MFMA path:
several 256-wide tiles, ragged M/N/K tails, both weight layouts, batched
attention products, and the terminal softmax / row-sum reductions."""
import math

import numpy as np
import pytest
import torch

from helpers import describe, run_parity
from paper_2607_20501_amd import mk, workloads

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def op(kind, ins, ip=(), fp=()):
    return {"kind": kind, "in": list(ins), "ip": list(ip), "fp": list(fp)}


def gemm_module(M, N, K, layout, dtype="bf16", epi=(), std=0.5):
    w = [N, K] if layout == 0 else [K, N]
    ops = [op("GEMM", [0, 1], [layout])]
    inputs = [[M, K], w]
    recipes = [(0, 0.0, 1.0), (0, 0.0, std / math.sqrt(K))]
    for e in epi:
        v = len(inputs) + len(ops) - 1
        if e == "BIAS":
            inputs.append([N])
            recipes.append((1, -0.5, 0.5))
            ops.append(op("BIAS", [v, None]))
        elif e == "ADD":
            inputs.append([M, N])
            recipes.append((0, 0.0, 1.0))
            ops.append(op("ADD", [v, None]))
        elif e == "SCALE":
            ops.append(op("SCALE", [v], fp=[0.75]))
        else:
            ops.append(op(e, [v]))
    # value ids of the extra operands are assigned after all inputs are known
    n_in = len(inputs)
    extra = 2
    for i, o in enumerate(ops):
        if i > 0:
            o["in"][0] = n_in + i - 1
        if None in o["in"]:
            o["in"][1] = extra
            extra += 1
    return {"name": "gemm", "dtype": dtype, "inputs": inputs, "recipes": recipes, "ops": ops}


# (K of 8, 32, 64 and 96 give 1, 1, 2 and 3 K slices: fewer than the ring's
# leading slices)
SHAPES = [(256, 256, 64), (513, 264, 136), (300, 520, 200), (1000, 1024, 1024), (64, 8, 8),
          (777, 1536, 328), (128, 512, 32), (300, 512, 96)]


@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("shape", SHAPES)
def test_gemm_plain(shape, layout):
    M, N, K = shape
    print(f"gemm {shape} layout {layout}", flush=True)
    module = gemm_module(M, N, K, layout)
    rep, m, *_ = run_parity(module, [0])
    assert m.subkernels()[0]["family"] == "GEMM"
    assert rep["pass"], describe(rep)


@pytest.mark.parametrize("layout", [0, 1])
def test_gemm_epilogue_chain(layout):
    module = gemm_module(700, 600, 264, layout, epi=("BIAS", "GELU_ERF", "SCALE", "ADD"))
    rep, *_ = run_parity(module, [0, 0, 0, 0, 0])
    assert rep["pass"], describe(rep)
    module = gemm_module(700, 600, 264, layout, epi=("BIAS", "GELU_TANH", "RELU"))
    rep, *_ = run_parity(module, [0, 0, 0, 0])
    assert rep["pass"], describe(rep)


@pytest.mark.parametrize("term", ["SOFTMAX", "ROWSUM"])
@pytest.mark.parametrize("N", [256, 600, 1024])
def test_gemm_terminal(term, N):
    module = gemm_module(333, N, 192, 1, epi=("BIAS", "GELU_TANH", "SCALE", term))
    rep, m, out, ref, stages = run_parity(module, [0] * 5)
    assert rep["pass"], describe(rep)
    if term == "SOFTMAX":
        np.testing.assert_allclose(mk.to_float64(out).sum(-1), 1.0, atol=1e-2)


def test_gemm_ln_prologue():
    module = workloads.mlp_block(M=300, D=256, F=512, affine=((0, 1.0, 0.5), (0, 0.0, 0.3)))
    for groups in ([0, 0, 0, 1, 1], [0, 0, 1, 2, 2]):
        rep, *_ = run_parity(module, groups)
        assert rep["pass"], describe(rep)


@pytest.mark.parametrize("S,dh,H", [(256, 128, 2), (300, 64, 3), (520, 128, 1)])
def test_attention_products_split(S, dh, H):
    """QK^T (weight layout [N,K] over packed K) and PV (layout [K,N] over packed V)
    as batched MFMA GEMMs, with the mask and softmax in between."""
    module = workloads.transformer_layer(B=2, S=S, D=H * dh, H=H, F=2 * H * dh)
    g = mk.mk_decomposition_preset(module, "split")
    rep, *_ = run_parity(module, g)
    assert rep["pass"], describe(rep)


def test_split_and_fused_agree_with_their_own_references():
    """Both decompositions of one module match their oracle references; the
    two references differ only by the rounding of materialised stages."""
    module = workloads.gemm_gelu_softmax(M=512, K=512, N=1024)
    outs = []
    for dec in ("split", "fused"):
        rep, m, out, ref, stages = run_parity(module, dec)
        assert rep["pass"], describe(rep)
        outs.append(mk.to_float64(out))
    np.testing.assert_allclose(outs[0], outs[1], rtol=5e-2, atol=2e-5)


F32_SHAPES = [(256, 256, 64), (513, 264, 132), (300, 520, 200), (128, 256, 256),
              (1000, 1024, 1028), (64, 4, 4), (256, 256, 16), (300, 512, 32)]


@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("shape", F32_SHAPES)
def test_gemm_plain_f32(shape, layout):
    """fp32 operands on the fp32 matrix cores (32x32x2 MFMA), ragged tails
    included, to the fp32 tolerance."""
    M, N, K = shape
    print(f"gemm f32 {shape} layout {layout}", flush=True)
    module = gemm_module(M, N, K, layout, dtype="f32")
    rep, m, *_ = run_parity(module, [0])
    assert m.subkernels()[0]["uses_mfma"]
    assert rep["pass"], describe(rep)


@pytest.mark.parametrize("term", ["SOFTMAX", "ROWSUM", None])
def test_gemm_epilogue_f32(term):
    epi = ("BIAS", "GELU_ERF", "SCALE") + ((term,) if term else ("ADD",))
    module = gemm_module(333, 600, 196, 0, dtype="f32", epi=epi)
    rep, m, *_ = run_parity(module, [0] * (len(epi) + 1))
    assert m.subkernels()[0]["uses_mfma"]
    assert rep["pass"], describe(rep)


def test_linear_relu_rowsum_f32_both_impls():
    """The fp32 Linear + bias + ReLU + row-sum module: tuned (MFMA) and simple
    subkernels, fused and split."""
    module = workloads.linear_relu_rowsum()
    for dec in ("fused", "split"):
        for impl in (mk.IMPL_TUNED, mk.IMPL_SIMPLE):
            g = mk.mk_decomposition_preset(module, dec)
            rep, m, *_ = run_parity(module, g, impls={i: impl for i in range(max(g) + 1)})
            assert rep["pass"], f"{dec} impl {impl}: " + describe(rep)
            assert m.subkernels()[0]["uses_mfma"] == (impl == mk.IMPL_TUNED)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("dec", ["fused", "split"])
@pytest.mark.parametrize("shape", [(300, 256, 512), (257, 600, 264), (64, 1000, 128)])
def test_post_ln_ffn_block(shape, dec, dtype):
    """CvT post-LN ReLU FFN, LN(x + W2 relu(W1 x + b1) + b2): fused, the
    second GEMM ends in the LayerNorm terminal (per-tile moments, then the
    finisher); ragged row lengths leave partial column tiles."""
    M, D, F = shape
    print(f"cvt ffn {shape} {dec} {dtype}", flush=True)
    module = workloads.cvt_ffn_block(M=M, D=D, F=F, dtype=dtype)
    rep, m, *_ = run_parity(module, dec)
    assert rep["pass"], describe(rep)
    if dec == "fused":
        assert m.subkernels()[1]["uses_mfma"] and m.subkernels()[1]["n_launches"] == 2
    rep, *_ = run_parity(module, dec, impls={i: mk.IMPL_SIMPLE for i in range(m.n)})
    assert rep["pass"], "simple: " + describe(rep)


# At least 64 tiles of 256 x 256 (smaller problems take the 64 x 64 kernel),
# ragged in M and N; the chains compiled into their own epilogues (none, exact
# GELU, residual add, column bias, bias + tanh GELU + scale + softmax
# partials) and the
# interpreted chain.  N = 2053 makes the output rows unaligned for 16-byte
# stores (element-wise tail path).
BIG_CHAINS = [(), ("GELU_ERF",), ("ADD",), ("BIAS",), ("BIAS", "GELU_TANH", "SCALE", "SOFTMAX"),
              ("BIAS", "GELU_ERF", "SCALE", "ADD"), ("ROWSUM",)]


@pytest.mark.parametrize("epi", BIG_CHAINS, ids=lambda e: "+".join(e) or "none")
@pytest.mark.parametrize("M,N,layout", [(2100, 2056, 0), (2100, 2056, 1), (2071, 2053, 0)])
def test_gemm_big_tiles(M, N, layout, epi):
    print(f"gemm big {M}x{N} layout {layout} {epi}", flush=True)
    module = gemm_module(M, N, 136, layout, epi=epi)
    rep, m, out, *_ = run_parity(module, [0] * (1 + len(epi)))
    assert m.subkernels()[0]["uses_mfma"]
    assert rep["pass"], describe(rep)
    if "SOFTMAX" in epi:
        np.testing.assert_allclose(mk.to_float64(out).sum(-1), 1.0, atol=1e-2)


@pytest.mark.parametrize("epi", [(), ("BIAS", "GELU_TANH", "SCALE", "SOFTMAX")],
                         ids=lambda e: "+".join(e) or "none")
def test_gemm_big_tiles_f32(epi):
    module = gemm_module(2100, 2056, 72, 0, dtype="f32", epi=epi)
    rep, m, *_ = run_parity(module, [0] * (1 + len(epi)))
    assert rep["pass"], describe(rep)


# K a multiple of the 64-deep stage: the compiled chains without a terminal
# run on four waves of 128 x 128 each, the stage loop in groups of six; 1, 5,
# 6 and 7 stages cover a lone stage, the remainder, one whole group and a group
# plus one.  Ragged M and N, and N = 2053 for unaligned output rows.
FOUR_WAVE_CHAINS = [(), ("GELU_ERF",), ("ADD",), ("BIAS",), ("BIAS", "GELU_TANH", "SCALE")]


@pytest.mark.parametrize("epi", FOUR_WAVE_CHAINS, ids=lambda e: "+".join(e) or "none")
@pytest.mark.parametrize("M,N,K", [(2100, 2056, 64), (2071, 2053, 320), (2048, 2048, 384),
                                   (2100, 2056, 448)])
def test_gemm_big_tiles_whole_stages(M, N, K, epi):
    print(f"gemm big {M}x{N}x{K} {epi}", flush=True)
    module = gemm_module(M, N, K, 0, epi=epi)
    rep, m, out, *_ = run_parity(module, [0] * (1 + len(epi)))
    assert m.subkernels()[0]["uses_mfma"]
    assert rep["pass"], describe(rep)
