"""Degenerate shapes of every family against the oracle: a single row, a
single output column, a contraction of depth 1, rows of length 1 (softmax ->
1, LayerNorm -> beta), a single-token sequence, a 1x1 image through a 3x3
conv, a single-element element-wise chain, and the smallest shapes the
matrix-core path accepts (K = 8 / 4, one slice)."""
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


def check(module, dec):
    rep, m, out, ref, stages = run_parity(module, dec)
    assert rep["pass"], describe(rep)
    return m, out


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("dec", ["fused", "split"])
def test_single_row_gemm_softmax(dtype, dec):
    check(workloads.gemm_gelu_softmax(M=1, K=64, N=300, dtype=dtype), dec)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (7, 1, 16), (5, 3, 1), (64, 64, 8), (33, 40, 4)])
def test_tiny_contractions(dtype, M, N, K):
    module = workloads.linear_relu_rowsum(M=M, K=K, N=N, dtype=dtype)
    for dec in ("fused", "split"):
        check(module, dec)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_rows_of_length_one(dtype):
    sm = {"name": "sm", "dtype": dtype, "inputs": [[9, 1]], "recipes": [(0, 0.0, 3.0)],
          "ops": [op("SOFTMAX", [0])]}
    m, out = check(sm, "fused")
    assert np.all(mk.to_float64(out) == 1.0)
    ln = {"name": "ln", "dtype": dtype, "inputs": [[9, 1], [1], [1]],
          "recipes": [(0, 0.0, 3.0), (1, 0.5, 1.5), (1, -1.0, 1.0)],
          "ops": [op("LAYERNORM", [0, 1, 2], fp=[1e-5])]}
    check(ln, "fused")
    rs = {"name": "rs", "dtype": dtype, "inputs": [[9, 1]], "recipes": [(0, 0.0, 3.0)],
          "ops": [op("ROWSUM", [0])]}
    check(rs, "fused")


@pytest.mark.parametrize("causal", [True, False])
def test_single_token_sequence(causal):
    B, S, H, dh = 2, 1, 2, 128
    ops = [op("QK", [0], [B, H, dh, S], [1 / math.sqrt(dh)])]
    v = 1
    if causal:
        ops.append(op("CAUSAL_MASK", [v]))
        v += 1
    ops += [op("SOFTMAX", [v]), op("PV", [v + 1, 0], [B, H, dh, S])]
    module = {"name": "attn1", "dtype": "bf16", "inputs": [[B * S, 3 * H * dh]],
              "recipes": [(0, 0.0, 1.0)], "ops": ops}
    for g in ([0] * len(ops), list(range(len(ops)))):
        m, out = check(module, g)


@pytest.mark.parametrize("pool", ["GAP", "GMP", "LPPOOL"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_one_pixel_image(pool, dtype):
    module = workloads.conv_relu_gap(N=2, C=32, H=1, W=1, K=8, dtype=dtype, pool=pool)
    for dec in ("fused", "split"):
        check(module, dec)


def test_single_element_chain():
    module = {"name": "ew1", "dtype": "bf16", "inputs": [[1, 1], [1]],
              "recipes": [(0, 0.0, 1.0), (1, -1.0, 1.0)],
              "ops": [op("BIAS", [0, 1]), op("GELU_ERF", [2]), op("SCALE", [3], fp=[0.5])]}
    for dec in ("fused", "split"):
        check(module, dec)


def test_ragged_element_wise_tail():
    """numel not a multiple of the 8-element group: the tail is finished by
    block 0 of the vector kernel."""
    module = {"name": "ew", "dtype": "bf16", "inputs": [[37, 11], [11]],
              "recipes": [(0, 0.0, 1.0), (1, -1.0, 1.0)],
              "ops": [op("BIAS", [0, 1]), op("GELU_TANH", [2])]}
    for dec in ("fused", "split"):
        check(module, dec)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_verify_rejects_an_unwritten_output_row(dtype):
    """mk_verify poisons the output buffer: a final-stage kernel that leaves
    its last row unwritten fails, even when the buffer already holds a
    correct output from an earlier run of the same module."""
    from paper_2607_20501_amd import inputs
    import oracle
    from helpers import TOL
    module = workloads.gemm_gelu_softmax(M=70, K=64, N=300, dtype=dtype)
    groups = mk.mk_decomposition_preset(module, "split")
    host = inputs.make_inputs(module, 0)
    ref = oracle.run(module, groups, host, keep={len(groups) - 1})[-1]
    m = mk.Module(module, groups)
    ins, _, ws = mk.device_buffers(module, host, m.workspace_size())
    out = mk.out_tensor(module, m.info["out_shape"])
    rtol, atol = TOL[dtype]
    checks = [{"stage": m.n - 1, "expect": ref.reshape(-1), "rtol": rtol, "atol": atol}]
    assert m.verify(ins, out, ws, checks)["pass"]
    m.run(ins, out, ws)                      # a correct output now sits in `out`
    torch.cuda.synchronize()
    m.select(m.n - 1, 110)                   # the softmax rows kernel skips the last row
    rep = m.verify(ins, out, ws, checks)
    assert not rep["pass"]
    r = rep["results"][0]
    assert r["n_nonfinite"] == 300 and r["worst_index"] >= 69 * 300, describe(rep)
