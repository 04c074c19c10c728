"""GPU parity: every decomposition of the five workload structures, at sizes
the oracle finishes quickly that still span several tiles and ragged tails,
compared stage by stage with the oracle through mk_verify."""
import numpy as np
import pytest
import torch

from helpers import describe, run_parity
from paper_2607_20501_amd import mk, workloads

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def small(k, dtype):
    if k == 1:
        return workloads.linear_relu_rowsum(M=200, K=300, N=333, dtype=dtype)
    if k == 2:
        return workloads.gemm_gelu_softmax(M=300, K=200, N=520, dtype=dtype)
    if k == 3:
        return workloads.conv_relu_gap(N=3, C=7, H=11, W=9, K=10, dtype=dtype)
    if k == 4:
        return workloads.mlp_block(M=150, D=192, F=320, dtype=dtype,
                                   affine=((0, 1.0, 0.5), (0, 0.0, 0.3)))
    return workloads.transformer_layer(B=2, S=70, D=128, H=2, F=256, dtype=dtype,
                                       affine=((0, 1.0, 0.5), (0, 0.0, 0.3)))


CASES = [(k, dt, dec) for k in range(1, 6) for dt in ("f32", "bf16")
         for dec in ("split", "fused")]


@pytest.mark.parametrize("k,dtype,dec", CASES)
def test_parity_tuned(k, dtype, dec):
    print(f"parity tuned k={k} {dtype} {dec}", flush=True)
    rep, *_ = run_parity(small(k, dtype), dec, seed=k)
    assert rep["pass"], describe(rep)


@pytest.mark.parametrize("k,dtype,dec", CASES)
def test_parity_simple(k, dtype, dec):
    print(f"parity simple k={k} {dtype} {dec}", flush=True)
    module = small(k, dtype)
    g = mk.mk_decomposition_preset(module, dec)
    n = max(g) + 1
    rep, *_ = run_parity(module, g, seed=10 + k, impls={i: mk.IMPL_SIMPLE for i in range(n)})
    assert rep["pass"], describe(rep)


@pytest.mark.parametrize("seed", range(5))
def test_five_inputs_protocol(seed):
    """Five random inputs per correctness check, as in the evaluation protocol."""
    print(f"five-input seed={seed}", flush=True)
    for k in (2, 4):
        rep, *_ = run_parity(small(k, "bf16"), "fused", seed=seed)
        assert rep["pass"], describe(rep)


def test_softmax_rows_sum_to_one():
    rep, m, out, ref, stages = run_parity(small(2, "bf16"), "fused", seed=3)
    assert rep["pass"], describe(rep)
    o = mk.to_float64(out)
    np.testing.assert_allclose(o.sum(-1), 1.0, atol=1e-2)


def test_uniform_softmax_mutant_fails_strict_check():
    """A softmax that outputs 1/N everywhere passes the vacuous bf16 atol but
    fails the row-length-scaled check (logits spread widened by the scale)."""
    from paper_2607_20501_amd import inputs
    module = workloads.gemm_gelu_softmax(M=64, K=200, N=520, scale=8.0)
    rep, m, out, ref, stages = run_parity(module, "fused", seed=1)
    assert rep["pass"], describe(rep)
    n_row = ref[stages[-1]].shape[-1]
    uniform = np.full(ref[stages[-1]].size, 1.0 / n_row)
    loose = {"stage": 0, "expect": uniform, "rtol": 2e-2, "atol": 2e-2}
    strict = {"stage": 0, "expect": uniform, "rtol": 2e-2, "atol": 2e-2 / n_row}
    ins, _, ws = mk.device_buffers(module, inputs.make_inputs(module, 1), m.workspace_size())
    r = m.verify(ins, out, ws, [loose, strict])
    assert r["results"][0]["pass"] and not r["results"][1]["pass"]
