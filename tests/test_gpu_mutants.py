"""The eleven injected bugs of App. D as test-only subkernel implementations
(ids >= 100), each swapped into one subkernel of the split form of its block
(MinGPT causal attention; Transformer FFN), in fp32: the per-stage check
against the oracle must reject every one, while the same module with the
correct subkernels passes.  (The tile-boundary and accumulator-dtype bugs
are one implementation each, applied to q.k^T / fc1 and q.k^T / fc2.)"""
import pytest
import torch

from helpers import describe, run_parity
from paper_2607_20501_amd import mk, workloads

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

UNSAFE_SOFTMAX, MASK_OFF_BY_ONE, TILE_BOUNDARY, BF16_ACCUM = 101, 102, 103, 104
SOFTMAX_DIM, UNSAFE_LN, GELU_SIGMOID, NO_RESIDUAL, RELU_GELU = 105, 106, 107, 108, 109


def attention():
    return workloads.causal_attention_block(B=2, S=128, D=256, H=2, dtype="f32")


def large_logits():
    """A softmax stage whose logits (60..120) overflow exp() unless the row
    max is subtracted first."""
    return {"name": "softmax_large_logits", "dtype": "f32", "inputs": [[64, 512]],
            "recipes": [(1, 60.0, 120.0)],
            "ops": [{"kind": "SOFTMAX", "in": [0], "ip": [], "fp": []}]}


def ffn():
    # x ~ N(0, 1) plus an offset so that skipping the centring matters
    m = workloads.mlp_block(M=256, D=256, F=512, dtype="f32")
    m["recipes"][0] = (0, 3.0, 1.0)
    return m


# (bug, module factory, op index whose split subkernel gets the mutant)
CASES = [
    ("unsafe softmax", UNSAFE_SOFTMAX, large_logits, 0),
    ("mask off-by-one", MASK_OFF_BY_ONE, attention, 2),
    ("tile boundary (K)", TILE_BOUNDARY, attention, 1),
    ("wrong acc dtype (QK)", BF16_ACCUM, attention, 1),
    ("softmax dim=-2", SOFTMAX_DIM, attention, 3),
    ("unsafe LayerNorm", UNSAFE_LN, ffn, 0),
    ("GELU sigmoid approx", GELU_SIGMOID, ffn, 2),
    ("tile boundary (fc1)", TILE_BOUNDARY, ffn, 1),
    ("wrong acc dtype (fc2)", BF16_ACCUM, ffn, 3),
    ("missing residual", NO_RESIDUAL, ffn, 3),
    ("ReLU not GELU", RELU_GELU, ffn, 2),
]


@pytest.mark.parametrize("name,impl,make,op", CASES, ids=[c[0] for c in CASES])
def test_mutant_is_caught_per_stage(name, impl, make, op):
    module = make()
    groups = mk.mk_decomposition_preset(module, "split")
    sk = groups[op]
    print(f"mutant {impl} ({name}) on subkernel {sk} of {module['name']}", flush=True)
    rep, m, *_ = run_parity(module, groups, strict_softmax=False)
    assert rep["pass"], "correct subkernels must pass: " + describe(rep)
    rep, m, *_ = run_parity(module, groups, impls={sk: impl}, strict_softmax=False)
    assert m.subkernels()[sk]["impl"] == impl
    assert not rep["pass"], f"{name} was not caught"
    # the first failing stage is the mutated subkernel itself
    first = min(r["stage"] for r in rep["results"] if not r["pass"])
    assert first == sk, describe(rep)


def test_mutants_only_where_they_apply():
    module = ffn()
    groups = mk.mk_decomposition_preset(module, "split")
    m = mk.Module(module, groups)
    with pytest.raises(mk.MkError):
        m.select(0, SOFTMAX_DIM)      # LayerNorm subkernel has no softmax
    with pytest.raises(mk.MkError):
        m.select(2, BF16_ACCUM)       # element-wise subkernel has no contraction
