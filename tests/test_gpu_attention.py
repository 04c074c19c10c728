"""GPU parity of the attention family: the fused (flash) subkernel and the
split QK^T / mask / softmax / PV chain, causal and not, with ragged sequence
lengths, against the oracle; plus the causal-mask off-by-one mutant."""
import math

import numpy as np
import pytest
import torch

from helpers import describe, run_parity
from paper_2607_20501_amd import mk

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def attn_module(B, S, H, dh, causal=True, dtype="bf16"):
    ops = [{"kind": "QK", "in": [0], "ip": [B, H, dh, S], "fp": [1 / math.sqrt(dh)]}]
    v = 1
    if causal:
        ops.append({"kind": "CAUSAL_MASK", "in": [v], "ip": [], "fp": []})
        v += 1
    ops.append({"kind": "SOFTMAX", "in": [v], "ip": [], "fp": []})
    ops.append({"kind": "PV", "in": [v + 1, 0], "ip": [B, H, dh, S], "fp": []})
    return {"name": "attention", "dtype": dtype, "inputs": [[B * S, 3 * H * dh]],
            "recipes": [(0, 0.0, 1.0)], "ops": ops}


CASES = [(2, 256, 2, 128, True), (1, 300, 3, 128, True), (2, 200, 2, 64, True),
         (1, 128, 1, 128, False), (2, 333, 2, 64, False), (1, 1024, 2, 128, True),
         (3, 77, 2, 128, True)]


@pytest.mark.parametrize("B,S,H,dh,causal", CASES)
def test_fused_attention(B, S, H, dh, causal):
    print(f"fused attention B={B} S={S} H={H} dh={dh} causal={causal}", flush=True)
    module = attn_module(B, S, H, dh, causal)
    g = [0] * len(module["ops"])
    rep, m, *_ = run_parity(module, g)
    assert m.subkernels()[0]["family"] == "ATTN"
    assert rep["pass"], describe(rep)


@pytest.mark.parametrize("B,S,H,dh,causal", CASES[:3])
def test_split_attention(B, S, H, dh, causal):
    module = attn_module(B, S, H, dh, causal)
    g = list(range(len(module["ops"])))
    rep, *_ = run_parity(module, g)
    assert rep["pass"], describe(rep)


def test_mask_off_by_one_mutant_is_caught():
    """App. D's 'causal mask off-by-one' bug: masking the diagonal too.  The
    output stage must fail against the oracle (row 0 has no key left)."""
    module = attn_module(1, 256, 2, 128, True)
    g = [0] * len(module["ops"])
    rep, *_ = run_parity(module, g, impls={0: 102})
    assert not rep["pass"]
    rep, *_ = run_parity(module, g, impls={0: mk.IMPL_SIMPLE})
    assert rep["pass"], describe(rep)


def test_fused_attention_growing_scores():
    """Keys whose scale grows along the sequence (and a few large spikes), so
    that the running maximum of a query's scores rises by many units after
    the first key blocks: the fused kernel moves its softmax reference (and
    rescales the partial output) only when the maximum exceeds it by more
    than a fixed margin, and must still match the oracle."""
    from paper_2607_20501_amd import inputs
    B, S, H, dh = 1, 1024, 2, 128
    module = attn_module(B, S, H, dh, True)
    x = inputs.bf16_bits_to_f32(inputs.make_inputs(module, 3)[0]).reshape(B * S, 3 * H * dh)
    key = np.arange(B * S) % S
    ramp = (1.0 + 6.0 * key / S).astype(np.float32)[:, None]
    x[:, H * dh:2 * H * dh] *= ramp                       # K grows along the keys
    x[[100, 400, 700, 900], H * dh:2 * H * dh] *= 4.0     # and jumps at a few keys
    bits = (x.astype(np.float32).view(np.uint32) + 0x7FFF + ((x.view(np.uint32) >> 16) & 1)) >> 16
    rep, *_ = run_parity(module, [0] * len(module["ops"]), host=[bits.astype(np.uint16).ravel()])
    assert rep["pass"], describe(rep)
