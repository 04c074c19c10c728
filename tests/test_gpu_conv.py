"""GPU parity of the conv family: implicit-GEMM MFMA path (bf16 and fp32;
padded-NHWC gather, NCHW store or fused GAP over tiles that straddle images)
and the simple direct conv, against the oracle."""
import pytest
import torch

from helpers import describe, run_parity
from paper_2607_20501_amd import mk, workloads
from paper_2607_20501_amd.inputs import NORMAL, UNIFORM

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

# (bf16 with C % 64 == 0 and at least 256 positions per image takes the
# persistent 256 x 256 kernel: C=64 and C=128 below, ragged in channels and in
# position tiles that straddle images)
CASES = [dict(N=3, C=32, H=20, W=20, K=40), dict(N=2, C=64, H=16, W=16, K=300),
         dict(N=2, C=32, H=31, W=31, K=64, stride=2), dict(N=1, C=96, H=24, W=24, K=256),
         dict(N=2, C=8, H=9, W=7, K=5), dict(N=3, C=64, H=20, W=20, K=40),
         dict(N=2, C=128, H=20, W=20, K=264)]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", CASES)
@pytest.mark.parametrize("dec", ["fused", "split"])
def test_conv_parity(shape, dec, dtype):
    print(f"conv {shape} {dec} {dtype}", flush=True)
    module = workloads.conv_relu_gap(dtype=dtype, **shape)
    rep, m, *_ = run_parity(module, dec)
    assert m.subkernels()[0]["uses_mfma"] == (shape["C"] % 32 == 0)
    assert rep["pass"], describe(rep)


def test_conv_impls_agree():
    module = workloads.conv_relu_gap(N=2, C=32, H=20, W=20, K=40)
    rep, m, *_ = run_parity(module, "fused", impls={0: mk.IMPL_SIMPLE})
    assert rep["pass"], describe(rep)
    assert m.subkernels()[0]["n_launches"] == 1
    rep, m, *_ = run_parity(module, "fused")
    assert rep["pass"], describe(rep)
    assert m.subkernels()[0]["n_launches"] == 3   # pack, GEMM, pool finish


POOL_CASES = [dict(N=3, C=32, H=20, W=20, K=40), dict(N=2, C=64, H=16, W=16, K=300),
              dict(N=2, C=8, H=9, W=7, K=5)]


# Persistent bf16 conv with a split last round.  294 position tiles of 256:
# the 38 tiles past the last whole round of 256 workgroups run as 64-row
# sub-tiles, K=40 leaving the second row-wave of each sub-tile 8 rows.  40
# tiles (fewer than the CUs): all cut into 64-row sub-tiles, K=100 giving a
# full first sub-tile, a ragged second one (36 rows) and two empty ones.
# K=300: two tile rows (294 tiles, the second row 44 channels deep), so the
# split round mixes full sub-tiles, a ragged one and empty ones.
@pytest.mark.parametrize("shape", [dict(N=24, C=64, H=56, W=56, K=40),
                                   dict(N=10, C=64, H=32, W=32, K=100),
                                   dict(N=12, C=64, H=56, W=56, K=300)])
def test_conv_tail_split(shape):
    print(f"conv tail split {shape}", flush=True)
    module = workloads.conv_relu_gap(dtype="bf16", **shape)
    rep, m, *_ = run_parity(module, "fused")
    assert rep["pass"], describe(rep)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("pool,p", [("GMP", 2.0), ("LPPOOL", 2.0), ("LPPOOL", 3.0)])
@pytest.mark.parametrize("shape", POOL_CASES)
@pytest.mark.parametrize("dec", ["fused", "split"])
def test_pooling_variants(shape, dec, pool, p, dtype):
    """Max and LP pooling in place of the average (Sec. 4 adaptation): fused
    into the conv GEMM's per-tile partials (tiles straddle images) and as a
    row subkernel after the split conv."""
    print(f"conv {shape} {dec} {pool} p={p} {dtype}", flush=True)
    module = workloads.conv_relu_gap(dtype=dtype, pool=pool, p=p, **shape)
    rep, m, *_ = run_parity(module, dec)
    assert rep["pass"], describe(rep)
    for impl in (mk.IMPL_SIMPLE,):
        rep, *_ = run_parity(module, dec, impls={i: impl for i in range(m.n)})
        assert rep["pass"], "simple: " + describe(rep)


def _chain_module(kind, dtype):
    """Conv modules whose fused epilogue runs longer chains: two channel
    biases around tanh-GELU and a scale, or a residual add before ReLU."""
    x, w = [2, 32, 20, 20], [40, 32, 3, 3]
    rx, rw, rb = (NORMAL, 0.0, 1.0), (NORMAL, 0.0, 0.02), (UNIFORM, -0.1, 0.1)
    conv = {"kind": "CONV2D", "in": [0, 1], "ip": [1, 1], "fp": []}
    if kind == "gelu_scale_bias2":
        return {"name": f"conv_chain_a_{dtype}", "dtype": dtype,
                "inputs": [x, w, [40], [40]], "recipes": [rx, rw, rb, rb],
                "ops": [conv, {"kind": "BIAS_CHANNEL", "in": [4, 2], "ip": [], "fp": []},
                        {"kind": "GELU_TANH", "in": [5], "ip": [], "fp": []},
                        {"kind": "SCALE", "in": [6], "ip": [], "fp": [0.5]},
                        {"kind": "BIAS_CHANNEL", "in": [7, 3], "ip": [], "fp": []},
                        {"kind": "GAP", "in": [8], "ip": [], "fp": []}]}
    return {"name": f"conv_chain_b_{dtype}", "dtype": dtype,
            "inputs": [x, w, [40], [2, 40, 20, 20]], "recipes": [rx, rw, rb, rx],
            "ops": [conv, {"kind": "BIAS_CHANNEL", "in": [4, 2], "ip": [], "fp": []},
                    {"kind": "ADD", "in": [5, 3], "ip": [], "fp": []},
                    {"kind": "RELU", "in": [6], "ip": [], "fp": []},
                    {"kind": "GMP", "in": [7], "ip": [], "fp": []}]}


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kind", ["gelu_scale_bias2", "residual_gmp"])
@pytest.mark.parametrize("dec", ["fused", "split"])
def test_conv_chain_variants(kind, dec, dtype):
    """Every chain step the conv epilogue supports, ahead of the pool (400
    positions per image: column blocks of 32 straddle image boundaries)."""
    print(f"conv chain {kind} {dec} {dtype}", flush=True)
    module = _chain_module(kind, dtype)
    rep, m, *_ = run_parity(module, dec)
    assert m.subkernels()[0]["uses_mfma"]
    if dec == "fused":
        assert len(m.subkernels()) == 1
    assert rep["pass"], describe(rep)
