"""GPU parity of the conv family: implicit-GEMM MFMA path (bf16 and fp32;
padded-NHWC gather, NCHW store or fused GAP over tiles that straddle images)
and the simple direct conv, against the oracle."""
import pytest
import torch

from helpers import describe, run_parity
from paper_2607_20501_amd import mk, workloads

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

CASES = [dict(N=3, C=32, H=20, W=20, K=40), dict(N=2, C=64, H=16, W=16, K=300),
         dict(N=2, C=32, H=31, W=31, K=64, stride=2), dict(N=1, C=96, H=24, W=24, K=256),
         dict(N=2, C=8, H=9, W=7, K=5)]


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
    assert m.subkernels()[0]["n_launches"] == 4


POOL_CASES = [dict(N=3, C=32, H=20, W=20, K=40), dict(N=2, C=64, H=16, W=16, K=300),
              dict(N=2, C=8, H=9, W=7, K=5)]


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
