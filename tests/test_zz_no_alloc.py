"""mk_run_noalloc (the entry point for callers that cannot allocate device
memory) against mk_run with a caller workspace: the same module and seeded
inputs must give the same output bytes, and both must match the oracle.  Two
calls in a row share the library's static workspace, the second on a smaller
module, so a kernel that read bytes the first call left behind would show."""
import numpy as np
import pytest

import oracle
from helpers import TOL
from paper_2607_20501_amd import inputs, mk, workloads

PAIRS = {
    # [K,N] weight transposed into scratch, softmax over rows
    "gemm_gelu_softmax": (workloads.gemm_gelu_softmax(M=520, K=512, N=1024),
                          workloads.gemm_gelu_softmax(M=200, K=256, N=640)),
    # NHWC / KRSC packs and per-tile pool partials in scratch
    "conv_relu_gap": (workloads.conv_relu_gap(N=4, C=64, H=20, W=20, K=128),
                      workloads.conv_relu_gap(N=2, C=64, H=12, W=12, K=64)),
    # LayerNorm prologue of the first GEMM in scratch
    "mlp_block": (workloads.mlp_block(M=520, D=512, F=1024),
                  workloads.mlp_block(M=130, D=256, F=512)),
    # every intermediate of the split layer in the workspace
    "transformer_layer": (workloads.transformer_layer(B=2, S=256, D=256, H=2, F=512),
                          workloads.transformer_layer(B=1, S=200, D=256, H=2, F=512)),
}
PRESET = {"gemm_gelu_softmax": "fused", "conv_relu_gap": "fused", "mlp_block": "fused",
          "transformer_layer": "split"}


def _oracle_out(module, groups, host):
    return oracle.run(module, groups, host, keep={len(module["ops"]) - 1})[-1]


def test_rejects_a_workspace_beyond_the_static_array():
    """Host-side size check: a module whose workspace exceeds the static array
    is refused before any device work (full-size MLP block: 128 MiB and more)."""
    module = workloads.mlp_block()
    m = mk.Module(module, "fused")
    assert m.workspace_size() > mk.NOALLOC_WS_BYTES
    with pytest.raises(mk.MkError) as e:
        mk.mk_run_noalloc(m.h, [0] * len(module["inputs"]), 0, 0)
    assert e.value.status == mk.STATUS.index("MK_E_WORKSPACE")


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(PAIRS))
def test_noalloc_matches_mk_run_on_two_calls(name):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    outs = []
    for module in PAIRS[name]:
        groups = mk.mk_decomposition_preset(module, PRESET[name])
        m = mk.Module(module, groups)
        assert 0 < m.workspace_size() <= mk.NOALLOC_WS_BYTES
        host = inputs.make_inputs(module, 3)
        ins, _, ws = mk.device_buffers(module, host, m.workspace_size())
        out_na = mk.out_tensor(module, m.info["out_shape"])
        m.run_noalloc(ins, out_na)
        outs.append((module, groups, host, m, ins, ws, out_na))
    torch.cuda.synchronize()
    # the reference runs come after both static-workspace calls
    for module, groups, host, m, ins, ws, out_na in outs:
        out_ref = mk.out_tensor(module, m.info["out_shape"])
        m.run(ins, out_ref, ws)
        torch.cuda.synchronize()
        a, b = mk.to_float64(out_na), mk.to_float64(out_ref)
        assert np.isfinite(a).all(), module["name"]
        assert np.array_equal(a, b), f"{module['name']}: max diff {np.abs(a - b).max()}"
        ref = _oracle_out(module, groups, host)
        rtol, atol = TOL[module["dtype"]]
        err = np.abs(a - ref)
        assert (err <= atol + rtol * np.abs(ref)).all(), f"{module['name']}: {err.max()}"
