"""Parity at the full workload sizes, in the launch configuration the
benchmark times: tuned subkernels, fused and split presets, the whole module
run once through the C ABI on inputs resident in HBM.

The oracle cannot evaluate these modules whole in seconds, but each of them is
independent per row (GEMM + GELU + softmax, MLP block), per image (conv +
ReLU + GAP) or per sequence (transformer layer), and causal attention makes a
prefix of a sequence depend on nothing after it.  So the oracle evaluates the
same module and grouping on sampled rows (first, last, both sides of the
256-row tile boundaries, about a thousand seeded random rows), on sampled
images (including images whose positions straddle a GEMM column tile), and on
the whole first and last sequences, and those outputs are compared element by
element with the full-size GPU output.  Each fused module is also run twice
into NaN-filled buffers and the two outputs compared bit for bit.  Properties that hold at any size (finite
values, softmax rows summing to 1, pooled ReLU outputs >= 0) are checked on the
whole output."""
import copy

import numpy as np
import pytest
import torch

import oracle
from paper_2607_20501_amd import inputs, mk, workloads

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

TOL = {"f32": (1e-4, 1e-5), "bf16": (2e-2, 2e-2)}
_HOST = {}


def host_inputs(cfg, module):
    if cfg not in _HOST:
        _HOST.clear()          # keep one workload's host inputs at a time
        _HOST[cfg] = inputs.make_inputs(module, 0)
    return _HOST[cfg]


def run_full(module, host, decomp):
    """Run the whole module on the GPU; returns the output tensor (device)."""
    m = mk.Module(module, decomp)
    ins, _, ws = mk.device_buffers(module, host, m.workspace_size())
    out = mk.out_tensor(module, m.info["out_shape"])
    m.run(ins, out, ws)
    torch.cuda.synchronize()
    del ins, ws
    return out, mk.mk_decomposition_preset(module, decomp)


def compare(got, ref, dtype, atol=None):
    rtol, a = TOL[dtype]
    atol = a if atol is None else atol
    err = np.abs(got - ref)
    bad = ~(err <= atol + rtol * np.abs(ref))
    ratio = err / (atol + rtol * np.abs(ref))
    k = int(np.argmax(ratio))
    msg = (f"{int(bad.sum())} of {ref.size} outside tolerance; worst ratio "
           f"{ratio.reshape(-1)[k]:.3g} at flat {k}: got {got.reshape(-1)[k]:.6g} "
           f"expect {ref.reshape(-1)[k]:.6g}")
    return not bad.any(), msg


def sampled_rows(M, n_random, seed=1234):
    fixed = [0, 1, 255, 256, M // 2 - 1, M // 2, M - 2, M - 1]
    rng = np.random.default_rng(seed)
    extra = rng.choice(M, size=n_random, replace=False).tolist()
    return sorted(set(fixed + extra))


def row_oracle(module, groups, host, rows):
    """Oracle on the given rows of input 0 (row-independent modules)."""
    sub = copy.deepcopy(module)
    M, K = module["inputs"][0]
    sub["inputs"][0] = [len(rows), K]
    x = np.asarray(host[0]).reshape(M, K)[rows].reshape(-1)
    return oracle.run(sub, groups, [x] + list(host[1:]),
                      keep={len(module["ops"]) - 1})[-1]


@pytest.mark.parametrize("decomp", ["fused", "split"])
def test_gemm_gelu_softmax_full_size(decomp):
    module = workloads.full_size(2)
    print(f"full-size {module['name']} {decomp}", flush=True)
    host = host_inputs(2, module)
    out, groups = run_full(module, host, decomp)
    M, N = out.shape
    # properties over the whole output
    o32 = out.float()
    assert torch.isfinite(o32).all()
    sums = o32.sum(dim=1)
    assert (sums - 1).abs().max().item() < 1e-2, "softmax rows must sum to 1"
    assert o32.min().item() >= 0
    rows = sampled_rows(M, 1024)
    ref = row_oracle(module, groups, host, rows)
    got = mk.to_float64(out[rows])
    ok, msg = compare(got, ref, "bf16")
    assert ok, msg
    # probabilities are ~1/N: the official atol is vacuous, so also check
    # with atol scaled by the row length
    ok, msg = compare(got, ref, "bf16", atol=2e-2 / N)
    assert ok, "strict softmax check: " + msg


@pytest.mark.parametrize("decomp", ["fused", "split"])
def test_mlp_block_full_size(decomp):
    module = workloads.full_size(4)
    print(f"full-size {module['name']} {decomp}", flush=True)
    host = host_inputs(4, module)
    out, groups = run_full(module, host, decomp)
    assert torch.isfinite(out.float()).all()
    rows = sampled_rows(out.shape[0], 512)
    ref = row_oracle(module, groups, host, rows)
    ok, msg = compare(mk.to_float64(out[rows]), ref, "bf16")
    assert ok, msg


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("decomp", ["fused", "split"])
def test_conv_relu_gap_full_size(decomp, dtype):
    module = workloads.conv_relu_gap(dtype=dtype)
    print(f"full-size {module['name']} {decomp}", flush=True)
    host = host_inputs((3, dtype), module)
    out, groups = run_full(module, host, decomp)
    o32 = out.float()
    assert torch.isfinite(o32).all() and o32.min().item() >= 0
    N, C, H, W = module["inputs"][0]
    # image 1 starts inside a 128-position column tile (56*56 = 24.5 tiles);
    # on the persistent bf16 kernel (784 tiles of 256) images 7 and N-1 lie
    # in tiles of the last, split round
    imgs = [0, 1, 7, 37, N - 1]
    sub = copy.deepcopy(module)
    sub["inputs"][0] = [len(imgs), C, H, W]
    x = np.asarray(host[0]).reshape(N, -1)[imgs].reshape(-1)
    ref = oracle.run(sub, groups, [x] + list(host[1:]), keep={len(module["ops"]) - 1})[-1]
    ok, msg = compare(mk.to_float64(out[imgs]), ref, dtype)
    assert ok, msg


@pytest.mark.parametrize("decomp", ["fused", "split"])
def test_transformer_layer_full_size(decomp):
    module = workloads.full_size(5)
    print(f"full-size {module['name']} {decomp}", flush=True)
    host = host_inputs(5, module)
    out, groups = run_full(module, host, decomp)
    assert torch.isfinite(out.float()).all()
    B, S, D = module["inputs"][0]
    x = np.asarray(host[0]).reshape(B, S, D)
    # whole sequences (every query position, up to 32 key blocks of the flash
    # kernel, every row of the GEMMs of that sequence): the first and the last
    for b in (0, B - 1):
        sub = copy.deepcopy(module)
        sub["inputs"][0] = [1, S, D]
        for op in sub["ops"]:
            if op["kind"] in ("QK", "PV"):
                op["ip"][0] = 1
        ref = oracle.run(sub, groups, [x[b].reshape(-1)] + list(host[1:]),
                         keep={len(module["ops"]) - 1})[-1]
        got = mk.to_float64(out[b])
        ok, msg = compare(got, ref.reshape(got.shape), "bf16")
        assert ok, f"sequence {b}: {msg}"
        print(f"sequence {b} of {B}: whole {S} tokens match", flush=True)


def poisoned_run(m, ins, out, ws):
    """Output and workspace filled with NaN bytes, one run, synchronised."""
    out.view(torch.uint8).fill_(0xFF)
    ws.fill_(0xFF)
    m.run(ins, out, ws)
    torch.cuda.synchronize()
    return out.clone()


@pytest.mark.parametrize("cfg,dtype", [(2, "bf16"), (3, "bf16"), (3, "f32"), (4, "bf16"),
                                       (5, "bf16")])
def test_full_size_fused_runs_are_bitwise_repeatable(cfg, dtype):
    """Every kernel of the fused full-size modules is deterministic (no
    atomics, fixed reduction orders): two runs into NaN-filled outputs and
    workspaces give the same bits, and every output element is written.  A
    race between the persistent GEMM's prefetch of the next tile and the
    epilogue of the current one, or an unwritten tile, shows here."""
    module = workloads.conv_relu_gap(dtype=dtype) if cfg == 3 else workloads.full_size(cfg)
    print(f"run twice: {module['name']} fused", flush=True)
    host = host_inputs((cfg, dtype), module)
    m = mk.Module(module, "fused")
    ins, _, ws = mk.device_buffers(module, host, m.workspace_size())
    out = mk.out_tensor(module, m.info["out_shape"])
    a = poisoned_run(m, ins, out, ws)
    b = poisoned_run(m, ins, out, ws)
    assert torch.isfinite(a.float()).all()
    ia = a.view(torch.int16 if a.dtype == torch.bfloat16 else torch.int32)
    ib = b.view(torch.int16 if b.dtype == torch.bfloat16 else torch.int32)
    n_diff = int((ia != ib).sum().item())
    assert n_diff == 0, f"{n_diff} of {ia.numel()} elements differ between two runs"
