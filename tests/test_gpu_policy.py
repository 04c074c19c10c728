"""The swap policy on the GPU (Sec. 3 "Swap"): mk_swap times every subkernel
with its selected and its reference implementation, applies the rule of
mk_swap_decide to those times, and leaves a module that still matches the
oracle."""
import pytest
import torch

from helpers import describe, run_parity
from paper_2607_20501_amd import inputs, mk, workloads

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


@pytest.mark.parametrize("make,dec", [(workloads.linear_relu_rowsum, "split"),
                                      (lambda: workloads.gemm_gelu_softmax(M=512, K=512, N=1024),
                                       "split")])
@pytest.mark.parametrize("tau", [0.9, 1e9])
def test_swap_applies_its_rule(make, dec, tau):
    module = make()
    print(f"swap {module['name']} {dec} tau={tau}", flush=True)
    m = mk.Module(module, dec)
    host = inputs.make_inputs(module, 0)
    ins, _, ws = mk.device_buffers(module, host, m.workspace_size())
    out = mk.out_tensor(module, m.info["out_shape"])
    r = m.swap(ins, out, ws, reference_impl=mk.IMPL_SIMPLE, tau=tau, n_runs=3)
    assert all(t > 0 for t in r["ms_selected"]) and all(t > 0 for t in r["ms_reference"])
    sw, trig = mk.mk_swap_decide(r["ms_selected"], r["ms_reference"], tau)
    assert (sw, trig) == (r["swapped"], r["triggered"])
    impls = [s["impl"] for s in m.subkernels()]
    assert impls == [mk.IMPL_SIMPLE if x else mk.IMPL_TUNED for x in sw]
    if tau > 1e8 and trig:
        assert all(sw)                       # every subkernel is below an enormous tau
    # the swapped composition is still correct
    rep, *_ = run_parity(module, m.groups, impls={i: v for i, v in enumerate(impls)})
    assert rep["pass"], describe(rep)
    shares = mk.mk_budget_shares(r["ms_selected"])
    assert sum(shares) == pytest.approx(1.0, abs=1e-5)


def test_launch_profile_every_launch_and_one_launch():
    """mk_profile_begin / end: every launch of every run in launch order, the
    max_launches cap, and one launch per run (the rest back to back)."""
    module = workloads.gemm_gelu_softmax(M=1024, K=512, N=1024)
    print(f"profile {module['name']}", flush=True)
    m = mk.Module(module, "fused", strict=True)
    host = inputs.make_inputs(module, 0)
    ins, _, ws = mk.device_buffers(module, host, m.workspace_size())
    out = mk.out_tensor(module, m.info["out_shape"])
    per_run = m.launches_per_run()
    assert per_run == 3                      # weight transpose, GEMM, softmax rows
    runs = 6
    m.run(ins, out, ws)
    m.profile_begin(per_run * runs)
    for _ in range(runs):
        m.run(ins, out, ws)
    every = m.profile_end(per_run * runs)
    assert len(every) == per_run * runs and all(t > 0 for t in every)
    m.profile_begin(4)                       # cap: later launches are not recorded
    for _ in range(2):
        m.run(ins, out, ws)
    assert len(m.profile_end(16)) == 4
    for k in range(per_run):
        m.profile_begin(runs, only_launch=k)
        for _ in range(runs):
            m.run(ins, out, ws)
        one = m.profile_end(runs)
        assert len(one) == runs and all(t > 0 for t in one)
        mean_every = sum(every[k::per_run]) / runs
        assert 0.2 < (sum(one) / runs) / mean_every < 5, (k, one, every[k::per_run])
    with pytest.raises(mk.MkError):
        m.profile_begin(4, only_launch=per_run)
