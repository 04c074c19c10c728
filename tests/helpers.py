"""Shared helpers of the GPU parity tests: run a module through the C ABI and
compare every materialised stage with the oracle on the same seeded bytes."""
import numpy as np

import oracle
from paper_2607_20501_amd import inputs, mk

TOL = {"f32": (1e-4, 1e-5), "bf16": (2e-2, 2e-2)}


def stage_ops(module, groups):
    """Index of the last op of each group (its output is the stage)."""
    n = len(groups)
    return [i for i in range(n) if i == n - 1 or groups[i + 1] != groups[i]]


def softmax_stage(module, op_index):
    k = module["ops"][op_index]["kind"]
    return k == "SOFTMAX"


def run_parity(module, groups, seed=0, impls=None, host=None, strict_softmax=True,
               extra_checks=None):
    """Returns (report, module handle, device output, oracle stage values)."""
    import torch
    if isinstance(groups, str):
        groups = mk.mk_decomposition_preset(module, groups)
    host = host if host is not None else inputs.make_inputs(module, seed)
    stages = stage_ops(module, groups)
    ref = oracle.run(module, groups, host, keep=set(stages))
    m = mk.Module(module, groups)
    for i, impl in (impls or {}).items():
        m.select(i, impl)
    ins, _, ws = mk.device_buffers(module, host, m.workspace_size())
    out = mk.out_tensor(module, m.info["out_shape"])
    rtol, atol = TOL[module["dtype"]]
    checks = []
    for s, op in enumerate(stages):
        e = ref[op].reshape(-1)
        checks.append({"stage": s, "expect": e, "rtol": rtol, "atol": atol})
        if strict_softmax and softmax_stage(module, op) and module["dtype"] == "bf16":
            # atol 2e-2 is vacuous for probabilities ~1/N; also check against
            # atol scaled by the row length.
            n_row = ref[op].shape[-1]
            checks.append({"stage": s, "expect": e, "rtol": rtol, "atol": atol / n_row})
    checks += extra_checks or []
    rep = m.verify(ins, out, ws, checks)
    torch.cuda.synchronize()
    return rep, m, out, ref, stages


def describe(rep):
    lines = []
    for r in rep["results"]:
        lines.append(f"stage {r['stage']}: pass={r['pass']} viol={r['n_violations']}/"
                     f"{r['n_checked']} nonfinite={r['n_nonfinite']} max_abs={r['max_abs_err']:.3g}"
                     f" worst_ratio={r['worst_ratio']:.3g} at {r['worst_index']} "
                     f"got={r['got_at_worst']:.6g} expect={r['expect_at_worst']:.6g}")
    return "\n".join(lines)
