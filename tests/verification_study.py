"""Decomposed vs end-to-end verification of composed modules (App. D),
reproduced with this library's kernels on the GPU against the oracle.

For each block -- MinGPT causal attention (QKV projection, scaled q.k^T,
causal mask, softmax, PV, output projection) and the Transformer FFN block
(LayerNorm, Linear, GELU, Linear, residual) -- and each dtype:

  * calibration: the correct module (split form, every op materialised) on
    `n_cal` seeds; for every stage the max absolute error against the oracle
    (rtol = 0), and the stage tolerance max + 3 sigma over those runs;
  * evaluation: on `n_eval` other seeds, the correct module and the module
    with each injected bug swapped into its subkernel; the decomposed check
    catches a run if any stage exceeds its tolerance, the end-to-end (E2E)
    check if the output exceeds a fixed atol;
  * feasibility gap of a bug at a stage: min over buggy runs of the error
    minus max over correct runs (E2E: at the output; decomposed: the best
    stage).  A positive gap means some tolerance separates the two.

Run on a GPU machine:  python tests/verification_study.py --out <dir>
(writes verification_study.json and verification_study.md).  The oracle
gives the reference of every stage; its rounding model (round to the module
dtype where a stage is stored) is the same for correct and buggy runs.
"""
import argparse
import json
import math
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))

import oracle  # noqa: E402
from paper_2607_20501_amd import inputs, mk, workloads  # noqa: E402

E2E_ATOLS = [1e-5, 1e-3, 1e-2, 1e-1]

# name, mutant id, op index that carries the bug
ATTN_BUGS = [("Unsafe softmax", 101, 3), ("Mask off-by-one", 102, 2),
             ("Tile boundary (K)", 103, 1), ("Wrong acc dtype (QK)", 104, 1),
             ("Softmax dim=-2", 105, 3)]
FFN_BUGS = [("Unsafe LayerNorm", 106, 0), ("GELU sigmoid approx", 107, 2),
            ("Tile boundary (fc1)", 103, 1), ("Wrong acc dtype (fc2)", 104, 3),
            ("Missing residual", 108, 3), ("ReLU not GELU", 109, 2)]


# The unsafe softmax only fails where exp overflows (scores above ~88.7 in
# fp32), which N(0, 1) tokens never reach; a third block scales the tokens so
# that the largest scores exceed it (scores grow as x_std^2: with these
# weights the largest score of a run is about 0.4 x_std^2 at D 256 and 1.7
# x_std^2 at D 768).
LARGE_BUGS = [("Unsafe softmax", 101, 3)]


def blocks(dtype, small):
    if small:
        attn = workloads.causal_attention_block(B=1, S=128, D=256, H=2, dtype=dtype)
        large = workloads.causal_attention_block(B=1, S=128, D=256, H=2, dtype=dtype,
                                                 x_std=20.0)
        ffn = workloads.mlp_block(M=128, D=256, F=512, dtype=dtype)
    else:
        attn = workloads.causal_attention_block(B=2, S=512, D=768, H=8, dtype=dtype)
        large = workloads.causal_attention_block(B=2, S=512, D=768, H=8, dtype=dtype,
                                                 x_std=10.0)
        ffn = workloads.mlp_block(M=1024, D=768, F=3072, dtype=dtype)
    return [("attention", attn, ATTN_BUGS), ("ffn", ffn, FFN_BUGS),
            ("attention_large_scores", large, LARGE_BUGS)]


class Runner:
    """One module in split form with a Module handle per implementation."""

    def __init__(self, module, bugs):
        import torch
        self.torch = torch
        self.module = module
        self.groups = mk.mk_decomposition_preset(module, "split")
        n = len(module["ops"])
        self.stage_ops = [i for i in range(n) if i == n - 1 or self.groups[i + 1] != self.groups[i]]
        self.handles = {"correct": mk.Module(module, self.groups)}
        for name, impl, op in bugs:
            h = mk.Module(module, self.groups)
            h.select(self.groups[op], impl)
            self.handles[name] = h
        ws = max(h.workspace_size() for h in self.handles.values())
        self.ws = torch.empty(max(1, ws), dtype=torch.uint8, device="cuda")
        self.out = mk.out_tensor(module, self.handles["correct"].info["out_shape"])

    def errors(self, seed):
        """{variant: [max abs error of each stage]} for one seed (inf for a
        stage with non-finite values)."""
        host = inputs.make_inputs(self.module, seed)
        ref = oracle.run(self.module, self.groups, host, keep=set(self.stage_ops))
        ins, _, _ = mk.device_buffers(self.module, host, 1)
        checks = [{"stage": s, "expect": ref[op].reshape(-1), "rtol": 0.0, "atol": 0.0}
                  for s, op in enumerate(self.stage_ops)]
        res = {}
        for name, h in self.handles.items():
            rep = h.verify(ins, self.out, self.ws, checks)
            errs = []
            for r in sorted(rep["results"], key=lambda r: r["stage"]):
                errs.append(math.inf if r["n_nonfinite"] else float(r["max_abs_err"]))
            res[name] = errs
        self.torch.cuda.synchronize()
        return res


def study_block(module, bugs, n_cal, n_eval, seed0):
    run = Runner(module, bugs)
    cal = [run.errors(seed0 + i)["correct"] for i in range(n_cal)]
    cal = np.array(cal)                                   # [n_cal, stages]
    tol = cal.max(axis=0) + 3 * cal.std(axis=0)
    ev = [run.errors(seed0 + 1000 + i) for i in range(n_eval)]
    names = ["correct"] + [b[0] for b in bugs]
    err = {n: np.array([e[n] for e in ev]) for n in names}   # [n_eval, stages]
    out = {"module": module["name"], "stages": [module["ops"][i]["kind"] for i in run.stage_ops],
           "tolerance": tol.tolist(), "calibration_max": cal.max(axis=0).tolist(),
           "variants": {}}
    corr = err["correct"]
    for n in names:
        e = err[n]
        dec = int((e > tol).any(axis=1).sum())
        e2e = {str(a): int((e[:, -1] > a).sum()) for a in E2E_ATOLS}
        v = {"decomposed_caught": dec, "e2e_caught": e2e,
             "output_err_min": float(e[:, -1].min()), "output_err_max": float(e[:, -1].max())}
        if n != "correct":
            gaps = e.min(axis=0) - corr.max(axis=0)
            v["gap_e2e"] = float(gaps[-1])
            v["gap_dec"] = float(gaps.max())
            v["gap_dec_stage"] = int(gaps.argmax())
        out["variants"][n] = v
    return out


def best_usable(block, dtype):
    """Smallest fixed E2E atol that rejects no correct run (fp32: 1e-5 first)."""
    cands = E2E_ATOLS if dtype == "f32" else E2E_ATOLS[1:]
    for a in cands:
        if block["variants"]["correct"]["e2e_caught"][str(a)] == 0:
            return a
    return cands[-1]


def to_markdown(res):
    n = res["n_eval"]
    lines = [f"Calibration {res['n_cal']} runs, evaluation {n} runs per variant; "
             f"tolerances max + 3 sigma, rtol 0.  Sizes: {res['sizes']}.", ""]
    for blk in ("attention", "ffn", "attention_large_scores"):
        for dt in ("f32", "bf16"):
            b = res["blocks"][f"{blk}_{dt}"]
            lines.append(f"### {b['module']}")
            lines.append("")
            lines.append("| stage | " + " | ".join(b["stages"]) + " |")
            lines.append("|---|" + "---|" * len(b["stages"]))
            lines.append("| tolerance | " + " | ".join(f"{t:.3g}" for t in b["tolerance"]) + " |")
            lines.append("")
            a_best = best_usable(b, dt)
            hdr = "| variant | " + " | ".join(f"E2E atol={a:g}" for a in E2E_ATOLS) + \
                  f" | E2E best ({a_best:g}) | decomposed | gap E2E | gap dec (stage) |"
            lines.append(hdr)
            lines.append("|---" * (len(E2E_ATOLS) + 5) + "|")
            for name, v in b["variants"].items():
                cells = [f"{v['e2e_caught'][str(a)]}/{n}" for a in E2E_ATOLS]
                cells.append(f"{v['e2e_caught'][str(a_best)]}/{n}")
                cells.append(f"{v['decomposed_caught']}/{n}")
                if name == "correct":
                    cells += ["", ""]
                else:
                    cells.append(f"{v['gap_e2e']:.3g}")
                    cells.append(f"{v['gap_dec']:.3g} ({b['stages'][v['gap_dec_stage']]})")
                lines.append(f"| {name} | " + " | ".join(cells) + " |")
            lines.append("")
    return "\n".join(lines)


def run_study(n_cal=20, n_eval=20, small=False, seed0=10000, log=print):
    res = {"n_cal": n_cal, "n_eval": n_eval, "blocks": {},
           "sizes": "small" if small else "attention B2 S512 D768 H8; FFN M1024 D768 F3072"}
    for dt in ("f32", "bf16"):
        for name, module, bugs in blocks(dt, small):
            t = time.time()
            res["blocks"][f"{name}_{dt}"] = study_block(module, bugs, n_cal, n_eval, seed0)
            log(f"{name} {dt}: {time.time() - t:.1f} s")
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--out", required=True)
    ap.add_argument("--n-cal", type=int, default=20)
    ap.add_argument("--n-eval", type=int, default=20)
    ap.add_argument("--small", action="store_true")
    args = ap.parse_args()
    res = run_study(args.n_cal, args.n_eval, args.small, log=lambda *a: print(*a, flush=True))
    os.makedirs(args.out, exist_ok=True)
    with open(os.path.join(args.out, "verification_study.json"), "w") as f:
        json.dump(res, f, indent=1)
    with open(os.path.join(args.out, "verification_study.md"), "w") as f:
        f.write(to_markdown(res) + "\n")
    print(to_markdown(res))


if __name__ == "__main__":
    main()
