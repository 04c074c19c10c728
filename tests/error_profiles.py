"""Error profiles of this library's kernels (App. D, Tables "error profiles",
"input dependence" and "dimension scaling"), measured on the GPU against the
oracle.

The paper compares GPU kernels with an fp32 CPU reference over 30 runs of
random inputs and reports the largest and the mean absolute error per run.
Here the reference is the oracle evaluated in fp64 on the unrounded fp32
inputs (module dtype f32, so nothing is rounded to bf16 anywhere in it); the
GPU runs the same module in fp32, or in bf16 on the same inputs rounded to
bf16 (the generator's round to nearest even).  A bf16 error therefore
contains the rounding of the inputs, of the output and the kernel's own
arithmetic, as in the paper's BF16 columns.

  * profiles: matmul 512 x 512 x 512, softmax 128 x 1024, LayerNorm 128 x
    1024 (gamma 1, beta 0, eps 1e-5) and a 3x3 conv (8 x 64 x 32 x 32 -> 64
    channels, stride 1, pad 1, weights as a framework layer initialises
    them); N(0, 1) inputs.  The paper names no LayerNorm or conv shape;
    CrossEntropy has no subkernel here and is left out.
  * input dependence: matmul 1024^3 with both operands from N(0, 0.01^2),
    N(0, 1), N(0, 10^2), U(0, 1), U(-100, 100), and "sparse": N(0, 1) with
    95% of the entries set to zero (a second seeded uniform stream picks the
    5% kept; the paper does not define its sparse inputs).
  * dimension scaling: square matmul N = 64 .. 4096, N(0, 1); for N >= 2048
    the oracle evaluates the first 256 rows of each run (the mean over them
    estimates the mean; their maximum is a lower bound of the full maximum).

Run on a GPU machine:  python tests/error_profiles.py --out <dir>
(writes error_profiles.json and error_profiles.md).
"""
import argparse
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))

import oracle  # noqa: E402
from paper_2607_20501_amd import inputs, mk  # noqa: E402

NORMAL, UNIFORM = inputs.NORMAL, inputs.UNIFORM


def op(kind, ins, ip=(), fp=()):
    return {"kind": kind, "in": list(ins), "ip": list(ip), "fp": list(fp)}


def matmul(M, N, K, recipe=(NORMAL, 0.0, 1.0)):
    return {"name": f"matmul_{M}x{N}x{K}", "dtype": "f32", "inputs": [[M, K], [N, K]],
            "recipes": [recipe, recipe], "ops": [op("GEMM", [0, 1], [0])]}


def softmax(R, C):
    return {"name": f"softmax_{R}x{C}", "dtype": "f32", "inputs": [[R, C]],
            "recipes": [(NORMAL, 0.0, 1.0)], "ops": [op("SOFTMAX", [0])]}


def layernorm(R, C):
    return {"name": f"layernorm_{R}x{C}", "dtype": "f32", "inputs": [[R, C], [C], [C]],
            "recipes": [(NORMAL, 0.0, 1.0), (UNIFORM, 1.0, 1.0), (UNIFORM, 0.0, 0.0)],
            "ops": [op("LAYERNORM", [0, 1, 2], fp=[1e-5])]}


def conv2d(N, C, H, W, K):
    """N(0, 1) input; weights uniform within +-1/sqrt(fan in), the default
    initialisation of a framework conv layer (the paper calls its inputs
    N(0, 1) and says nothing of the conv's weights)."""
    bound = 1.0 / (C * 9) ** 0.5
    return {"name": f"conv2d_{N}x{C}x{H}x{W}_k{K}", "dtype": "f32",
            "inputs": [[N, C, H, W], [K, C, 3, 3]],
            "recipes": [(NORMAL, 0.0, 1.0), (UNIFORM, -bound, bound)],
            "ops": [op("CONV2D", [0, 1], [1, 1])]}


def with_dtype(module, dtype):
    m = dict(module)
    m["dtype"] = dtype
    m["name"] = module["name"] + "_" + dtype
    return m


def gen_inputs(module, seed, sparse=0.0):
    """(fp32 arrays, bf16 bit arrays) of the module's inputs under `seed`; with
    sparse > 0 all but that fraction of every input is zeroed (in both)."""
    f32, b16 = [], []
    for tid, (shape, (dist, p0, p1)) in enumerate(zip(module["inputs"], module["recipes"])):
        n = int(np.prod(shape))
        a = inputs.fill(seed, tid, dist, p0, p1, "f32", n)
        b = inputs.fill(seed, tid, dist, p0, p1, "bf16", n)
        if sparse > 0:
            keep = inputs.fill(seed, 100 + tid, UNIFORM, 0.0, 1.0, "f32", n) < sparse
            a = np.where(keep, a, np.float32(0))
            b = np.where(keep, b, np.uint16(0))
        f32.append(a)
        b16.append(b)
    return f32, b16


class GpuModule:
    def __init__(self, module):
        import torch
        self.torch = torch
        self.module = module
        self.m = mk.Module(module, "fused")
        self.ws = torch.empty(max(1, self.m.workspace_size()), dtype=torch.uint8, device="cuda")
        self.out = mk.out_tensor(module, self.m.info["out_shape"])

    def run(self, host):
        ins, _, _ = mk.device_buffers(self.module, host, 1)
        self.m.run(ins, self.out, self.ws)
        self.torch.cuda.synchronize()
        return mk.to_float64(self.out)


def reference(module32, host32, rows=None):
    """The oracle on fp32 inputs (all of them, or the first `rows` rows of the
    first input when it is row-independent)."""
    groups = [0] * len(module32["ops"])
    if rows is not None:
        sub = json.loads(json.dumps(module32))
        sub["inputs"][0][0] = rows
        k = int(np.prod(module32["inputs"][0][1:]))
        host32 = [host32[0][:rows * k]] + list(host32[1:])
        module32 = sub
    return oracle.run(module32, groups, host32, keep={len(module32["ops"]) - 1})[-1]


def profile(module32, runs, seed0, sparse=0.0, rows=None, dtypes=("f32", "bf16")):
    """Per dtype: lists of (max abs, mean abs) over `runs` seeds."""
    gpu = {dt: GpuModule(with_dtype(module32, dt)) for dt in dtypes}
    res = {dt: {"max": [], "mean": []} for dt in dtypes}
    for r in range(runs):
        f32, b16 = gen_inputs(module32, seed0 + r, sparse)
        ref = reference(module32, f32, rows)
        for dt in dtypes:
            got = gpu[dt].run(f32 if dt == "f32" else b16)
            if rows is not None:
                got = got.reshape(module32["inputs"][0][0], -1)[:rows]
            err = np.abs(got.reshape(-1) - ref.reshape(-1))
            res[dt]["max"].append(float(err.max()))
            res[dt]["mean"].append(float(err.mean()))
    return res


DISTS = [("N(0, 0.01^2)", (NORMAL, 0.0, 0.01), 0.0), ("N(0, 1)", (NORMAL, 0.0, 1.0), 0.0),
         ("N(0, 10^2)", (NORMAL, 0.0, 10.0), 0.0), ("U(0, 1)", (UNIFORM, 0.0, 1.0), 0.0),
         ("U(-100, 100)", (UNIFORM, -100.0, 100.0), 0.0),
         ("sparse 5% (N(0, 1))", (NORMAL, 0.0, 1.0), 0.05)]
DIMS = [64, 128, 256, 512, 1024, 2048, 4096]


def run_all(runs=30, seed0=20000, log=print, dims=DIMS, quick=False):
    out = {"runs": runs, "profiles": {}, "input_dependence": {}, "dimension_scaling": {}}
    t = time.time()
    cases = [("Matmul 512^2", matmul(512, 512, 512)), ("Softmax 128x1024", softmax(128, 1024)),
             ("LayerNorm 128x1024", layernorm(128, 1024)),
             ("Conv2d 8x64x32x32 -> 64, 3x3", conv2d(8, 64, 32, 32, 64))]
    for name, mod in cases:
        out["profiles"][name] = profile(mod, runs, seed0)
        log(f"{name}: {time.time() - t:.1f} s")
    n = 256 if quick else 1024
    for name, recipe, sparse in DISTS:
        out["input_dependence"][name] = profile(matmul(n, n, n, recipe), runs, seed0, sparse)
        log(f"matmul {n}^3 {name}: {time.time() - t:.1f} s")
    out["input_dependence_n"] = n
    for d in dims:
        rows = 256 if d >= 2048 else None
        out["dimension_scaling"][str(d)] = profile(matmul(d, d, d), runs, seed0, rows=rows)
        out["dimension_scaling"][str(d)]["rows_sampled"] = rows
        log(f"matmul {d}^3: {time.time() - t:.1f} s")
    return out


def rng(v):
    lo, hi = min(v), max(v)
    return f"{lo:.2g}" if lo == hi else f"{lo:.2g} - {hi:.2g}"


def to_markdown(res):
    L = [f"{res['runs']} runs per row; errors are |GPU - oracle| (oracle: fp64 on the fp32 "
         "inputs); ranges are min - max over the runs of the per-run value.", "",
         "### Error profiles (App. D, Table 'error profiles')", "",
         "| operation | fp32 max abs | fp32 mean abs | bf16 max abs | bf16 mean abs |",
         "|---|---|---|---|---|"]
    for name, r in res["profiles"].items():
        L.append(f"| {name} | {rng(r['f32']['max'])} | {np.mean(r['f32']['mean']):.2g} | "
                 f"{rng(r['bf16']['max'])} | {np.mean(r['bf16']['mean']):.2g} |")
    n = res["input_dependence_n"]
    L += ["", f"### Input dependence, matmul {n}^3 (App. D, Table 'input dependence')", "",
          "| inputs | fp32 max abs | bf16 max abs |", "|---|---|---|"]
    for name, r in res["input_dependence"].items():
        L.append(f"| {name} | {rng(r['f32']['max'])} | {rng(r['bf16']['max'])} |")
    L += ["", "### Dimension scaling, matmul N^3, N(0, 1) (App. D, Table 'dimension scaling')",
          "", "| N | fp32 avg max abs | fp32 avg mean abs | bf16 avg max abs | bf16 avg mean abs |"
          " rows compared |", "|---|---|---|---|---|---|"]
    for d, r in res["dimension_scaling"].items():
        rows = r.get("rows_sampled") or "all"
        L.append(f"| {d} | {np.mean(r['f32']['max']):.2g} | {np.mean(r['f32']['mean']):.2g} | "
                 f"{np.mean(r['bf16']['max']):.2g} | {np.mean(r['bf16']['mean']):.2g} | {rows} |")
    return "\n".join(L)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--out", required=True)
    ap.add_argument("--runs", type=int, default=30)
    args = ap.parse_args()
    res = run_all(args.runs, log=lambda *a: print(*a, flush=True))
    os.makedirs(args.out, exist_ok=True)
    with open(os.path.join(args.out, "error_profiles.json"), "w") as f:
        json.dump(res, f, indent=1)
    with open(os.path.join(args.out, "error_profiles.md"), "w") as f:
        f.write(to_markdown(res) + "\n")
    print(to_markdown(res))


if __name__ == "__main__":
    main()
