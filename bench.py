#!/usr/bin/env python3
"""Composed-module benchmark on one MI355X.

A step is one run of the whole composed module (every subkernel of the
chosen decomposition) over one batch of synthetic, seeded input that is
already resident in HBM.  Default workload: the bf16 transformer MLP block
x[16384,4096] -> LayerNorm -> Linear 4096->14336 -> exact GELU -> Linear
14336->4096 -> + x, fused (the largest of the five workloads); --config
selects the others.

Prints ONE JSON line with the throughput of the fused composition (TFLOP/s of
the module's algorithmic flops), the split composition beside it, the
roofline of the dominant kernel (from a HIP event pair around that launch,
recorded over as many runs as the timed steps, the other launches back to
back) and the oracle's CPU throughput on a bounded
sample of independent units -- rows, images or sequences -- which also checks
those units of the GPU output).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6    # 256 CU x 2.4 GHz x 4096 flop/clk/CU, dense
PEAK_F32_TFLOPS = 157.3      # fp32 matrix
PEAK_HBM_GBS = 8000.0

def log(*a):
    print(*a, file=sys.stderr, flush=True)


def build_module(cfg, dtype):
    from paper_2607_20501_amd import workloads
    if cfg == 3:
        return workloads.conv_relu_gap(dtype=dtype or "bf16")
    m = workloads.full_size(cfg)
    if dtype:
        m["dtype"] = dtype
    return m


def launch_names(mod):
    """Name of every kernel launch of one run, in order.  A GEMM subkernel runs
    [layernorm prologue] [transpose of a [K,N] weight] gemm [row finisher]."""
    names = []
    for s in mod.subkernels():
        ops = [o["kind"] for o in mod.desc["ops"][s["op_begin"]:s["op_end"]]]
        n = s["n_launches"]
        if s["family"] == "GEMM":
            ln = ops[0] == "LAYERNORM"
            fin = ops[-1] in ("SOFTMAX", "ROWSUM", "LAYERNORM")
            seq = ["row_kernel (layernorm prologue)"] if ln else []
            if n - len(seq) - (2 if fin else 1) == 1:
                seq.append("transpose_b_kernel")
            seq.append("gemm_mfma_kernel (" + ",".join(ops) + ")")
            if fin:
                # (a softmax over rows one wave holds runs as a row pass over
                # the stored values; otherwise a finisher over partials)
                row_pass = ops[-1] == "SOFTMAX" and s.get("out_shape", [0])[-1] * (
                    2 if mod.desc["dtype"] == "bf16" else 4) <= 8192
                seq.append("row_wave_kernel (softmax)" if row_pass
                           else ops[-1].lower() + "_finish_kernel")
            names += seq
        elif s["family"] == "CONV" and n >= 2:
            names += ["pack_nhwc_kernel (+ weight repack)",
                      "gemm_mfma_kernel (conv: " + ",".join(ops) + ")"]
            names += ["gap_finish_kernel"] * (n - 2)
        elif s["family"] == "ATTN":
            names += ["attn_fwd_pipe_kernel (" + ",".join(ops) + ")"] * n
        else:
            names += [s["family"].lower() + " subkernel (" + ",".join(ops) + ")"] * n
    return names


def source_digest(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


GEMM_SOURCES = ["paper_2607_20501_amd/csrc/k_gemm_mfma.hip", "paper_2607_20501_amd/csrc/dev.hpp",
                "paper_2607_20501_amd/csrc/kernels.hpp", "paper_2607_20501_amd/csrc/plan_codes.hpp"]


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    counter summary, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        table = json.load(fh)
    rec = table.get(workload, {})
    rec = rec.get(kernel) or rec.get(kernel.split(" ")[0])
    if not rec or rec.get("source_digest") != source_digest(GEMM_SOURCES):
        return None
    return rec["hbm_bytes_per_launch"]


def warmup_steps(mod, ins, out, ws, warmup):
    """Run the untimed warm-up: exactly `warmup` steps when given, otherwise
    at least 10 steps and at least 100 ms of them (after an idle period the
    chip needs tens of milliseconds under load to reach its steady clock;
    10 steps of a 250-us module are 2.5 ms).  Returns the count run."""
    import torch
    if warmup is not None:
        for _ in range(warmup):
            mod.run(ins, out, ws)
        torch.cuda.synchronize()
        return warmup
    n, t0 = 0, time.perf_counter()
    while n < 10 or time.perf_counter() - t0 < 0.1:
        for _ in range(10):
            mod.run(ins, out, ws)
        n += 10
        torch.cuda.synchronize()
    return n


def time_module(mod, ins, out, ws, steps, warmup):
    """ms per step over `steps` back-to-back runs (after the untimed warm-up,
    see warmup_steps), bracketed by device synchronisation; then, for each
    launch k of a run, `steps` more runs with a HIP event pair around launch k
    alone (the other launches run back to back, as in the timed steps) for
    per-launch durations.  An event pair adds the launch's dispatch time (a
    few microseconds) to its figure, so the pairs stay out of the timed
    region.  Returns (ms, per-launch ms, warm-up steps run)."""
    import torch
    warmed = warmup_steps(mod, ins, out, ws, warmup)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        mod.run(ins, out, ws)
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    per_launch = []
    for k in range(mod.launches_per_run()):
        mod.profile_begin(steps, only_launch=k)
        for _ in range(steps):
            mod.run(ins, out, ws)
        torch.cuda.synchronize()
        launch_ms = mod.profile_end(steps)
        per_launch.append(sum(launch_ms) / len(launch_ms))
    return ms, per_launch, warmed


def median_flushed(mod, ins, out, ws, runs, flush):
    """Median time (ms) of `runs` individually timed runs, each preceded by a
    write of the `flush` buffer so that no operand is served from L2 or the
    256 MB Infinity Cache."""
    import statistics
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(runs)]
    for i, (a, b) in enumerate(ev):
        flush.fill_(i & 0x7F)
        a.record()
        mod.run(ins, out, ws)
        b.record()
    torch.cuda.synchronize()
    return statistics.median(a.elapsed_time(b) for a, b in ev)


TOL = {"f32": (1e-4, 1e-5), "bf16": (2e-2, 2e-2)}


def sample_module(module, n):
    """The same module over n independent units of its leading dimension
    (rows of a row-wise module, images of the conv module, sequences of the
    transformer layer): the first input's leading size and the batch
    parameter of attention ops become n."""
    sub = json.loads(json.dumps(module))
    sub["inputs"][0][0] = n
    for o in sub["ops"]:
        if o["kind"] in ("QK", "PV"):
            o["ip"][0] = n
    return sub


def cpu_baseline(module, host, units, out_dev, unit_name):
    """The oracle on the units `units` of the leading dimension (each unit is
    independent of the others), timed on the host cores; also compares those
    units of the GPU output element by element at the module dtype's
    tolerance (softmax outputs also against atol / row length)."""
    import numpy as np
    import oracle
    from paper_2607_20501_amd import mk
    n_all = module["inputs"][0][0]
    per = int(np.prod(module["inputs"][0][1:]))
    sub = sample_module(module, len(units))
    sub_host = [np.concatenate([host[0][u * per:(u + 1) * per] for u in units])] + list(host[1:])
    groups = mk.mk_decomposition_preset(module, "fused")
    threads = int(os.environ.get("OMP_NUM_THREADS") or len(os.sched_getaffinity(0)))
    t = time.perf_counter()
    ref = oracle.run(sub, groups, sub_host, keep={len(module["ops"]) - 1}, nthreads=threads)[-1]
    dt = time.perf_counter() - t
    flops = oracle.plan(sub, groups)["flops"]
    import torch
    got = mk.to_float64(out_dev[torch.tensor(units, device=out_dev.device)])
    rtol, atol = TOL[module["dtype"]]
    err = np.abs(got - ref)
    ok = err <= atol + rtol * np.abs(ref)
    if module["ops"][-1]["kind"] == "SOFTMAX":
        ok &= err <= atol / ref.shape[-1] + rtol * np.abs(ref)
    span = (f"units {units[0]}..{units[-1]}" if units == list(range(units[0], units[-1] + 1))
            else "units " + ",".join(map(str, units)))
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(units)} of {n_all} {unit_name} ({span.replace('units', unit_name)})"
                      f" of the same fused module (fp64 oracle, {flops / 1e9:.1f} GFLOP in "
                      f"{dt:.1f} s)",
            "seconds": dt,
            "parity_units_checked": len(units), "parity_max_abs_err": float(err.max()),
            "parity_pass": bool(ok.all())}


def baseline_units(cfg, module, flops, cpu_units):
    """Which units the oracle leg evaluates: about 800 GFLOP of rows (row-wise
    modules), every image (conv, 118 GFLOP), the first and the last sequence
    (transformer, 223 GFLOP each)."""
    n = module["inputs"][0][0]
    if cfg == 3:
        k = cpu_units or n
        return list(range(min(k, n))), "images"
    if cfg == 5:
        k = cpu_units or 2
        return (list(range(k - 1)) + [n - 1]) if k < n else list(range(n)), "sequences"
    k = cpu_units or max(1, min(n, int(800e9 / (flops / n))))
    return list(range(min(k, n))), "rows"


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed warm-up steps (default: at least 10 and at least 100 ms of "
                         "steps, so that the chip has reached its steady clock)")
    ap.add_argument("--config", type=int, default=4, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--dtype", default=None, choices=[None, "f32", "bf16"])
    ap.add_argument("--decomp", default="fused", choices=["fused", "split"])
    ap.add_argument("--no-split", action="store_true", help="skip timing the split form")
    ap.add_argument("--cpu-units", type=int, default=None,
                    help="units of the oracle sample: rows, images or sequences (default: "
                         "about 800 GFLOP of rows, every image, first and last sequence)")
    ap.add_argument("--calibration-copy-mb", type=int, default=0,
                    help="run one plain device copy of this size first (counter calibration)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--protocol-runs", type=int, default=100,
                    help="individually timed runs (1 GiB cache flush before each) for the "
                         "median; 0 skips")
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the composed-module hot path is "
              "single-GPU (no collectives); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_20501_amd import inputs, mk

    torch.cuda.set_device(0)
    module = build_module(args.config, args.dtype)
    t0 = time.perf_counter()
    host = inputs.make_inputs(module, args.seed)
    log(f"inputs generated in {time.perf_counter() - t0:.1f} s")
    fused = mk.Module(module, args.decomp, strict=True)
    split = None if args.no_split else mk.Module(module, "split", strict=True)
    ws_bytes = max(fused.workspace_size(), split.workspace_size() if split else 0)
    ins, _, ws = mk.device_buffers(module, host, ws_bytes)
    out = mk.out_tensor(module, fused.info["out_shape"])
    flops = fused.info["flops"]
    if args.calibration_copy_mb:
        n = args.calibration_copy_mb << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: {n} bytes")
        del src, dst

    ms, per_launch, warmed = time_module(fused, ins, out, ws, args.steps, args.warmup)
    log(f"{args.decomp}: {ms * 1e3:.1f} us/step, launches (us): "
        f"{[round(x * 1e3, 1) for x in per_launch]}")
    result = {}
    if split is not None:
        out_s = mk.out_tensor(module, split.info["out_shape"])
        ms_s, per_s, _ = time_module(split, ins, out_s, ws, args.steps, args.warmup)
        log(f"split: {ms_s * 1e3:.1f} us/step, launches (us): {[round(x * 1e3, 1) for x in per_s]}")
        result["split"] = {"ms_per_step": ms_s, "value": flops / (ms_s * 1e-3) / 1e12,
                           "launch_us": [round(x * 1e3, 2) for x in per_s]}
        result["fused_vs_split_speedup"] = ms_s / ms
        # the split run overwrote nothing the fused output depends on; rerun fused
        fused.run(ins, out, ws)
        torch.cuda.synchronize()

    if args.protocol_runs:
        flush = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        med = {"runs": args.protocol_runs, "flush_bytes": 1 << 30,
               "fused_median_ms": median_flushed(fused, ins, out, ws, args.protocol_runs, flush)}
        if split is not None:
            out_s = mk.out_tensor(module, split.info["out_shape"])
            med["split_median_ms"] = median_flushed(split, ins, out_s, ws, args.protocol_runs,
                                                    flush)
            med["fused_vs_split_speedup"] = med["split_median_ms"] / med["fused_median_ms"]
            del out_s
            fused.run(ins, out, ws)
        med["fused_tflops"] = flops / (med["fused_median_ms"] * 1e-3) / 1e12
        del flush
        torch.cuda.synchronize()
        result["median_protocol"] = med
        log(f"median protocol: {med}")

    # dominant kernel of the timed composition
    names = launch_names(fused)
    k = max(range(len(per_launch)), key=lambda i: per_launch[i])
    sk = fused.subkernels()
    launch_to_sub = [i for i, s in enumerate(sk) for _ in range(s["n_launches"])]
    sub = sk[launch_to_sub[k]]
    sub_ms = [0.0] * len(sk)
    for i, t in enumerate(per_launch):
        sub_ms[launch_to_sub[i]] += t
    result["subkernel_us"] = [round(t * 1e3, 2) for t in sub_ms]
    # runtime attribution of the composition (the share a budget allocation by
    # runtime would give each subkernel)
    result["subkernel_share"] = [round(x, 4) for x in mk.mk_budget_shares(sub_ms)]
    bf = module["dtype"] == "bf16"
    if sub["flops"] > 0:
        achieved = sub["flops"] / (per_launch[k] * 1e-3) / 1e12
        peak = PEAK_BF16_TFLOPS if bf else PEAK_F32_TFLOPS
        roof = {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                "frac": achieved / peak,
                "traffic": measured_traffic(module["name"], names[k])}
    else:
        achieved = sub["alg_bytes"] / (per_launch[k] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS, "traffic": None}
    roof["kernel"] = names[k]
    roof["kernel_us"] = per_launch[k] * 1e3
    roof["per_launch_flops"] = sub["flops"]
    roof["per_launch_alg_bytes"] = sub["alg_bytes"]

    line = {
        "metric": "composed-module TFLOP/s (fused), % of MI355X roofline, fused vs split speedup",
        "value": flops / (ms * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": warmed,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf else "f32",
        "data": "synthetic (seeded SplitMix64 / Box-Muller inputs, resident in HBM)",
        "config": {"workload": module["name"], "decomposition": args.decomp,
                   "module_flops": flops, "module_alg_bytes": fused.info["alg_bytes"],
                   "launches_per_step": len(per_launch), "parallelism": "single GPU"},
        "roofline": roof,
        "launch_us": [round(x * 1e3, 2) for x in per_launch],
    }
    line.update(result)
    if not args.no_cpu_baseline:
        units, unit_name = baseline_units(args.config, module, flops, args.cpu_units)
        line["cpu_baseline"] = cpu_baseline(module, host, units, out, unit_name)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
