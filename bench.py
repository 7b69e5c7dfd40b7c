"""Throughput of batched dynamic-routing inference on one MI355X.

One step = one dycl_run of a whole batch through the compiled dynamic
network: sub-network convolutions, decision heads, compaction, row
gathers / scatters and the count-only host module.  Inputs are resident in
HBM before the timed region; the plan (weights, workspace) is built before.

Prints one JSON line:
  value        samples/s over exactly --steps timed steps (HIP events on the
               run's stream, bracketed by device synchronisation);
  roofline     the dominant kernel class (the MFMA convolutions), timed per
               launch with HIP events in a second, profiled pass of the same
               steps: algorithmic FLOPs of the executed rows / kernel time,
               against the bf16 dense MFMA peak;
  cpu_baseline the oracle (plain per-sample CPU interpreter) on a bounded
               sample of the same workload.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "samples/sec of batched dynamic-routing inference + % of bf16 MFMA / HBM peak"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
PEAK_F32_TFLOPS = 157.3


def cpu_baseline(wl, seconds: float):
    import numpy as np
    import torch
    from oracle import dycl_oracle as O
    o = O.from_workload(wl)
    x, aux = wl.inputs_f32(64)
    n, t0 = 0, time.perf_counter()
    while True:
        o.run_sample(x[n % 64], None if aux is None else float(aux[n % 64]))
        n += 1
        el = time.perf_counter() - t0
        if (el >= seconds and n >= 2) or el >= 4 * seconds:
            break
    _ = np
    return {"value": n / el, "unit": "samples/s", "cores": torch.get_num_threads(), "kind": "oracle",
            "sample": f"{n} samples of {wl.name} run one by one (float64 accumulation, bf16 storage), {el:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="resnet18_exit")
    ap.add_argument("--batch", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(samples are independent, so a multi-GPU run would shard the batch; not built)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2307_04963_amd import runtime
    from workloads import configs

    wl = configs.build(args.workload)
    B = args.batch or configs.DEFAULT_BATCH[args.workload]
    plan = runtime.Plan.from_workload(wl, B)
    x, aux = wl.inputs(B)
    xt, at = runtime.device_inputs(wl, x, aux)
    logits = torch.empty((B, plan.n_out), dtype=torch.float32, device="cuda")
    rec = torch.empty((B, 4), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        plan.run(xt, at, logits, rec, stream)
    torch.cuda.synchronize()

    # timed region: exactly --steps steps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        plan.run(xt, at, logits, rec, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = e0.elapsed_time(e1) / args.steps
    counts = plan.counts()

    # profiled pass: per-launch HIP events around every kernel on the run's stream
    plan.profile(True)
    for _ in range(args.steps):
        plan.run(xt, at, logits, rec, stream)
    torch.cuda.synchronize()
    prof = plan.profile_read()
    plan.profile(False)
    conv = prof["conv_bf16_mfma"]
    conv_ms = conv["ms"] / max(conv["launches"], 1)
    conv_flops = conv["flops"] / max(conv["launches"], 1)
    achieved = conv["flops"] / (conv["ms"] * 1e-3) / 1e12 if conv["ms"] > 0 else 0.0
    kernels = {k: {"launches_per_step": v["launches"] / args.steps, "ms_per_step": v["ms"] / args.steps,
                   "tflops": (v["flops"] / (v["ms"] * 1e-3) / 1e12) if v["ms"] else 0.0,
                   "gbs": (v["bytes"] / (v["ms"] * 1e-3) / 1e9) if v["ms"] else 0.0}
               for k, v in prof.items() if v["launches"]}

    out = {
        "metric": METRIC,
        "value": B / (ms * 1e-3),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "wall_ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.arch["dtype"],
        "data": "synthetic (seeded N(0,1) inputs, seeded random-init weights, calibrated BN/heads)",
        "config": {"workload": args.workload, "batch": B, "input": list(wl.arch["input"]),
                   "branch_counts": counts, "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "kernel": "conv_bf16_mfma (implicit-GEMM conv / linear)",
                     "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None,
                     "avg_launch_ms": conv_ms, "avg_launch_flops": conv_flops},
        "kernels": kernels,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    plan.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
