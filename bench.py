"""Throughput of batched dynamic-routing inference on one MI355X.

One step = one dycl_run of a whole batch through the compiled dynamic
network: sub-network convolutions, decision heads, compaction, row
gathers / scatters and the count-only host module.  Inputs are resident in
HBM before the timed region; the plan (weights, workspace) is built before.

Prints one JSON line:
  value        samples/s over exactly --steps timed steps (HIP events on the
               run's stream, bracketed by device synchronisation) in the
               host mode --host-mode;
  host_modes   the same --steps timed in each host mode: sync (branch counts
               read back at every decision point), device (counts stay on the
               device, count-guarded launches) and graph (device mode
               replayed from a captured HIP graph), with the host-module cost
               per decision point that the device modes remove;
  roofline     the dominant kernel class (the MFMA convolutions), timed per
               launch with HIP events in a second, profiled pass of the same
               steps: algorithmic FLOPs of the executed rows / kernel time,
               against the bf16 dense MFMA peak;
  cpu_baseline the oracle (plain per-sample CPU interpreter) on a bounded
               sample of the same workload, on every host core (parallel
               across samples) and on one core;
  other_workloads  samples/s of every other workload at its own batch
               (device host mode, same step count);
  hbm_kernels  the routing primitives at HBM-bound sizes: the 2^26-flag
               partition (flags to row indices, and carrying ids) and a
               gather of 1.5 MiB rows.
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


def measured_traffic(workload: str, batch: int):
    """HBM bytes per conv launch from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy), or None when there is
    none for this workload or the conv kernel source changed since the
    counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"conv_bf16_mfma__{workload}_b{batch}__traffic.md")
    if not os.path.exists(path):
        return None, "no counter summary for this workload"
    kv = {}
    for line in open(path):
        if " = " in line:
            k, v = line.strip().split(" = ", 1)
            kv[k] = v
    # the conv class spans several sources: the hash is over their bytes in
    # the order listed
    srcs = [os.path.join(ROOT, f) for f in kv.get("kernel_source", "").split()]
    if not srcs or not all(os.path.isfile(f) for f in srcs):
        return None, "kernel source named by the summary is missing"
    h = hashlib.sha256()
    for f in srcs:
        h.update(open(f, "rb").read())
    if h.hexdigest() != kv.get("kernel_source_sha256"):
        return None, "conv kernel changed since the counters were taken"
    return float(kv["traffic_bytes_per_launch"]), os.path.relpath(path, ROOT)


def _cpu_info():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    smt = None
    try:
        smt = open("/sys/devices/system/cpu/smt/active").read().strip() == "1"
    except OSError:
        pass
    return model, os.cpu_count(), smt


def _oracle_worker(args):
    """One host core: the float64 oracle on samples start, start + stride, ...
    of the workload's batch (cycled), one by one, for about `seconds`."""
    name, batch, start, stride, seconds = args
    import torch
    torch.set_num_threads(1)
    from oracle import dycl_oracle as O
    from workloads import configs
    wl = configs.build(name)
    rows = list(range(start, batch, stride)) or [start % batch]
    x, aux = wl.inputs_f32(max(rows) + 1)
    o = O.from_workload(wl, "f64")
    n, t0 = 0, time.perf_counter()
    while True:
        i = rows[n % len(rows)]
        o.run_sample(x[i], None if aux is None else float(aux[i]))
        n += 1
        el = time.perf_counter() - t0
        if (el >= seconds and n >= 2) or el >= 4 * seconds:
            return n, el


def cpu_baseline(wl, batch: int, seconds: float):
    """The oracle (the plain per-sample interpreter, float64 accumulation,
    bf16 storage) on this host's cores, parallel across samples (one process
    per core, one thread each), and on one core alone."""
    import multiprocessing as mp
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    cores = max(1, min(cores, 16))
    span = min(batch, 256)           # the first samples of the batch, in their routing mix
    with mp.get_context("spawn").Pool(cores) as pool:
        par = pool.map(_oracle_worker, [(wl.name, span, r, cores, seconds) for r in range(cores)])
        single = pool.map(_oracle_worker, [(wl.name, span, 0, 1, seconds)])[0]
    value = sum(n / el for n, el in par)
    model, ncpu, smt = _cpu_info()
    done = sum(n for n, _ in par)
    return {"value": value, "unit": "samples/s", "cores": cores, "kind": "oracle",
            "sample": f"{done} samples of {wl.name} (the first {span} of the batch, cycled, split over {cores} "
                      f"processes of one thread) run one by one with float64 accumulation and bf16 storage, "
                      f"about {seconds:.0f} s per process",
            "single_core_value": single[0] / single[1],
            "single_core_sample": f"{single[0]} samples in {single[1]:.1f} s on one thread",
            "cpu_model": model, "logical_cpus": ncpu, "smt_active": smt}


def hbm_kernels(stream, reps: int = 10):
    """Routing primitives at sizes where HBM bandwidth is the bound, timed
    with HIP events on `stream`: the large-n compaction of 2^26 flags (set
    with probability 1/2; without ids, and again carrying original ids) and
    the gather of ResNet-50 stage-1 activation rows (56x56x256 bf16 =
    1.5 MiB per sample)."""
    import ctypes as C
    import numpy as np
    import torch
    from paper_2307_04963_amd import _lib
    L = _lib.lib
    out = {}
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731

    n = 1 << 26
    g = torch.Generator(device="cuda").manual_seed(3)
    flags = (torch.rand(n, device="cuda", generator=g) < 0.5).to(torch.uint8)
    orig = torch.randperm(n, device="cuda", generator=g).to(torch.int32)
    outs = [torch.empty(n, dtype=torch.int32, device="cuda") for _ in range(4)]
    counts = torch.empty(2, dtype=torch.int32, device="cuda")
    wsb = L.dycl_op_compact_workspace(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    p = lambda t: C.c_void_p(t.data_ptr())  # noqa: E731

    def timed(args):
        _lib.check(L.dycl_op_compact(*args))
        a, b = ev(), ev()
        a.record(stream)
        for _ in range(reps):
            _lib.check(L.dycl_op_compact(*args))
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / reps

    tail = [p(counts), p(ws), wsb, C.c_void_p(stream.cuda_stream)]
    # the partition as the method needs it: a flag read and one 4-byte row
    # index written per element (no ids carried)
    us = timed([p(flags), None, n, p(outs[0]), None, p(outs[2]), None] + tail)
    nbytes = n * (1 + 4)
    out["compaction_2^26"] = {"us": us, "algorithmic_bytes": nbytes, "gbs": nbytes / (us * 1e-6) / 1e9,
                              "frac": nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS,
                              "form": "flags -> row indices (1 B read + 4 B written per element)"}
    # the same with original ids carried (the plan's nested-decision form):
    # ids read and one id written per element on top
    us = timed([p(flags), p(orig), n] + [p(t) for t in outs] + tail)
    moved = n * (1 + 4 + 8)
    out["compaction_ids_2^26"] = {"us": us, "algorithmic_bytes": moved, "gbs": moved / (us * 1e-6) / 1e9,
                                  "frac": moved / (us * 1e-6) / 1e9 / PEAK_HBM_GBS,
                                  "form": "flags + ids -> row indices + ids (13 B per element)"}
    del flags, orig, outs, ws

    row, rows, total = 56 * 56 * 256 * 2, 182, 256
    src = torch.empty(total * row // 2, dtype=torch.int16, device="cuda")
    dst = torch.empty(rows * row // 2, dtype=torch.int16, device="cuda")
    idx = torch.from_numpy(np.sort(np.random.default_rng(5).choice(total, rows, replace=False)).astype(np.int32)).cuda()
    args = [C.c_void_p(dst.data_ptr()), None, C.c_void_p(src.data_ptr()), C.c_void_p(idx.data_ptr()), row, rows,
            C.c_void_p(stream.cuda_stream)]
    _lib.check(L.dycl_op_move_rows(*args))
    a, b = ev(), ev()
    a.record(stream)
    for _ in range(reps):
        _lib.check(L.dycl_op_move_rows(*args))
    b.record(stream)
    torch.cuda.synchronize()
    us = a.elapsed_time(b) * 1e3 / reps
    nbytes = 2 * row * rows + 4 * rows
    out["gather_rows_1.5MiB"] = {"us": us, "rows": rows, "row_bytes": row, "algorithmic_bytes": nbytes,
                                 "gbs": nbytes / (us * 1e-6) / 1e9, "frac": nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS}
    return out


def copy_probe():
    """A plain 1 GiB device copy (torch's copy kernel), three times: the
    reference for scaling the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    a = torch.empty(1 << 29, dtype=torch.int16, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": 2 * a.numel(), "copies": 3}), flush=True)


def other_workloads(skip: str, steps: int, warmup: int, stream):
    """Samples/s of every other workload at its own batch, in device host
    mode, timed like the headline (HIP events around exactly `steps` runs)."""
    import torch
    from paper_2307_04963_amd import runtime
    from workloads import configs
    res = {}
    for name in configs.NAMES:
        if name == skip:
            continue
        wl = configs.build(name)
        B = configs.DEFAULT_BATCH[name]
        plan = runtime.Plan.from_workload(wl, B)
        x, aux = wl.inputs(B)
        xt, at = runtime.device_inputs(wl, x, aux)
        logits, rec, tok = plan.outputs(B)
        plan.set_host_mode("device")
        for _ in range(warmup):
            plan.run(xt, at, logits, rec, stream, tok)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            plan.run(xt, at, logits, rec, stream, tok)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        res[name] = {"batch": B, "dtype": wl.arch["dtype"], "ms_per_step": ms, "samples_per_s": B / (ms * 1e-3),
                     "branch_counts": plan.counts(), "host_mode": "device"}
        plan.close()
        del xt, at, logits, rec, tok
    return res


RIDGE = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)   # FLOP per HBM byte where the two bounds meet


def layer_table(wl, plan, xt, at, logits, rec, stream, warmup, tok=None):
    """One profiled sync-mode step: each conv launch with its algorithmic
    FLOPs and bytes (executed rows only) and its HIP-event time; the bound
    is the layer's attainable rate min(peak, intensity x HBM peak)."""
    import torch
    plan.set_host_mode("sync")
    for _ in range(max(warmup, 1)):
        plan.run(xt, at, logits, rec, stream, tok)
    plan.profile(True)
    plan.run(xt, at, logits, rec, stream, tok)
    torch.cuda.synchronize()
    every = plan.profile_launches()
    launches = [r for r in every if r["class"] in ("conv_bf16_mfma", "linear_f32")]
    heads = [r for r in every if r["class"] in ("decision_heads", "gather_scatter", "compaction")]
    plan.profile(False)
    rows, cb_f, cb_t = [], 0.0, 0.0
    for i, r in enumerate(launches):
        inten = r["flops"] / r["bytes"] if r["bytes"] else 0.0
        tf = r["flops"] / (r["ms"] * 1e-3) / 1e12 if r["ms"] else 0.0
        attain = min(PEAK_BF16_TFLOPS, inten * PEAK_HBM_GBS / 1e3)
        bound = "mfma" if inten >= RIDGE else "hbm"
        if bound == "mfma":
            cb_f += r["flops"]
            cb_t += r["ms"]
        rows.append({"layer": r["label"], "us": round(r["ms"] * 1e3, 1),
                     "gflop": round(r["flops"] / 1e9, 3), "mb": round(r["bytes"] / 1e6, 2),
                     "flop_per_byte": round(inten, 1), "bound": bound, "tflops": round(tf, 1),
                     "frac_peak": round(tf / PEAK_BF16_TFLOPS, 4), "frac_attainable": round(tf / attain, 4) if attain else None})
    cb = cb_f / (cb_t * 1e-3) / 1e12 if cb_t else 0.0
    # HBM-bound routing steps of the same step: heads (pooling reads), compaction, row moves
    hb = [{"class": r["class"], "node": r["label"], "us": round(r["ms"] * 1e3, 1), "mb": round(r["bytes"] / 1e6, 2),
           "gbs": round(r["bytes"] / (r["ms"] * 1e-3) / 1e9, 0) if r["ms"] else 0.0,
           "frac_hbm": round(r["bytes"] / (r["ms"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4) if r["ms"] else 0.0}
          for r in heads]
    return {"workload": wl.name, "batch": int(xt.shape[0]), "branch_counts": plan.counts(), "ridge_flop_per_byte": RIDGE,
            "hbm_steps": hb,
            "mfma_bound_layers": sum(r["bound"] == "mfma" for r in rows),
            "mfma_bound_flop_weighted_tflops": cb, "mfma_bound_frac_peak": cb / PEAK_BF16_TFLOPS, "layers": rows}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="resnet50_exit")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="skip the device-mode throughput of the other workloads")
    ap.add_argument("--batch", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-hbm-kernels", action="store_true")
    ap.add_argument("--copy-probe", action="store_true", help="only run the counter-scaling copy")
    ap.add_argument("--layers", action="store_true",
                    help="only the per-layer table: one profiled sync-mode step, every conv launch timed")
    ap.add_argument("--host-mode", default="device", choices=["sync", "device", "graph", "persistent"],
                    help="host mode of the headline value (all three are timed)")
    args = ap.parse_args()
    if args.copy_probe:
        copy_probe()
        return
    if args.gpus != 1:
        print(f"bench.py: the executor runs on one GPU; --gpus {args.gpus} is not supported "
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
    logits, rec, tok = plan.outputs(B)
    stream = torch.cuda.current_stream()

    if args.layers:
        print(json.dumps(layer_table(wl, plan, xt, at, logits, rec, stream, args.warmup, tok)), flush=True)
        return

    def timed(mode):
        plan.set_host_mode(mode)
        for _ in range(args.warmup):
            plan.run(xt, at, logits, rec, stream, tok)
        torch.cuda.synchronize()
        # timed region: exactly --steps steps
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        e0.record(stream)
        for _ in range(args.steps):
            plan.run(xt, at, logits, rec, stream, tok)
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        return e0.elapsed_time(e1) / args.steps, wall * 1e3 / args.steps, plan.counts()

    modes = {}
    all_modes = ("sync", "device", "graph") + (("persistent",) if args.workload == "act_loop" else ())
    for mode in [m for m in all_modes if m != args.host_mode] + [args.host_mode]:
        modes[mode] = timed(mode)
    ms, wall_ms, counts = modes[args.host_mode]
    assert all(m[2] == counts for m in modes.values()), "host modes disagree on the branch counts"
    plan.set_host_mode("sync")
    decisions = sum(1 for a, b in counts if a + b > 0)
    host_modes = {m: {"ms_per_step": v[0], "wall_ms_per_step": v[1], "samples_per_s": B / (v[0] * 1e-3)}
                  for m, v in modes.items()}
    host_modes["decision_points_reached"] = decisions
    host_modes["us_per_decision_sync_minus_device"] = (
        (modes["sync"][0] - modes["device"][0]) * 1e3 / decisions if decisions else None)
    host_modes["us_per_decision_sync_minus_graph"] = (
        (modes["sync"][0] - modes["graph"][0]) * 1e3 / decisions if decisions else None)

    # profiled pass: per-launch HIP events around every kernel on the run's stream
    plan.profile(True)
    for _ in range(args.steps):
        plan.run(xt, at, logits, rec, stream, tok)
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

    traffic, traffic_src = measured_traffic(args.workload, B)
    out = {
        "metric": METRIC,
        "value": B / (ms * 1e-3),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "wall_ms_per_step": wall_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.arch["dtype"],
        "data": "synthetic (seeded N(0,1) inputs, seeded random-init weights, calibrated BN/heads)",
        "config": {"workload": args.workload, "batch": B, "input": list(wl.arch["input"]),
                   "branch_counts": counts, "host_mode": args.host_mode, "parallelism": "single GPU"},
        "host_modes": host_modes,
        "roofline": {"bound": "mfma", "kernel": "conv_bf16_mfma (bf16 MFMA convolutions and linears: halo-tiled, narrow, RGB stem, implicit GEMM)",
                     "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic,
                     "traffic_unit": "HBM bytes per launch", "traffic_source": traffic_src,
                     "algorithmic_bytes_per_launch": conv["bytes"] / max(conv["launches"], 1),
                     "avg_launch_ms": conv_ms, "avg_launch_flops": conv_flops},
        "kernels": kernels,
    }
    plan.close()
    del xt, at, logits, rec, tok
    if not args.no_other_workloads:
        out["other_workloads"] = other_workloads(args.workload, args.steps, args.warmup, stream)
    if not args.no_hbm_kernels:
        out["hbm_kernels"] = hbm_kernels(stream)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, B, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
