"""Decision-noise floor of each workload.  TEST INFRASTRUCTURE (oracle side).

A routing decision compares a float32 statistic (an exit head's largest
softmax probability, a gate's sigmoid, an accumulated halting probability)
with a threshold.  Two correct implementations that accumulate the same
bf16-stored network in different orders drift apart by an amount that
grows with depth; a decision whose margin is inside that drift is not
determined by the network, only by rounding.

This script measures the drift with the oracle alone: it runs each workload
with float64 and with float32 accumulation and takes, for each decision
position (exit head k, gate i, loop step t) and over all samples, the largest
difference between corresponding decision statistics (up to the first
decision where the two runs part ways).  The floors written to
``tests/golden/decision_floor.json`` are SAFETY times those drifts; the
parity tests treat a sample as a near-tie when one of its decisions k lies
closer to its threshold than max(1e-3, floor[k]).

Run: ``python -m oracle.floor [names...]``.
"""

from __future__ import annotations

import json
import os
import sys

import numpy as np
import torch

from .dycl_oracle import from_workload

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
from workloads import configs  # noqa: E402

SAFETY = 4.0
SAMPLES = {"mlp_exit": 1024, "resnet18_exit": 384, "skipnet38": 384, "resnet50_exit": 96, "act_loop": 1024}
OUT = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "tests", "golden",
                   "decision_floor.json")


def drift(r64, r32, positions):
    worst, diverged = [0.0] * positions, 0
    for t64, t32, e64, e32, i64, i32, s64, s32 in zip(r64["trail"], r32["trail"], r64["exit_index"],
                                                      r32["exit_index"], r64["iterations"], r32["iterations"],
                                                      r64["skip_mask"], r32["skip_mask"]):
        n = min(len(t64), len(t32))
        for k, (a, b) in enumerate(zip(t64[:n], t32[:n])):
            worst[k] = max(worst[k], abs(a - b))
        if (e64, i64, s64) != (e32, i32, s32):
            diverged += 1
    return worst, diverged


def n_positions(arch):
    fam = arch["family"]
    if fam == "seq_decoder":
        return arch["max_len"]
    if fam == "early_exit_mlp":
        return len(arch["layers"]) - 1
    if fam == "early_exit_resnet":
        return len(arch["stages"]) - 1
    if fam == "skipnet":
        return len(arch["blocks"])
    return arch["max_steps"] - 1


def thresholds(arch):
    fam = arch["family"]
    if fam == "skipnet":
        return float(np.float32(arch["gate_threshold"]))
    if fam == "seq_decoder":
        return 0.0      # the statistic is the gap between the two largest logits
    return float(np.float32(arch["tau"]))


def near_tie(trail, thr, floors, base=1e-3):
    """True when some decision k of the trail is within max(base, floors[k])."""
    return any(abs(v - thr) < max(base, floors[k]) for k, v in enumerate(trail))


def measure(name: str):
    wl = configs.build(name)
    n = SAMPLES[name]
    x, aux = wl.inputs_f32(n)
    r64 = from_workload(wl, "f64").run(x, aux)
    r32 = from_workload(wl, "f32").run(x, aux)
    worst, diverged = drift(r64, r32, n_positions(wl.arch))
    floors = [SAFETY * w for w in worst]
    thr = thresholds(wl.arch)
    frac = float(np.mean([near_tie(t, thr, floors) for t in r64["trail"]]))
    return {"samples": n, "max_stat_drift_f32_vs_f64": worst, "routing_diverged": diverged,
            "safety": SAFETY, "floor": floors, "threshold": thr, "near_tie_fraction": frac}


if __name__ == "__main__":
    torch.set_num_threads(max(1, os.cpu_count() or 1))
    names = sys.argv[1:] or configs.NAMES
    data = {}
    if os.path.exists(OUT):
        with open(OUT) as f:
            data = json.load(f)
    for nm in names:
        data[nm] = measure(nm)
        print(nm, data[nm], flush=True)
    data["_about"] = ("written by oracle/floor.py: SAFETY x the largest difference between the float32- and "
                      "float64-accumulating oracle's decision statistics")
    with open(OUT, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
