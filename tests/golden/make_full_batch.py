"""Writes the full-batch oracle results the GPU parity tests compare against.

For every workload at its full batch (and, for the four calibrated ones,
their literal form: BatchNorm at its eval defaults, heads and gates as
drawn), the oracle runs every sample with float64 accumulation (the
reference) and with each of its four float32 accumulation orders (other
correct evaluations of the same network).  Stored per sample: the float64
run's logits, exit index, iteration count, skip mask, emitted tokens (the
decoder; -1 past the end), decision margin (the
smallest |statistic - threshold| over the decisions it evaluated) and
decision trail, and whether some float32 order routed the sample
differently ("oracle-unstable": a property of the network, measured without
the GPU), with the library float32 order's own flag beside it.  A fingerprint of the inputs and weight bytes ties each
file to the workload it was computed from.

Only the oracle and the seeded workload generator are called here.  Samples
are independent (the oracle's batch-split invariance is pinned), so they are
spread over worker processes.

Run: ``python -m tests.golden.make_full_batch [name[:literal] ...]``
"""

from __future__ import annotations

import hashlib
import multiprocessing as mp
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from workloads import configs  # noqa: E402

OUT_DIR = os.path.join(ROOT, "tests", "golden", "full_batch")
LITERAL = ["mlp_exit", "resnet18_exit", "skipnet38", "resnet50_exit"]


def golden_path(name: str, literal: bool = False) -> str:
    return os.path.join(OUT_DIR, f"{name}{'_literal' if literal else ''}.npz")


def fingerprint(wl, batch: int) -> str:
    """SHA-256 over the batch's input bytes, its aux values and the weight blob."""
    x, aux = wl.inputs(batch)
    h = hashlib.sha256()
    h.update(np.ascontiguousarray(x).tobytes())
    if aux is not None:
        h.update(np.ascontiguousarray(aux).tobytes())
    h.update(wl.blob()[0])
    return h.hexdigest()


def _worker(args):
    name, literal, acc, lo, hi = args
    import torch
    torch.set_num_threads(1)
    from oracle import dycl_oracle as O
    wl = configs.build(name, calibrated=not literal)
    x, aux = wl.inputs_f32(hi)
    return lo, O.from_workload(wl, acc).run(x, aux, indices=range(lo, hi))


def run_oracle(name, literal, acc, batch, procs):
    step = max(1, (batch + 4 * procs - 1) // (4 * procs))
    jobs = [(name, literal, acc, lo, min(batch, lo + step)) for lo in range(0, batch, step)]
    with mp.get_context("spawn").Pool(procs) as pool:
        parts = sorted(pool.map(_worker, jobs), key=lambda t: t[0])
    out = {}
    for k in ("logits", "exit_index", "iterations", "skip_mask", "margin", "tokens"):
        out[k] = np.concatenate([p[k] for _, p in parts])
    out["trail"] = [t for _, p in parts for t in p["trail"]]
    return out


def make(name: str, literal: bool, procs: int):
    wl = configs.build(name, calibrated=not literal)
    B = configs.DEFAULT_BATCH[name]
    t0 = time.time()
    from oracle.dycl_oracle import ACC_F32
    r64 = run_oracle(name, literal, "f64", B, procs)
    diff = {}
    for acc in ACC_F32:
        r = run_oracle(name, literal, acc, B, procs)
        diff[acc] = ((r64["exit_index"] != r["exit_index"]) | (r64["iterations"] != r["iterations"])
                     | (r64["skip_mask"] != r["skip_mask"]) | (r64["tokens"] != r["tokens"]).any(axis=1))
        if acc == "f32":
            r32 = r
    same = ~np.logical_or.reduce([diff[a] for a in ACC_F32])
    same32 = ~diff["f32"] & same
    P = max([len(t) for t in r64["trail"]] + [1])
    trail = np.full((B, P), np.nan)
    for i, t in enumerate(r64["trail"]):
        trail[i, :len(t)] = t
    floor = (float(np.abs(r64["logits"][same32].astype(np.float64) - r32["logits"][same32]).max())
             if same32.any() else 0.0)
    np.savez_compressed(
        golden_path(name, literal), fingerprint=np.array(fingerprint(wl, B)), batch=np.array(B),
        logits=r64["logits"].astype(np.float32), exit_index=r64["exit_index"], iterations=r64["iterations"],
        skip_mask=r64["skip_mask"], tokens=r64["tokens"], margin=r64["margin"], trail=trail, unstable=~same,
        unstable_f32=diff["f32"], **{f"routed_apart_{a}": diff[a] for a in ACC_F32},
        logit_floor_f32_vs_f64=np.array(floor))
    print(f"{name}{' (literal)' if literal else ''}: B={B} unstable={int((~same).sum())} "
          f"({', '.join(f'{a}: {int(diff[a].sum())}' for a in ACC_F32)}) "
          f"near_tie={int((r64['margin'] < 1e-3).sum())} logit_floor={floor:.3g} {time.time() - t0:.0f}s", flush=True)


def main(argv):
    procs = max(1, min(16, os.cpu_count() or 1))
    todo = []
    for a in argv or [*configs.NAMES, *[n + ":literal" for n in LITERAL]]:
        nm, _, lit = a.partition(":")
        todo.append((nm, lit == "literal"))
    os.makedirs(OUT_DIR, exist_ok=True)
    for nm, lit in todo:
        make(nm, lit, procs)


if __name__ == "__main__":
    main(sys.argv[1:])
