"""GPU-vs-oracle comparison used by the parity tests and the smoke check.

The contract (Eq. 2: the compiled host program equals the dynamic network on
every input; RQ1, Table 3: zero inconsistent outputs) is checked per sample.
A sample falls in one of these categories:

  exact       routing (exit index, iteration count, skip mask, and a
              decoder's emitted tokens) identical to the oracle's;
  near-tie    some decision the float64 oracle evaluated lies within 1e-3 of
              its threshold (its fp32 margin is below 1e-3);
  unstable    one of the oracle's float32 accumulation orders routes the
              sample differently from its float64 run: two correct
              accumulation orders of the same bf16-stored network disagree,
              so its routing is not fixed by the network (a property
              measured without the GPU; the count for the library float32
              order alone is printed beside it);
  mismatch    routing differs from the oracle's although the sample is
              neither near-tie nor unstable: a failure.

Logits are compared on every sample whose routing matches, against 2e-2
absolute for bf16 workloads and 1e-4 for the fp32 one.  The older
drift-based band (4x the float32-vs-float64 drift of each decision
position) is reported as a diagnostic count only.
"""

from __future__ import annotations

import json
import os

import numpy as np

from oracle import dycl_oracle as O
from oracle.floor import near_tie as _in_drift_band, thresholds

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
with open(os.path.join(ROOT, "tests", "golden", "decision_floor.json")) as _f:
    FLOORS = json.load(_f)

NEAR_TIE = 1e-3
LOGIT_TOL = {"bf16": 2e-2, "f32": 1e-4}
ROUTE_KEYS = ("exit_index", "iterations", "skip_mask")


def _route_keys(ref):
    """Routing fields: the records, and a decoder's emitted tokens."""
    return ROUTE_KEYS + (("tokens",) if np.asarray(ref.get("tokens", np.zeros((0, 0)))).shape[-1] else ())


def _differ(a, b):
    a, b = np.asarray(a), np.asarray(b)
    d = a != b
    return d.any(axis=1) if d.ndim == 2 else d


def oracle_ref(wl, x_f32, aux, indices=None):
    """Float64 oracle results for `indices` plus the unstable flags from the
    oracle's float32 accumulation orders on the same samples."""
    r64 = O.from_workload(wl, "f64").run(x_f32, aux, indices=indices)
    apart = {}
    for acc in O.ACC_F32:
        r = O.from_workload(wl, acc).run(x_f32, aux, indices=indices)
        d = np.zeros(len(r64["exit_index"]), dtype=bool)
        for k in _route_keys(r64):
            d |= _differ(r64[k], r[k])
        apart[acc] = d
    r64["unstable"] = np.logical_or.reduce([apart[a] for a in O.ACC_F32])
    r64["unstable_f32"] = apart["f32"]
    return r64


def load_golden(wl, literal: bool = False):
    """The stored full-batch oracle results of a workload, checked against
    the workload's current input and weight bytes."""
    from tests.golden.make_full_batch import fingerprint, golden_path
    from workloads import configs
    path = golden_path(wl.name, literal)
    with np.load(path, allow_pickle=False) as z:
        g = {k: z[k] for k in z.files}
    B = int(g["batch"])
    assert B == configs.DEFAULT_BATCH[wl.name]
    assert str(g["fingerprint"]) == fingerprint(wl, B), f"{path} is stale: regenerate it with make_full_batch"
    return g


def histogram(ref, arch):
    fam = arch["family"]
    if fam in ("early_exit_mlp", "early_exit_resnet"):
        return np.bincount(ref["exit_index"], minlength=len(arch.get("heads", []))).tolist()
    if fam == "act":
        return np.bincount(ref["iterations"], minlength=arch["max_steps"] + 1)[1:].tolist()
    if fam == "seq_decoder":
        return np.bincount(ref["iterations"], minlength=arch["max_len"] + 1)[1:].tolist()
    bits = [(np.asarray(ref["skip_mask"], dtype=np.uint64) >> np.uint64(i)) & np.uint64(1)
            for i in range(len(arch["blocks"]))]
    return [int(b.sum()) for b in bits]           # samples that skip each gate


def compare(wl, gpu: dict, ref: dict, rows=None, logit_tol=None):
    """gpu: results for the whole batch; ref: oracle results for `rows`
    (default: all), with an `unstable` flag per row when known."""
    rows = np.arange(len(ref["exit_index"])) if rows is None else np.asarray(rows)
    keys = _route_keys(ref)
    g = {k: np.asarray(gpu[k])[rows] for k in ("logits",) + keys}
    route_ok = np.ones(len(rows), dtype=bool)
    for k in keys:
        route_ok &= ~_differ(g[k], ref[k])
    tie = np.asarray(ref["margin"]) < NEAR_TIE
    unstable = np.asarray(ref.get("unstable", np.zeros(len(rows), dtype=bool)), dtype=bool)
    bad_route = ~route_ok & ~tie & ~unstable
    tol = LOGIT_TOL[wl.arch["dtype"]] if logit_tol is None else logit_tol
    err = np.abs(g["logits"][route_ok].astype(np.float64) - np.asarray(ref["logits"])[route_ok].astype(np.float64))
    max_err = float(err.max()) if err.size else 0.0
    finite = bool(np.isfinite(g["logits"]).all())
    # diagnostic: the drift-based band of the decision-floor file
    thr = thresholds(wl.arch)
    floors = FLOORS.get(wl.name, {}).get("floor")
    trails = ref.get("trail")
    band = None
    if floors is not None and trails is not None:
        tl = [t[~np.isnan(t)] if isinstance(t, np.ndarray) else t for t in trails]
        band = int(sum(_in_drift_band(list(t), thr, floors) for t in tl))
    rep = {
        "samples": int(len(rows)), "exact": int(route_ok.sum()), "near_tie": int(tie.sum()),
        "oracle_unstable": int(unstable.sum()),
        "oracle_unstable_f32_library_order": int(np.asarray(ref.get("unstable_f32", unstable)).sum()),
        "near_tie_mismatch": int((~route_ok & tie).sum()),
        "unstable_mismatch": int((~route_ok & unstable & ~tie).sum()), "mismatch": int(bad_route.sum()),
        "max_abs_logit_err": max_err, "tol": tol, "finite": finite,
        "delta": O.delta(g["logits"][route_ok], np.asarray(ref["logits"])[route_ok]),
        "eta": O.eta(g["logits"][route_ok], np.asarray(ref["logits"])[route_ok]),
        "routing_histogram_oracle": histogram(ref, wl.arch), "routing_histogram_gpu": histogram(g, wl.arch),
        "drift_band_diagnostic": band,
    }
    rep["ok"] = bool(rep["mismatch"] == 0 and max_err <= tol and finite)
    return rep
