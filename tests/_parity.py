"""GPU-vs-oracle comparison used by the parity tests and the smoke check.

Categories of a sample (see the decision-floor script beside the oracle):
  exact     routing identical to the oracle's;
  near-tie  some decision of the oracle lies within max(1e-3, floor[k]) of
            its threshold, where floor[k] is the measured drift of decision
            position k between two correct accumulation orders;
  mismatch  routing differs although no decision is a near-tie (a failure).
Logits are compared on every sample whose routing matches.
"""

from __future__ import annotations

import json
import os

import numpy as np

from oracle import dycl_oracle as O
from oracle.floor import near_tie, thresholds

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
with open(os.path.join(ROOT, "tests", "golden", "decision_floor.json")) as _f:
    FLOORS = json.load(_f)

LOGIT_TOL = {"bf16": 2e-2, "f32": 1e-4}


def compare(wl, gpu: dict, ref: dict, rows=None, floors=None):
    """gpu: results for the whole batch; ref: oracle results for `rows`."""
    rows = np.arange(len(ref["exit_index"])) if rows is None else np.asarray(rows)
    floors = FLOORS[wl.name]["floor"] if floors is None else floors
    thr = thresholds(wl.arch)
    g = {k: gpu[k][rows] for k in ("logits", "exit_index", "iterations", "skip_mask")}
    route_ok = ((g["exit_index"] == ref["exit_index"]) & (g["iterations"] == ref["iterations"])
                & (g["skip_mask"] == ref["skip_mask"]))
    tie = np.array([near_tie(t, thr, floors) for t in ref["trail"]], dtype=bool)
    bad_route = ~route_ok & ~tie
    tol = LOGIT_TOL[wl.arch["dtype"]]
    err = np.abs(g["logits"][route_ok].astype(np.float64) - ref["logits"][route_ok].astype(np.float64))
    max_err = float(err.max()) if err.size else 0.0
    finite = bool(np.isfinite(g["logits"]).all())
    rep = {
        "samples": int(len(rows)), "exact": int(route_ok.sum()), "near_tie": int(tie.sum()),
        "near_tie_mismatch": int((~route_ok & tie).sum()), "mismatch": int(bad_route.sum()),
        "max_abs_logit_err": max_err, "tol": tol, "finite": finite,
        "delta": O.delta(g["logits"][route_ok], ref["logits"][route_ok]),
        "eta": O.eta(g["logits"][route_ok], ref["logits"][route_ok]),
    }
    rep["ok"] = bool(rep["mismatch"] == 0 and max_err <= tol and finite)
    return rep
