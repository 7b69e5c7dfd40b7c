"""The stored full-batch oracle results (written by the script beside them,
which calls only the oracle) against the oracle itself, on the CPU: each
file belongs to the workload's current input and weight bytes, and a few
rows recomputed one by one reproduce the stored routing, margins and logits
bit for bit; the unstable flags are consistent with the per-order flags."""

import numpy as np
import pytest

from oracle import dycl_oracle as O
from tests._parity import load_golden
from workloads import configs

CASES = [(n, False) for n in configs.NAMES] + [(n, True) for n in
                                                ("mlp_exit", "resnet18_exit", "skipnet38", "resnet50_exit")]


@pytest.mark.parametrize("name,literal", CASES)
def test_golden_rows_reproduce(name, literal):
    wl = configs.build(name, calibrated=not literal)
    g = load_golden(wl, literal)                     # checks the fingerprint
    B = int(g["batch"])
    rows = sorted({0, B // 2, B - 1})
    x, aux = wl.inputs_f32(B)
    r = O.from_workload(wl, "f64").run(x, aux, indices=rows)
    np.testing.assert_array_equal(r["logits"], g["logits"][rows])
    for k in ("exit_index", "iterations", "skip_mask", "margin"):
        np.testing.assert_array_equal(r[k], g[k][rows])
    if "tokens" in g:
        np.testing.assert_array_equal(r["tokens"], g["tokens"][rows])
    for j, i in enumerate(rows):
        t = g["trail"][i]
        np.testing.assert_array_equal(np.asarray(r["trail"][j]), t[~np.isnan(t)])
    anyorder = np.logical_or.reduce([g[f"routed_apart_{a}"] for a in O.ACC_F32])
    np.testing.assert_array_equal(g["unstable"], anyorder)
    np.testing.assert_array_equal(g["unstable_f32"], g["routed_apart_f32"])
    assert g["logits"].shape == (B, wl.arch["n_out"])
