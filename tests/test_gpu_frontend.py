"""Plans compiled by the front-end from the PyTorch modules run on the GPU
and give the same bits as the plans of the hand lowering, and agree with
the oracle."""

import json

import numpy as np
import pytest

from oracle import dycl_oracle as O
from tests._parity import compare, oracle_ref
from tests.dynn_modules import module_for, input_shape

pytestmark = pytest.mark.gpu

SMALL = {"mlp_exit": 37, "resnet18_exit": 37, "skipnet38": 45, "resnet50_exit": 5, "act_loop": 300}


@pytest.mark.parametrize("name", list(SMALL))
def test_frontend_plan_runs_like_the_lowered_one(name):
    import torch
    assert torch.cuda.is_available()
    from paper_2307_04963_amd import runtime
    from paper_2307_04963_amd.frontend import compile_module
    m, wl = module_for(name)
    spec, blob = compile_module(m, input_shape(wl), wl.arch["dtype"])
    B = SMALL[name]
    print(f"[frontend] {name} B={B}", flush=True)
    pf = runtime.Plan(json.dumps(spec), blob, B)
    pl = runtime.Plan.from_workload(wl, B)
    x, aux = wl.inputs(B)
    a = runtime.run_numpy(pf, wl, x, aux)
    b = runtime.run_numpy(pl, wl, x, aux)
    assert np.array_equal(a["logits"], b["logits"], equal_nan=True)
    for k in ("exit_index", "iterations", "skip_mask"):
        assert np.array_equal(a[k], b[k]), k
    assert a["counts"] == b["counts"]
    ref = oracle_ref(wl, *wl.inputs_f32(B))
    rep = compare(wl, a, ref)
    assert rep["ok"], rep
