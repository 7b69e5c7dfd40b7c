"""GPU parity: the HIP path through the C ABI against the oracle.

* every workload at a small batch (several tiles, ragged tails), element by
  element;
* every workload at its full batch, in the launch configuration the
  benchmark times, on sampled rows the oracle recomputes one by one;
* edge cases: empty batch, one sample, over-sized batch, forced routing of
  every density (nobody / everybody leaves at a decision), and branch
  counts that agree with the per-sample records.
"""

import numpy as np
import pytest

from oracle import dycl_oracle as O
from tests._parity import compare
from workloads import configs

pytestmark = pytest.mark.gpu

SMALL = {"mlp_exit": 37, "resnet18_exit": 37, "skipnet38": 45, "resnet50_exit": 5, "act_loop": 300}
SAMPLED = {"mlp_exit": 64, "resnet18_exit": 24, "skipnet38": 24, "resnet50_exit": 4, "act_loop": 64}

_cache = {}


def _rt():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2307_04963_amd import runtime
    return runtime


def _plan(name, wl=None, max_batch=None):
    rt = _rt()
    key = (name, max_batch, id(wl) if wl is not None else None)
    if key not in _cache:
        wl = wl or configs.build(name)
        _cache[key] = (wl, rt.Plan.from_workload(wl, max_batch or configs.DEFAULT_BATCH[name]))
    return _cache[key]


def _check_counts(wl, gpu):
    counts, fam = gpu["counts"], wl.arch["family"]
    B = len(gpu["exit_index"])
    if fam in ("early_exit_mlp", "early_exit_resnet"):
        assert sum(c[0] for c in counts) == B          # every sample leaves once
        for k, (ex, stay) in enumerate(counts):
            assert ex == int((gpu["exit_index"] == k).sum())
    elif fam == "skipnet":
        for i, (run, skip) in enumerate(counts[:-1]):
            bits = (gpu["skip_mask"] >> np.uint64(i)) & np.uint64(1)
            assert run == int((bits == 0).sum()) and skip == int((bits == 1).sum())
    else:
        for t, (halt, stay) in enumerate(counts):
            assert halt == int((gpu["iterations"] == t + 1).sum())
        assert gpu["iterations"].min() >= 1 and gpu["iterations"].max() <= wl.arch["max_steps"]


@pytest.mark.parametrize("name", configs.NAMES)
def test_small_batch_parity(name):
    rt = _rt()
    wl, plan = _plan(name)
    B = SMALL[name]
    print(f"[parity-small] {name} B={B}", flush=True)
    x, aux = wl.inputs(B)
    gpu = rt.run_numpy(plan, wl, x, aux)
    xf, auxf = wl.inputs_f32(B)
    ref = O.from_workload(wl).run(xf, auxf)
    rep = compare(wl, gpu, ref)
    print(name, rep, flush=True)
    assert rep["ok"], rep
    _check_counts(wl, gpu)


@pytest.mark.parametrize("name", configs.NAMES)
def test_full_batch_sampled_parity(name):
    rt = _rt()
    wl, plan = _plan(name)
    B = configs.DEFAULT_BATCH[name]
    print(f"[parity-full] {name} B={B}", flush=True)
    x, aux = wl.inputs(B)
    gpu = rt.run_numpy(plan, wl, x, aux)
    rng = np.random.default_rng(7)
    k = min(B, SAMPLED[name])
    rows = np.unique(np.concatenate([[0, B - 1], rng.choice(B, k - 2, replace=False)]))
    xf, auxf = wl.inputs_f32(B)
    ref = O.from_workload(wl).run(xf, auxf, indices=rows)
    rep = compare(wl, gpu, ref, rows)
    print(name, rep, "counts", gpu["counts"], flush=True)
    assert rep["ok"], rep
    _check_counts(wl, gpu)


def test_empty_one_and_oversized_batches():
    rt = _rt()
    import torch
    from paper_2307_04963_amd._lib import DyclError
    wl, plan = _plan("resnet18_exit")
    x, _ = wl.inputs(1)
    xt, _ = rt.device_inputs(wl, x, None)
    logits = torch.full((1, plan.n_out), float("nan"), device="cuda")
    rec = torch.zeros((1, 4), dtype=torch.int32, device="cuda")
    plan.run(xt[:0], None, logits, rec)               # batch 0: nothing happens
    torch.cuda.synchronize()
    assert torch.isnan(logits).all()
    gpu = rt.run_numpy(plan, wl, x)
    ref = O.from_workload(wl).run(*wl.inputs_f32(1))
    assert compare(wl, gpu, ref)["ok"]
    big = torch.zeros((plan.max_batch + 1, 32, 32, 3), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(DyclError) as e:
        plan.run(big, None, logits, rec)
    assert e.value.code == -4


@pytest.mark.parametrize("tau,want", [(0.0, 0), (1.5, 2)])
def test_forced_exits_mlp(tau, want):
    rt = _rt()
    wl = configs.build("mlp_exit")
    wl.arch = dict(wl.arch, tau=tau)
    _, plan = _plan("mlp_exit", wl, 64)
    x, _ = wl.inputs(50)
    gpu = rt.run_numpy(plan, wl, x)
    assert (gpu["exit_index"] == want).all()
    ref = O.from_workload(wl).run(x)
    assert compare(wl, gpu, ref)["ok"]


@pytest.mark.parametrize("v,mask", [(50.0, 0), (-50.0, (1 << 18) - 1)])
def test_forced_gates_skipnet(v, mask):
    rt = _rt()
    wl = configs.build("skipnet38")
    for b in wl.arch["blocks"]:
        t = wl.tensors[b["gate"] + ".v"]
        wl.tensors[b["gate"] + ".v"] = configs.Tensor(t.name, t.dtype, t.shape, np.array([v], dtype=np.float32))
    _, plan = _plan("skipnet38", wl, 64)
    x, _ = wl.inputs(19)
    gpu = rt.run_numpy(plan, wl, x)
    assert (gpu["skip_mask"] == np.uint64(mask)).all()
    ref = O.from_workload(wl).run(wl.inputs_f32(19)[0])
    rep = compare(wl, gpu, ref)
    assert rep["ok"], rep


@pytest.mark.parametrize("bias,steps", [(10.0, 1), (-30.0, 16)])
def test_forced_halting_act(bias, steps):
    rt = _rt()
    wl, plan = _plan("act_loop")
    x, _ = wl.inputs(70)
    aux = np.full(70, bias, dtype=np.float32)
    gpu = rt.run_numpy(plan, wl, x, aux)
    assert (gpu["iterations"] == steps).all()
    ref = O.from_workload(wl).run(wl.inputs_f32(70)[0][:8], aux[:8])
    rep = compare(wl, {k: v[:8] for k, v in gpu.items() if k != "counts"}, ref)
    assert rep["ok"], rep
