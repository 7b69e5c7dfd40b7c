"""GPU parity: the HIP path through the C ABI against the oracle.

* every workload at a small batch (several tiles, ragged tails), element by
  element, with the float32-accumulating oracle run beside it to mark the
  oracle-unstable samples;
* every workload at its full batch, in the launch configuration the
  benchmark times (device host mode), on EVERY row, against the stored
  full-batch oracle results (written by the script beside them, which calls
  only the oracle); the calibrated workloads and the four literal ones;
* edge cases: empty batch, one sample, over-sized batch, forced routing of
  every density (nobody / everybody leaves at a decision), and branch
  counts that agree with the per-sample records.

Routing must be bit-exact except on near-tie samples (a decision within 1e-3
of its threshold) and oracle-unstable ones (float32 and float64 oracle runs
disagree); every category is printed.  Eq. 2 and RQ1 (Table 3: no
inconsistent output) are the statements these check.
"""

import os

import numpy as np
import pytest

from oracle import dycl_oracle as O
from tests._parity import compare, load_golden, oracle_ref
from workloads import configs

pytestmark = pytest.mark.gpu

SMALL = {"mlp_exit": 37, "resnet18_exit": 37, "skipnet38": 45, "resnet50_exit": 5, "act_loop": 300,
         "lstm_decoder": 77}
LITERAL = ["mlp_exit", "resnet18_exit", "skipnet38", "resnet50_exit"]

_cache = {}


def _rt():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2307_04963_amd import runtime
    return runtime


def _plan(name, wl=None, max_batch=None, literal=False):
    rt = _rt()
    key = (name, max_batch, id(wl) if wl is not None else None, literal)
    if key not in _cache:
        wl = wl or configs.build(name, calibrated=not literal)
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
        bound = wl.arch["max_steps"] if fam == "act" else wl.arch["max_len"]
        for t, (halt, stay) in enumerate(counts):
            assert halt == int((gpu["iterations"] == t + 1).sum())
        assert gpu["iterations"].min() >= 1 and gpu["iterations"].max() <= bound
        if fam == "seq_decoder":   # tokens up to each sample's length, -1 after it
            L = np.arange(bound)[None, :]
            assert ((gpu["tokens"] >= 0) == (L < gpu["iterations"][:, None])).all()


@pytest.mark.parametrize("name", configs.NAMES)
def test_small_batch_parity(name):
    rt = _rt()
    wl, plan = _plan(name)
    B = SMALL[name]
    print(f"[parity-small] {name} B={B}", flush=True)
    x, aux = wl.inputs(B)
    gpu = rt.run_numpy(plan, wl, x, aux)
    xf, auxf = wl.inputs_f32(B)
    ref = oracle_ref(wl, xf, auxf)
    rep = compare(wl, gpu, ref)
    print(name, rep, flush=True)
    assert rep["ok"], rep
    _check_counts(wl, gpu)


def _full_batch(name, literal):
    rt = _rt()
    wl, plan = _plan(name, literal=literal)
    B = configs.DEFAULT_BATCH[name]
    ref = load_golden(wl, literal)
    print(f"[parity-full] {name}{' literal' if literal else ''} B={B} every row, device host mode", flush=True)
    x, aux = wl.inputs(B)
    plan.set_host_mode("device")
    try:
        gpu = rt.run_numpy(plan, wl, x, aux)
    finally:
        plan.set_host_mode("sync")
    dump = os.environ.get("DYCL_PARITY_DUMP")
    if dump:   # the GPU results, for inspection beside the stored oracle results
        os.makedirs(dump, exist_ok=True)
        np.savez_compressed(os.path.join(dump, f"{name}{'_literal' if literal else ''}.npz"),
                            **{k: v for k, v in gpu.items() if k != "counts"})
    return wl, gpu, ref


@pytest.mark.parametrize("name", configs.NAMES)
def test_full_batch_every_row_parity(name):
    wl, gpu, ref = _full_batch(name, False)
    rep = compare(wl, gpu, ref)
    print(name, rep, "counts", gpu["counts"], flush=True)
    assert rep["samples"] == configs.DEFAULT_BATCH[name]
    assert rep["ok"], rep
    _check_counts(wl, gpu)


@pytest.mark.parametrize("name", LITERAL)
def test_literal_variant_full_batch_parity(name):
    """The literal reading of the workload descriptions (BatchNorm at its
    eval defaults, heads and gates as drawn).  Its logits reach 10^2-10^3,
    where 2e-2 absolute is below float32's own spacing; the logits bound is
    four times the distance between the oracle's float32- and
    float64-accumulating runs (the floor of two correct accumulation orders),
    and never below 2e-2.  Routing is held to the same rule as everywhere."""
    wl, gpu, ref = _full_batch(name, True)
    tol = max(2e-2, 4.0 * float(ref["logit_floor_f32_vs_f64"]))
    rep = compare(wl, gpu, ref, logit_tol=tol)
    print(name, "literal", rep, "counts", gpu["counts"], flush=True)
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


@pytest.mark.parametrize("shift,length", [(1e4, 1), (-1e4, 24)])
def test_forced_end_token_decoder(shift, length):
    # the end token always / never the most likely: every sequence is one
    # token long / runs to the length bound, in every host mode
    rt = _rt()
    wl = configs.build("lstm_decoder")
    b = wl.tensors["out.b"]
    v = b.value.copy()
    v[wl.arch["eos"]] += np.float32(shift)
    wl.tensors["out.b"] = configs.Tensor(b.name, b.dtype, b.shape, v)
    _, plan = _plan("lstm_decoder", wl, 64)
    x, _ = wl.inputs(40)
    ref = oracle_ref(wl, *wl.inputs_f32(40))
    for mode in ("sync", "device", "graph"):
        print(f"[decoder-forced] shift={shift} mode={mode}", flush=True)
        plan.set_host_mode(mode)
        try:
            gpu = rt.run_numpy(plan, wl, x)
        finally:
            plan.set_host_mode("sync")
        assert (gpu["iterations"] == length).all()
        if length == 1:
            assert (gpu["tokens"][:, 0] == wl.arch["eos"]).all() and (gpu["tokens"][:, 1:] == -1).all()
        else:
            assert (gpu["tokens"] != wl.arch["eos"]).all() and (gpu["tokens"] >= 0).all()
        rep = compare(wl, gpu, ref)
        assert rep["ok"], rep
