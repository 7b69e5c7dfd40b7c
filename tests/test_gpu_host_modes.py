"""The three host modes give the same results.

DYCL_HOST_SYNC reads every decision's branch counts back and launches the
next kernels on exactly that many rows; DYCL_HOST_DEVICE leaves the counts
on the device and launches count-guarded kernels sized for the rows that
reached the decision; DYCL_HOST_GRAPH replays a captured HIP graph of the
device-mode run.  Every kernel takes the same per-element arithmetic at any
launch size, so the modes agree bit for bit: logits, records and branch
counts.  Also checked here: device mode against the oracle, forced routing
in which a branch is empty (kernels launched with no live row), graph
replays over new input contents with eager work between them, and
re-capture when the batch size changes.
"""

import numpy as np
import pytest

from oracle import dycl_oracle as O
from tests._parity import compare, oracle_ref
from workloads import configs

pytestmark = pytest.mark.gpu

SMALL = {"mlp_exit": 37, "resnet18_exit": 37, "skipnet38": 45, "resnet50_exit": 5, "act_loop": 300,
         "lstm_decoder": 77}

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


def _run(rt, plan, wl, x, aux, mode):
    plan.set_host_mode(mode)
    try:
        return rt.run_numpy(plan, wl, x, aux)
    finally:
        plan.set_host_mode("sync")


def _same(a, b):
    assert np.array_equal(a["logits"], b["logits"], equal_nan=True)
    for k in ("exit_index", "iterations", "skip_mask") + (("tokens",) if "tokens" in a else ()):
        assert np.array_equal(a[k], b[k]), k
    assert a["counts"] == b["counts"]


@pytest.mark.parametrize("name", configs.NAMES)
@pytest.mark.parametrize("size", ["small", "full"])
def test_modes_agree_bitwise(name, size):
    rt = _rt()
    wl, plan = _plan(name)
    B = SMALL[name] if size == "small" else configs.DEFAULT_BATCH[name]
    print(f"[host-modes] {name} B={B}", flush=True)
    x, aux = wl.inputs(B)
    ref = _run(rt, plan, wl, x, aux, "sync")
    for mode in ("device", "graph", "persistent"):
        got = _run(rt, plan, wl, x, aux, mode)
        _same(ref, got)
    print(name, "counts", ref["counts"], flush=True)


@pytest.mark.parametrize("name", ["mlp_exit", "resnet18_exit", "skipnet38", "act_loop"])
def test_device_mode_stale_hints(name):
    # device mode picks tile shapes from an earlier run's branch counts; a
    # run whose routing is nothing like the earlier one (every row the same
    # sample, at another batch size) must still give the sync results
    rt = _rt()
    wl, plan = _plan(name)
    B = configs.DEFAULT_BATCH[name]
    x, aux = wl.inputs(B)
    want = _run(rt, plan, wl, x, aux, "sync")
    xs = np.repeat(x[:1], 33, axis=0)
    auxs = np.repeat(aux[:1], 33, axis=0) if aux is not None else None
    plan.set_host_mode("device")
    try:
        rt.run_numpy(plan, wl, xs, auxs)          # skewed counts become the hint
        got = rt.run_numpy(plan, wl, x, aux)
    finally:
        plan.set_host_mode("sync")
    _same(want, got)


@pytest.mark.parametrize("name", configs.NAMES)
def test_device_mode_oracle_parity(name):
    rt = _rt()
    wl, plan = _plan(name)
    B = SMALL[name]
    print(f"[device-parity] {name} B={B}", flush=True)
    x, aux = wl.inputs(B)
    gpu = _run(rt, plan, wl, x, aux, "device")
    xf, auxf = wl.inputs_f32(B)
    ref = oracle_ref(wl, xf, auxf)
    rep = compare(wl, gpu, ref)
    print(name, rep, flush=True)
    assert rep["ok"], rep


def test_large_batch_partition_all_modes():
    # above 16384 rows a decision's partition takes the chained single-pass
    # kernel; device and graph modes hand it the live count on the device
    rt = _rt()
    B = 40000
    wl, plan = _plan("mlp_exit", max_batch=B)
    print(f"[host-modes] mlp_exit B={B} (large partition)", flush=True)
    x, aux = wl.inputs(B)
    ref = _run(rt, plan, wl, x, aux, "sync")
    for mode in ("device", "graph"):
        _same(ref, _run(rt, plan, wl, x, aux, mode))
    rows = np.arange(0, B, 37)
    xf, auxf = wl.inputs_f32(B)
    oref = oracle_ref(wl, xf[rows], None if auxf is None else auxf[rows])
    rep = compare(wl, ref, oref, rows=rows)
    print(rep, flush=True)
    assert rep["ok"], rep


@pytest.mark.parametrize("tau,want", [(0.0, 0), (1.5, 2)])
def test_device_mode_forced_exits(tau, want):
    # tau 0: every row leaves at the first head and later kernels find no
    # live row; tau 1.5: nobody leaves before the final head
    rt = _rt()
    wl = configs.build("mlp_exit")
    wl.arch = dict(wl.arch, tau=tau)
    _, plan = _plan("mlp_exit", wl, 64)
    x, _ = wl.inputs(50)
    for mode in ("device", "graph"):
        gpu = _run(rt, plan, wl, x, None, mode)
        assert (gpu["exit_index"] == want).all()
        assert gpu["counts"][want] == (50, 0)
        assert all(c == (0, 0) for c in gpu["counts"][want + 1:])
        assert compare(wl, gpu, O.from_workload(wl).run(x))["ok"]


@pytest.mark.parametrize("v,mask", [(50.0, 0), (-50.0, (1 << 18) - 1)])
def test_device_mode_forced_gates(v, mask):
    rt = _rt()
    wl = configs.build("skipnet38")
    for b in wl.arch["blocks"]:
        t = wl.tensors[b["gate"] + ".v"]
        wl.tensors[b["gate"] + ".v"] = configs.Tensor(t.name, t.dtype, t.shape, np.array([v], dtype=np.float32))
    _, plan = _plan("skipnet38", wl, 64)
    x, _ = wl.inputs(19)
    sync = _run(rt, plan, wl, x, None, "sync")
    for mode in ("device", "graph"):
        gpu = _run(rt, plan, wl, x, None, mode)
        assert (gpu["skip_mask"] == np.uint64(mask)).all()
        _same(sync, gpu)


@pytest.mark.parametrize("bias,steps", [(10.0, 1), (-30.0, 16)])
def test_device_mode_forced_halting(bias, steps):
    rt = _rt()
    wl, plan = _plan("act_loop")
    x, _ = wl.inputs(70)
    aux = np.full(70, bias, dtype=np.float32)
    sync = _run(rt, plan, wl, x, aux, "sync")
    for mode in ("device", "graph"):
        gpu = _run(rt, plan, wl, x, aux, mode)
        assert (gpu["iterations"] == steps).all()
        _same(sync, gpu)


def test_graph_replays_new_contents_and_recaptures():
    # one capture serves every run with the same batch and buffers, whatever
    # the buffers hold, with torch work between the replays; a new batch
    # size captures again
    rt = _rt()
    import torch
    wl, plan = _plan("resnet18_exit")
    B = 96
    xs = [wl.inputs(B, start=start)[0] for start in (0, 500, 1000)]
    wants = [rt.run_numpy(plan, wl, x, None) for x in xs]     # sync mode
    xt = torch.empty((B, 32, 32, 3), dtype=torch.bfloat16, device="cuda")
    logits = torch.empty((B, plan.n_out), device="cuda")
    rec = torch.empty((B, 4), dtype=torch.int32, device="cuda")
    caps0 = plan.info()["graph_captures"]
    plan.set_host_mode("graph")
    try:
        def check(want, b):
            ex, it, sk = rt.decode_records(rec[:b].cpu().numpy())
            got = {"logits": logits[:b].cpu().numpy(), "exit_index": ex, "iterations": it, "skip_mask": sk}
            for k in got:
                assert np.array_equal(got[k], want[k][:b], equal_nan=True), k

        for x, want in zip(xs, wants):
            xt.copy_(rt.device_inputs(wl, x, None)[0])
            logits.fill_(float("nan"))
            rec.fill_(-7)
            plan.run(xt, None, logits, rec)
            junk = torch.randn(2048, 2048, device="cuda") @ torch.randn(2048, 2048, device="cuda")
            torch.cuda.synchronize()
            del junk
            check(want, B)
            assert plan.counts() == want["counts"]
        assert plan.info()["graph_captures"] - caps0 == 1
        # rows are independent: the first 40 rows alone give the same results
        logits.fill_(float("nan"))
        plan.run(xt[:40], None, logits[:40], rec[:40])
        torch.cuda.synchronize()
        check(wants[-1], 40)
        plan.run(xt, None, logits, rec)
        torch.cuda.synchronize()
        check(wants[-1], B)
        assert plan.info()["graph_captures"] - caps0 == 3
    finally:
        plan.set_host_mode("sync")


def test_host_mode_errors():
    _rt()
    from paper_2307_04963_amd._lib import lib
    _, plan = _plan("mlp_exit")
    with pytest.raises(ValueError):
        plan.set_host_mode("async")
    rc = lib.dycl_plan_set_host_mode(plan._h, 7)
    assert rc == -1
    assert plan.set_host_mode("sync") == "sync"
    assert plan.info()["host_mode"] == 0
    assert plan.set_host_mode("device") == "sync"
    assert plan.info()["host_mode"] == 1
    plan.set_host_mode("sync")
