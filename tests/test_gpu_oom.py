"""Plan creation that cannot get its device memory (include/dycl.h,
DYCL_E_OOM): with all but about 2 GiB of the GPU held by another
allocation, a ResNet-50 plan for 2048 images (activation buffers of several
GiB each) cannot be built.  The call returns DYCL_E_OOM with a message
naming the allocation, hands back no plan, frees what it had allocated
(device free memory is where it was, over repeated attempts), and leaves
the runtime usable: once the other allocation is gone, a plan of a normal
size builds and runs."""

import ctypes as C

import pytest

pytestmark = pytest.mark.gpu

DYCL_E_OOM = -5


def test_oversized_plan_returns_oom_and_leaks_nothing():
    import torch
    assert torch.cuda.is_available()
    from paper_2307_04963_amd import _lib, runtime
    from paper_2307_04963_amd.lowering import lower_json
    from workloads import configs

    wl = configs.build("resnet50_exit")
    blob, man = wl.blob()
    spec = lower_json(wl.arch, man).encode()
    buf = C.create_string_buffer(blob, len(blob))
    torch.cuda.synchronize()
    free, _ = torch.cuda.mem_get_info()
    hold = torch.empty(max(free - (2 << 30), 0), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    print(f"[oom] holding {hold.numel() >> 20} MiB, {free0 >> 20} MiB free", flush=True)
    for attempt in range(3):
        print(f"[oom] resnet50_exit max_batch=2048 attempt {attempt}", flush=True)
        h = C.c_void_p(1)
        rc = _lib.lib.dycl_plan_create(spec, C.cast(buf, C.c_void_p), len(blob), 2048, 0, C.byref(h))
        assert rc == DYCL_E_OOM, (rc, _lib.last_error())
        assert not h.value
        assert "hipMalloc" in _lib.last_error()
    torch.cuda.synchronize()
    free1 = torch.cuda.mem_get_info()[0]
    assert abs(free1 - free0) < (64 << 20), (free0, free1)
    del hold
    torch.cuda.empty_cache()

    print("[oom] a normal plan afterwards", flush=True)
    plan = runtime.Plan.from_workload(wl, 4)
    x, aux = wl.inputs(4)
    xt, at = runtime.device_inputs(wl, x, aux)
    logits, rec, tok = plan.outputs(4)
    plan.run(xt, at, logits, rec, torch.cuda.current_stream(), tok)
    torch.cuda.synchronize()
    assert torch.isfinite(logits).all()
    plan.close()
