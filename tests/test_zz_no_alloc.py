"""The allocation-free compaction entry point (static device scratch)
through the C ABI against dycl_op_compact with a caller workspace: two
calls in a row on the same GPU, the second smaller (so the scratch holds the
first call's block offsets when the second starts), then a single-workgroup
size with no id outputs (ids routed into the scratch), then an empty input.
Bit-exact: the two entry points run the same kernels."""

import ctypes as C

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _lib():
    import torch
    assert torch.cuda.is_available()
    from paper_2307_04963_amd import _lib
    return _lib


def _with_workspace(L, f, o, n):
    import torch
    outs = [torch.full((max(n, 1),), -7, dtype=torch.int32, device="cuda") for _ in range(4)]
    counts = torch.full((2,), -9, dtype=torch.int32, device="cuda")
    wsb = L.lib.dycl_op_compact_workspace(n)
    ws = torch.empty(max(wsb, 8), dtype=torch.uint8, device="cuda")
    L.check(L.lib.dycl_op_compact(C.c_void_p(f.data_ptr()), C.c_void_p(o.data_ptr()) if o is not None else None, n,
                                  *[C.c_void_p(t.data_ptr()) for t in outs], C.c_void_p(counts.data_ptr()),
                                  C.c_void_p(ws.data_ptr()), wsb, None))
    return outs, counts


def _noalloc(L, f, o, n, with_ids=True):
    import torch
    outs = [torch.full((max(n, 1),), -7, dtype=torch.int32, device="cuda") for _ in range(4)]
    counts = torch.full((2,), -9, dtype=torch.int32, device="cuda")
    ptr = [C.c_void_p(t.data_ptr()) for t in outs]
    if not with_ids:
        ptr[1] = ptr[3] = None
    L.check(L.lib.dycl_op_compact_noalloc(C.c_void_p(f.data_ptr()), C.c_void_p(o.data_ptr()) if o is not None else None,
                                          n, *ptr, C.c_void_p(counts.data_ptr()), None))
    return outs, counts


@pytest.mark.parametrize("sizes", [((1 << 22) + 4099, 40007, 5000), ((1 << 20) + 7, 16385, 64)])
def test_noalloc_compact_matches_workspace_form(sizes):
    import torch
    L = _lib()
    for step, n in enumerate(sizes):
        print(f"[noalloc] call {step} n={n}", flush=True)
        rng = np.random.default_rng(n)
        flags = (rng.random(n) < 0.37).astype(np.uint8) * rng.integers(1, 256, n).astype(np.uint8)
        f = torch.from_numpy(flags).cuda()
        o = torch.from_numpy(rng.permutation(n).astype(np.int32)).cuda()
        small_no_ids = n <= 16384
        want, wc = _with_workspace(L, f, o, n)
        got, gc = _noalloc(L, f, o, n, with_ids=not small_no_ids)
        torch.cuda.synchronize()
        assert gc.tolist() == wc.tolist()
        c1, c0 = wc.tolist()
        assert c1 + c0 == n and c1 == int((flags != 0).sum())
        for k, m in ((0, c1), (1, c1), (2, c0), (3, c0)):
            if small_no_ids and k in (1, 3):
                continue
            assert torch.equal(got[k][:m], want[k][:m]), (n, k)
        # the partition itself, independently of the other entry point
        np.testing.assert_array_equal(got[0][:c1].cpu().numpy(), np.flatnonzero(flags))
        np.testing.assert_array_equal(got[2][:c0].cpu().numpy(), np.flatnonzero(flags == 0))


def test_noalloc_compact_empty_and_limit():
    import torch
    L = _lib()
    counts = torch.full((2,), -9, dtype=torch.int32, device="cuda")
    L.check(L.lib.dycl_op_compact_noalloc(None, None, 0, None, None, None, None, C.c_void_p(counts.data_ptr()), None))
    torch.cuda.synchronize()
    assert counts.tolist() == [0, 0]
    rc = L.lib.dycl_op_compact_noalloc(None, None, (1 << 28) + 1, None, None, None, None,
                                       C.c_void_p(counts.data_ptr()), None)
    assert rc == -1
