"""Routing primitives through include/dycl_ops.h on the GPU: the stable
two-way partition (single-workgroup form up to 16384 rows, one chained pass
over blocks of 4096 above) bit-exact against numpy at every density (none,
rare, half, all set) and ragged sizes, also on a reused workspace that
starts out dirty, and row gathers / scatters byte-exact."""

import ctypes as C

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _lib():
    import torch
    assert torch.cuda.is_available()
    from paper_2307_04963_amd import _lib
    return _lib


@pytest.mark.parametrize("n", [1, 63, 64, 1000, 4096, 16384, 16385, 100003, (1 << 20) + 7, 1 << 24])
@pytest.mark.parametrize("density", [0.0, 1 / 64, 0.5, 1.0])
def test_compact_is_a_stable_partition(n, density):
    import torch
    L = _lib()
    print(f"[compact] n={n} density={density}", flush=True)
    rng = np.random.default_rng(n + int(density * 1000))
    flags = (rng.random(n) < density).astype(np.uint8) * rng.integers(1, 256, n).astype(np.uint8)
    orig = rng.permutation(n).astype(np.int32)
    f = torch.from_numpy(flags).cuda()
    o = torch.from_numpy(orig).cuda()
    outs = [torch.full((n,), -7, dtype=torch.int32, device="cuda") for _ in range(4)]
    counts = torch.zeros(2, dtype=torch.int32, device="cuda")
    ws_bytes = L.lib.dycl_op_compact_workspace(n)
    ws = torch.zeros(max(ws_bytes, 8), dtype=torch.uint8, device="cuda")
    L.check(L.lib.dycl_op_compact(C.c_void_p(f.data_ptr()), C.c_void_p(o.data_ptr()), n,
                                  *[C.c_void_p(t.data_ptr()) for t in outs], C.c_void_p(counts.data_ptr()),
                                  C.c_void_p(ws.data_ptr()), ws_bytes, None))
    torch.cuda.synchronize()
    ones = np.nonzero(flags)[0].astype(np.int32)
    zeros = np.nonzero(flags == 0)[0].astype(np.int32)
    c = counts.cpu().numpy()
    assert (c[0], c[1]) == (len(ones), len(zeros))
    i1, g1, i0, g0 = [t.cpu().numpy() for t in outs]
    np.testing.assert_array_equal(i1[:len(ones)], ones)
    np.testing.assert_array_equal(g1[:len(ones)], orig[ones])
    np.testing.assert_array_equal(i0[:len(zeros)], zeros)
    np.testing.assert_array_equal(g0[:len(zeros)], orig[zeros])


def test_compact_scan_carries_across_rounds():
    # 2^26 + 4097 rows: 16385 blocks of 4096 flags, so a block's prefix is
    # carried through many look-back windows of 64 blocks, and the last,
    # all-set block starts from the total of all the others
    import torch
    L = _lib()
    n = (1 << 26) + 4097
    print(f"[compact] n={n} (16385 chained blocks)", flush=True)
    rng = np.random.default_rng(26)
    flags = (rng.random(n, dtype=np.float32) < 0.5).astype(np.uint8)
    flags[-4097:] = 1                       # the second round's block: all set
    f = torch.from_numpy(flags).cuda()
    o = torch.arange(n, dtype=torch.int32, device="cuda").flip(0).contiguous()
    outs = [torch.empty((n,), dtype=torch.int32, device="cuda") for _ in range(4)]
    counts = torch.zeros(2, dtype=torch.int32, device="cuda")
    ws_bytes = L.lib.dycl_op_compact_workspace(n)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    L.check(L.lib.dycl_op_compact(C.c_void_p(f.data_ptr()), C.c_void_p(o.data_ptr()), n,
                                  *[C.c_void_p(t.data_ptr()) for t in outs], C.c_void_p(counts.data_ptr()),
                                  C.c_void_p(ws.data_ptr()), ws_bytes, None))
    torch.cuda.synchronize()
    ones = np.flatnonzero(flags).astype(np.int32)
    zeros = np.flatnonzero(flags == 0).astype(np.int32)
    assert counts.cpu().tolist() == [len(ones), len(zeros)]
    i1, g1, i0, g0 = [t.cpu().numpy() for t in outs]
    np.testing.assert_array_equal(i1[:len(ones)], ones)
    np.testing.assert_array_equal(g1[:len(ones)], n - 1 - ones)
    np.testing.assert_array_equal(i0[:len(zeros)], zeros)
    np.testing.assert_array_equal(g0[:len(zeros)], n - 1 - zeros)


def test_compact_reuses_a_dirty_workspace():
    # every call clears the block status words and the ticket it uses: a
    # workspace full of garbage, then reused by a smaller call, gives exact
    # partitions
    import torch
    L = _lib()
    ws_bytes = L.lib.dycl_op_compact_workspace(300007)
    ws = torch.full((ws_bytes,), 0xC3, dtype=torch.uint8, device="cuda")
    for n, density in ((300007, 0.3), (70001, 0.7)):
        print(f"[compact] dirty workspace n={n} density={density}", flush=True)
        rng = np.random.default_rng(n)
        flags = (rng.random(n) < density).astype(np.uint8)
        orig = rng.permutation(n).astype(np.int32)
        f, o = torch.from_numpy(flags).cuda(), torch.from_numpy(orig).cuda()
        outs = [torch.full((n,), -7, dtype=torch.int32, device="cuda") for _ in range(4)]
        counts = torch.zeros(2, dtype=torch.int32, device="cuda")
        L.check(L.lib.dycl_op_compact(C.c_void_p(f.data_ptr()), C.c_void_p(o.data_ptr()), n,
                                      *[C.c_void_p(t.data_ptr()) for t in outs], C.c_void_p(counts.data_ptr()),
                                      C.c_void_p(ws.data_ptr()), ws_bytes, None))
        torch.cuda.synchronize()
        ones, zeros = np.nonzero(flags)[0], np.nonzero(flags == 0)[0]
        assert counts.cpu().tolist() == [len(ones), len(zeros)]
        i1, g1, i0, g0 = [t.cpu().numpy() for t in outs]
        np.testing.assert_array_equal(i1[:len(ones)], ones)
        np.testing.assert_array_equal(g1[:len(ones)], orig[ones])
        np.testing.assert_array_equal(i0[:len(zeros)], zeros)
        np.testing.assert_array_equal(g0[:len(zeros)], orig[zeros])


def test_compact_empty_and_null_ids():
    import torch
    L = _lib()
    counts = torch.full((2,), 5, dtype=torch.int32, device="cuda")
    L.check(L.lib.dycl_op_compact(None, None, 0, None, None, None, None, C.c_void_p(counts.data_ptr()), None, 0,
                                  None))
    torch.cuda.synchronize()
    assert counts.cpu().tolist() == [0, 0]
    n = 50000
    flags = torch.from_numpy((np.arange(n) % 3 == 0).astype(np.uint8)).cuda()
    i1 = torch.empty(n, dtype=torch.int32, device="cuda")
    i0 = torch.empty(n, dtype=torch.int32, device="cuda")
    ws_bytes = L.lib.dycl_op_compact_workspace(n)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    L.check(L.lib.dycl_op_compact(C.c_void_p(flags.data_ptr()), None, n, C.c_void_p(i1.data_ptr()), None,
                                  C.c_void_p(i0.data_ptr()), None, C.c_void_p(counts.data_ptr()),
                                  C.c_void_p(ws.data_ptr()), ws_bytes, None))
    torch.cuda.synchronize()
    k = (n + 2) // 3
    np.testing.assert_array_equal(i1[:k].cpu().numpy(), np.arange(0, n, 3))
    assert counts.cpu().tolist() == [k, n - k]


def test_compact_without_ids_at_full_size():
    # the form the partition itself needs (flags in, row indices out, no
    # ids), at 2^26 + 12345 rows, as the bandwidth measurement runs it
    import torch
    L = _lib()
    n = (1 << 26) + 12345
    print(f"[compact] n={n} without ids", flush=True)
    g = torch.Generator(device="cuda").manual_seed(3)
    f = (torch.rand(n, device="cuda", generator=g) < 0.5).to(torch.uint8)
    i1 = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    i0 = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    counts = torch.zeros(2, dtype=torch.int32, device="cuda")
    ws_bytes = L.lib.dycl_op_compact_workspace(n)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    L.check(L.lib.dycl_op_compact(C.c_void_p(f.data_ptr()), None, n, C.c_void_p(i1.data_ptr()), None,
                                  C.c_void_p(i0.data_ptr()), None, C.c_void_p(counts.data_ptr()),
                                  C.c_void_p(ws.data_ptr()), ws_bytes, None))
    torch.cuda.synchronize()
    flags = f.cpu().numpy()
    ones = np.flatnonzero(flags).astype(np.int32)
    zeros = np.flatnonzero(flags == 0).astype(np.int32)
    assert counts.cpu().tolist() == [len(ones), len(zeros)]
    np.testing.assert_array_equal(i1.cpu().numpy()[:len(ones)], ones)
    np.testing.assert_array_equal(i0.cpu().numpy()[:len(zeros)], zeros)


@pytest.mark.parametrize("row_bytes,n,rows", [(16, 7, 10), (2048, 333, 1000), (128 * 1024, 40, 64)])
def test_gather_and_scatter_rows(row_bytes, n, rows):
    import torch
    L = _lib()
    rng = np.random.default_rng(row_bytes)
    src = torch.from_numpy(rng.integers(0, 256, rows * row_bytes, dtype=np.uint8)).cuda()
    idx = torch.from_numpy(rng.choice(rows, n, replace=False).astype(np.int32)).cuda()
    g = torch.zeros(n * row_bytes, dtype=torch.uint8, device="cuda")
    L.check(L.lib.dycl_op_move_rows(C.c_void_p(g.data_ptr()), None, C.c_void_p(src.data_ptr()),
                                    C.c_void_p(idx.data_ptr()), row_bytes, n, None))
    back = torch.zeros(rows * row_bytes, dtype=torch.uint8, device="cuda")
    L.check(L.lib.dycl_op_move_rows(C.c_void_p(back.data_ptr()), C.c_void_p(idx.data_ptr()),
                                    C.c_void_p(g.data_ptr()), None, row_bytes, n, None))
    torch.cuda.synchronize()
    s = src.cpu().numpy().reshape(rows, row_bytes)
    ii = idx.cpu().numpy()
    np.testing.assert_array_equal(g.cpu().numpy().reshape(n, row_bytes), s[ii])
    b = back.cpu().numpy().reshape(rows, row_bytes)
    np.testing.assert_array_equal(b[ii], s[ii])
    rest = np.setdiff1d(np.arange(rows), ii)
    assert (b[rest] == 0).all()
