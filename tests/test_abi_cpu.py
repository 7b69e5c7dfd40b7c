"""C-ABI checks that need no GPU: the library loads, exports what the
header declares, and rejects bad specs / sizes / pointers before any HIP
call; the front-end lowers every workload to a spec the host-side
validator accepts with the expected HCFG shape."""

import ctypes as C
import json
import os
import re

import pytest

from paper_2307_04963_amd import _lib, lowering
from workloads import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
lib = _lib.lib


def _declared(header):
    with open(os.path.join(ROOT, "include", header)) as f:
        text = f.read()
    # function declarations only (return type at the start of the line)
    return sorted(set(re.findall(r"^(?:int|size_t|void|const char\s*\*)\s*(dycl_[a-z_]+)\s*\(", text, re.M)))


def test_exports_match_headers():
    for header, exported in (("dycl.h", _lib.EXPORTS), ("dycl_ops.h", _lib.OPS_EXPORTS)):
        names = _declared(header)
        assert names == sorted(exported), header
        for n in names:
            assert hasattr(lib, n), n


def test_ops_reject_bad_arguments_without_gpu():
    assert lib.dycl_op_compact_workspace(0) == 0
    assert lib.dycl_op_compact_workspace(100) == 0
    assert lib.dycl_op_compact_workspace(1 << 20) >= (1 << 20) // 8192 * 8   # one status word per block
    assert lib.dycl_op_compact(None, None, -1, None, None, None, None, None, None, 0, None) == -1
    assert lib.dycl_op_compact(None, None, 5, None, None, None, None, None, None, 0, None) == -1
    assert lib.dycl_op_move_rows(None, None, None, None, 16, 3, None) == -1
    assert lib.dycl_op_move_rows(C.c_void_p(16), None, C.c_void_p(32), None, 24, 3, None) == -1   # row_bytes % 16
    assert lib.dycl_op_move_rows(None, None, None, None, 16, 0, None) == 0
    # the allocation-free compaction rejects sizes beyond its static scratch
    # and bad pointers before touching a device
    big = lib.DYCL_OP_COMPACT_NOALLOC_MAX_N if hasattr(lib, "DYCL_OP_COMPACT_NOALLOC_MAX_N") else (1 << 28)
    assert lib.dycl_op_compact_noalloc(None, None, big + 1, None, None, None, None, C.c_void_p(16), None) == -1
    assert "static scratch" in _lib.last_error()
    assert lib.dycl_op_compact_noalloc(None, None, -1, None, None, None, None, C.c_void_p(16), None) == -1
    assert lib.dycl_op_compact_noalloc(None, None, 5, None, None, None, None, C.c_void_p(16), None) == -1
    assert lib.dycl_op_compact_noalloc(None, None, 5, None, None, None, None, None, None) == -1
    assert lib.dycl_op_compact_noalloc(C.c_void_p(17), None, 5, C.c_void_p(64), None, C.c_void_p(64), None,
                                       C.c_void_p(64), None) == -1                     # misaligned flags


def _check(spec, blob_bytes, max_batch=8):
    buf = C.create_string_buffer(512)
    rc = lib.dycl_spec_check(spec.encode() if isinstance(spec, str) else spec, blob_bytes, max_batch, buf, 512)
    return rc, (buf.value.decode() if rc == 0 else _lib.last_error())


@pytest.mark.parametrize("name", configs.NAMES)
def test_every_workload_spec_validates(name):
    wl = configs.build(name)
    blob, man = wl.blob()
    spec = lowering.lower(wl.arch, man)
    rc, msg = _check(json.dumps(spec), len(blob), configs.DEFAULT_BATCH[name])
    assert rc == 0, msg
    decisions = int(re.search(r"decisions=(\d+)", msg).group(1))
    want = {"mlp_exit": 3, "resnet18_exit": 4, "skipnet38": 19, "resnet50_exit": 4, "act_loop": 16,
            "lstm_decoder": 24}[name]
    assert decisions == want
    # row moves fused into the convolutions: exit carries read in place, gate
    # gathers / scatters of bodies that run on the implicit GEMM
    fg = int(re.search(r"fused_gathers=(\d+)", msg).group(1))
    fgt = int(re.search(r"fused_gates=(\d+)", msg).group(1))
    assert (fg, fgt) == {"mlp_exit": (0, 0), "resnet18_exit": (3, 0), "skipnet38": (0, 18),
                         "resnet50_exit": (3, 0), "act_loop": (30, 0), "lstm_decoder": (23, 0)}[name]
    # the ImageNet stem's max-pool runs in the stem kernel's epilogue
    fp = int(re.search(r"fused_pools=(\d+)", msg).group(1))
    assert fp == (1 if name == "resnet50_exit" else 0)
    # each stage's projection shortcut (stride 1, then 2) folds into its block's last 1x1 conv
    fpr = int(re.search(r"fused_projections=(\d+)", msg).group(1))
    assert fpr == (4 if name == "resnet50_exit" else 0)
    # block boundaries run as one-launch pairs: both of the first stage (256 -> 64
    # channels, one with a folded projection) and the two plain ones of the second
    # (512 -> 128)
    fpa = int(re.search(r"fused_pairs=(\d+)", msg).group(1))
    assert fpa == (4 if name == "resnet50_exit" else 0)
    # the bounded loop is unrolled: one halting test per step (Sec. 5.2 rewriting)
    if name == "act_loop":
        assert sum(n["op"] == "halt" for n in spec["nodes"]) == 16


def test_exit_gathers_fused_only_into_plain_conv_readers():
    # an exit's carried copy is never made when only convolutions read it,
    # as their main input, before the next decision; any other reader (a
    # residual here) keeps the copy
    wl = configs.build("resnet18_exit")
    blob, man = wl.blob()
    spec = lowering.lower(wl.arch, man)
    rc, msg = _check(json.dumps(spec), len(blob), 64)
    assert rc == 0 and "fused_gathers=3" in msg, msg
    # a carried tensor that is also a residual keeps its copy
    toy = {"version": 1, "dtype": "bf16", "input": {"name": "x", "shape": [8, 8, 64]}, "n_out": 10, "nodes": [
        {"op": "conv", "src": "x", "dst": "a", "k": 1, "cout": 64, "act": "relu", "w": {"off": 0}},
        {"op": "exit", "src": "a", "w": 8192, "b": 8192 + 2560, "T": 8192 + 2600, "ncls": 10, "tau": 0.5,
         "index": 0, "final": False, "carry": [["a", "ac"]]},
        {"op": "conv", "src": "ac", "dst": "b", "k": 1, "cout": 64, "act": "relu", "w": {"off": 0}},
        {"op": "conv", "src": "b", "dst": "c", "k": 1, "cout": 64, "act": "relu", "w": {"off": 0}, "res": "ac"},
        {"op": "exit", "src": "c", "w": 8192, "b": 8192 + 2560, "ncls": 10, "index": 1, "final": True}]}
    rc, msg = _check(json.dumps(toy), 16384)
    assert rc == 0 and "fused_gathers=0" in msg, msg
    toy["nodes"][3]["res"] = None
    rc, msg = _check(json.dumps(toy), 16384)
    assert rc == 0 and "fused_gathers=1" in msg, msg


def test_stem_pool_fused_only_when_the_pool_is_the_only_reader():
    # 7x7 / 2 ReLU stem on a 3-channel input, then a 3x3 / 2 max-pool
    wb = 64 * 147 * 2
    head = {"op": "exit", "w": wb, "b": wb + 64 * 10 * 4, "ncls": 10, "index": 0, "final": True}

    def spec(act="relu", extra_reader=False):
        nodes = [{"op": "conv", "src": "x", "dst": "s", "k": 7, "stride": 2, "pad": 3, "cout": 64, "act": act,
                  "w": {"off": 0}},
                 {"op": "maxpool", "src": "s", "dst": "p"},
                 dict(head, src="p")]
        if extra_reader:
            nodes.insert(2, {"op": "conv", "src": "s", "dst": "t", "k": 1, "cout": 64, "act": "relu",
                             "w": {"off": 0, "ldk": 147, "k0": 0}})
        return {"version": 1, "dtype": "bf16", "input": {"name": "x", "shape": [64, 64, 3]}, "n_out": 10,
                "nodes": nodes}

    nb = wb + 64 * 10 * 4 + 64
    for sp, want in ((spec(), 1), (spec(act="none"), 0), (spec(extra_reader=True), 0)):
        rc, msg = _check(json.dumps(sp), nb)
        assert rc == 0, msg
        assert f"fused_pools={want}" in msg, msg


def test_projection_folded_only_into_its_sole_linear_reader():
    # h = relu(conv1x1(x)); p = conv1x1(x) (the projection); y = relu(conv1x1(h) + p)
    wb = 64 * 64 * 2

    def spec(p_act="none", p_stride=1, extra_reader=False, decision_between=False):
        head = {"op": "exit", "w": wb, "b": wb + 64 * 10 * 4, "ncls": 10, "final": True}
        nodes = [{"op": "conv", "src": "x", "dst": "h", "k": 1, "cout": 64, "act": "relu", "w": {"off": 0}},
                 {"op": "conv", "src": "x", "dst": "p", "k": 1, "stride": p_stride, "cout": 64, "act": p_act,
                  "w": {"off": 0}},
                 {"op": "conv", "src": "h" if p_stride == 1 else "hs", "dst": "y", "k": 1, "cout": 64,
                  "act": "relu", "w": {"off": 0}, "res": "p"},
                 dict(head, src="y", index=1)]
        if p_stride != 1:
            nodes.insert(2, {"op": "conv", "src": "h", "dst": "hs", "k": 1, "stride": 2, "cout": 64, "act": "relu",
                             "w": {"off": 0}})
        if extra_reader:
            nodes.insert(-1, {"op": "conv", "src": "p", "dst": "z", "k": 1, "cout": 64, "act": "relu",
                              "w": {"off": 0}})
            nodes[-1]["src"] = "z"
        if decision_between:
            nodes.insert(2, dict(head, src="p", final=False, tau=0.5, index=0, T=wb + 64 * 10 * 4,
                                 carry=[["h", "hc"], ["p", "pc"]]))
            nodes[3]["src"], nodes[3]["res"] = "hc", "pc"
        return {"version": 1, "dtype": "bf16", "input": {"name": "x", "shape": [8, 8, 64]}, "n_out": 10,
                "nodes": nodes}

    nb = wb + 64 * 10 * 4 + 64
    cases = ((spec(), 1), (spec(p_act="relu"), 0), (spec(p_stride=2), 1), (spec(extra_reader=True), 0),
             (spec(decision_between=True), 0))
    for sp, want in cases:
        rc, msg = _check(json.dumps(sp), nb)
        assert rc == 0, msg
        assert f"fused_projections={want}" in msg, (want, msg)


def test_pointwise_pairs_only_where_the_second_reads_only_the_first():
    # y = relu(bn(conv1x1(x, 64 -> 256)) + r); z = relu(bn(conv1x1(y, 256 -> 64)))
    w3 = 256 * 64 * 2
    w1 = 64 * 256 * 2
    vec = w3 + w1                       # four float32 vectors, 256 floats apart
    head_w = vec + 4 * 256 * 4

    def spec(second_res=False, second_k=1, c3=256, first_res=True, switch=None, between=False):
        v = lambda i: vec + i * 1024  # noqa: E731
        nodes = [{"op": "conv", "src": "x", "dst": "r", "k": 1, "cout": c3, "act": "relu", "w": {"off": 0}},
                 {"op": "conv", "src": "r", "dst": "a", "k": 1, "cout": 64, "act": "relu", "w": {"off": w3}},
                 {"op": "conv", "src": "a", "dst": "y", "k": 1, "cout": c3, "act": "relu", "w": {"off": 0},
                  "scale": v(0), "shift": v(1), "res": "r" if first_res else None},
                 {"op": "conv", "src": "y", "dst": "z", "k": second_k, "pad": second_k // 2, "cout": 64,
                  "act": "relu", "w": {"off": w3}, "scale": v(2), "shift": v(3),
                  "res": "a" if second_res else None},
                 {"op": "exit", "src": "z", "w": head_w, "b": head_w + 64 * 10 * 4, "ncls": 10, "index": 0,
                  "final": True}]
        if between:
            nodes.insert(3, {"op": "maxpool", "src": "y", "dst": "yp"})
            nodes[4]["src"] = "yp"
        sp = {"version": 1, "dtype": "bf16", "input": {"name": "x", "shape": [8, 8, 64]}, "n_out": 10,
              "nodes": nodes}
        if switch is not None:
            sp["pair_pointwise"] = switch
        return sp

    nb = head_w + 64 * 10 * 4 + 64 + 64 * 256 * 9 * 2
    cases = ((spec(), 1), (spec(first_res=False), 1), (spec(switch=False), 0), (spec(second_res=True), 0),
             (spec(second_k=3), 0), (spec(c3=128), 0), (spec(between=True), 0))
    for sp, want in cases:
        rc, msg = _check(json.dumps(sp), nb)
        assert rc == 0, msg
        assert f"fused_pairs={want}" in msg, (want, msg)


def _mlp_spec():
    wl = configs.build("mlp_exit")
    blob, man = wl.blob()
    return lowering.lower(wl.arch, man), len(blob)


def test_error_paths_before_any_hip_call():
    spec, nb = _mlp_spec()
    assert _check("{not json", nb)[0] == -2
    assert _check(json.dumps(spec), nb - 4096)[0] == -3           # blob too small
    assert _check(json.dumps(spec), nb, max_batch=0)[0] == -4
    bad = json.loads(json.dumps(spec))
    bad["nodes"][0]["src"] = "nope"
    rc, msg = _check(json.dumps(bad), nb)
    assert rc == -2 and "unknown tensor" in msg
    # a tensor from before an exit, used after it without being carried
    bad = json.loads(json.dumps(spec))
    bad["nodes"][2]["src"] = bad["nodes"][0]["dst"]
    rc, msg = _check(json.dumps(bad), nb)
    assert rc == -2 and "carry" in msg
    bad = json.loads(json.dumps(spec))
    bad["nodes"][0]["k"] = 5
    assert _check(json.dumps(bad), nb)[0] == -2
    assert lib.dycl_spec_check(None, 0, 1, None, 0) == -1


def test_plan_create_rejects_bad_arguments_without_gpu():
    spec, nb = _mlp_spec()
    out = C.c_void_p()
    blob = C.create_string_buffer(nb)
    assert lib.dycl_plan_create(None, blob, nb, 8, 0, C.byref(out)) == -1
    assert lib.dycl_plan_create(json.dumps(spec).encode(), blob, nb, 0, 0, C.byref(out)) == -4
    assert lib.dycl_plan_create(b"[]", blob, nb, 8, 0, C.byref(out)) == -2
    assert out.value is None
    assert lib.dycl_run(None, None, 1, None, None, None, None) == -1
    assert lib.dycl_last_counts(None, None, 0) == -1
    assert lib.dycl_plan_set_host_mode(None, 1) == -1
    assert lib.dycl_plan_info(None, None, 0) == -1
    lib.dycl_plan_destroy(None)
    assert lib.dycl_profile_class(99) == b""
    assert lib.dycl_profile_class(0) == b"conv_bf16_mfma"


def test_conv_pack_and_validation():
    """dycl_op_conv_pack lays out [cout_pad][Kp] with zero padding; the conv
    entry point rejects bad arguments before touching the device."""
    import ctypes as C

    import numpy as np
    from paper_2307_04963_amd import _lib
    lib = _lib.lib
    assert lib.dycl_op_conv_packed_bytes(64, 3, 64) == 64 * 576 * 2
    assert lib.dycl_op_conv_packed_bytes(24, 3, 3) == 32 * 64 * 2        # K 27 -> 64, Cout 24 -> 32
    assert lib.dycl_op_conv_packed_bytes(300, 1, 100) == 512 * 128 * 2   # Cout >= 256 pads to 256s
    assert lib.dycl_op_conv_packed_bytes(64, 5, 64) == 0
    assert lib.dycl_op_conv_packed_bytes(0, 3, 64) == 0
    rng = np.random.default_rng(0)
    w = rng.integers(0, 65535, (24, 3, 3, 3), dtype=np.uint16)
    nb = lib.dycl_op_conv_packed_bytes(24, 3, 3)
    out = np.full(nb // 2, 7, np.uint16)
    assert lib.dycl_op_conv_pack(w.ctypes.data, 24, 3, 3, out.ctypes.data, nb) == 0
    ref = np.zeros((32, 64), np.uint16)
    ref[:24, :27] = w.reshape(24, 27)
    assert (out.reshape(32, 64) == ref).all()
    assert lib.dycl_op_conv_pack(w.ctypes.data, 24, 3, 3, out.ctypes.data, nb - 2) == -1
    assert lib.dycl_op_conv_pack(None, 24, 3, 3, out.ctypes.data, nb) == -1
    p16 = C.c_void_p(256)
    args = lambda **kw: [kw.get("x", p16), kw.get("n", 2), 8, 8, 64, kw.get("w", p16), 64, kw.get("k", 3),  # noqa: E731
                         kw.get("s", 1), kw.get("pad", 1), None, None, kw.get("res"), kw.get("act", 1),
                         kw.get("y", p16), kw.get("ws"), kw.get("wsb", 0), None]
    assert lib.dycl_op_conv(*args(n=-1)) == -1
    assert lib.dycl_op_conv(*args(k=5)) == -1
    assert lib.dycl_op_conv(*args(pad=3)) == -1
    assert lib.dycl_op_conv(*args(act=3)) == -1
    assert lib.dycl_op_conv(*args(x=None)) == -1
    assert lib.dycl_op_conv(*args(y=C.c_void_p(258))) == -1               # misaligned
    assert lib.dycl_op_conv(*args(res=C.c_void_p(264))) == -1
    assert "aligned" in _lib.last_error()
    assert lib.dycl_op_conv(*args(ws=C.c_void_p(264), wsb=4096)) == -1   # misaligned workspace
    assert lib.dycl_op_conv(*args(n=0)) == 0                              # nothing to do
    # K split workspace: deep K on at most 64 output pixels per image only,
    # sized by S * n * Ho * Wo * cout fp32
    assert lib.dycl_op_conv_workspace_bytes(255, 14, 14, 512, 512, 3, 2, 1) == 4 * 255 * 49 * 512 * 4
    assert lib.dycl_op_conv_workspace_bytes(255, 6, 6, 4608, 256, 1, 1, 0) == 4 * 255 * 36 * 256 * 4
    assert lib.dycl_op_conv_workspace_bytes(255, 4, 4, 512, 512, 3, 1, 1) == 4 * 255 * 16 * 512 * 4
    assert lib.dycl_op_conv_workspace_bytes(255, 8, 8, 512, 512, 3, 2, 1) == 4 * 255 * 16 * 512 * 4
    assert lib.dycl_op_conv_workspace_bytes(255, 8, 8, 256, 512, 3, 2, 1) == 0     # K = 2304
    assert lib.dycl_op_conv_workspace_bytes(255, 16, 16, 512, 512, 3, 1, 1) == 0   # 256 pixels per image
    assert lib.dycl_op_conv_workspace_bytes(255, 4, 4, 128, 512, 3, 1, 1) == 0     # K = 1152
    assert lib.dycl_op_conv_workspace_bytes(255, 4, 4, 512, 128, 3, 1, 1) == 0     # cout < 256
    assert lib.dycl_op_conv_workspace_bytes(0, 4, 4, 512, 512, 3, 1, 1) == 0
    # the fused stem + max-pool takes the ImageNet stem shape with ReLU only
    mp = lambda **kw: lib.dycl_op_conv_maxpool(kw.get("x", p16), kw.get("n", 2), kw.get("H", 32), kw.get("W", 32),  # noqa: E731
                                                kw.get("cin", 3), p16, kw.get("cout", 64), kw.get("k", 7),
                                                kw.get("s", 2), kw.get("pad", 3), None, None, kw.get("act", 1),
                                                kw.get("y", p16), None)
    assert mp(act=0) == -1 and mp(act=2) == -1
    assert mp(cin=8) == -1 and mp(cout=128) == -1 and mp(k=3) == -1 and mp(s=1) == -1
    assert mp(W=36) == -1                                                  # W % 8
    assert mp(W=256) == -1                                                 # rows of more than 112 outputs
    assert mp(n=-1) == -1 and mp(x=None) == -1 and mp(y=C.c_void_p(264)) == -1
    assert mp(n=0) == 0
