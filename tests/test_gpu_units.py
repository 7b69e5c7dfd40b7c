"""Kernel-level GPU checks on hand-built specs (single conv + classifier):
stems on narrow inputs (padded to 8 channels inside the plan) and wide
inputs, fused and unfused exit heads, against a numpy float64 reference
with the same bf16 storage points."""

import json

import numpy as np
import pytest

from workloads.configs import bf16_bits_to_f32, to_bf16_bits

pytestmark = pytest.mark.gpu


def q(v):
    return bf16_bits_to_f32(to_bf16_bits(np.asarray(v, np.float32))).astype(np.float64)


def conv(x, w, s, p):
    H, W, Ci = x.shape
    Co, k, _, _ = w.shape
    xp = np.zeros((H + 2 * p, W + 2 * p, Ci))
    xp[p:p + H, p:p + W] = x
    Ho, Wo = (H + 2 * p - k) // s + 1, (W + 2 * p - k) // s + 1
    y = np.zeros((Ho, Wo, Co))
    for i in range(k):
        for j in range(k):
            y += xp[i:i + s * (Ho - 1) + 1:s, j:j + s * (Wo - 1) + 1:s] @ w[:, i, j, :].T
    return y


@pytest.mark.parametrize("cin,ncls,k,stride", [(3, 10, 3, 1), (8, 10, 3, 1), (3, 2000, 3, 1), (16, 10, 3, 2),
                                               (3, 10, 7, 2), (64, 100, 1, 1)])
def test_single_conv_and_classifier(cin, ncls, k, stride):
    import torch
    from paper_2307_04963_amd import runtime
    rng = np.random.default_rng(cin * 1000 + ncls + k)
    B, HW, cout = 5, 12, 16
    blob, man = bytearray(), {}

    def add(name, arr, dt):
        blob.extend(b"\0" * ((-len(blob)) % 256))
        man[name] = len(blob)
        blob.extend(to_bf16_bits(arr).tobytes() if dt == "bf16" else np.asarray(arr, np.float32).tobytes())

    w = q(rng.uniform(-0.5, 0.5, (cout, k, k, cin)))
    a = rng.uniform(0.5, 1.5, cout).astype(np.float32)
    b = rng.uniform(-0.2, 0.2, cout).astype(np.float32)
    add("w", w, "bf16"); add("a", a, "f32"); add("b", b, "f32")
    hw = rng.uniform(-1, 1, (ncls, cout)).astype(np.float32)
    hb = rng.uniform(-1, 1, ncls).astype(np.float32)
    add("hw", hw, "f32"); add("hb", hb, "f32")
    spec = {"version": 1, "dtype": "bf16", "input": {"name": "x", "shape": [HW, HW, cin]}, "n_out": ncls,
            "nodes": [{"op": "conv", "src": "x", "dst": "y", "k": k, "stride": stride, "pad": k // 2, "cout": cout,
                       "act": "relu", "w": {"off": man["w"]}, "scale": man["a"], "shift": man["b"]},
                      {"op": "exit", "src": "y", "w": man["hw"], "b": man["hb"], "ncls": ncls, "index": 0,
                       "final": True}]}
    plan = runtime.Plan(json.dumps(spec), bytes(blob), 8)
    x = q(rng.standard_normal((B, HW, HW, cin)))
    xt = torch.from_numpy(to_bf16_bits(x.astype(np.float32)).view(np.int16).copy()).view(torch.bfloat16).cuda()
    logits = torch.zeros((B, ncls), device="cuda")
    rec = torch.zeros((B, 4), dtype=torch.int32, device="cuda")
    plan.run(xt, None, logits, rec)
    torch.cuda.synchronize()
    got = logits.cpu().numpy()
    ref = []
    for i in range(B):
        y = q(np.maximum(conv(x[i], w, stride, k // 2) * a + b, 0.0))
        ref.append(hw.astype(np.float64) @ y.reshape(-1, cout).mean(0) + hb)
    ref = np.stack(ref)
    # one bf16 rounding of y may flip between accumulation orders: bound by a
    # few bf16 ulps of the pooled features propagated through the head
    assert np.abs(got - ref).max() <= 1e-3 * max(1.0, np.abs(ref).max()), np.abs(got - ref).max()
    assert (rec.cpu().numpy()[:, 0] == 0).all()


@pytest.mark.parametrize("stride,tiny", [(1, False), (2, False), (1, True)])
def test_folded_projection_with_zero_scales(stride, tiny):
    # h = relu(1x1(x)) and the projection p = 1x1(x) (linear), both at
    # `stride`; y = relu(1x1(h) + p) with a third of the block's scales 0:
    # the plan folds p into y's convolution (the projection's K steps
    # first, its sum scaled, shifted and rounded to bf16 as the unfused
    # projection stores it, then carried into the block's sum; a channel of
    # scale 0 keeps only p).  The reference keeps the unfused layers, so the
    # two differ only by accumulation order.  `tiny`: one block scale is an
    # fp32 denormal, whose inverse would overflow; the plan must not fold
    # then, and the result stays finite and equal.
    import torch
    from paper_2307_04963_amd import runtime
    rng = np.random.default_rng(70 + stride)
    B, HW, cin, cmid, cout, ncls = 5, 8, 64, 64, 64, 10
    blob, man = bytearray(), {}

    def add(name, arr, dt):
        blob.extend(b"\0" * ((-len(blob)) % 256))
        man[name] = len(blob)
        blob.extend(to_bf16_bits(arr).tobytes() if dt == "bf16" else np.asarray(arr, np.float32).tobytes())

    wh = q(rng.uniform(-0.3, 0.3, (cmid, 1, 1, cin)))
    wp = q(rng.uniform(-0.3, 0.3, (cout, 1, 1, cin)))
    wc = q(rng.uniform(-0.3, 0.3, (cout, 1, 1, cmid)))
    ah, bh = rng.uniform(0.5, 1.5, cmid).astype(np.float32), rng.uniform(-0.2, 0.2, cmid).astype(np.float32)
    ap, bp = rng.uniform(0.5, 1.5, cout).astype(np.float32), rng.uniform(-0.2, 0.2, cout).astype(np.float32)
    ac, bc = rng.uniform(0.5, 1.5, cout).astype(np.float32), rng.uniform(-0.2, 0.2, cout).astype(np.float32)
    ac[::3] = 0.0
    if tiny:
        ac[1] = 1e-40
    for name, arr, dt in (("wh", wh, "bf16"), ("wp", wp, "bf16"), ("wc", wc, "bf16"), ("ah", ah, "f32"),
                          ("bh", bh, "f32"), ("ap", ap, "f32"), ("bp", bp, "f32"), ("ac", ac, "f32"),
                          ("bc", bc, "f32")):
        add(name, arr, dt)
    hw = rng.uniform(-1, 1, (ncls, cout)).astype(np.float32)
    hb = rng.uniform(-1, 1, ncls).astype(np.float32)
    add("hw", hw, "f32"); add("hb", hb, "f32")
    spec = {"version": 1, "dtype": "bf16", "input": {"name": "x", "shape": [HW, HW, cin]}, "n_out": ncls,
            "nodes": [{"op": "conv", "src": "x", "dst": "h", "k": 1, "stride": stride, "cout": cmid, "act": "relu",
                       "w": {"off": man["wh"]}, "scale": man["ah"], "shift": man["bh"]},
                      {"op": "conv", "src": "x", "dst": "p", "k": 1, "stride": stride, "cout": cout, "act": "none",
                       "w": {"off": man["wp"]}, "scale": man["ap"], "shift": man["bp"]},
                      {"op": "conv", "src": "h", "dst": "y", "k": 1, "cout": cout, "act": "relu", "res": "p",
                       "w": {"off": man["wc"]}, "scale": man["ac"], "shift": man["bc"]},
                      {"op": "exit", "src": "y", "w": man["hw"], "b": man["hb"], "ncls": ncls, "index": 0,
                       "final": True}]}
    plan = runtime.Plan(json.dumps(spec), bytes(blob), 8)
    print(f"[fold] stride={stride} tiny={tiny}", flush=True)
    x = q(rng.standard_normal((B, HW, HW, cin)))
    xt = torch.from_numpy(to_bf16_bits(x.astype(np.float32)).view(np.int16).copy()).view(torch.bfloat16).cuda()
    logits = torch.zeros((B, ncls), device="cuda")
    rec = torch.zeros((B, 4), dtype=torch.int32, device="cuda")
    plan.run(xt, None, logits, rec)
    torch.cuda.synchronize()
    got = logits.cpu().numpy()
    ref = []
    for i in range(B):
        h = q(np.maximum(conv(x[i], wh, stride, 0) * ah + bh, 0.0))
        p = q(conv(x[i], wp, stride, 0) * ap + bp)
        y = q(np.maximum(conv(h, wc, 1, 0) * ac + bc + p, 0.0))
        ref.append(hw.astype(np.float64) @ y.reshape(-1, cout).mean(0) + hb)
    ref = np.stack(ref)
    assert np.isfinite(got).all()
    # one bf16 rounding of y (or of p) may flip between accumulation orders
    assert np.abs(got - ref).max() <= 1e-3 * max(1.0, np.abs(ref).max()), np.abs(got - ref).max()
    plan.close()
