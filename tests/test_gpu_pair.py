"""Two 1x1 convolutions in one launch: a bottleneck block's last 1x1 layer
and the next block's first 1x1 layer, which reads nothing but its output
(dycl_op_conv_pair; dycl_run runs such pairs this way by default).

* dycl_op_conv_pair against dycl_op_conv called twice, bit for bit on every
  element (ragged last tile, one row, several K steps, with and without the
  residual, the full ResNet-50 first-stage shape at batch 256; 512 -> 128
  channels in chunks, up to the second-stage shape at the rows that reach
  it), and both of
  its outputs against the oracle's float64 convolutions on sampled images
  within the fp32 accumulation bound (the second layer's reference takes the
  first layer's bf16 output as its input, as the network does).
* The ResNet-50 early-exit plan at its benchmark batch and at 37 images: the same logits,
  records and branch counts with the pairing on and off
  ("pair_pointwise": false), in the sync and device host modes; the pairing
  covers both first-stage boundaries, one of them a block whose projection
  shortcut is folded into the pair's first layer, and the two plain
  second-stage boundaries (512 channels, taken 128 at a time).
"""

import json

import numpy as np
import pytest
import torch

from oracle import dycl_oracle as O
from workloads import configs
from workloads.configs import bf16_bits_to_f32, to_bf16_bits

pytestmark = pytest.mark.gpu


def _bits(a):
    return torch.from_numpy(to_bf16_bits(np.asarray(a, np.float32)).view(np.int16).copy())


def _f64(t):
    return bf16_bits_to_f32(t.cpu().view(torch.int16).numpy().view(np.uint16)).astype(np.float64)


def _check_1x1(x, w, sc, sh, r, got, imgs, what):
    """got[i] against act(sc * (x[i] w^T) + sh (+ r[i])) in float64, ReLU;
    bound: gamma_K * sum |x w| * |sc| + fp32 epilogue roundings + half a bf16
    ulp of the result."""
    K = w.shape[1]
    gamma = K * 2.0 ** -24 / (1 - K * 2.0 ** -24)
    for i in imgs:
        xi = x[i].reshape(-1, K).astype(np.float64)
        acc = xi @ w.T.astype(np.float64)
        mag = np.abs(xi) @ np.abs(w.T.astype(np.float64))
        v = acc * sc + sh + (r[i].reshape(acc.shape) if r is not None else 0.0)
        v = np.maximum(v, 0.0)
        tol = (2.0 ** -8 * 1.001 * np.abs(v) + gamma * mag * np.abs(sc) +
               2.0 ** -22 * (np.abs(acc * sc) + np.abs(sh) + (np.abs(r[i].reshape(acc.shape)) if r is not None else 0)))
        err = np.abs(got[i].reshape(acc.shape) - v)
        bad = np.argwhere(err > tol)
        assert bad.size == 0, f"{what} image {i}: {len(bad)} elements out of bound, first {tuple(bad[0])}"


CASES = [
    # n, H, W, cin, residual, c3, c1
    (2, 7, 7, 64, True, 256, 64),         # 98 rows: a ragged second tile
    (1, 1, 1, 64, True, 256, 64),         # one row
    (3, 9, 9, 128, False, 256, 64),       # two K steps, no residual
    (5, 14, 14, 1024, True, 256, 64),     # sixteen K steps
    (256, 56, 56, 64, True, 256, 64),     # ResNet-50's first stage at batch 256
    (3, 7, 7, 128, True, 512, 128),       # 512 channels in chunks of 128: ragged last tile
    (2, 5, 5, 128, False, 512, 128),      # no residual
    (182, 28, 28, 128, True, 512, 128),   # ResNet-50's second stage at the rows that reach it
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "n{}_{}x{}_cin{}_res{}_c{}".format(*c[:6]))
def test_conv_pair_op(case):
    from paper_2307_04963_amd import runtime
    n, H, W, cin, residual, c3, c1 = case
    print(f"[pair-op] n={n} {H}x{W} cin={cin} residual={residual}", flush=True)
    rng = np.random.default_rng(n * 1000 + cin)
    x = bf16_bits_to_f32(to_bf16_bits(rng.standard_normal((n, H, W, cin)).astype(np.float32)))
    w3 = bf16_bits_to_f32(to_bf16_bits(rng.uniform(-1, 1, (c3, cin)).astype(np.float32) * np.sqrt(6.0 / cin)))
    w1 = bf16_bits_to_f32(to_bf16_bits(rng.uniform(-1, 1, (c1, c3)).astype(np.float32) * np.sqrt(6.0 / c3)))
    sc3, sh3 = rng.uniform(0.5, 1.5, c3).astype(np.float32), rng.uniform(-0.3, 0.3, c3).astype(np.float32)
    sc1, sh1 = rng.uniform(0.5, 1.5, c1).astype(np.float32), rng.uniform(-0.3, 0.3, c1).astype(np.float32)
    r = bf16_bits_to_f32(to_bf16_bits(rng.standard_normal((n, H, W, c3)).astype(np.float32))) if residual else None
    p3 = torch.from_numpy(runtime.pack_conv_weights(to_bf16_bits(w3.reshape(c3, 1, 1, cin))).view(np.int16)).cuda()
    p1 = torch.from_numpy(runtime.pack_conv_weights(to_bf16_bits(w1.reshape(c1, 1, 1, c3))).view(np.int16)).cuda()
    xt = _bits(x).cuda().view(torch.bfloat16)
    rt = _bits(r).cuda().view(torch.bfloat16) if residual else None
    v = [torch.from_numpy(a).cuda() for a in (sc3, sh3, sc1, sh1)]
    y3, y1 = runtime.conv_pair(xt, p3, v[0], v[1], rt, c3, p1, v[2], v[3], c1)
    u3 = runtime.conv(xt, p3, c3, 1, 1, 0, v[0], v[1], rt, 1)
    u1 = runtime.conv(u3, p1, c1, 1, 1, 0, v[2], v[3], None, 1)
    torch.cuda.synchronize()
    assert torch.equal(y3.view(torch.int16), u3.view(torch.int16)), "first layer: fused and unfused bits differ"
    assert torch.equal(y1.view(torch.int16), u1.view(torch.int16)), "second layer: fused and unfused bits differ"
    g3, g1 = _f64(y3), _f64(y1)
    imgs = np.arange(n) if n <= 8 else np.unique(np.linspace(0, n - 1, 4).astype(int))
    _check_1x1(x, w3, sc3, sh3, r, g3, imgs, "first layer")
    _check_1x1(g3, w1, sc1, sh1, None, g1, imgs, "second layer")


def test_conv_pair_op_rejects_other_shapes():
    from paper_2307_04963_amd import runtime
    from paper_2307_04963_amd._lib import DyclError
    x = torch.zeros((1, 4, 4, 64), dtype=torch.bfloat16, device="cuda")
    p = torch.zeros(1 << 16, dtype=torch.int16, device="cuda")
    v = torch.ones(512, dtype=torch.float32, device="cuda")
    with pytest.raises(DyclError):
        runtime.conv_pair(x, p, v, v, None, 512, p, v, v, 128)   # 512 -> 128 takes cin 128 only
    with pytest.raises(DyclError):
        runtime.conv_pair(x[..., :32].contiguous(), p, v, v, None, 256, p, v, v, 64)   # cin % 64 != 0


@pytest.mark.parametrize("batch", [None, 37], ids=["benchmark_batch", "b37"])
def test_resnet50_plan_same_bits_with_and_without_pairs(batch):
    """At the benchmark batch and at 37 images (ragged last tiles at every
    stage; the exits leave odd live counts, read on the device)."""
    from paper_2307_04963_amd import lowering, runtime
    name = "resnet50_exit"
    B = batch or configs.DEFAULT_BATCH[name]
    wl = configs.build(name)
    blob, man = wl.blob()
    spec = lowering.lower(wl.arch, man)
    on = runtime.Plan(json.dumps(spec), blob, B)
    off = runtime.Plan(json.dumps(dict(spec, pair_pointwise=False)), blob, B)
    x, aux = wl.inputs(B)
    # the pairing took both first-stage boundaries and two of the second stage
    # (labels of the profiled launches; the second stage's pairs run when
    # some rows reach it)
    on.profile(True)
    res = runtime.run_numpy(on, wl, x, aux)
    labels = [r["label"] for r in on.profile_launches() if " + " in r["label"]]
    on.profile(False)
    assert len(labels) == (4 if res["counts"][0][1] > 0 else 2), labels
    for mode in ("sync", "device"):
        print(f"[pair-plan] {name} B={B} mode={mode}", flush=True)
        on.set_host_mode(mode)
        off.set_host_mode(mode)
        a = runtime.run_numpy(on, wl, x, aux)
        b = runtime.run_numpy(off, wl, x, aux)
        assert np.array_equal(a["logits"], b["logits"], equal_nan=True)
        for k in ("exit_index", "iterations", "skip_mask"):
            assert np.array_equal(a[k], b[k]), k
        assert a["counts"] == b["counts"]
    on.close()
    off.close()
