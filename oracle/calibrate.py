"""Calibration of the synthetic workloads.  TEST INFRASTRUCTURE (oracle side).

Writes ``workloads/calib/<name>.npz``: the constants a random-weight network
needs so that its activations stay O(1) and its routing is mixed.  Run it
with ``python -m oracle.calibrate [names...]``; it calls only the oracle's
primitives and the seeded generator, on a calibration batch drawn from its
own input stream (never the evaluation inputs).

Per workload (the choices are listed with their reasons in the design notes):

* BatchNorm (CNNs): every conv's BatchNorm takes the per-channel mean and
  variance of that conv's output over the calibration batch (beta 0,
  eps 1e-5), layer by layer in program order, with the earlier layers
  already calibrated; it is folded to a float32 scale and shift.  gamma is 1,
  except on the last BatchNorm of each residual branch, where it is
  GAMMA_LAST (small, as in trained residual networks): with gamma 1 the
  random network amplifies rounding perturbations by ~2.4x per block, which
  makes deep exit decisions depend on accumulation order.
* Exit heads (CNNs): head weights keep their seeded draw; the bias is minus
  the mean head output over the samples that reach the head (centring), and
  the head's softmax temperature is chosen by bisection so that about
  1 / (number of heads left) of those samples exit there.  The final head is
  centred and always exits.
* Exit heads (MLP): the head weight is scaled by s_k, found by bisection, so
  that about a third of the batch exits at each of the first two heads.
* Gates (SkipNet): with every block executed, BatchNorm is calibrated as
  above; then, gate by gate in order, the gate pre-activation u.GAP(x) is
  standardised over the calibration batch as routed by the earlier gates,
  and the seeded N(0, 1.5) offset is added.
* End token (LSTM decoder): the output bias of the end token is raised by an
  offset found by bisection so that the greedy decodings of the calibration
  batch are DECODER_MEAN_LEN tokens long on average (with the drawn bias the
  end token is almost never the most likely one, and every sequence would
  run to the length bound).
"""

from __future__ import annotations

import math
import os
import sys

import numpy as np
import torch
import torch.nn.functional as F

from .dycl_oracle import q, f32

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
from workloads import configs  # noqa: E402

BN_EPS = configs.BN_EPS
GAMMA_LAST = 0.1
CALIB_BATCH = {"mlp_exit": 4096, "resnet18_exit": 512, "skipnet38": 1024, "resnet50_exit": 64, "lstm_decoder": 256}
DECODER_MEAN_LEN = 8.0


def _bisect(frac_fn, target, lo, hi, increasing=True, iters=60):
    for _ in range(iters):
        mid = 0.5 * (lo + hi) if hi / max(lo, 1e-30) < 4 else math.sqrt(max(lo, 1e-30) * hi)
        f = frac_fn(mid)
        if (f < target) == increasing:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def _maxprob_rows(z, T):
    z = z / T
    return 1.0 / torch.exp(z - z.max(dim=1, keepdim=True).values).sum(dim=1)


class _CNN:
    """Batched static forward used only to collect calibration statistics."""

    def __init__(self, wl):
        self.wl = wl
        self.W = {k: torch.from_numpy(v).to(torch.float64) for k, v in wl.weights_f32().items()}
        self.out = {}

    def conv_bn(self, x, c, relu=True, res=None, calibrate=True):
        w = self.W[c["name"] + ".w"].permute(0, 3, 1, 2)
        y = F.conv2d(x, w, stride=c["stride"], padding=c["pad"])
        if calibrate:
            mu = y.mean(dim=(0, 2, 3))
            var = y.var(dim=(0, 2, 3), unbiased=False)
            gamma = GAMMA_LAST if res is not None else 1.0
            a = f32(gamma / torch.sqrt(var + BN_EPS))
            b = f32(-mu * a)
            self.out[c["name"] + ".a"] = a.numpy().astype(np.float32)
            self.out[c["name"] + ".b"] = b.numpy().astype(np.float32)
        a = torch.from_numpy(self.out[c["name"] + ".a"]).to(torch.float64)
        b = torch.from_numpy(self.out[c["name"] + ".b"]).to(torch.float64)
        y = y * a[None, :, None, None] + b[None, :, None, None]
        if res is not None:
            y = y + res
        if relu:
            y = torch.clamp_min(y, 0.0)
        return q(y)

    def block(self, x, b):
        sc = self.conv_bn(x, b["proj"], relu=False) if b["proj"] is not None else x
        if b["type"] == "basic":
            t = self.conv_bn(x, b["c1"])
            return self.conv_bn(t, b["c2"], res=sc)
        t = self.conv_bn(x, b["c1"])
        t = self.conv_bn(t, b["c2"])
        return self.conv_bn(t, b["c3"], res=sc)


def _inputs(wl, n):
    x, _ = wl.inputs_f32(n, 0, stream="calib")
    return torch.from_numpy(x).to(torch.float64)


def calibrate_mlp(wl, n):
    a = wl.arch
    W = {k: torch.from_numpy(v).to(torch.float64) for k, v in wl.weights_f32().items()}
    h = _inputs(wl, n)
    alive = torch.ones(n, dtype=torch.bool)
    out, K = {}, len(a["layers"])
    for k, (L, H) in enumerate(zip(a["layers"], a["heads"])):
        h = f32(torch.clamp_min(h @ W[L["name"] + ".w"].T + W[L["name"] + ".b"], 0.0))
        if k == K - 1:
            break
        wz = h[alive] @ W[H["name"] + ".w"].T
        c = W[H["name"] + ".b"]

        def frac(s):
            return float((_maxprob_rows(s * wz + c, 1.0) >= np.float32(a["tau"])).double().mean())

        s = _bisect(frac, 1.0 / (K - k), 1e-3, 1e3)
        out[H["name"] + ".w"] = (s * W[H["name"] + ".w"]).numpy().astype(np.float32)
        z = s * (h @ W[H["name"] + ".w"].T) + c
        ex = (_maxprob_rows(z, 1.0) >= np.float32(a["tau"])) & alive
        alive &= ~ex
    return out


def calibrate_resnet(wl, n):
    a, net = wl.arch, _CNN(wl)
    x = _inputs(wl, n).permute(0, 3, 1, 2)
    y = net.conv_bn(x, a["stem"])
    if a["maxpool"]:
        y = F.max_pool2d(y, 3, 2, 1)
    alive = torch.ones(n, dtype=torch.bool)
    K = len(a["stages"])
    for s, stage in enumerate(a["stages"]):
        for b in stage:
            y = net.block(y, b)
        H = a["heads"][s]
        g = y.mean(dim=(2, 3))
        wz = g[alive] @ net.W[H["name"] + ".w"].T
        c = -wz.mean(dim=0)
        net.out[H["name"] + ".b"] = c.numpy().astype(np.float32)
        z = wz + c
        T = 1.0
        if s < K - 1:
            def frac(t):
                return float((_maxprob_rows(z, t) >= np.float32(a["tau"])).double().mean())
            T = _bisect(frac, 1.0 / (K - s), 1e-4, 1e3, increasing=False)
            zz = g @ net.W[H["name"] + ".w"].T + c
            ex = (_maxprob_rows(zz, T) >= np.float32(a["tau"])) & alive
            alive &= ~ex
        net.out[H["name"] + ".T"] = np.array([T], dtype=np.float32)
    return net.out


def calibrate_skipnet(wl, n):
    a, net = wl.arch, _CNN(wl)
    x0 = _inputs(wl, n).permute(0, 3, 1, 2)
    # BatchNorm with every block executed
    y = net.conv_bn(x0, a["stem"])
    for b in a["blocks"]:
        y = net.block(y, b)
    # gates, in order, on the routed batch
    y = net.conv_bn(x0, a["stem"], calibrate=False)
    for b in a["blocks"]:
        g = y.mean(dim=(2, 3))
        u = net.W[b["gate"] + ".u"]
        v = net.W[b["gate"] + ".v"][0]
        s = g @ u
        mu, sd = s.mean(), s.std(unbiased=False)
        u2 = f32(u / sd)
        v2 = f32(-mu / sd + v)
        net.out[b["gate"] + ".u"] = u2.numpy().astype(np.float32)
        net.out[b["gate"] + ".v"] = np.array([float(v2)], dtype=np.float32)
        qv = 1.0 / (1.0 + torch.exp(-(g @ u2 + v2)))
        run = qv > np.float32(a["gate_threshold"])
        prev = net.conv_bn(y, b["proj"], relu=False, calibrate=False) if b["proj"] is not None else y
        t = net.conv_bn(y, b["c1"], calibrate=False)
        yb = net.conv_bn(t, b["c2"], res=prev, calibrate=False)
        y = torch.where(run[:, None, None, None], yb, prev)
    return net.out


def _decoder_lengths(args):
    """Greedy decoding lengths of calibration samples [lo, hi) with the end
    token's bias raised by `offset` (one worker process)."""
    name, offset, lo, hi = args
    torch.set_num_threads(1)
    from .dycl_oracle import Oracle
    wl = configs.raw_workload(name)
    W = wl.weights_f32()
    W["out.b"] = W["out.b"].copy()
    W["out.b"][wl.arch["eos"]] += np.float32(offset)
    x, _ = wl.inputs_f32(hi, 0, stream="calib")
    return Oracle(wl.arch, W).run(x, None, indices=range(lo, hi))["iterations"]


def calibrate_decoder(wl, n):
    import multiprocessing as mp
    procs = max(1, min(16, os.cpu_count() or 1))
    step = (n + procs - 1) // procs
    with mp.get_context("spawn").Pool(procs) as pool:
        def mean_len(offset):
            parts = pool.map(_decoder_lengths, [(wl.name, offset, lo, min(n, lo + step)) for lo in range(0, n, step)])
            return float(np.concatenate(parts).mean())
        off = _bisect(mean_len, DECODER_MEAN_LEN, 0.0, 32.0, increasing=False, iters=24)
    b = wl.weights_f32()["out.b"].copy()
    b[wl.arch["eos"]] += np.float32(off)
    return {"out.b": b, "_eos_offset": np.array(off)}


def calibrate(name: str):
    wl = configs.raw_workload(name)
    n = CALIB_BATCH[name]
    torch.set_num_threads(max(1, os.cpu_count() or 1))
    fam = wl.arch["family"]
    if fam == "early_exit_mlp":
        out = calibrate_mlp(wl, n)
    elif fam == "early_exit_resnet":
        out = calibrate_resnet(wl, n)
    elif fam == "skipnet":
        out = calibrate_skipnet(wl, n)
    elif fam == "seq_decoder":
        out = calibrate_decoder(wl, n)
    else:
        raise ValueError(f"{name} needs no calibration")
    os.makedirs(configs.CALIB_DIR, exist_ok=True)
    path = os.path.join(configs.CALIB_DIR, f"{name}.npz")
    np.savez_compressed(path, **out)
    return path


if __name__ == "__main__":
    names = sys.argv[1:] or ["mlp_exit", "resnet18_exit", "skipnet38", "resnet50_exit"]
    for nm in names:
        print("calibrated", nm, "->", calibrate(nm), flush=True)
