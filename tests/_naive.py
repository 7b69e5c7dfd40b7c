"""Independent numpy references used to pin the oracle on tiny networks.

Nothing here calls the oracle or torch: convolutions are sums of shifted
matrix products over an explicitly padded image, bf16 rounding is a numpy
bit operation, and every dynamic network is evaluated as a *static*
network along a path that the caller fixes.  The tests then enumerate all
paths and check that exactly one is self-consistent and that the oracle
picked it.
"""

from __future__ import annotations

import math

import numpy as np


def q_np(v):
    """float64 -> float32 -> bf16 (nearest even) -> float64, numpy only."""
    f = np.asarray(v, dtype=np.float32)
    b = f.view(np.uint32).astype(np.uint64)
    r = (((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16).astype(np.uint64)
    r = (r & 0xFFFFFFFF).astype(np.uint32)
    out = r.view(np.float32).astype(np.float64)
    return np.where(np.isnan(f), np.nan, out)


def f32_np(v):
    return np.asarray(v, dtype=np.float32).astype(np.float64)


def conv_shift(x, w, stride, pad):
    """x: [H, W, Ci]; w: [Co, kh, kw, Ci] -> [Ho, Wo, Co] as sum of tap products."""
    H, W, Ci = x.shape
    Co, kh, kw, _ = w.shape
    xp = np.zeros((H + 2 * pad, W + 2 * pad, Ci))
    xp[pad:pad + H, pad:pad + W] = x
    Ho = (H + 2 * pad - kh) // stride + 1
    Wo = (W + 2 * pad - kw) // stride + 1
    y = np.zeros((Ho, Wo, Co))
    for i in range(kh):
        for j in range(kw):
            win = xp[i:i + stride * (Ho - 1) + 1:stride, j:j + stride * (Wo - 1) + 1:stride, :]
            y += win @ w[:, i, j, :].T
    return y


def conv_loops(x, w, stride, pad):
    """Same as conv_shift with scalar loops (for the smallest shapes only)."""
    H, W, Ci = x.shape
    Co, kh, kw, _ = w.shape
    Ho = (H + 2 * pad - kh) // stride + 1
    Wo = (W + 2 * pad - kw) // stride + 1
    y = np.zeros((Ho, Wo, Co))
    for co in range(Co):
        for oh in range(Ho):
            for ow in range(Wo):
                s = 0.0
                for i in range(kh):
                    for j in range(kw):
                        ih, iw = oh * stride - pad + i, ow * stride - pad + j
                        if 0 <= ih < H and 0 <= iw < W:
                            for ci in range(Ci):
                                s += x[ih, iw, ci] * w[co, i, j, ci]
                y[oh, ow, co] = s
    return y


def maxpool_loops(x):
    H, W, C = x.shape
    Ho, Wo = (H + 2 - 3) // 2 + 1, (W + 2 - 3) // 2 + 1
    y = np.full((Ho, Wo, C), -np.inf)
    for oh in range(Ho):
        for ow in range(Wo):
            for i in range(3):
                for j in range(3):
                    ih, iw = 2 * oh - 1 + i, 2 * ow - 1 + j
                    if 0 <= ih < H and 0 <= iw < W:
                        y[oh, ow] = np.maximum(y[oh, ow], x[ih, iw])
    return y


def softmax_max(z, T):
    e = np.exp((z - z.max()) / T)
    return float(np.float32(e.max() / e.sum()))


def sigmoid_np(v):
    return float(np.float32(1.0 / (1.0 + math.exp(-v))))


def erf_series(x):
    """erf by its Maclaurin series, 2/sqrt(pi) * sum (-1)^n x^(2n+1) / (n! (2n+1)).

    Accurate to ~1e-13 for |x| <= 3; beyond that Python's libm erf (not the
    library the oracle uses) takes over."""
    if abs(x) > 3.0:
        return math.erf(x)
    s, term, n = 0.0, x, 0
    while True:
        add = term / (2 * n + 1)
        s += add
        if abs(add) < 1e-17 * max(1.0, abs(s)):
            break
        n += 1
        term *= -x * x / n
    return 2.0 / math.sqrt(math.pi) * s


class NaiveCNN:
    def __init__(self, W, store):
        self.W, self.store = W, store

    def conv_bn(self, x, c, relu=True, res=None):
        y = conv_shift(x, self.W[c["name"] + ".w"].astype(np.float64), c["stride"], c["pad"])
        y = y * self.W[c["name"] + ".a"].astype(np.float64) + self.W[c["name"] + ".b"].astype(np.float64)
        if res is not None:
            y = y + res
        if relu:
            y = np.maximum(y, 0.0)
        return self.store(y)

    def block(self, x, b):
        sc = self.conv_bn(x, b["proj"], relu=False) if b["proj"] is not None else x
        if b["type"] == "basic":
            return self.conv_bn(self.conv_bn(x, b["c1"]), b["c2"], res=sc)
        t = self.conv_bn(self.conv_bn(x, b["c1"]), b["c2"])
        return self.conv_bn(t, b["c3"], res=sc)


def resnet_exit_static(arch, W, x):
    """All stages executed; returns [(z_k, p_k)] for every head."""
    net = NaiveCNN(W, q_np)
    y = net.conv_bn(x.astype(np.float64), arch["stem"])
    if arch["maxpool"]:
        y = maxpool_loops(y)
    out = []
    for s, stage in enumerate(arch["stages"]):
        for b in stage:
            y = net.block(y, b)
        H = arch["heads"][s]
        g = y.reshape(-1, y.shape[-1]).sum(axis=0) / (y.shape[0] * y.shape[1])
        z = W[H["name"] + ".w"].astype(np.float64) @ g + W[H["name"] + ".b"].astype(np.float64)
        out.append((z, softmax_max(z, float(W[H["name"] + ".T"][0]))))
    return out


def mlp_static(arch, W, x):
    h = x.astype(np.float64)
    out = []
    for L, H in zip(arch["layers"], arch["heads"]):
        h = f32_np(np.maximum(W[L["name"] + ".w"].astype(np.float64) @ h + W[L["name"] + ".b"], 0.0))
        z = W[H["name"] + ".w"].astype(np.float64) @ h + W[H["name"] + ".b"].astype(np.float64)
        out.append((z, softmax_max(z, float(W[H["name"] + ".T"][0]))))
    return out


def skipnet_path(arch, W, x, path):
    """Run with gate i forced to path[i] (1 = execute).  Returns (z, [q_i])."""
    net = NaiveCNN(W, q_np)
    y = net.conv_bn(x.astype(np.float64), arch["stem"])
    qs = []
    for i, b in enumerate(arch["blocks"]):
        g = y.reshape(-1, y.shape[-1]).sum(axis=0) / (y.shape[0] * y.shape[1])
        qs.append(sigmoid_np(float(W[b["gate"] + ".u"].astype(np.float64) @ g) + float(W[b["gate"] + ".v"][0])))
        sc = net.conv_bn(y, b["proj"], relu=False) if b["proj"] is not None else y
        if path[i]:
            y = net.conv_bn(net.conv_bn(y, b["c1"]), b["c2"], res=sc)
        else:
            y = sc
    g = y.reshape(-1, y.shape[-1]).sum(axis=0) / (y.shape[0] * y.shape[1])
    z = W["fc.w"].astype(np.float64) @ g + W["fc.b"].astype(np.float64)
    return z, qs


def act_static(arch, W, x, b_s):
    """The loop run for all max_steps; returns [(h_t, S_t)] and W2/b2 map."""
    Hd = arch["hidden"]
    h = np.zeros(Hd)
    S = np.float32(0.0)
    out = []
    W1 = W["W1"].astype(np.float64)
    for t in range(arch["max_steps"]):
        u = W1 @ np.concatenate([h, x.astype(np.float64)]) + W["b1"].astype(np.float64)
        gel = np.array([0.5 * v * (1.0 + erf_series(v / math.sqrt(2.0))) for v in u])
        h = q_np(gel)
        p = np.float32(sigmoid_np(float(W["w_halt"].astype(np.float64) @ h) + float(b_s)))
        S = np.float32(S + p)
        out.append((h, float(S)))
    return out


def lstm_step(Wl, bl, h, e, c):
    """One LSTM cell on [h; e] in float64, no rounding: gates input, forget,
    cell, output in blocks of H.  Returns (h', c')."""
    H = h.shape[0]
    g = Wl @ np.concatenate([h, e]) + bl
    sg = 1.0 / (1.0 + np.exp(-g))
    i, f, u, o = sg[:H], sg[H:2 * H], np.tanh(g[2 * H:3 * H]), sg[3 * H:]
    c2 = f * c + i * u
    return o * np.tanh(c2), c2


def decoder_path(arch, W, x, toks):
    """The decoder run along a fixed token sequence `toks` (the token fed at
    step t + 1 is toks[t]), with the storage points of the workload: gate
    pre-activations and the cell state rounded to float32, h to bf16, logits
    float32.  Returns the logits of every step."""
    H = arch["hidden"]
    f64 = lambda k: W[k].astype(np.float64)  # noqa: E731
    h = q_np(np.tanh(f64("enc.w") @ x.astype(np.float64) + f64("enc.b")))
    c = np.zeros(H)
    prev, zs = arch["bos"], []
    for tok in toks:
        g = f32_np(f64("lstm.w") @ np.concatenate([h, f64("emb")[prev]]) + f64("lstm.b"))
        sg = 1.0 / (1.0 + np.exp(-g))
        i, f, u, o = sg[:H], sg[H:2 * H], np.tanh(g[2 * H:3 * H]), sg[3 * H:]
        c = f32_np(f * c + i * u)
        h = q_np(o * np.tanh(c))
        zs.append(f32_np(f64("out.w") @ h + f64("out.b")))
        prev = tok
    return zs
