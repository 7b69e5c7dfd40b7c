"""Oracle for batched dynamic-routing inference.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this module.  The GPU product path never calls it, and it shares no
code with the GPU path: both only read the same seeded workload bytes.

What it computes.  DyCL compiles a dynamic network P_DyNN into a host
program P_Host whose result equals the original for every input (Sec. 5,
Eq. 2).  The plain definition of that result is the original dynamic
network, the "vendor" program V of Sec. 3.2, run one input at a time with
ordinary ``if`` and ``for`` statements: the condition nodes read an
intermediate tensor (an exit confidence, a gate value; Sec. 2.2) and pick
the branch for that input alone.  Each family below is that program for one
kind of dynamic network:

  early_exit_mlp / early_exit_resnet  layer-wise early stopping (Table 1,
      Shallow-Deep): after each stage an exit head; leave when confident.
  skipnet  block-wise selective execution (Table 1; the SkipNet forward of
      Sec. 4): a gate before each residual block picks execute or identity;
      at a down-sampling block the skipped sample takes the shortcut
      projection.
  act  a bounded loop (Sec. 2.2: loops carry a constant maximum iteration
      count); a halting unit stops the loop per input.
  seq_decoder  a generative network (Table 1, En-Decoder: an encoder state
      fed to an LSTM that emits one token per step): greedy decoding, each
      step's token read back as the next step's input, until the end token
      or the length bound (the bounded loop of Sec. 2.2 again); the token
      choice is the per-input decision.

Numerics.  Contractions accumulate in float64 (``acc="f64"``, the
reference) or in one of four float32 orders, used only to find the samples
whose routing two correct accumulation orders of the same network disagree
on (Eq. 2 fixes the result only up to the order of rounding):
``"f32"`` the library's float32 convolution / product, ``"f32r"`` the same
over the input channels in reverse order, ``"f32c"`` the input channels in
blocks of 16 (each block's sum over its channels and taps exact, rounded to
float32, the blocks added in float32 in channel order: the shape of a
16-deep matrix-core step), ``"f32n"`` the library's float32 convolution
without its oneDNN path (im2col and a matrix product).  The bf16 workloads store every
conv / linear output in bf16: ``q`` rounds to float32, then to bf16 with
round-to-nearest-even, exactly where the GPU stores bf16.  Heads (global
average pool, head linear, softmax / sigmoid) and the final logits stay
float32-or-better and are never rounded to bf16.  Every decision compares a
float32 statistic with a float32 threshold, the precision the GPU decides in.

The margin of a sample is the smallest distance between a decision
statistic it evaluated and that decision's threshold (forced decisions - the
last exit head, the last loop step - carry none).  A decoder's decision is
the argmax over the step's float32 logits (ties to the lowest index); its
statistic is the gap between the two largest logits, whose threshold is 0,
and every step's choice counts (the last step's token is still emitted).

Parity pins for every function here live in the CPU test-suite: brute-force
loops on tiny inputs, closed forms, invariants and path enumeration.
"""

from __future__ import annotations

import math
import warnings
from dataclasses import dataclass

import numpy as np
import torch
import torch.nn.functional as F

NO_EXIT = -1

# --------------------------------------------------------------------------
# primitives
# --------------------------------------------------------------------------


ACC_F32 = ("f32", "f32r", "f32c", "f32n")


def _dt(acc):
    if acc == "f64":
        return torch.float64
    if acc in ACC_F32:
        return torch.float32
    raise ValueError(acc)


def _chunked(f, x, w, ci_axis_w, block=16):
    """sum over input-channel blocks of f(x[block], w[block]) computed in
    float64, each block rounded to float32, the blocks added in float32."""
    out = None
    for c0 in range(0, x.shape[0], block):
        xs = x[c0:c0 + block].to(torch.float64)
        ws = w.narrow(ci_axis_w, c0, min(block, x.shape[0] - c0)).to(torch.float64)
        part = f(xs, ws).to(torch.float32)
        out = part if out is None else out + part
    return out


def q(t: torch.Tensor) -> torch.Tensor:
    """bf16 storage: round to float32, then to bf16 (nearest, ties to even).

    Returns float64 holding the bf16 value.  NaN stays NaN, overflow goes to
    +-inf as IEEE rounding requires.
    """
    f = t.to(torch.float32)
    b = f.view(torch.int32).to(torch.int64) & 0xFFFFFFFF
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    r = torch.where(r >= 2 ** 31, r - 2 ** 32, r).to(torch.int32)
    out = r.view(torch.float32)
    out = torch.where(torch.isnan(f), f, out)
    return out.to(torch.float64)


def f32(t):
    """Round to float32 (nearest even) and return float64."""
    if isinstance(t, torch.Tensor):
        return t.to(torch.float32).to(torch.float64)
    return float(np.float32(t))


def conv2d(x: torch.Tensor, w: torch.Tensor, stride: int, pad: int, acc="f64") -> torch.Tensor:
    """y[co, oh, ow] = sum_{kh, kw, ci} x[ci, oh*s - p + kh, ow*s - p + kw] * w[co, ci, kh, kw]

    x: [Ci, H, W]; w: [Co, Ci, kh, kw]; zero padding.  Returns [Co, Ho, Wo]
    in the accumulation precision (a library convolution is the step).
    """
    dt = _dt(acc)
    if acc == "f32r":
        return F.conv2d(x.to(dt).flip(0)[None], w.to(dt).flip(1), stride=stride, padding=pad)[0]
    if acc == "f32c":
        return _chunked(lambda a, b: F.conv2d(a[None], b, stride=stride, padding=pad)[0], x, w, 1)
    if acc == "f32n":
        with warnings.catch_warnings():
            warnings.simplefilter("ignore")
            with torch.backends.mkldnn.flags(enabled=False):
                return F.conv2d(x.to(dt)[None], w.to(dt), stride=stride, padding=pad)[0]
    return F.conv2d(x.to(dt)[None], w.to(dt), stride=stride, padding=pad)[0]


def linear(W: torch.Tensor, v: torch.Tensor, acc="f64") -> torch.Tensor:
    """W @ v in the accumulation precision (``"f32n"``: the library's float32
    product, as ``"f32"``)."""
    dt = _dt(acc)
    if acc == "f32r":
        return W.to(dt).flip(-1) @ v.to(dt).flip(0)
    if acc == "f32c":
        return _chunked(lambda a, b: b @ a, v, W, W.dim() - 1)
    return W.to(dt) @ v.to(dt)


def gap(x: torch.Tensor, acc="f64") -> torch.Tensor:
    """Global average pool of [C, H, W] -> [C]: sum over H*W, divided by H*W."""
    dt = _dt(acc)
    c = x.shape[0]
    return x.to(dt).reshape(c, -1).sum(dim=1) / (x.shape[1] * x.shape[2])


def maxpool3s2(x: torch.Tensor) -> torch.Tensor:
    """3x3 window, stride 2, padding 1 with -inf."""
    return F.max_pool2d(x[None], kernel_size=3, stride=2, padding=1)[0]


def maxprob(z: torch.Tensor, T: float, acc="f64") -> float:
    """Largest softmax probability of z / T: 1 / sum_j exp((z_j - max z) / T)."""
    dt = _dt(acc)
    z = z.to(dt)
    s = torch.exp((z - z.max()) / torch.tensor(T, dtype=dt)).sum()
    return float(f32(1.0 / s))


def sigmoid(v, acc="f64") -> float:
    dt = _dt(acc)
    v = torch.as_tensor(v, dtype=dt)
    return float(f32(1.0 / (1.0 + torch.exp(-v))))


def gelu(u: torch.Tensor, acc="f64") -> torch.Tensor:
    """Exact (erf) GELU: u/2 * (1 + erf(u / sqrt 2))."""
    dt = _dt(acc)
    u = u.to(dt)
    return 0.5 * u * (1.0 + torch.erf(u / math.sqrt(2.0)))


# --------------------------------------------------------------------------
# per-sample programs
# --------------------------------------------------------------------------


@dataclass
class Result:
    logits: np.ndarray         # float32 [n_out]
    exit_index: int            # head that produced the logits, -1 if none
    iterations: int            # loop steps executed, 0 if no loop
    skip_mask: int             # bit i set <=> gate i chose identity / shortcut
    margin: float              # min |statistic - threshold| over decisions
    trail: tuple = ()          # the non-forced decision statistics, in order
    tokens: tuple = ()         # tokens a decoder emitted, in order


class Oracle:
    """Runs one workload's dynamic network sample by sample.

    arch: the architecture description; weights: name -> float32 numpy array
    (bf16 tensors already hold their exact bf16 values).
    """

    def __init__(self, arch: dict, weights: dict, acc: str = "f64"):
        self.arch, self.acc = arch, acc
        self.W = {}
        for k, v in weights.items():
            t = torch.from_numpy(np.asarray(v, dtype=np.float32)).to(torch.float64)
            if t.dim() == 4:                 # conv [Co, kh, kw, Ci] -> [Co, Ci, kh, kw]
                t = t.permute(0, 3, 1, 2).contiguous()
            self.W[k] = t
        self.bf16 = arch["dtype"] == "bf16"
        self.store = q if self.bf16 else f32

    # ---- layers ---------------------------------------------------------
    def conv_bn(self, x, c, relu=True, res=None):
        """store(ReLU(a * conv(x) + b [+ res])) with BatchNorm folded into a, b."""
        y = conv2d(x, self.W[c["name"] + ".w"], c["stride"], c["pad"], self.acc).to(torch.float64)
        y = y * self.W[c["name"] + ".a"][:, None, None] + self.W[c["name"] + ".b"][:, None, None]
        if res is not None:
            y = y + res
        if relu:
            y = torch.clamp_min(y, 0.0)
        return self.store(y)

    def basic(self, x, b):
        sc = self.conv_bn(x, b["proj"], relu=False) if b["proj"] is not None else x
        t = self.conv_bn(x, b["c1"])
        return self.conv_bn(t, b["c2"], res=sc)

    def bottleneck(self, x, b):
        sc = self.conv_bn(x, b["proj"], relu=False) if b["proj"] is not None else x
        t = self.conv_bn(x, b["c1"])
        t = self.conv_bn(t, b["c2"])
        return self.conv_bn(t, b["c3"], res=sc)

    def head_logits(self, g, name):
        return linear(self.W[name + ".w"], g, self.acc).to(torch.float64) + self.W[name + ".b"]

    # ---- families -------------------------------------------------------
    def run_sample(self, x: np.ndarray, aux: float | None = None) -> Result:
        fam = self.arch["family"]
        xt = torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.float64)
        if fam == "early_exit_mlp":
            return self._mlp(xt)
        if fam == "early_exit_resnet":
            return self._resnet_exit(xt.permute(2, 0, 1))
        if fam == "skipnet":
            return self._skipnet(xt.permute(2, 0, 1))
        if fam == "act":
            return self._act(xt, aux)
        if fam == "seq_decoder":
            return self._decoder(xt)
        raise ValueError(fam)

    def _mlp(self, h):
        a, tau = self.arch, np.float32(self.arch["tau"])
        margin, last, trail = math.inf, len(a["layers"]) - 1, []
        for k, (L, H) in enumerate(zip(a["layers"], a["heads"])):
            h = f32(torch.clamp_min(linear(self.W[L["name"] + ".w"], h, self.acc).to(torch.float64)
                                    + self.W[L["name"] + ".b"], 0.0))
            z = self.head_logits(h, H["name"])
            p = np.float32(maxprob(z, float(self.W[H["name"] + ".T"][0]), self.acc))
            if k == last:
                return Result(f32(z).numpy().astype(np.float32), k, 0, 0, margin, tuple(trail))
            margin = min(margin, abs(float(p) - float(tau)))
            trail.append(float(p))
            if p >= tau:
                return Result(f32(z).numpy().astype(np.float32), k, 0, 0, margin, tuple(trail))
        raise AssertionError("unreachable")

    def _resnet_exit(self, x):
        a, tau = self.arch, np.float32(self.arch["tau"])
        y = self.conv_bn(x, a["stem"])
        if a["maxpool"]:
            y = maxpool3s2(y)
        margin, last, trail = math.inf, len(a["stages"]) - 1, []
        for s, stage in enumerate(a["stages"]):
            for b in stage:
                y = self.basic(y, b) if b["type"] == "basic" else self.bottleneck(y, b)
            H = a["heads"][s]
            z = self.head_logits(gap(y, self.acc).to(torch.float64), H["name"])
            p = np.float32(maxprob(z, float(self.W[H["name"] + ".T"][0]), self.acc))
            if s == last:
                return Result(f32(z).numpy().astype(np.float32), s, 0, 0, margin, tuple(trail))
            margin = min(margin, abs(float(p) - float(tau)))
            trail.append(float(p))
            if p >= tau:
                return Result(f32(z).numpy().astype(np.float32), s, 0, 0, margin, tuple(trail))
        raise AssertionError("unreachable")

    def _skipnet(self, x):
        a = self.arch
        thr = np.float32(a["gate_threshold"])
        x = self.conv_bn(x, a["stem"])
        mask, margin, trail = 0, math.inf, []
        for i, b in enumerate(a["blocks"]):
            g = gap(x, self.acc)
            u = self.W[b["gate"] + ".u"]
            qv = np.float32(sigmoid(float(linear(u[None], g, self.acc)[0]) + float(self.W[b["gate"] + ".v"][0]),
                                    self.acc))
            margin = min(margin, abs(float(qv) - float(thr)))
            trail.append(float(qv))
            # the shortcut (identity, or the down-sampling projection) is what a
            # skipped block passes on
            prev = self.conv_bn(x, b["proj"], relu=False) if b["proj"] is not None else x
            if qv > thr:
                t = self.conv_bn(x, b["c1"])
                x = self.conv_bn(t, b["c2"], res=prev)
            else:
                x = prev
                mask |= 1 << i
        z = self.head_logits(gap(x, self.acc).to(torch.float64), "fc")
        return Result(f32(z).numpy().astype(np.float32), NO_EXIT, 0, mask, margin, tuple(trail))

    def _act(self, x, b_s):
        a = self.arch
        tau, T = np.float32(a["tau"]), a["max_steps"]
        h = torch.zeros(a["hidden"], dtype=torch.float64)
        S, margin, trail = np.float32(0.0), math.inf, []
        W1, b1, w = self.W["W1"], self.W["b1"], self.W["w_halt"]
        for t in range(1, T + 1):
            u = linear(W1, torch.cat([h, x]), self.acc).to(torch.float64) + b1
            h = q(gelu(u, self.acc))
            p = np.float32(sigmoid(float(linear(w[None], h, self.acc)[0]) + float(b_s), self.acc))
            S = np.float32(S + p)
            if t < T:
                margin = min(margin, abs(float(S) - float(tau)))
                trail.append(float(S))
            if S >= tau or t == T:
                z = linear(self.W["W2"], h, self.acc).to(torch.float64) + self.W["b2"]
                return Result(f32(z).numpy().astype(np.float32), NO_EXIT, t, 0, margin, tuple(trail))
        raise AssertionError("unreachable")

    def _decoder(self, x):
        a, W = self.arch, self.W
        H, L, eos = a["hidden"], a["max_len"], a["eos"]
        dt = _dt(self.acc)

        def sig(v):
            return 1.0 / (1.0 + torch.exp(-v.to(dt)))

        # encoder state: h0 = bf16(tanh(W_enc x + b_enc)), c0 = 0
        h = q(torch.tanh(linear(W["enc.w"], x, self.acc).to(dt) + W["enc.b"].to(dt)))
        c = torch.zeros(H, dtype=torch.float64)
        tok, toks, margin, trail = a["bos"], [], math.inf, []
        for t in range(1, L + 1):
            # LSTM step on [h; embedding of the previous token]; gate order
            # input, forget, cell, output.  The cell is the epilogue of the
            # gate linear layer: its pre-activations stay float32, and what
            # the layer stores is the cell state (float32) and h (bf16)
            g = f32(linear(W["lstm.w"], torch.cat([h, W["emb"][tok]]), self.acc).to(dt) + W["lstm.b"].to(dt))
            i, f, u, o = sig(g[:H]), sig(g[H:2 * H]), torch.tanh(g[2 * H:3 * H]), sig(g[3 * H:])
            c = f32(f * c.to(dt) + i * u)                   # cell state kept in float32
            h = q(o * torch.tanh(c.to(dt)))                 # hidden state stored in bf16
            z = f32(linear(W["out.w"], h, self.acc).to(dt) + W["out.b"].to(dt))   # float32 logits
            zmax = float(z.max())
            tok = int(torch.nonzero(z == zmax)[0, 0])       # ties: the lowest index
            second = float(torch.cat([z[:tok], z[tok + 1:]]).max())
            gap = zmax - second
            margin = min(margin, gap)
            trail.append(gap)
            toks.append(tok)
            if tok == eos or t == L:
                return Result(z.numpy().astype(np.float32), NO_EXIT, t, 0, margin, tuple(trail), tuple(toks))
        raise AssertionError("unreachable")

    # ---- batch ----------------------------------------------------------
    def run(self, X: np.ndarray, AUX: np.ndarray | None = None, indices=None):
        """Run the samples ``indices`` (default: all) one after another.

        Returns a dict of stacked results in the order of ``indices``.
        """
        idx = range(X.shape[0]) if indices is None else indices
        res = [self.run_sample(X[i], None if AUX is None else float(AUX[i])) for i in idx]
        return {
            "logits": np.stack([r.logits for r in res]) if res else np.zeros((0, self.arch["n_out"]), np.float32),
            "exit_index": np.array([r.exit_index for r in res], dtype=np.int32),
            "iterations": np.array([r.iterations for r in res], dtype=np.int32),
            "skip_mask": np.array([r.skip_mask for r in res], dtype=np.uint64),
            "margin": np.array([r.margin for r in res], dtype=np.float64),
            "trail": [r.trail for r in res],
            "tokens": _pad_tokens([r.tokens for r in res], self.arch.get("max_len", 0)),
        }


def _pad_tokens(seqs, width):
    """[n, width] int32: each sequence's tokens, then -1."""
    out = np.full((len(seqs), width), -1, dtype=np.int32)
    for i, s in enumerate(seqs):
        out[i, :len(s)] = s
    return out


def from_workload(wl, acc="f64") -> Oracle:
    return Oracle(wl.arch, wl.weights_f32(), acc)


# --------------------------------------------------------------------------
# correctness metrics of Eq. 1 (Sec. 3.2)
# --------------------------------------------------------------------------


def delta(c_before: np.ndarray, v_before: np.ndarray, eps: float = 1e-10) -> float:
    """Maximum numeric error: log10(max_i ||C(x_i) - V(x_i)|| + eps).

    The norm is taken per input over its output vector (Euclidean); an
    error of zero gives -10 with eps = 1e-10.
    """
    if c_before.shape[0] == 0:
        return math.log10(eps)
    err = np.linalg.norm(c_before.astype(np.float64) - v_before.astype(np.float64), axis=1).max()
    return math.log10(err + eps)


def eta(c_before: np.ndarray, v_before: np.ndarray) -> float:
    """Final inconsistent rate: fraction of inputs whose argmax label differs."""
    if c_before.shape[0] == 0:
        return 0.0
    return float(np.mean(np.argmax(c_before, axis=1) != np.argmax(v_before, axis=1)))
