"""Synthetic DyNN workloads: architecture descriptions, seeded weights, inputs.

The five workloads stand in for the paper's dynamic networks (an early-exit
network in the style of Shallow-Deep, a block-skipping SkipNet and a bounded
loop; Table 1 and the bounded-loop restriction of Sec. 2.2).  The paper's
datasets and trained weights are not available, so every tensor here is drawn
from the counter-based generator in ``rng``:

  mlp_exit      early-exit MLP, fp32, 784-256-256-256, three exit heads
  resnet18_exit early-exit ResNet-18-style CNN, bf16, 32x32 inputs, 4 heads
  skipnet38     SkipNet-style ResNet-38, bf16, 18 gated basic blocks
  resnet50_exit early-exit ResNet-50-style bottleneck CNN, bf16, 224x224
  act_loop      adaptive-computation-time loop, bf16, hidden 1024, <=16 steps
  lstm_decoder  greedy LSTM decoder, bf16, hidden 512, vocabulary 4096,
                <=24 tokens (a generative network: Table 1's En-Decoder)

This module holds no part of the executed method.  Parameters that have to
be calibrated on the network itself (folded BatchNorm statistics, exit-head
centring and temperatures, gate standardisation, the MLP head scales) are
read from ``calib/<name>.npz``; those files are written by the calibration
script that sits beside the oracle.  Without them a workload is built in its
literal form (BatchNorm at PyTorch's eval defaults, heads uncentred).
"""

from __future__ import annotations

import json
import math
import os
from collections import OrderedDict
from dataclasses import dataclass, field

import numpy as np

from . import rng

SEED = 0
CALIB_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "calib")
BN_EPS = 1e-5

NAMES = ["mlp_exit", "resnet18_exit", "skipnet38", "resnet50_exit", "act_loop", "lstm_decoder"]
DEFAULT_BATCH = {"mlp_exit": 64, "resnet18_exit": 1024, "skipnet38": 2048,
                 "resnet50_exit": 256, "act_loop": 4096, "lstm_decoder": 1024}


# --------------------------------------------------------------------------
# bf16 bytes.  Inputs and weights of the bf16 workloads are handed to both
# sides as bf16 bit patterns (round-to-nearest-even of the float32 draw).
# --------------------------------------------------------------------------

def to_bf16_bits(v: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(v, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    r = ((b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)
    return r


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Tensor:
    name: str
    dtype: str            # "bf16" or "f32"
    shape: tuple
    value: np.ndarray     # float32 values (bf16 tensors hold bf16-representable values)


@dataclass
class Workload:
    name: str
    arch: dict
    tensors: "OrderedDict[str, Tensor]" = field(default_factory=OrderedDict)
    calibrated: bool = False

    # ---- inputs ---------------------------------------------------------
    @property
    def in_shape(self):
        return tuple(self.arch["input"])

    @property
    def in_dtype(self):
        return self.arch["dtype"]

    @property
    def has_aux(self):
        return self.arch["family"] == "act"

    @property
    def n_out(self):
        return self.arch["n_out"]

    def inputs(self, batch: int, start: int = 0, stream: str = "x"):
        """Sample i of any batch is drawn from counters i*D .. i*D+D-1 only.

        Returns (x, aux): x is float32 (fp32 workloads) or uint16 bf16 bits,
        shaped [batch, *in_shape]; aux is float32 [batch] or None.
        """
        d = int(np.prod(self.in_shape))
        key = rng.stream_key(SEED + 1, f"{self.name}/{stream}")
        v = rng.normal(key, start * d, batch * d).astype(np.float32)
        v = v.reshape((batch,) + self.in_shape)
        x = v if self.in_dtype == "f32" else to_bf16_bits(v)
        aux = None
        if self.has_aux:
            # per-sample halting bias b ~ N(-1, 1)
            ka = rng.stream_key(SEED + 1, f"{self.name}/{stream}/halt_bias")
            aux = (rng.normal(ka, start, batch) - 1.0).astype(np.float32)
        return x, aux

    def inputs_f32(self, batch: int, start: int = 0, stream: str = "x"):
        x, aux = self.inputs(batch, start, stream)
        if self.in_dtype == "bf16":
            x = bf16_bits_to_f32(x)
        return x, aux

    # ---- weight blob ----------------------------------------------------
    def blob(self):
        """(bytes, manifest): tensors packed at 256-byte aligned offsets."""
        parts, manifest, off = [], OrderedDict(), 0
        for t in self.tensors.values():
            if t.dtype == "bf16":
                raw = to_bf16_bits(t.value).tobytes()
            else:
                raw = np.ascontiguousarray(t.value, dtype=np.float32).tobytes()
            pad = (-off) % 256
            if pad:
                parts.append(b"\0" * pad)
                off += pad
            manifest[t.name] = {"dtype": t.dtype, "shape": list(t.shape),
                                "offset": off, "nbytes": len(raw)}
            parts.append(raw)
            off += len(raw)
        return b"".join(parts), manifest

    def weights_f32(self):
        """name -> float32 array (bf16 tensors as their exact bf16 values)."""
        out = {}
        for t in self.tensors.values():
            v = np.asarray(t.value, dtype=np.float32)
            if t.dtype == "bf16":
                v = bf16_bits_to_f32(to_bf16_bits(v)).reshape(v.shape)
            out[t.name] = v
        return out


# --------------------------------------------------------------------------
# initialisers
# --------------------------------------------------------------------------

def _u(wl_name, tname, n):
    return rng.uniform(rng.stream_key(SEED, f"{wl_name}/{tname}"), 0, n)


def _n(wl_name, tname, n):
    return rng.normal(rng.stream_key(SEED, f"{wl_name}/{tname}"), 0, n)


def kaiming_uniform(wl, tname, shape, fan_in):
    """U(-b, b) with b = sqrt(6 / fan_in): gain sqrt(2), mode fan_in."""
    b = math.sqrt(6.0 / fan_in)
    n = int(np.prod(shape))
    return ((2.0 * _u(wl, tname, n) - 1.0) * b).astype(np.float32).reshape(shape)


def linear_default(wl, tname, shape, fan_in):
    """PyTorch nn.Linear's default weight init, U(-1/sqrt(fan_in), 1/sqrt(fan_in))."""
    b = 1.0 / math.sqrt(fan_in)
    n = int(np.prod(shape))
    return ((2.0 * _u(wl, tname, n) - 1.0) * b).astype(np.float32).reshape(shape)


# --------------------------------------------------------------------------
# architectures
# --------------------------------------------------------------------------

def _conv(name, k, stride, cin, cout):
    return {"name": name, "k": k, "stride": stride, "pad": k // 2, "cin": cin, "cout": cout}


def _basic(name, cin, cout, stride, gate=None):
    b = {"type": "basic", "name": name, "cin": cin, "cout": cout, "stride": stride,
         "c1": _conv(name + ".c1", 3, stride, cin, cout),
         "c2": _conv(name + ".c2", 3, 1, cout, cout),
         "proj": _conv(name + ".proj", 1, stride, cin, cout) if (stride != 1 or cin != cout) else None}
    if gate is not None:
        b["gate"] = gate
    return b


def _bottleneck(name, cin, mid, cout, stride):
    return {"type": "bottleneck", "name": name, "cin": cin, "mid": mid, "cout": cout, "stride": stride,
            "c1": _conv(name + ".c1", 1, 1, cin, mid),
            "c2": _conv(name + ".c2", 3, stride, mid, mid),
            "c3": _conv(name + ".c3", 1, 1, mid, cout),
            "proj": _conv(name + ".proj", 1, stride, cin, cout) if (stride != 1 or cin != cout) else None}


def arch_mlp_exit(dims=(784, 256, 256, 256), n_classes=10, tau=0.9):
    layers = [{"name": f"fc{k + 1}", "cin": dims[k], "cout": dims[k + 1]} for k in range(len(dims) - 1)]
    heads = [{"name": f"exit{k + 1}", "cin": dims[k + 1]} for k in range(len(dims) - 1)]
    return {"family": "early_exit_mlp", "dtype": "f32", "input": [dims[0]], "layers": layers,
            "heads": heads, "n_classes": n_classes, "n_out": n_classes, "tau": tau}


def arch_resnet_exit(kind, hw, widths, blocks, n_classes, tau, stem_k, stem_stride, maxpool,
                     stem_out=None, expansion=4):
    stem_out = stem_out or widths[0]
    stages, heads, cin = [], [], stem_out
    for s, (w, nb) in enumerate(zip(widths, blocks)):
        bl = []
        for j in range(nb):
            stride = 2 if (j == 0 and s > 0) else 1
            name = f"s{s + 1}.b{j}"
            if kind == "basic":
                bl.append(_basic(name, cin, w, stride))
                cin = w
            else:
                bl.append(_bottleneck(name, cin, w, w * expansion, stride))
                cin = w * expansion
        stages.append(bl)
        heads.append({"name": f"head{s + 1}", "cin": cin})
    return {"family": "early_exit_resnet", "dtype": "bf16", "input": [hw, hw, 3],
            "stem": _conv("stem", stem_k, stem_stride, 3, stem_out), "maxpool": maxpool,
            "stages": stages, "heads": heads, "n_classes": n_classes, "n_out": n_classes, "tau": tau}


def arch_skipnet(hw=32, widths=(16, 32, 64), per_stage=6, n_classes=10):
    blocks, cin, i = [], widths[0], 0
    for s, w in enumerate(widths):
        for j in range(per_stage):
            stride = 2 if (j == 0 and s > 0) else 1
            blocks.append(_basic(f"s{s + 1}.b{j}", cin, w, stride, gate=f"gate{i}"))
            cin, i = w, i + 1
    return {"family": "skipnet", "dtype": "bf16", "input": [hw, hw, 3],
            "stem": _conv("stem", 3, 1, 3, widths[0]), "blocks": blocks,
            "fc": {"name": "fc", "cin": cin}, "n_classes": n_classes, "n_out": n_classes,
            "gate_threshold": 0.5}


def arch_act(hidden=1024, d_in=1024, d_out=1024, max_steps=16, tau=0.99):
    return {"family": "act", "dtype": "bf16", "input": [d_in], "hidden": hidden,
            "n_out": d_out, "max_steps": max_steps, "tau": tau}


def arch_decoder(d_in=512, hidden=512, embed=256, vocab=4096, max_len=24, eos=0, bos=1, out_gain=32.0):
    """Greedy LSTM decoder: h0 = tanh(W_enc x + b_enc), c0 = 0, then one token
    per step until the end token `eos` or `max_len` tokens; the first step
    reads the start token `bos`.  The output layer is drawn with gain
    `out_gain` over nn.Linear's default range (a trained decoder's output
    distribution is peaked; at gain 1 the two largest logits of a step lie
    ~1e-2 apart)."""
    return {"family": "seq_decoder", "dtype": "bf16", "input": [d_in], "hidden": hidden, "embed": embed,
            "vocab": vocab, "n_out": vocab, "max_len": max_len, "eos": eos, "bos": bos, "out_gain": out_gain}


ARCHS = {
    "mlp_exit": lambda: arch_mlp_exit(),
    "resnet18_exit": lambda: arch_resnet_exit("basic", 32, [64, 128, 256, 512], [2, 2, 2, 2], 100, 0.8,
                                              3, 1, False),
    "skipnet38": lambda: arch_skipnet(),
    "resnet50_exit": lambda: arch_resnet_exit("bottleneck", 224, [64, 128, 256, 512], [3, 4, 6, 3], 1000,
                                              0.7, 7, 2, True, stem_out=64),
    "act_loop": lambda: arch_act(),
    "lstm_decoder": lambda: arch_decoder(),
}


def all_convs(arch):
    """Every conv of a CNN architecture in program order."""
    out = [arch["stem"]]
    blocks = arch.get("blocks") or [b for st in arch.get("stages", []) for b in st]
    for b in blocks:
        keys = ["c1", "c2"] + (["c3"] if b["type"] == "bottleneck" else [])
        if b["proj"] is not None:
            keys = ["proj"] + keys
        out += [b[k] for k in keys]
    return out


# --------------------------------------------------------------------------
# weights
# --------------------------------------------------------------------------

def _add(wl, name, dtype, value):
    value = np.asarray(value, dtype=np.float32)
    wl.tensors[name] = Tensor(name, dtype, tuple(value.shape), value)


def _load_calib(name):
    path = os.path.join(CALIB_DIR, f"{name}.npz")
    if not os.path.exists(path):
        return None
    with np.load(path, allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


def raw_workload(name: str, arch: dict | None = None) -> Workload:
    """The workload before calibration (literal reading of its description)."""
    arch = arch or ARCHS[name]()
    wl = Workload(name, arch)
    fam = arch["family"]
    if fam == "early_exit_mlp":
        for L in arch["layers"]:
            _add(wl, L["name"] + ".w", "f32", kaiming_uniform(name, L["name"] + ".w", (L["cout"], L["cin"]), L["cin"]))
            _add(wl, L["name"] + ".b", "f32", np.zeros(L["cout"]))
        for h in arch["heads"]:
            nc = arch["n_classes"]
            _add(wl, h["name"] + ".w", "f32", kaiming_uniform(name, h["name"] + ".w", (nc, h["cin"]), h["cin"]))
            _add(wl, h["name"] + ".b", "f32", 4.0 * _u(name, h["name"] + ".b", nc) - 2.0)   # U(-2, 2)
            _add(wl, h["name"] + ".T", "f32", np.ones(1))
    elif fam in ("early_exit_resnet", "skipnet"):
        for c in all_convs(arch):
            fan = c["k"] * c["k"] * c["cin"]
            _add(wl, c["name"] + ".w", "bf16",
                 kaiming_uniform(name, c["name"] + ".w", (c["cout"], c["k"], c["k"], c["cin"]), fan))
            # BatchNorm at eval defaults (gamma 1, beta 0, mean 0, var 1) folded to scale/shift
            _add(wl, c["name"] + ".a", "f32", np.full(c["cout"], 1.0 / math.sqrt(1.0 + BN_EPS)))
            _add(wl, c["name"] + ".b", "f32", np.zeros(c["cout"]))
        if fam == "early_exit_resnet":
            for h in arch["heads"]:
                nc = arch["n_classes"]
                _add(wl, h["name"] + ".w", "f32", linear_default(name, h["name"] + ".w", (nc, h["cin"]), h["cin"]))
                _add(wl, h["name"] + ".b", "f32", np.zeros(nc))
                _add(wl, h["name"] + ".T", "f32", np.ones(1))
        else:
            for b in arch["blocks"]:
                g, c = b["gate"], b["cin"]
                _add(wl, g + ".u", "f32", kaiming_uniform(name, g + ".u", (c,), c))
                _add(wl, g + ".v", "f32", 1.5 * _n(name, g + ".v", 1))            # N(0, 1.5)
            fc = arch["fc"]
            _add(wl, "fc.w", "f32", kaiming_uniform(name, "fc.w", (arch["n_classes"], fc["cin"]), fc["cin"]))
            _add(wl, "fc.b", "f32", np.zeros(arch["n_classes"]))
    elif fam == "act":
        H, D, O = arch["hidden"], arch["input"][0], arch["n_out"]
        _add(wl, "W1", "bf16", linear_default(name, "W1", (H, H + D), H + D))
        _add(wl, "b1", "f32", np.zeros(H))
        _add(wl, "w_halt", "f32", linear_default(name, "w_halt", (H,), H))
        _add(wl, "W2", "bf16", linear_default(name, "W2", (O, H), H))
        _add(wl, "b2", "f32", np.zeros(O))
    elif fam == "seq_decoder":
        H, D, E, V = arch["hidden"], arch["input"][0], arch["embed"], arch["vocab"]
        # PyTorch's defaults: nn.Linear U(+-1/sqrt(fan_in)) for the encoder,
        # nn.Embedding N(0, 1), nn.LSTM U(+-1/sqrt(hidden)) for weights and
        # both biases (summed here), nn.Linear for the output projection
        _add(wl, "enc.w", "bf16", linear_default(name, "enc.w", (H, D), D))
        _add(wl, "enc.b", "f32", linear_default(name, "enc.b", (H,), D))
        _add(wl, "emb", "bf16", _n(name, "emb", V * E).astype(np.float32).reshape(V, E))
        _add(wl, "lstm.w", "bf16", linear_default(name, "lstm.w", (4 * H, H + E), H))
        _add(wl, "lstm.b", "f32", linear_default(name, "lstm.b_ih", (4 * H,), H)
             + linear_default(name, "lstm.b_hh", (4 * H,), H))
        g = arch["out_gain"]
        _add(wl, "out.w", "bf16", g * linear_default(name, "out.w", (V, H), H))
        _add(wl, "out.b", "f32", g * linear_default(name, "out.b", (V,), H))
    else:
        raise ValueError(fam)
    return wl


def apply_calibration(wl: Workload, cal: dict) -> Workload:
    """Overwrite the calibrated tensors with the stored constants."""
    for k, v in cal.items():
        if k.startswith("_"):
            continue
        if k not in wl.tensors:
            raise KeyError(f"calibration constant {k} has no tensor in {wl.name}")
        t = wl.tensors[k]
        v = np.asarray(v, dtype=np.float32).reshape(t.shape)
        wl.tensors[k] = Tensor(k, t.dtype, t.shape, v)
    wl.calibrated = True
    return wl


def build(name: str, calibrated: bool = True) -> Workload:
    wl = raw_workload(name)
    if calibrated and name != "act_loop":
        cal = _load_calib(name)
        if cal is None:
            raise FileNotFoundError(f"calibration file for {name} missing in {CALIB_DIR}")
        apply_calibration(wl, cal)
    return wl


def arch_json(wl: Workload) -> str:
    return json.dumps(wl.arch, sort_keys=True)
