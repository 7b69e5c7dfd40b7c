"""The workload networks written as ordinary PyTorch dynamic networks (one
sample per call, conditionals and loops in Python), for the front-end
tests.  Weights come from the workload's tensors; BatchNorm is given the
folded scale / shift as its affine parameters with zero mean, unit variance
and eps 0, so that folding it back gives the same float32 values."""

from __future__ import annotations

import numpy as np
import torch
import torch.nn as nn
import torch.nn.functional as F

from workloads import configs


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))


def conv_bn(W, c):
    conv = nn.Conv2d(c["cin"], c["cout"], c["k"], c["stride"], c["pad"], bias=False)
    conv.weight.data = _t(W[c["name"] + ".w"].transpose(0, 3, 1, 2))     # [cout][kh][kw][cin] -> [cout][cin][kh][kw]
    bn = nn.BatchNorm2d(c["cout"], eps=0.0)
    bn.weight.data = _t(W[c["name"] + ".a"])
    bn.bias.data = _t(W[c["name"] + ".b"])
    bn.running_mean.zero_()
    bn.running_var.fill_(1.0)
    return nn.Sequential(conv, bn)


def linear(W, name, cin, cout, bias=True):
    m = nn.Linear(cin, cout, bias=bias)
    m.weight.data = _t(W[name + ".w"] if name + ".w" in W else W[name]).reshape(cout, cin)
    if bias:
        m.bias.data = _t(W[name + ".b"])
    return m


class Basic(nn.Module):
    def __init__(self, W, b):
        super().__init__()
        self.cb1 = conv_bn(W, b["c1"])
        self.cb2 = conv_bn(W, b["c2"])
        self.proj = conv_bn(W, b["proj"]) if b["proj"] is not None else None

    def forward(self, x):
        sc = x if self.proj is None else self.proj(x)
        y = F.relu(self.cb1(x))
        y = self.cb2(y)
        return F.relu(y + sc)


class GatedBasic(nn.Module):
    """A SkipNet block: the shortcut comes in from outside (every sample
    needs it, executed or skipped)."""

    def __init__(self, W, b):
        super().__init__()
        self.cb1 = conv_bn(W, b["c1"])
        self.cb2 = conv_bn(W, b["c2"])
        self.proj = conv_bn(W, b["proj"]) if b["proj"] is not None else None

    def forward(self, x, sc):
        y = F.relu(self.cb1(x))
        y = self.cb2(y)
        return F.relu(y + sc)


class Bottleneck(nn.Module):
    def __init__(self, W, b):
        super().__init__()
        self.cb1 = conv_bn(W, b["c1"])
        self.cb2 = conv_bn(W, b["c2"])
        self.cb3 = conv_bn(W, b["c3"])
        self.proj = conv_bn(W, b["proj"]) if b["proj"] is not None else None

    def forward(self, x):
        sc = x if self.proj is None else self.proj(x)
        y = F.relu(self.cb1(x))
        y = F.relu(self.cb2(y))
        y = self.cb3(y)
        return F.relu(y + sc)


class EarlyExitResNet(nn.Module):
    def __init__(self, wl):
        super().__init__()
        a, W = wl.arch, wl.weights_f32()
        self.stem = conv_bn(W, a["stem"])
        self.pool = a["maxpool"]
        Block = Basic if a["stages"][0][0]["type"] == "basic" else Bottleneck
        self.stages = nn.ModuleList([nn.Sequential(*[Block(W, b) for b in st]) for st in a["stages"]])
        self.heads = nn.ModuleList([linear(W, h["name"], h["cin"], a["n_classes"]) for h in a["heads"]])
        self.register_buffer("T", _t(np.concatenate([W[h["name"] + ".T"] for h in a["heads"]])))
        self.tau = a["tau"]

    def forward(self, x):
        x = F.relu(self.stem(x))
        if self.pool:
            x = F.max_pool2d(x, 3, 2, 1)
        last = len(self.stages) - 1
        for s in range(len(self.stages)):
            x = self.stages[s](x)
            z = self.heads[s](torch.flatten(F.adaptive_avg_pool2d(x, 1), 1))
            if s == last:
                return z
            if torch.max(F.softmax(z / self.T[s], dim=1)) >= self.tau:
                return z


class SkipNet(nn.Module):
    def __init__(self, wl):
        super().__init__()
        a, W = wl.arch, wl.weights_f32()
        self.stem = conv_bn(W, a["stem"])
        self.blocks = nn.ModuleList([GatedBasic(W, b) for b in a["blocks"]])
        gates = []
        for b in a["blocks"]:
            g = nn.Linear(b["cin"], 1)
            g.weight.data = _t(W[b["gate"] + ".u"]).reshape(1, -1)
            g.bias.data = _t(W[b["gate"] + ".v"])
            gates.append(g)
        self.gates = nn.ModuleList(gates)
        self.fc = linear(W, "fc", a["fc"]["cin"], a["n_classes"])
        self.thr = a["gate_threshold"]

    def forward(self, x):
        x = F.relu(self.stem(x))
        for i in range(len(self.blocks)):
            b = self.blocks[i]
            sc = x if b.proj is None else b.proj(x)
            g = torch.sigmoid(self.gates[i](torch.flatten(F.adaptive_avg_pool2d(x, 1), 1)))
            if g > self.thr:
                x = b(x, sc)
            else:
                x = sc
        return self.fc(torch.flatten(F.adaptive_avg_pool2d(x, 1), 1))


class EarlyExitMLP(nn.Module):
    def __init__(self, wl):
        super().__init__()
        a, W = wl.arch, wl.weights_f32()
        self.layers = nn.ModuleList([linear(W, L["name"], L["cin"], L["cout"]) for L in a["layers"]])
        self.heads = nn.ModuleList([linear(W, h["name"], h["cin"], a["n_classes"]) for h in a["heads"]])
        self.register_buffer("T", _t(np.concatenate([W[h["name"] + ".T"] for h in a["heads"]])))
        self.tau = a["tau"]

    def forward(self, x):
        last = len(self.layers) - 1
        for k in range(len(self.layers)):
            x = F.relu(self.layers[k](x))
            z = self.heads[k](x)
            if k == last:
                return z
            if torch.max(F.softmax(z / self.T[k], dim=-1)) >= self.tau:
                return z


class AdaptiveLoop(nn.Module):
    """Adaptive computation time: the state is updated until the running
    halting probability reaches tau, at most max_steps times; the second
    input is the sample's halting bias."""

    def __init__(self, wl):
        super().__init__()
        a, W = wl.arch, wl.weights_f32()
        H, D, O = a["hidden"], a["input"][0], a["n_out"]
        self.H, self.T, self.tau = H, a["max_steps"], a["tau"]
        self.W1 = nn.Linear(H + D, H)
        self.W1.weight.data = _t(W["W1"])
        self.W1.bias.data = _t(W["b1"])
        self.halt = nn.Linear(H, 1, bias=False)
        self.halt.weight.data = _t(W["w_halt"]).reshape(1, H)
        self.W2 = nn.Linear(H, O)
        self.W2.weight.data = _t(W["W2"])
        self.W2.bias.data = _t(W["b2"])

    def forward(self, x, b):
        h = torch.zeros(1, self.H)
        S = 0
        for t in range(self.T):
            h = F.gelu(self.W1(torch.cat((h, x), dim=1)))
            S = S + torch.sigmoid(self.halt(h) + b)
            if S >= self.tau:
                break
        return self.W2(h)


MODULES = {"mlp_exit": EarlyExitMLP, "resnet18_exit": EarlyExitResNet, "resnet50_exit": EarlyExitResNet,
           "skipnet38": SkipNet, "act_loop": AdaptiveLoop}


def module_for(name, wl=None):
    wl = wl or configs.build(name)
    return MODULES[name](wl).eval(), wl


def input_shape(wl):
    s = wl.arch["input"]
    return (s[2], s[0], s[1]) if len(s) == 3 else (s[0],)
