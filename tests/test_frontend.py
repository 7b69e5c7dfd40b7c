"""The front-end (the compiler half: rewriting, HCFG, graph optimisation,
shape propagation) against the hand lowering of the same networks.

Each workload network is written as an ordinary PyTorch module
(tests/dynn_modules.py) and compiled from its forward's source.  The
resulting spec must describe the same program as the architecture lowering:
the same node kinds in the same order with the same layer parameters,
decisions, carries, gathers and scatters (tensor names aside), and every
weight the spec references must hold the same bytes.  The GPU test then runs
both plans on the same inputs: bit-identical results."""

import json

import numpy as np
import pytest

from paper_2307_04963_amd.frontend import FrontendError, compile_module
from paper_2307_04963_amd.lowering import lower
from tests.dynn_modules import module_for, input_shape
from workloads import configs

NAMES = ["mlp_exit", "resnet18_exit", "skipnet38", "resnet50_exit", "act_loop"]


def _shapes(spec):
    """tensor name -> (H, W, C), propagated like the plan builder does."""
    s = spec["input"]["shape"]
    sh = {"x": tuple(s) if len(s) == 3 else (1, 1, s[0])}

    def walk(nodes):
        for n in nodes:
            op = n["op"]
            if op == "conv":
                H, W, C = sh[n["src"]]
                if n.get("src2"):
                    C += sh[n["src2"]][2]
                k, st, p = n.get("k", 1), n.get("stride", 1), n.get("pad", 0)
                sh[n["dst"]] = ((H + 2 * p - k) // st + 1, (W + 2 * p - k) // st + 1, n["cout"])
                n["_cin"] = C
            elif op == "maxpool":
                H, W, C = sh[n["src"]]
                sh[n["dst"]] = ((H - 1) // 2 + 1, (W - 1) // 2 + 1, C)
            for key in ("carry", "gather"):
                for a, b in n.get(key, []):
                    sh[b] = sh[a]
            if op == "halt":
                sh[n["park"][1]] = sh[n["park"][0]]
            walk(n.get("body", []))
    walk(spec["nodes"])
    return sh


def _canon(spec, blob):
    """The spec with tensor names replaced by first-appearance numbers and
    every weight offset by the bytes it refers to."""
    spec = json.loads(json.dumps(spec))
    sh = _shapes(spec)
    names = {"x": "x", "h_final": "h_final"}
    esz = 2 if spec["dtype"] == "bf16" else 4

    def nm(t):
        if t is None:
            return None
        if t not in names:
            names[t] = f"t{len(names)}"
        return names[t]

    def raw(off, n):
        return bytes(blob[off:off + n])

    out = []

    def walk(nodes, dst):
        for n in nodes:
            op = n["op"]
            c = {"op": op}
            if op == "conv":
                K = n["k"] * n["k"] * n["_cin"]
                w = n["w"]
                ldk, k0 = w.get("ldk", K), w.get("k0", 0)
                rows = [raw(w["off"] + (r * ldk + k0) * esz, K * esz) for r in range(n["cout"])]
                c.update(src=nm(n["src"]), src2=nm(n.get("src2")), res=nm(n.get("res")), k=n["k"],
                         stride=n.get("stride", 1), pad=n.get("pad", 0), cout=n["cout"], act=n.get("act", "none"),
                         w=b"".join(rows),
                         scale=raw(n["scale"], 4 * n["cout"]) if n.get("scale") is not None else None,
                         shift=raw(n["shift"], 4 * n["cout"]) if n.get("shift") is not None else None)
                c["dst"] = nm(n["dst"])
            elif op == "maxpool":
                c.update(src=nm(n["src"]), dst=nm(n["dst"]))
            elif op == "exit":
                C = sh[n["src"]][2]
                c.update(src=nm(n["src"]), w=raw(n["w"], 4 * n["ncls"] * C), b=raw(n["b"], 4 * n["ncls"]),
                         ncls=n["ncls"], index=n["index"], final=n["final"],
                         tau=None if n["final"] else n["tau"], T=None if n["final"] else raw(n["T"], 4),
                         carry=[[nm(a), nm(b)] for a, b in n.get("carry", [])])
            elif op == "gate":
                C = sh[n["src"]][2]
                c.update(src=nm(n["src"]), u=raw(n["u"], 4 * C), v=raw(n["v"], 4), thr=n["threshold"],
                         index=n["index"], gather=[[nm(a), nm(b)] for a, b in n["gather"]])
                body = []
                walk(n["body"], body)
                c["body"] = body
                c["scatter"] = [[nm(a), nm(b)] for a, b in n["scatter"]]
            elif op == "halt":
                C = sh[n["src"]][2]
                c.update(src=nm(n["src"]), w=raw(n["w"], 4 * C), tau=n["tau"], step=n["step"],
                         max_steps=n["max_steps"], park=[nm(n["park"][0]), nm(n["park"][1])],
                         carry=[[nm(a), nm(b)] for a, b in n.get("carry", [])])
            elif op == "output":
                C = sh[n["src"]][2]
                c.update(src=nm(n["src"]), w=raw(n["w"]["off"], 2 * n["cout"] * C), bias=raw(n["bias"], 4 * n["cout"]),
                         cout=n["cout"])
            dst.append(c)
    walk(spec["nodes"], out)
    return {"dtype": spec["dtype"], "input": spec["input"]["shape"], "n_out": spec["n_out"],
            "aux": bool(spec.get("aux")), "nodes": out}


@pytest.mark.parametrize("name", NAMES)
def test_frontend_matches_lowering(name):
    m, wl = module_for(name)
    spec, blob = compile_module(m, input_shape(wl), wl.arch["dtype"])
    rblob, man = wl.blob()
    ref = lower(wl.arch, man)
    a, b = _canon(spec, blob), _canon(ref, rblob)
    assert len(a["nodes"]) == len(b["nodes"])
    for i, (x, y) in enumerate(zip(a["nodes"], b["nodes"])):
        assert x == y, f"node {i}: {x['op']} differs: " + ", ".join(
            k for k in set(x) | set(y) if x.get(k) != y.get(k))
    assert a == b


def test_frontend_rejects_what_no_kernel_runs():
    import torch
    import torch.nn as nn
    import torch.nn.functional as F

    class Tanh(nn.Module):
        def __init__(self):
            super().__init__()
            self.fc = nn.Linear(8, 4)

        def forward(self, x):
            return self.fc(torch.tanh(x))

    class DataLoop(nn.Module):
        def __init__(self):
            super().__init__()
            self.fc = nn.Linear(8, 8)
            self.head = nn.Linear(8, 4)

        def forward(self, x):
            while x.sum() > 0:
                x = self.fc(x)
            return self.head(x)

    class BadExit(nn.Module):
        def __init__(self):
            super().__init__()
            self.fc = nn.Linear(8, 8)
            self.head = nn.Linear(8, 4)

        def forward(self, x):
            z = self.head(F.relu(self.fc(x)))
            if torch.max(F.softmax(z, dim=1)) >= 0.5:
                return x
            return z

    for M in (Tanh, DataLoop, BadExit):
        with pytest.raises(FrontendError):
            compile_module(M(), (8,), "f32")


def test_frontend_constant_propagation_and_unrolling():
    # conditions on Python values are decided at compile time (no node), a
    # loop over a ModuleList unrolls, a zero state drops its weight columns
    import torch
    import torch.nn as nn
    import torch.nn.functional as F

    class Net(nn.Module):
        def __init__(self):
            super().__init__()
            self.layers = nn.ModuleList([nn.Linear(16, 16) for _ in range(3)])
            self.use_last = False
            self.head = nn.Linear(16, 4)

        def forward(self, x):
            for i, L in enumerate(self.layers):
                if i < 2 or self.use_last:
                    x = F.relu(L(x))
            return self.head(x)

    spec, _ = compile_module(Net(), (16,), "f32")
    ops = [n["op"] for n in spec["nodes"]]
    assert ops == ["conv", "conv", "exit"]
    assert spec["nodes"][-1]["final"] and spec["nodes"][-1]["index"] == -1
