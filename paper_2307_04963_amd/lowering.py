"""Front-end: lower a dynamic network's description to the plan spec.

This is the host-side counterpart of the paper's rewriting and HCFG
construction (Sec. 5.2-5.3, Alg. 1) for the network families used here:
every loop is unrolled (the bounded loop of an adaptive-computation network
becomes max_steps copies of its body), and the program is split into
sub-DNN nodes (runs of convolutions / linear layers) and logic nodes (one
conditional each: an exit test, a gate, a halting test, a decoder's token
choice).  The identity path
of a skipped block (Sec. 5.4, first strategy) needs no node at all: a
skipped sample's row is left where it is.

Input: the architecture dict and the weight manifest (tensor name ->
offset / dtype / shape in the blob).  Output: the JSON spec read by
``dycl_plan_create``.
"""

from __future__ import annotations

import json


class _Lower:
    def __init__(self, arch, manifest):
        self.arch, self.man = arch, manifest
        self.nodes = []
        self.n = 0

    def fresh(self, base):
        self.n += 1
        return f"{base}.{self.n}"

    def off(self, name):
        return self.man[name]["offset"]

    def conv(self, src, c, act, res=None, out=None, nodes=None):
        dst = out or self.fresh(c["name"])
        (self.nodes if nodes is None else nodes).append({
            "op": "conv", "src": src, "dst": dst, "res": res, "k": c["k"], "stride": c["stride"], "pad": c["pad"],
            "cout": c["cout"], "act": act, "w": {"off": self.off(c["name"] + ".w")},
            "scale": self.off(c["name"] + ".a"), "shift": self.off(c["name"] + ".b")})
        return dst

    def exit(self, src, head, index, final, tau, T=True):
        node = {"op": "exit", "src": src, "w": self.off(head + ".w"), "b": self.off(head + ".b"),
                "ncls": self.arch["n_out"], "tau": tau, "index": index, "final": final}
        if T:
            node["T"] = self.off(head + ".T")
        out = src
        if not final:
            out = self.fresh(src.split(".")[0] + "_c")
            node["carry"] = [[src, out]]
        self.nodes.append(node)
        return out

    # ---- families -------------------------------------------------------
    def mlp(self):
        a = self.arch
        h = "x"
        last = len(a["layers"]) - 1
        for k, (L, H) in enumerate(zip(a["layers"], a["heads"])):
            d = self.fresh(L["name"])
            self.nodes.append({"op": "conv", "src": h, "dst": d, "k": 1, "cout": L["cout"], "act": "relu",
                               "w": {"off": self.off(L["name"] + ".w")}, "shift": self.off(L["name"] + ".b")})
            h = self.exit(d, H["name"], k, k == last, a["tau"])

    def block(self, x, b, nodes=None, src_override=None, res_override=None):
        src = src_override or x
        if b["type"] == "basic":
            t = self.conv(src, b["c1"], "relu", nodes=nodes)
            return self.conv(t, b["c2"], "relu", res=res_override, nodes=nodes)
        t = self.conv(src, b["c1"], "relu", nodes=nodes)
        t = self.conv(t, b["c2"], "relu", nodes=nodes)
        return self.conv(t, b["c3"], "relu", res=res_override, nodes=nodes)

    def resnet_exit(self):
        a = self.arch
        y = self.conv("x", a["stem"], "relu")
        if a["maxpool"]:
            p = self.fresh("pool")
            self.nodes.append({"op": "maxpool", "src": y, "dst": p})
            y = p
        last = len(a["stages"]) - 1
        for s, stage in enumerate(a["stages"]):
            for b in stage:
                sc = self.conv(y, b["proj"], "none") if b["proj"] is not None else y
                y = self.block(y, b, res_override=sc)
            y = self.exit(y, a["heads"][s]["name"], s, s == last, a["tau"])

    def skipnet(self):
        a = self.arch
        x = self.conv("x", a["stem"], "relu")
        for i, b in enumerate(a["blocks"]):
            body = []
            xg = self.fresh("xg")
            gather = [[x, xg]]
            if b["proj"] is not None:
                # the shortcut projection is what every sample of this block
                # needs (a skipped sample's output, an executed one's residual)
                y = self.conv(x, b["proj"], "none")
                pg = self.fresh("pg")
                gather.append([y, pg])
                res = pg
            else:
                y, res = x, xg
            yg = self.block(None, b, nodes=body, src_override=xg, res_override=res)
            self.nodes.append({"op": "gate", "src": x, "u": self.off(b["gate"] + ".u"),
                               "v": self.off(b["gate"] + ".v"), "threshold": a["gate_threshold"], "index": i,
                               "gather": gather, "body": body, "scatter": [[yg, y]]})
            x = y
        self.exit(x, "fc", -1, True, 0.0, T=False)

    def act(self):
        a = self.arch
        H, T = a["hidden"], a["max_steps"]
        ldk = H + a["input"][0]
        x, h = "x", None
        for t in range(1, T + 1):
            d = f"h{t}"
            node = {"op": "conv", "src": h if h else x, "dst": d, "k": 1, "cout": H, "act": "gelu",
                    "shift": self.off("b1")}
            if h is None:        # h0 = 0: only the x columns of W1 contribute
                node["w"] = {"off": self.off("W1"), "ldk": ldk, "k0": H}
            else:
                node["src2"] = x
                node["w"] = {"off": self.off("W1"), "ldk": ldk, "k0": 0}
            self.nodes.append(node)
            halt = {"op": "halt", "src": d, "w": self.off("w_halt"), "tau": a["tau"], "step": t, "max_steps": T,
                    "park": [d, "h_final"]}
            if t < T:
                h, xn = f"h{t}c", f"x{t}"
                halt["carry"] = [[d, h], [x, xn]]
                x = xn
            self.nodes.append(halt)
        self.nodes.append({"op": "output", "src": "h_final", "w": {"off": self.off("W2")}, "bias": self.off("b2"),
                           "cout": a["n_out"]})


    def decoder(self):
        # greedy decoding unrolled to max_len steps: each step an LSTM cell
        # (a linear layer over [h; embedding of the previous token] whose
        # epilogue is the cell) and a logic node choosing the token, whose
        # end test moves finished rows out; h and the cell state are carried
        a = self.arch
        H, L = a["hidden"], a["max_len"]
        self.nodes.append({"op": "conv", "src": "x", "dst": "h0", "k": 1, "cout": H, "act": "tanh",
                           "w": {"off": self.off("enc.w")}, "shift": self.off("enc.b")})
        h, c = "h0", None
        for t in range(1, L + 1):
            hn, cn = f"h{t}", f"c{t}"
            self.nodes.append({"op": "conv", "act": "lstm", "src": h, "cell_in": c, "dst": hn, "cell_out": cn,
                               "cout": 4 * H, "w": {"off": self.off("lstm.w")}, "shift": self.off("lstm.b"),
                               "emb": {"off": self.off("emb"), "rows": a["vocab"], "dim": a["embed"]}})
            node = {"op": "decode", "src": hn, "w": {"off": self.off("out.w")}, "b": self.off("out.b"),
                    "eos": a["eos"], "step": t}
            if t < L:
                h, c = f"h{t}c", f"c{t}c"
                node["carry"] = [[hn, h], [cn, c]]
            self.nodes.append(node)


def lower(arch: dict, manifest: dict) -> dict:
    """Spec dict for one architecture and its blob manifest."""
    L = _Lower(arch, manifest)
    fam = arch["family"]
    {"early_exit_mlp": L.mlp, "early_exit_resnet": L.resnet_exit, "skipnet": L.skipnet, "act": L.act,
     "seq_decoder": L.decoder}[fam]()
    spec = {"version": 1, "dtype": arch["dtype"], "input": {"name": "x", "shape": list(arch["input"])},
            "n_out": arch["n_out"], "aux": fam == "act", "nodes": L.nodes}
    if fam == "seq_decoder":
        spec["decode"] = {"max_len": arch["max_len"], "bos": arch["bos"]}
    return spec


def lower_json(arch: dict, manifest: dict) -> str:
    return json.dumps(lower(arch, manifest))
