"""Front-end: compile a dynamic network written as a PyTorch module into the
plan spec and weight blob that ``dycl_plan_create`` reads.

This is the compiler half of DyCL (Sec. 5), for programs whose tensor
statements are the layers the executor runs and whose conditionals are the
three decisions it evaluates on the device:

* program rewriting (Sec. 5.2): the module's ``forward`` is interpreted
  from its source (``ast``), not traced, so every ``for`` loop with a
  trip count known at compile time is unrolled, Python values are
  propagated as constants (loop indices, ``len(self.blocks)``, conditions
  on them), and calls of user sub-modules are inlined.  A tensor known to
  be zero (``torch.zeros``) is propagated too: a linear layer applied to a
  concatenation with a zero block keeps only the columns of the other part.
* HCFG construction (Sec. 5.3, Alg. 1): tensor statements form sub-DNN
  nodes; an ``if`` whose condition depends on tensor data is a logic node.
  Three shapes of conditional are recognised from the condition's dataflow:
    - exit:  ``if max(softmax(z / T)) >= tau: return z`` with
             z = Linear(flatten(avgpool(x))) (or Linear(x) on vectors);
    - gate:  ``if sigmoid(Linear(flatten(avgpool(x)))) > thr: <assignments>``
             with an optional ``else`` (Linear with one output);
    - halt:  ``S = S + sigmoid(Linear(h) + b)`` then
             ``if S >= tau: break`` inside an unrolled loop, where ``b`` is
             the module's second input (a per-sample bias).
  An unconditional final ``return Linear(...)`` is a final exit (or, after
  a halting loop, the output layer on the parked states).
* graph optimisation (Sec. 5.4): a gate's ``else`` value that is a tensor
  that already exists (the identity path) costs nothing: the executed rows'
  results are written over it in place; values computed only on the
  ``else`` path (a shortcut projection) are hoisted in front of the gate,
  because the executed rows need them too.
* shape propagation (Alg. 2): every value carries its per-sample shape from
  the input on, and each layer checks its operands against it.
* sub-DNN compilation: convolution, BatchNorm (folded into a per-channel
  scale / shift), residual addition and activation fuse into one conv node
  (one kernel with its epilogue); weights go to a blob (bf16 for
  convolutions and bf16 linear layers in K order (kh, kw, ci), float32 for
  heads, folded BatchNorm, biases).

Anything outside this subset is rejected with FrontendError naming the
source line.
"""

from __future__ import annotations

import ast
import inspect
import json
import math
import textwrap
from dataclasses import dataclass, field

import numpy as np
import torch
import torch.nn as nn
import torch.nn.functional as F


class FrontendError(Exception):
    pass


# ------------------------------------------------------------- values ----

@dataclass(eq=False)
class Sym:
    """A per-sample tensor value of the program (batch dimension 1)."""
    op: str
    args: tuple = ()
    attrs: dict = field(default_factory=dict)
    shape: tuple = ()
    uses: int = 0

    def __repr__(self):
        return f"Sym({self.op}, {self.shape})"


class Aux:
    """The module's second input: one float per sample."""


@dataclass
class Decision:
    kind: str            # exit | gate | halt
    attrs: dict


class _Break(Exception):
    pass


class _Return(Exception):
    def __init__(self, value):
        self.value = value


_TORCH_FUNCS = {
    torch.relu: "relu", F.relu: "relu", F.gelu: "gelu", torch.sigmoid: "sigmoid", F.softmax: "softmax",
    torch.softmax: "softmax", torch.max: "max", torch.cat: "cat", torch.flatten: "flatten",
    F.adaptive_avg_pool2d: "gap", torch.zeros: "zeros", torch.zeros_like: "zeros_like", F.max_pool2d: "max_pool2d",
}


def _bf16_bits(a: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    return ((b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


# -------------------------------------------------------- interpreter ----

class _Interp:
    """Runs ``forward`` on symbolic tensors and records the program as a
    trace: tensor values (Syms) and decisions in program order."""

    def __init__(self):
        self.trace = []          # list of ("sym", Sym) | ("decision", Decision) | ("return", Sym)
        self.loop_halts = None   # halts of the loop being unrolled
        self.n_exits = 0

    # ---- values -------------------------------------------------------
    def sym(self, op, args=(), shape=(), **attrs):
        s = Sym(op, tuple(args), attrs, tuple(shape))
        for a in args:
            if isinstance(a, Sym):
                a.uses += 1
        self.trace.append(("sym", s))
        return s

    def fail(self, node, msg):
        line = getattr(node, "lineno", "?")
        raise FrontendError(f"line {line} of forward: {msg}")

    # ---- module calls ---------------------------------------------------
    def call_module(self, m, args, node):
        if isinstance(m, nn.Sequential):
            v = args[0]
            for sub in m:
                v = self.call_module(sub, [v], node)
            return v
        if isinstance(m, nn.Identity):
            return args[0]
        x = args[0] if args else None
        if isinstance(m, nn.Conv2d):
            if not isinstance(x, Sym) or len(x.shape) != 4:
                self.fail(node, "Conv2d needs an image tensor")
            if m.groups != 1 or m.dilation != (1, 1) or m.kernel_size[0] != m.kernel_size[1] or \
                    m.stride[0] != m.stride[1] or m.padding[0] != m.padding[1] or m.padding_mode != "zeros":
                self.fail(node, "Conv2d must be square, ungrouped, undilated, zero-padded")
            k, s, p = m.kernel_size[0], m.stride[0], m.padding[0]
            _, C, H, W = x.shape
            if C != m.in_channels:
                self.fail(node, f"Conv2d expects {m.in_channels} channels, gets {C}")
            Ho, Wo = (H + 2 * p - k) // s + 1, (W + 2 * p - k) // s + 1
            return self.sym("conv", (x,), (1, m.out_channels, Ho, Wo), mod=m)
        if isinstance(m, nn.BatchNorm2d):
            if not isinstance(x, Sym) or x.shape[1] != m.num_features:
                self.fail(node, "BatchNorm2d on a tensor of another width")
            return self.sym("bn", (x,), x.shape, mod=m)
        if isinstance(m, nn.ReLU):
            return self.sym("relu", (x,), x.shape)
        if isinstance(m, nn.GELU):
            if m.approximate != "none":
                self.fail(node, "only the exact GELU is supported")
            return self.sym("gelu", (x,), x.shape)
        if isinstance(m, nn.MaxPool2d):
            return self.max_pool(x, m.kernel_size, m.stride, m.padding, node)
        if isinstance(m, nn.Linear):
            if not isinstance(x, Sym) or x.shape[-1] != m.in_features or len(x.shape) != 2:
                self.fail(node, f"Linear({m.in_features}) on {getattr(x, 'shape', x)}")
            return self.sym("linear", (x,), (1, m.out_features), mod=m)
        if isinstance(m, nn.Module):
            return self.inline(m, args, node)
        self.fail(node, f"cannot call {type(m).__name__}")

    def max_pool(self, x, k, s, p, node):
        norm = lambda v: v if isinstance(v, int) else (v[0] if v[0] == v[1] else None)  # noqa: E731
        if (norm(k), norm(s), norm(p)) != (3, 2, 1):
            self.fail(node, "only 3x3 / stride 2 / pad 1 max pooling is supported")
        _, C, H, W = x.shape
        return self.sym("maxpool", (x,), (1, C, (H - 1) // 2 + 1, (W - 1) // 2 + 1))

    def inline(self, m, args, node):
        fn = type(m).forward
        try:
            src = textwrap.dedent(inspect.getsource(fn))
        except (OSError, TypeError):
            self.fail(node, f"no source for {type(m).__name__}.forward")
        fdef = ast.parse(src).body[0]
        params = [a.arg for a in fdef.args.args]
        if len(args) > len(params) - 1:
            self.fail(node, f"too many arguments for {type(m).__name__}.forward")
        defaults = fdef.args.defaults
        env = {params[0]: m}
        for i, name in enumerate(params[1:]):
            if i < len(args):
                env[name] = args[i]
            else:
                d = len(params) - 1 - len(defaults)
                if i < d:
                    self.fail(node, f"missing argument {name}")
                env[name] = self.expr(defaults[i - d], env)
        try:
            self.block(fdef.body, env)
        except _Return as r:
            return r.value
        return None

    # ---- statements -----------------------------------------------------
    def block(self, stmts, env):
        for st in stmts:
            self.stmt(st, env)

    def assign(self, target, value, env, node):
        if isinstance(target, ast.Name):
            env[target.id] = value
        elif isinstance(target, (ast.Tuple, ast.List)):
            if not isinstance(value, (tuple, list)) or len(value) != len(target.elts):
                self.fail(node, "tuple assignment of a non-tuple")
            for t, v in zip(target.elts, value):
                self.assign(t, v, env, node)
        else:
            self.fail(node, "only assignments to names are supported")

    def stmt(self, st, env):
        if isinstance(st, ast.Expr):
            if isinstance(st.value, ast.Constant):
                return   # docstring
            self.expr(st.value, env)
        elif isinstance(st, ast.Assign):
            v = self.expr(st.value, env)
            for t in st.targets:
                self.assign(t, v, env, st)
        elif isinstance(st, ast.AugAssign):
            cur = self.expr(st.target, env)
            self.assign(st.target, self.binop(st.op, cur, self.expr(st.value, env), st), env, st)
        elif isinstance(st, ast.Return):
            raise _Return(self.expr(st.value, env) if st.value is not None else None)
        elif isinstance(st, ast.Pass):
            pass
        elif isinstance(st, ast.Break):
            raise _Break()
        elif isinstance(st, ast.For):
            self.for_loop(st, env)
        elif isinstance(st, ast.If):
            self.if_stmt(st, env)
        else:
            self.fail(st, f"unsupported statement {type(st).__name__}")

    def for_loop(self, st, env):
        it = self.expr(st.iter, env)
        if isinstance(it, (nn.ModuleList, nn.Sequential)):
            it = list(it)
        if not isinstance(it, (range, list, tuple)):
            self.fail(st, "a loop must run over range(...), a list or a ModuleList with a trip count known here")
        if st.orelse:
            self.fail(st, "for ... else is not supported")
        items = list(it)
        outer = self.loop_halts
        self.loop_halts = {"halts": [], "n": len(items), "step": 0}
        try:
            for i, v in enumerate(items):
                self.loop_halts["step"] = i + 1
                self.assign(st.target, v, env, st)
                try:
                    self.block(st.body, env)
                except _Break:
                    break
            halts = self.loop_halts["halts"]
            if halts:
                self.close_halting_loop(halts, env, st)
        finally:
            self.loop_halts = outer

    def if_stmt(self, st, env):
        c = self.expr(st.test, env)
        if not isinstance(c, Sym):
            self.block(st.body if c else st.orelse, env)
            return
        kind = c.attrs.get("decision")
        if kind == "exit":
            self.exit_decision(st, c, env)
        elif kind == "gate":
            self.gate_decision(st, c, env)
        elif kind == "halt":
            self.halt_decision(st, c, env)
        else:
            self.fail(st, "a data-dependent condition must be an exit test (max softmax >= tau), a gate "
                          "(sigmoid(Linear(pool(x))) > thr) or a halting test (running sum >= tau)")

    # ---- decisions ------------------------------------------------------
    def exit_decision(self, st, c, env):
        if st.orelse or len(st.body) != 1 or not isinstance(st.body[0], ast.Return):
            self.fail(st, "an exit test must be followed by `return <the head's logits>` alone")
        z = self.expr(st.body[0].value, env)
        if z is not c.attrs["z"]:
            self.fail(st, "an exit must return the logits its test was computed from")
        self.trace.append(("decision", Decision("exit", {"z": z, "tau": c.attrs["tau"], "T": c.attrs["T"],
                                                         "index": self.n_exits})))
        z.uses += 1
        self.n_exits += 1

    def gate_decision(self, st, c, env):
        before = dict(env)
        # the else path runs first, on every row: its new values exist before
        # the gate (hoisted); then the executed rows' path is recorded apart
        else_env = dict(env)
        self.block(st.orelse, else_env)
        start = len(self.trace)
        then_env = dict(env)
        self.block(st.body, then_env)
        body = self.trace[start:]
        del self.trace[start:]
        merged = {}
        for name in set(then_env) | set(else_env):
            tv, ev = then_env.get(name), else_env.get(name)
            if tv is ev:
                continue
            if not isinstance(tv, Sym) or not isinstance(ev, Sym):
                self.fail(st, f"variable '{name}' must be a tensor on both paths of a gate")
            if tv.shape != ev.shape:
                self.fail(st, f"variable '{name}' has different shapes on the two paths of a gate")
            merged[name] = (tv, ev)
        if not merged:
            self.fail(st, "a gate must assign a tensor")
        outs = {}
        for name, (tv, ev) in merged.items():
            m = self.sym("merge", (ev, tv), ev.shape)
            outs[name] = m
        dec = Decision("gate", {"x": c.attrs["x"], "lin": c.attrs["lin"], "thr": c.attrs["thr"], "body": body,
                                "merges": list(outs.values()), "before": before})
        # the decision goes in front of the merge values it produces
        merges = [e for e in self.trace[-len(outs):]]
        del self.trace[-len(outs):]
        self.trace.append(("decision", dec))
        self.trace.extend(merges)
        c.attrs["x"].uses += 1
        env.update(else_env)
        env.update(outs)

    def halt_decision(self, st, c, env):
        if self.loop_halts is None:
            self.fail(st, "a halting test must sit in a loop")
        if st.orelse or len(st.body) != 1 or not isinstance(st.body[0], ast.Break):
            self.fail(st, "a halting test must be followed by `break` alone")
        L = self.loop_halts
        depth, v = 0, c.attrs["cum"]
        while v is not None:
            depth, v = depth + 1, v.attrs["prev"]
        if depth != L["step"]:
            self.fail(st, "the running sum must start at 0 before the loop and grow by one term per step")
        d = Decision("halt", {"h": c.attrs["h"], "lin": c.attrs["lin"], "tau": c.attrs["tau"], "step": L["step"],
                              "env": dict(env)})
        c.attrs["h"].uses += 1
        L["halts"].append(d)
        self.trace.append(("decision", d))

    def close_halting_loop(self, halts, env, st):
        L = self.loop_halts
        if len(halts) != L["n"] or [h.attrs["step"] for h in halts] != list(range(1, L["n"] + 1)):
            self.fail(st, "a halting loop needs one halting test per step")
        # the value every sample leaves the loop with: each step's own state
        # for the rows that halt there; the last step halts every row left
        states = []
        for d in halts:
            names = [n for n, v in d.attrs["env"].items() if v is d.attrs["h"]]
            if not names:
                self.fail(st, "the halting test must read the loop's state variable")
            states.append(names)
        common = set(states[0])
        for s in states[1:]:
            common &= set(s)
        if len(common) != 1:
            self.fail(st, "the halting test must read one state variable of the loop")
        name = common.pop()
        for d in halts:
            d.attrs["max_steps"] = L["n"]
        parked = self.sym("parked", tuple(d.attrs["h"] for d in halts), halts[0].attrs["h"].shape, halts=halts)
        env[name] = parked

    # ---- expressions ------------------------------------------------------
    def expr(self, e, env):
        if isinstance(e, ast.Constant):
            return e.value
        if isinstance(e, ast.Name):
            if e.id in env:
                return env[e.id]
            g = {"torch": torch, "F": F, "nn": nn, "range": range, "len": len, "enumerate": enumerate,
                 "int": int, "float": float, "min": min, "max": max, "True": True, "False": False, "None": None}
            if e.id in g:
                return g[e.id]
            self.fail(e, f"unknown name '{e.id}'")
        if isinstance(e, ast.Attribute):
            base = self.expr(e.value, env)
            if isinstance(base, Sym):
                return ("method", base, e.attr)
            if base is torch.nn.functional or base is torch or isinstance(base, nn.Module) or \
                    isinstance(base, (int, float, tuple)):
                return getattr(base, e.attr)
            self.fail(e, f"attribute '{e.attr}' of an unsupported value")
        if isinstance(e, ast.Subscript):
            base = self.expr(e.value, env)
            idx = self.expr(e.slice, env)
            if isinstance(base, Sym):
                self.fail(e, "tensor indexing is not supported")
            return base[idx]
        if isinstance(e, (ast.Tuple, ast.List)):
            return tuple(self.expr(x, env) for x in e.elts)
        if isinstance(e, ast.BinOp):
            return self.binop(e.op, self.expr(e.left, env), self.expr(e.right, env), e)
        if isinstance(e, ast.UnaryOp):
            v = self.expr(e.operand, env)
            if isinstance(v, Sym):
                self.fail(e, "unary operators on tensors are not supported")
            return {ast.Not: lambda a: not a, ast.USub: lambda a: -a, ast.UAdd: lambda a: a}[type(e.op)](v)
        if isinstance(e, ast.Compare):
            if len(e.ops) != 1:
                self.fail(e, "chained comparisons are not supported")
            return self.compare(e.ops[0], self.expr(e.left, env), self.expr(e.comparators[0], env), e)
        if isinstance(e, ast.BoolOp):
            vals = [self.expr(v, env) for v in e.values]
            syms = [v for v in vals if isinstance(v, Sym)]
            consts = [v for v in vals if not isinstance(v, Sym)]
            if isinstance(e.op, ast.Or):
                if any(consts):
                    return True
                if len(syms) == 1:
                    return syms[0]
            else:
                if consts and not all(consts):
                    return False
                if len(syms) == 1:
                    return syms[0]
            if not syms:
                return any(vals) if isinstance(e.op, ast.Or) else all(vals)
            self.fail(e, "a condition may combine one tensor test with constants only")
        if isinstance(e, ast.IfExp):
            c = self.expr(e.test, env)
            if isinstance(c, Sym):
                self.fail(e, "conditional expressions on tensor data are not supported; use an if statement")
            return self.expr(e.body if c else e.orelse, env)
        if isinstance(e, ast.Call):
            return self.call(e, env)
        self.fail(e, f"unsupported expression {type(e).__name__}")

    def binop(self, op, a, b, node):
        if not isinstance(a, (Sym, Aux)) and not isinstance(b, (Sym, Aux)):
            return {ast.Add: lambda: a + b, ast.Sub: lambda: a - b, ast.Mult: lambda: a * b,
                    ast.Div: lambda: a / b, ast.FloorDiv: lambda: a // b}[type(op)]()
        if isinstance(op, ast.Add):
            # the running halting sum: S = S + p (S starts at the number 0)
            if isinstance(b, Sym) and b.op == "sigmoid" and (
                    (not isinstance(a, (Sym, Aux)) and a == 0) or (isinstance(a, Sym) and a.op == "cum")):
                prev = a if isinstance(a, Sym) else None
                return self.sym("cum", (b,) if prev is None else (prev, b), (1, 1), prev=prev)
            if isinstance(a, Sym) and isinstance(b, Sym):
                if a.shape != b.shape:
                    self.fail(node, f"adding {a.shape} and {b.shape}")
                return self.sym("add", (a, b), a.shape)
            # the halting unit's pre-activation: Linear(h) + b
            if isinstance(a, Sym) and isinstance(b, Aux) and a.op == "linear" and a.shape == (1, 1):
                return self.sym("plus_aux", (a,), a.shape)
            self.fail(node, "unsupported addition")
        if isinstance(op, ast.Div) and isinstance(a, Sym) and not isinstance(b, Sym):
            return self.sym("div", (a,), a.shape, by=b)
        if isinstance(op, ast.Div) and isinstance(a, Sym) and isinstance(b, torch.Tensor):
            return self.sym("div", (a,), a.shape, by=b)
        self.fail(node, "unsupported arithmetic on tensors")

    def compare(self, op, a, b, node):
        if not isinstance(a, Sym):
            return {ast.Eq: lambda: a == b, ast.NotEq: lambda: a != b, ast.Lt: lambda: a < b,
                    ast.LtE: lambda: a <= b, ast.Gt: lambda: a > b, ast.GtE: lambda: a >= b,
                    ast.Is: lambda: a is b, ast.IsNot: lambda: a is not b}[type(op)]()
        thr = float(b)
        # exit: max softmax(z / T) >= tau
        if a.op == "max" and a.args[0].op == "softmax":
            if not isinstance(op, ast.GtE):
                self.fail(node, "an exit test is `>= tau` (the sample leaves when its confidence reaches tau)")
            sm = a.args[0]
            zz = sm.args[0]
            T = 1.0
            if zz.op == "div":
                T, zz = zz.attrs["by"], zz.args[0]
            if zz.op != "linear":
                self.fail(node, "the exit test must read a Linear head's logits")
            return self.sym("cond", (a,), (), decision="exit", z=zz, tau=thr, T=T)
        # gate: sigmoid(Linear(pool(x))) > thr
        if a.op == "sigmoid" and a.args[0].op == "linear" and a.args[0].shape == (1, 1):
            if not isinstance(op, ast.Gt):
                self.fail(node, "a gate test is `> thr` (the block runs when its score exceeds thr)")
            lin = a.args[0]
            x = self.pooled_source(lin.args[0], node)
            return self.sym("cond", (a,), (), decision="gate", x=x, lin=lin.attrs["mod"], thr=thr)
        # halt: running sum >= tau
        if a.op == "cum":
            if not isinstance(op, ast.GtE):
                self.fail(node, "a halting test is `>= tau`")
            sg = a.args[-1]
            pre = sg.args[0]
            if pre.op != "plus_aux":
                self.fail(node, "the halting probability must be sigmoid(Linear(h) + b) with b the second input")
            lin = pre.args[0]
            # the sum must run over this loop's steps one by one
            return self.sym("cond", (a,), (), decision="halt", h=lin.args[0], lin=lin.attrs["mod"], tau=thr, cum=a)
        self.fail(node, "unsupported comparison on tensor data")

    def pooled_source(self, v, node):
        if v.op == "flatten" and v.args[0].op == "gap":
            return v.args[0].args[0]
        if v.op == "gap_flat":
            return v.args[0]
        self.fail(node, "a gate must read flatten(adaptive_avg_pool2d(x, 1)) or x.mean((2, 3))")

    def call(self, e, env):
        f = self.expr(e.func, env)
        args = [self.expr(a, env) for a in e.args]
        kw = {k.arg: self.expr(k.value, env) for k in e.keywords}
        if isinstance(f, tuple) and f and f[0] == "method":
            return self.method(f[1], f[2], args, kw, e)
        if isinstance(f, nn.Module):
            return self.call_module(f, args, e)
        if f in (range, len, enumerate, int, float, min, max):
            if f is enumerate:
                seq = args[0]
                if isinstance(seq, (nn.ModuleList, nn.Sequential)):
                    seq = list(seq)
                return list(enumerate(seq))
            return f(*args, **kw)
        name = _TORCH_FUNCS.get(f)
        if name is None:
            self.fail(e, f"unsupported call {getattr(f, '__name__', f)}")
        return self.torch_call(name, args, kw, e)

    def torch_call(self, name, args, kw, e):
        x = args[0] if args else None
        if name in ("relu", "gelu"):
            if name == "gelu" and kw.get("approximate", "none") != "none":
                self.fail(e, "only the exact GELU is supported")
            return self.sym(name, (x,), x.shape)
        if name == "sigmoid":
            return self.sym("sigmoid", (x,), x.shape)
        if name == "softmax":
            dim = kw.get("dim", args[1] if len(args) > 1 else None)
            if dim not in (1, -1):
                self.fail(e, "softmax over the class dimension (dim=1 or -1) only")
            return self.sym("softmax", (x,), x.shape)
        if name == "max":
            if len(args) != 1 or kw:
                self.fail(e, "torch.max(p) over all classes only")
            return self.sym("max", (x,), ())
        if name == "flatten":
            start = kw.get("start_dim", args[1] if len(args) > 1 else 0)
            if x.op != "gap" or start != 1:
                self.fail(e, "flatten(adaptive_avg_pool2d(x, 1), 1) only")
            return self.sym("flatten", (x,), (1, x.shape[1]))
        if name == "gap":
            if (args[1] if len(args) > 1 else kw.get("output_size")) not in (1, (1, 1)):
                self.fail(e, "adaptive_avg_pool2d to 1x1 only")
            return self.sym("gap", (x,), (1, x.shape[1], 1, 1))
        if name == "max_pool2d":
            k = args[1] if len(args) > 1 else kw.get("kernel_size")
            s = args[2] if len(args) > 2 else kw.get("stride", k)
            p = args[3] if len(args) > 3 else kw.get("padding", 0)
            return self.max_pool(x, k, s, p, e)
        if name in ("zeros", "zeros_like"):
            shape = tuple(x.shape) if name == "zeros_like" else tuple(a for a in args)
            if len(shape) == 1 and isinstance(shape[0], (tuple, list)):
                shape = tuple(shape[0])
            return self.sym("zeros", (), tuple(shape))
        if name == "cat":
            parts = list(x)
            dim = kw.get("dim", args[1] if len(args) > 1 else 0)
            if dim not in (1, -1) or any(len(p.shape) != 2 for p in parts) or len(parts) != 2:
                self.fail(e, "torch.cat of two [1, D] vectors along the last dimension only")
            return self.sym("cat", tuple(parts), (1, parts[0].shape[1] + parts[1].shape[1]))
        self.fail(e, f"unsupported call {name}")

    def method(self, x, name, args, kw, e):
        if name == "mean":
            dims = args[0] if args else kw.get("dim")
            if tuple(dims) not in ((2, 3), (-2, -1)) or len(x.shape) != 4:
                self.fail(e, "x.mean((2, 3)) over the spatial dimensions only")
            return self.sym("gap_flat", (x,), (1, x.shape[1]))
        if name == "flatten":
            return self.torch_call("flatten", [x] + args, kw, e)
        if name in ("relu", "sigmoid"):
            return self.sym(name, (x,), x.shape)
        if name == "max" and not args and not kw:
            return self.sym("max", (x,), ())
        self.fail(e, f"unsupported tensor method .{name}")


# -------------------------------------------------------------- lower ----

class _Blob:
    def __init__(self):
        self.parts, self.off = [], 0
        self.seen = {}

    def add(self, arr: np.ndarray, dtype: str, key=None) -> int:
        """Offset of arr in the blob; a key already added (one parameter
        read by several unrolled steps) returns its first copy."""
        if key is not None and (key, dtype) in self.seen:
            return self.seen[(key, dtype)]
        if key is not None:
            self.seen[(key, dtype)] = self._put(arr, dtype)
            return self.seen[(key, dtype)]
        return self._put(arr, dtype)

    def _put(self, arr: np.ndarray, dtype: str) -> int:
        raw = (_bf16_bits(arr) if dtype == "bf16" else np.ascontiguousarray(arr, dtype=np.float32)).tobytes()
        pad = (-self.off) % 256
        if pad:
            self.parts.append(b"\0" * pad)
            self.off += pad
        at = self.off
        self.parts.append(raw)
        self.off += len(raw)
        return at

    def bytes(self) -> bytes:
        return b"".join(self.parts)


def _np(t) -> np.ndarray:
    return t.detach().to(torch.float64).cpu().numpy()


class _Lower:
    def __init__(self, interp: _Interp, dtype: str, image: bool):
        self.I, self.dt, self.image = interp, dtype, image
        self.blob = _Blob()
        self.names = {}          # Sym -> spec tensor name (current row group)
        self.count = 0
        self.nodes = []
        self.aux = False
        self.pos = {}            # Sym -> trace position (program order)
        self.overwritten = set() # values a gate wrote its executed rows over

    def fresh(self, base="t"):
        self.count += 1
        return f"{base}{self.count}"

    # ---- conv chains: conv -> [bn] -> [add residual] -> [act] -------------
    def chain(self, s):
        """The conv node a value is the end of, or None: (conv, bn, res, act)."""
        bn = res = act = None
        v = s
        if v.op in ("relu", "gelu"):
            act, v = v.op, v.args[0]
            if v.uses != 1:
                return None
        if v.op == "add":
            a, b = v.args
            # the addend computed last carries the epilogue; the other one must
            # exist before it as the residual
            if self.pos.get(a, -1) < self.pos.get(b, -1):
                a, b = b, a
            for cand, other in ((a, b), (b, a)):
                c = self._conv_bn(cand)
                if c is not None and cand.uses == 1:
                    res, v = other, cand
                    break
            else:
                return None
            if v.uses != 1:
                return None
        c = self._conv_bn(v)
        if c is None:
            return None
        conv, bn = c
        return conv, bn, res, act

    def _conv_bn(self, v):
        if v.op == "bn" and v.args[0].op == "conv" and v.args[0].uses == 1:
            return v.args[0], v
        if v.op == "conv":
            return v, None
        if v.op == "linear" and self.dt == "bf16":
            return v, None
        return None

    def emit_conv(self, s, nodes):
        ch = self.chain(s)
        if ch is None:
            return False
        conv, bn, res, act = ch
        m = conv.attrs["mod"]
        src = conv.args[0]
        # operands first, in program order
        ops = [v for v in (src, res) if v is not None]
        if src.op == "cat":
            ops = [v for v in src.args if v.op != "zeros"] + ([res] if res is not None else [])
        for v in sorted(ops, key=lambda v: self.pos.get(v, -1)):
            self.name(v, nodes)
        node = {"op": "conv", "k": 1, "stride": 1, "pad": 0, "cout": conv.shape[1],
                "act": {"relu": "relu", "gelu": "gelu", None: "none"}[act]}
        if isinstance(m, nn.Conv2d):
            w = _np(m.weight).transpose(0, 2, 3, 1)          # [cout][kh][kw][cin]: K order (kh, kw, ci)
            node.update(k=m.kernel_size[0], stride=m.stride[0], pad=m.padding[0])
            node["w"] = {"off": self.blob.add(w, "bf16", key=id(m.weight))}
            scale = np.ones(conv.shape[1])
            shift = _np(m.bias) if m.bias is not None else np.zeros(conv.shape[1])
            if bn is not None:
                b = bn.attrs["mod"]
                if b.training or b.running_mean is None:
                    raise FrontendError("BatchNorm must be in eval mode with running statistics")
                a = _np(b.weight) / np.sqrt(_np(b.running_var) + b.eps)
                scale, shift = a, _np(b.bias) + (shift - _np(b.running_mean)) * a
            node["scale"] = self.blob.add(scale, "f32")
            node["shift"] = self.blob.add(shift, "f32")
        else:   # a linear layer on vectors (k = 1 on 1x1 rows)
            W = _np(m.weight)
            wo = self.blob.add(W, "bf16", key=id(m.weight))
            if src.op == "cat":
                h, x = src.args
                if h.op == "zeros":     # a zero block contributes nothing: keep the other columns
                    node["w"] = {"off": wo, "ldk": W.shape[1], "k0": h.shape[1]}
                    src = x
                elif x.op == "zeros":
                    node["w"] = {"off": wo, "ldk": W.shape[1], "k0": 0}
                    if h.shape[1] != W.shape[1] - x.shape[1]:
                        raise FrontendError("concatenation widths do not match the linear layer")
                    raise FrontendError("a zero block after the data columns is not supported")
                else:
                    node["w"] = {"off": wo, "ldk": W.shape[1], "k0": 0}
                    node["src2"] = self.name(x, nodes)
                    src = h
            else:
                node["w"] = {"off": wo}
            if m.bias is not None:
                node["shift"] = self.blob.add(_np(m.bias), "f32", key=id(m.bias))
        node["src"] = self.name(src, nodes)
        if res is not None:
            node["res"] = self.name(res, nodes)
        node["dst"] = self.fresh("c")
        nodes.append(node)
        self.names[s] = node["dst"]
        return True

    def name(self, s, nodes):
        """The spec tensor holding value s, emitting what produces it."""
        if s in self.overwritten:
            raise FrontendError("a tensor is read after a gate wrote its executed rows over it; read the gate's "
                                "result instead")
        if s in self.names:
            return self.names[s]
        if self.emit_conv(s, nodes):
            return self.names[s]
        if s.op == "linear" and self.dt == "f32":
            m = s.attrs["mod"]
            node = {"op": "conv", "src": self.name(s.args[0], nodes), "dst": self.fresh("l"), "k": 1,
                    "cout": s.shape[1], "act": "none", "w": {"off": self.blob.add(_np(m.weight), "f32")}}
            if m.bias is not None:
                node["shift"] = self.blob.add(_np(m.bias), "f32")
            nodes.append(node)
            self.names[s] = node["dst"]
            return node["dst"]
        if s.op in ("relu",) and s.args[0].op == "linear" and self.dt == "f32" and s.args[0].uses == 1:
            lin = s.args[0]
            m = lin.attrs["mod"]
            node = {"op": "conv", "src": self.name(lin.args[0], nodes), "dst": self.fresh("l"), "k": 1,
                    "cout": s.shape[1], "act": "relu", "w": {"off": self.blob.add(_np(m.weight), "f32")}}
            if m.bias is not None:
                node["shift"] = self.blob.add(_np(m.bias), "f32")
            nodes.append(node)
            self.names[s] = node["dst"]
            return node["dst"]
        if s.op == "maxpool":
            node = {"op": "maxpool", "src": self.name(s.args[0], nodes), "dst": self.fresh("p")}
            nodes.append(node)
            self.names[s] = node["dst"]
            return node["dst"]
        raise FrontendError(f"no kernel computes {s.op} of {[a.op for a in s.args if isinstance(a, Sym)]} "
                            "(convolutions fuse BatchNorm, one residual addition and an activation)")

    # ---- heads ----------------------------------------------------------
    def head(self, z, nodes):
        """(source tensor name, W, b) of logits z = Linear(pool(x)) or Linear(x)."""
        m = z.attrs["mod"]
        v = z.args[0]
        if self.image:
            if v.op == "flatten" and v.args[0].op == "gap":
                v = v.args[0].args[0]
            elif v.op == "gap_flat":
                v = v.args[0]
            else:
                raise FrontendError("an image network's head must read flatten(adaptive_avg_pool2d(x, 1))")
        src = self.name(v, nodes)
        return src, _np(m.weight), (_np(m.bias) if m.bias is not None else np.zeros(m.out_features))

    def exit_node(self, z, tau, T, index, final, nodes):
        src, W, b = self.head(z, nodes)
        node = {"op": "exit", "src": src, "w": self.blob.add(W, "f32"), "b": self.blob.add(b, "f32"),
                "ncls": int(W.shape[0]), "tau": float(tau), "index": index, "final": final}
        if not final:
            Tv = float(T.detach().reshape(-1)[0]) if isinstance(T, torch.Tensor) else float(T)
            node["T"] = self.blob.add(np.array([Tv]), "f32")
        nodes.append(node)
        return node

    # ---- program ------------------------------------------------------------
    def run(self, trace):
        for k, v in trace:
            if k == "sym" and v.op == "input":
                self.names[v] = "x"
        for i, (k, v) in enumerate(trace):
            if k == "sym":
                self.pos[v] = i
            elif k == "decision" and v.kind == "gate":
                for j, (k2, v2) in enumerate(v.attrs["body"]):
                    if k2 == "sym":
                        self.pos[v2] = i + (j + 1) / (len(v.attrs["body"]) + 1)
        self.lower_seq(trace, self.nodes, top=True)
        return self.nodes

    # values that only feed a head or a decision test are never stored
    _TRANSIENT = ("gap", "gap_flat", "flatten", "softmax", "max", "div", "cond", "sigmoid", "plus_aux", "cum",
                  "zeros", "cat", "parked")

    def need(self, s, nodes):
        if s.op in ("cum", "cond"):
            return       # decision tests: the decision kernels compute them
        if s.op in self._TRANSIENT:
            for a in s.args:
                if isinstance(a, Sym) and s.op != "parked":
                    self.need(a, nodes)
            return
        if s.op == "linear" and s.uses == 0:
            return
        self.name(s, nodes)

    def materialize_before(self, trace, i, nodes):
        """Store every value computed before position i that is read after
        it, so that the decision at i can carry it."""
        def reads(item):
            kind, v = item
            if kind == "return":
                return [v]
            if kind == "sym":
                return [] if v.op == "parked" else [a for a in v.args if isinstance(a, Sym)]
            if v.kind == "gate":
                out = [v.attrs["x"]]
                for k2, s2 in v.attrs["body"]:
                    if k2 == "sym":
                        out += [a for a in s2.args if isinstance(a, Sym)]
                return out
            return [v.attrs["z"] if v.kind == "exit" else v.attrs["h"]]
        for item in trace[i + 1:]:
            for a in reads(item):
                if self.pos.get(a, -1) < i and a.op != "input":
                    self.need(a, nodes)

    def later_uses(self, trace, i):
        """Values defined before position i that the rest of the trace reads."""
        live = []
        seen = set()

        def reads(item):
            kind, v = item
            if kind == "sym":
                return [] if v.op == "parked" else [a for a in v.args if isinstance(a, Sym)]
            if kind == "return":
                return [v]
            d = v
            if d.kind == "exit":
                return [d.attrs["z"]]
            if d.kind == "gate":
                out = [d.attrs["x"]]
                for k2, s2 in d.attrs["body"]:
                    out += [a for a in s2.args if isinstance(a, Sym)] if k2 == "sym" else []
                return out
            return [d.attrs["h"]]

        defined_after = set(v for k, v in trace[i + 1:] if k == "sym")
        def walk(a):
            # a value read after i: stored ones are live; transient ones read
            # their own operands
            if a in seen:
                return
            seen.add(a)
            if a in self.names and a not in defined_after:
                live.append(a)
            elif a.op in self._TRANSIENT and a.op not in ("parked", "cum", "cond") and a not in defined_after:
                for b in a.args:
                    if isinstance(b, Sym):
                        walk(b)
        for item in trace[i + 1:]:
            for a in reads(item):
                walk(a)
        return live

    def lower_seq(self, trace, nodes, top):
        for i, (kind, v) in enumerate(trace):
            if kind == "sym":
                continue     # emitted on demand by the values that read them
            if kind == "return":
                self.final(v, nodes)
                return
            d = v
            self.materialize_before(trace, i, nodes)
            if d.kind == "exit":
                self.exit_node(d.attrs["z"], d.attrs["tau"], d.attrs["T"], d.attrs["index"], False, nodes)
                self.carry(nodes[-1], trace, i)
            elif d.kind == "gate":
                self.gate(d, trace, i, nodes)
            elif d.kind == "halt":
                self.halt(d, trace, i, nodes)

    def carry(self, node, trace, i):
        pairs = []
        for s in self.later_uses(trace, i):
            new = self.fresh("k")
            pairs.append([self.names[s], new])
            self.names[s] = new
        if pairs:
            node["carry"] = pairs

    def gate(self, d, trace, i, nodes):
        x = self.name(d.attrs["x"], nodes)
        merges = [v for k, v in trace[i + 1:] if k == "sym" and v.op == "merge"][:len(d.attrs["merges"])]
        # the values the merges fall back to exist for every row: produce them
        outer = [self.name(m.args[0], nodes) for m in merges]
        lin = d.attrs["lin"]
        node = {"op": "gate", "src": x, "u": self.blob.add(_np(lin.weight).reshape(-1), "f32"),
                "v": self.blob.add(_np(lin.bias).reshape(-1) if lin.bias is not None else np.zeros(1), "f32"),
                "threshold": d.attrs["thr"], "index": sum(1 for n in self.nodes if n["op"] == "gate")}
        # the body reads outer values through gathered copies
        body_syms = [v for k, v in d.attrs["body"] if k == "sym"]
        body_set = set(body_syms)
        outer_reads = []
        for s in body_syms:
            for a in s.args:
                if isinstance(a, Sym) and a not in body_set and a not in outer_reads:
                    outer_reads.append(a)
        for a in outer_reads:
            self.name(a, nodes)
        saved = dict(self.names)
        gather = []
        for a in outer_reads:
            nm = saved[a] if a.op != "input" else "x"
            if not any(g[0] == nm for g in gather):
                gather.append([nm, self.fresh("g")])
            self.names[a] = next(g[1] for g in gather if g[0] == nm)
        body = []
        for m in merges:
            self.name(m.args[1], body)
        node["gather"] = gather
        node["body"] = body
        node["scatter"] = [[self.names[m.args[1]], o] for m, o in zip(merges, outer)]
        self.names = saved
        for m, o in zip(merges, outer):
            self.names[m] = o
            if m.args[0].op != "input":
                self.overwritten.add(m.args[0])
        nodes.append(node)

    def halt(self, d, trace, i, nodes):
        h = self.name(d.attrs["h"], nodes)
        lin = d.attrs["lin"]
        if lin.bias is not None:
            raise FrontendError("the halting unit's Linear must have no bias (the per-sample input is its bias)")
        self.aux = True
        node = {"op": "halt", "src": h, "w": self.blob.add(_np(lin.weight).reshape(-1), "f32"),
                "tau": d.attrs["tau"], "step": d.attrs["step"], "max_steps": d.attrs["max_steps"],
                "park": [h, "h_final"]}
        nodes.append(node)
        if d.attrs["step"] < d.attrs["max_steps"]:
            self.carry(node, trace, i)

    def final(self, v, nodes):
        if v.op == "linear" and any(a.op == "parked" for a in v.args):
            m = v.attrs["mod"]
            nodes.append({"op": "output", "src": "h_final", "w": {"off": self.blob.add(_np(m.weight), "bf16", key=id(m.weight))},
                          "bias": self.blob.add(_np(m.bias) if m.bias is not None else np.zeros(m.out_features),
                                                "f32"),
                          "cout": m.out_features})
            return
        if v.op != "linear":
            raise FrontendError("the program must end by returning a Linear head's logits")
        index = self.I.n_exits if self.I.n_exits > 0 else -1
        self.exit_node(v, 0.0, 1.0, index, True, nodes)


# ------------------------------------------------------------ driver ----

def compile_module(module: nn.Module, input_shape, dtype: str = "bf16"):
    """Compile ``module`` (its ``forward(self, x[, b])`` for one sample:
    ``x`` of shape [1, C, H, W] or [1, D], ``b`` a per-sample scalar) into
    (spec dict, weight blob bytes)."""
    if dtype not in ("bf16", "f32"):
        raise FrontendError("dtype must be bf16 or f32")
    module = module.eval()
    I = _Interp()
    shape = (1,) + tuple(input_shape)
    image = len(shape) == 4
    x = Sym("input", (), {}, shape)
    I.trace.append(("sym", x))
    fn = type(module).forward
    fdef = ast.parse(textwrap.dedent(inspect.getsource(fn))).body[0]
    nargs = len(fdef.args.args) - 1
    args = [x] + ([Aux()] if nargs >= 2 else [])
    with torch.no_grad():
        out = I.inline(module, args, fdef)
    if out is None:
        raise FrontendError("forward must return the logits")
    I.trace.append(("return", out))
    L = _Lower(I, dtype, image)
    nodes = L.run(I.trace)
    n_out = next(n["ncls"] if n["op"] == "exit" else n["cout"] for n in reversed(nodes)
                 if n["op"] in ("exit", "output"))
    spec_shape = [shape[2], shape[3], shape[1]] if image else [shape[1]]
    spec = {"version": 1, "dtype": dtype, "input": {"name": "x", "shape": spec_shape}, "n_out": n_out,
            "aux": L.aux, "nodes": nodes}
    return spec, L.blob.bytes()


def compile_module_json(module: nn.Module, input_shape, dtype: str = "bf16"):
    spec, blob = compile_module(module, input_shape, dtype)
    return json.dumps(spec), blob


__all__ = ["FrontendError", "compile_module", "compile_module_json", "math"]
