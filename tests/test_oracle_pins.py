"""Pins of the oracle against things other than itself (CPU only).

* bf16 rounding: a library conversion over every upper half-word and the
  rounding-relevant lower half-words, plus hand-worked values.
* Layer primitives: scalar-loop brute force, closed forms, textbook values.
* Whole programs: on tiny networks every static path is evaluated with the
  independent numpy reference in ``_naive``; exactly one path must agree with
  its own decisions, and the oracle must take it, with the same logits.
* Invariants on the real workloads: batch-split and permutation invariance,
  forced routing, loop bounds, monotone halting sums.
* The correctness metrics of Eq. 1 on closed-form cases.
"""

import itertools
import math

import numpy as np
import pytest
import torch

from oracle import dycl_oracle as O
from workloads import configs
from tests import _naive as N

RNG = np.random.default_rng(1234)


# ---------------------------------------------------------------- bf16 ----

def test_q_matches_library_bf16_over_structured_exhaustive_set():
    hi = np.arange(65536, dtype=np.uint32) << np.uint32(16)
    lows = [0x0000, 0x0001, 0x7FFE, 0x7FFF, 0x8000, 0x8001, 0x8002, 0xFFFF, 0x4000, 0xC000]
    lows += list(RNG.integers(0, 65536, 6))
    bits = (hi[:, None] | np.array(lows, dtype=np.uint32)[None, :]).ravel()
    f = bits.view(np.float32)
    ours = O.q(torch.from_numpy(f)).to(torch.float32).numpy()
    lib = torch.from_numpy(f).to(torch.bfloat16).to(torch.float32).numpy()
    nan = np.isnan(f)
    assert np.isnan(ours[nan]).all()
    assert (ours[~nan].view(np.uint32) == lib[~nan].view(np.uint32)).all()


def test_q_hand_worked_values():
    ulp = 2.0 ** -7                       # bf16 spacing in [1, 2)
    cases = {1.0: 1.0, 1.0 + ulp / 2: 1.0,                  # tie -> even (1.0)
             1.0 + 3 * ulp / 2: 1.0 + 2 * ulp,              # tie -> even (1 + 2 ulp)
             1.0 + ulp / 2 + 2 ** -20: 1.0 + ulp,           # above the tie
             -2.5: -2.5, 3.3999e38: float("inf"),            # above the largest bf16 + half ulp
             1e-45: 0.0}                                    # fp32 denormal below bf16 half-ulp
    for v, want in cases.items():
        assert float(O.q(torch.tensor([v], dtype=torch.float64))[0]) == want, v


# ---------------------------------------------------------- primitives ----

@pytest.mark.parametrize("k,stride,pad", [(1, 1, 0), (3, 1, 1), (3, 2, 1), (1, 2, 0), (7, 2, 3)])
def test_conv2d_vs_scalar_loops(k, stride, pad):
    H = 9 if k == 7 else 6
    x = RNG.standard_normal((H, H + 1, 3))
    w = RNG.standard_normal((4, k, k, 3))
    ours = O.conv2d(torch.from_numpy(x).permute(2, 0, 1), torch.from_numpy(w).permute(0, 3, 1, 2),
                    stride, pad).permute(1, 2, 0).numpy()
    np.testing.assert_allclose(ours, N.conv_loops(x, w, stride, pad), rtol=1e-12, atol=1e-12)


def test_conv2d_delta_kernel_is_a_shift():
    x = RNG.standard_normal((2, 5, 5))
    w = np.zeros((2, 2, 3, 3))
    w[0, 0, 0, 0] = 1.0          # picks x[0, oh-1, ow-1]
    w[1, 1, 2, 1] = 1.0          # picks x[1, oh+1, ow]
    y = O.conv2d(torch.from_numpy(x), torch.from_numpy(w), 1, 1).numpy()
    xp = np.pad(x, ((0, 0), (1, 1), (1, 1)))
    np.testing.assert_array_equal(y[0], xp[0, 0:5, 0:5])
    np.testing.assert_array_equal(y[1], xp[1, 2:7, 1:6])


def test_gap_maxpool_vs_loops():
    x = RNG.standard_normal((3, 7, 5))
    g = O.gap(torch.from_numpy(x)).numpy()
    np.testing.assert_allclose(g, [x[c].sum() / 35.0 for c in range(3)], rtol=1e-14)
    mp = O.maxpool3s2(torch.from_numpy(x)).permute(1, 2, 0).numpy()
    np.testing.assert_array_equal(mp, N.maxpool_loops(x.transpose(1, 2, 0)))


def test_maxprob_closed_forms():
    assert O.maxprob(torch.zeros(10, dtype=torch.float64), 1.0) == pytest.approx(0.1, abs=1e-7)
    a = 2.0
    z = torch.tensor([a, 0, 0, 0], dtype=torch.float64)
    assert O.maxprob(z, 1.0) == pytest.approx(math.exp(a) / (math.exp(a) + 3), abs=1e-7)
    # temperature divides the logits
    assert O.maxprob(z, 2.0) == pytest.approx(math.exp(1.0) / (math.exp(1.0) + 3), abs=1e-7)
    # shift invariance, and the limit of a dominant logit
    assert O.maxprob(z + 123.0, 1.0) == O.maxprob(z, 1.0)
    assert O.maxprob(torch.tensor([100.0, 0.0], dtype=torch.float64), 1.0) == 1.0


def test_sigmoid_gelu_closed_forms():
    assert O.sigmoid(0.0) == 0.5
    for v in (0.3, 1.7, -4.0):
        assert O.sigmoid(v) + O.sigmoid(-v) == pytest.approx(1.0, abs=1e-7)
    assert O.sigmoid(math.log(3.0)) == pytest.approx(0.75, abs=1e-7)
    g = O.gelu(torch.tensor([0.0, 1.0, -1.0, 10.0, -10.0], dtype=torch.float64)).numpy()
    phi1 = 0.8413447460685429             # standard normal CDF at 1 (textbook table)
    np.testing.assert_allclose(g, [0.0, phi1, -(1 - phi1), 10.0, 0.0], atol=1e-15)
    for v in np.linspace(-4, 4, 17):
        want = 0.5 * v * (1.0 + N.erf_series(v / math.sqrt(2.0)))
        assert float(O.gelu(torch.tensor([v], dtype=torch.float64))[0]) == pytest.approx(want, abs=1e-12)


# -------------------------------------------------- whole tiny programs ----

def _tiny(name, arch):
    wl = configs.raw_workload(name, arch)
    return wl, wl.weights_f32()


def _first_exit(ps, tau):
    t = np.float32(tau)
    for k, p in enumerate(ps[:-1]):
        if np.float32(p) >= t:
            return k
    return len(ps) - 1


def _check_exit_network(arch, W, x, stats):
    res = O.Oracle(arch, W).run(x)
    seen = set()
    for i in range(x.shape[0]):
        ps = [p for _, p in stats[i]]
        consistent = [k for k in range(len(ps))
                      if all(np.float32(ps[j]) < np.float32(arch["tau"]) for j in range(k))
                      and (k == len(ps) - 1 or np.float32(ps[k]) >= np.float32(arch["tau"]))]
        assert len(consistent) == 1                      # exactly one self-consistent path
        k = consistent[0]
        assert res["exit_index"][i] == k == _first_exit(ps, arch["tau"])
        np.testing.assert_allclose(res["logits"][i], stats[i][k][0], rtol=1e-6, atol=1e-6)
        _check_trail(res, i, ps[:min(k + 1, len(ps) - 1)], arch["tau"])
        seen.add(k)
    return seen


def _check_trail(res, i, stats, thr):
    """The oracle's decision trail is the statistics of the decisions the
    enumerated path evaluates (forced ones excluded), in order, and its
    margin is their smallest distance to the threshold."""
    trail = res["trail"][i]
    assert len(trail) == len(stats)
    np.testing.assert_allclose(trail, np.asarray(stats, dtype=np.float64), rtol=2e-6, atol=1e-7)
    want = min((abs(float(np.float32(v)) - float(np.float32(thr))) for v in stats), default=math.inf)
    assert res["margin"][i] == pytest.approx(want, rel=1e-5, abs=2e-7)


def test_tiny_mlp_exit_paths():
    arch = configs.arch_mlp_exit(dims=(12, 8, 8, 8), n_classes=5, tau=0.5)
    wl, W = _tiny("tiny_mlp", arch)
    x, _ = wl.inputs_f32(40)
    stats = [N.mlp_static(arch, W, x[i]) for i in range(40)]
    p0 = np.sort([s[0][1] for s in stats])
    arch["tau"] = float(0.5 * (p0[13] + p0[14]))        # a third leaves at head 0
    seen = _check_exit_network(arch, W, x, stats)
    assert len(seen) >= 2


@pytest.mark.parametrize("kind", ["basic", "bottleneck"])
def test_tiny_resnet_exit_paths(kind):
    if kind == "basic":
        arch = configs.arch_resnet_exit("basic", 8, [4, 8], [1, 1], 5, 0.5, 3, 1, False)
    else:
        arch = configs.arch_resnet_exit("bottleneck", 12, [2, 4], [1, 1], 5, 0.5, 7, 2, True,
                                        stem_out=4, expansion=4)
    wl, W = _tiny("tiny_" + kind, arch)
    x, _ = wl.inputs_f32(12)
    stats = [N.resnet_exit_static(arch, W, x[i]) for i in range(12)]
    p0 = np.sort([s[0][1] for s in stats])
    arch["tau"] = float(0.5 * (p0[5] + p0[6]))
    seen = _check_exit_network(arch, W, x, stats)
    assert seen == {0, 1}


def test_tiny_skipnet_paths():
    arch = configs.arch_skipnet(hw=8, widths=(4, 8), per_stage=2, n_classes=5)
    wl, W = _tiny("tiny_skip", arch)
    n = 10
    x, _ = wl.inputs_f32(n)
    # centre every gate on the all-execute path so that routing is mixed
    for i, b in enumerate(arch["blocks"]):
        qs = [N.skipnet_path(arch, W, x[j], [1] * 4)[1][i] for j in range(n)]
        pre = np.log(np.array(qs) / (1 - np.array(qs))) - W[b["gate"] + ".v"][0]
        W[b["gate"] + ".v"] = np.array([-np.median(pre)], dtype=np.float32)
    res = O.Oracle(arch, W).run(x)
    masks = set()
    for j in range(n):
        consistent = []
        for path in itertools.product([0, 1], repeat=4):
            z, qs = N.skipnet_path(arch, W, x[j], path)
            if all((np.float32(qv) > np.float32(0.5)) == bool(d) for qv, d in zip(qs, path)):
                consistent.append((path, z))
        assert len(consistent) == 1
        path, z = consistent[0]
        want_mask = sum(1 << i for i, d in enumerate(path) if not d)
        assert int(res["skip_mask"][j]) == want_mask
        np.testing.assert_allclose(res["logits"][j], z, rtol=1e-6, atol=1e-6)
        _check_trail(res, j, N.skipnet_path(arch, W, x[j], path)[1], 0.5)
        masks.add(want_mask)
    assert len(masks) >= 3


def test_tiny_act_paths_and_one_step_closed_form():
    arch = configs.arch_act(hidden=8, d_in=8, d_out=6, max_steps=5, tau=0.99)
    wl, W = _tiny("tiny_act", arch)
    x, aux = wl.inputs_f32(24)
    res = O.Oracle(arch, W).run(x, aux)
    iters = set()
    for i in range(24):
        traj = N.act_static(arch, W, x[i], aux[i])
        Ns = [t + 1 for t in range(5) if (traj[t][1] >= np.float32(0.99) or t == 4)
              and all(traj[s][1] < np.float32(0.99) for s in range(t))]
        assert len(Ns) == 1
        n = Ns[0]
        assert res["iterations"][i] == n
        _check_trail(res, i, [traj[t][1] for t in range(min(n, 4))], 0.99)   # step 5 is forced
        z = W["W2"].astype(np.float64) @ traj[n - 1][0] + W["b2"]
        np.testing.assert_allclose(res["logits"][i], z, rtol=1e-6, atol=1e-6)
        iters.add(n)
    assert len(iters) >= 2
    # max_steps = 1: a two-layer MLP on [0; x]
    arch1 = dict(arch, max_steps=1)
    r1 = O.Oracle(arch1, W).run(x[:3], aux[:3])
    for i in range(3):
        u = W["W1"][:, 8:].astype(np.float64) @ x[i] + W["b1"]
        h = N.q_np([0.5 * v * (1 + N.erf_series(v / math.sqrt(2))) for v in u])
        np.testing.assert_allclose(r1["logits"][i], W["W2"].astype(np.float64) @ h + W["b2"], rtol=1e-6, atol=1e-6)
        assert r1["iterations"][i] == 1


# -------------------------------------------------- real workloads -------

def _same(a, b):
    for k in ("logits", "exit_index", "iterations", "skip_mask"):
        np.testing.assert_array_equal(a[k], b[k])


@pytest.mark.parametrize("name,B", [("mlp_exit", 64), ("act_loop", 24), ("skipnet38", 5)])
def test_batch_split_and_permutation_invariance(name, B):
    wl = configs.build(name)
    x, aux = wl.inputs_f32(B)
    o = O.from_workload(wl)
    full = o.run(x, aux)
    k = B // 3
    lo, hi = o.run(x[:k], None if aux is None else aux[:k]), o.run(x[k:], None if aux is None else aux[k:])
    for key in ("logits", "exit_index", "iterations", "skip_mask"):
        np.testing.assert_array_equal(np.concatenate([lo[key], hi[key]]), full[key])
    perm = RNG.permutation(B)
    pr = o.run(x[perm], None if aux is None else aux[perm])
    for key in ("logits", "exit_index", "iterations", "skip_mask"):
        np.testing.assert_array_equal(pr[key], full[key][perm])
    # sample i of a larger batch is the same sample
    x2, aux2 = wl.inputs_f32(B + 3)
    np.testing.assert_array_equal(x2[:B], x)


def test_exit_invariants_and_forced_thresholds():
    wl = configs.build("mlp_exit")
    x, _ = wl.inputs_f32(64)
    r = O.from_workload(wl).run(x)
    assert np.bincount(r["exit_index"], minlength=3).sum() == 64
    assert r["exit_index"].min() >= 0 and r["exit_index"].max() <= 2
    for tau, want in ((0.0, 0), (1.5, 2)):
        arch = dict(wl.arch, tau=tau)
        rr = O.Oracle(arch, wl.weights_f32()).run(x)
        assert (rr["exit_index"] == want).all()


def test_resnet_exit_forced_thresholds():
    wl = configs.build("resnet18_exit")
    x, _ = wl.inputs_f32(2)
    W = wl.weights_f32()
    r0 = O.Oracle(dict(wl.arch, tau=0.0), W).run(x)
    r1 = O.Oracle(dict(wl.arch, tau=1.5), W).run(x)
    assert (r0["exit_index"] == 0).all() and (r1["exit_index"] == 3).all()


def test_act_loop_bounds_and_monotone_halting_sum():
    wl = configs.build("act_loop")
    x, aux = wl.inputs_f32(48)
    r = O.from_workload(wl).run(x, aux)
    assert r["iterations"].min() >= 1 and r["iterations"].max() <= 16
    for tr, n in zip(r["trail"], r["iterations"]):
        assert all(b > a for a, b in zip(tr, tr[1:]))
        assert len(tr) == min(n, 15)
        assert all(s < np.float32(0.99) for s in tr[:n - 1])


def test_skipnet_forced_gates_reproduce_static_networks():
    wl = configs.build("skipnet38")
    x, _ = wl.inputs_f32(2)
    W = wl.weights_f32()
    arch = wl.arch
    for v, mask in ((50.0, 0), (-50.0, (1 << 18) - 1)):
        W2 = dict(W)
        for b in arch["blocks"]:
            W2[b["gate"] + ".v"] = np.array([v], dtype=np.float32)
        r = O.Oracle(arch, W2).run(x)
        assert (r["skip_mask"] == mask).all()
        if v < 0:     # every block skipped: stem, then the two shortcut projections, then fc
            for i in range(2):
                z, _ = N.skipnet_path(arch, W2, x[i], [0] * 18)
                np.testing.assert_allclose(r["logits"][i], z, rtol=1e-6, atol=1e-6)


# ---------------------------------------------------------- metrics -----

def test_eq1_metrics_closed_forms():
    a = RNG.standard_normal((5, 4)).astype(np.float32)
    assert O.delta(a, a) == pytest.approx(-10.0)
    b = a.copy()
    b[2, 1] += 0.001
    assert O.delta(b, a) == pytest.approx(math.log10(0.001 + 1e-10), abs=1e-4)
    assert O.eta(a, a) == 0.0
    c = a.copy()
    c[0] = -a[0] + 10 * (np.arange(4) == (np.argmin(a[0])))   # argmax moves
    assert O.eta(c, a) == pytest.approx(0.2)


# ------------------------------------------ float32 accumulation orders ----

@pytest.mark.parametrize("acc", O.ACC_F32)
def test_f32_orders_within_the_float32_summation_bound(acc):
    # every float32 order is a correct evaluation: within the textbook
    # bound of float32 recursive summation, gamma_K * sum |x| |w| with
    # gamma_K = K u / (1 - K u), u = 2^-24, of the exact (float64) sums
    g = torch.Generator().manual_seed(5)
    x = torch.randn(40, 7, 6, generator=g, dtype=torch.float64)
    w = torch.randn(5, 40, 3, 3, generator=g, dtype=torch.float64)
    y = O.conv2d(x, w, 1, 1, acc)
    assert y.dtype == torch.float32
    ref = O.conv2d(x, w, 1, 1, "f64")
    mag = O.conv2d(x.abs(), w.abs(), 1, 1, "f64")
    K, u = 40 * 9, 2.0 ** -24
    assert ((y.double() - ref).abs() <= K * u / (1 - K * u) * mag + 1e-300).all()
    W = torch.randn(9, 70, generator=g, dtype=torch.float64)
    v = torch.randn(70, generator=g, dtype=torch.float64)
    z = O.linear(W, v, acc)
    assert z.dtype == torch.float32
    assert ((z.double() - W @ v).abs() <= 70 * u / (1 - 70 * u) * (W.abs() @ v.abs())).all()


def test_f32_block_order_is_exact_below_one_block():
    # 16 input channels or fewer form one block: its sum is exact and is
    # rounded to float32 once, so it equals the float64 result rounded
    g = torch.Generator().manual_seed(6)
    x = torch.randn(16, 5, 5, generator=g, dtype=torch.float64)
    w = torch.randn(3, 16, 3, 3, generator=g, dtype=torch.float64)
    assert torch.equal(O.conv2d(x, w, 1, 1, "f32c"), O.conv2d(x, w, 1, 1, "f64").to(torch.float32))
    W = torch.randn(4, 16, generator=g, dtype=torch.float64)
    v = torch.randn(16, generator=g, dtype=torch.float64)
    assert torch.equal(O.linear(W, v, "f32c"), (W @ v).to(torch.float32))


def test_f32_orders_are_distinct_orders():
    # the orders are different summations of the same terms: on long sums
    # they differ somewhere in the last bits, and never by more than the bound
    g = torch.Generator().manual_seed(7)
    x = torch.randn(256, 6, 6, generator=g, dtype=torch.float64)
    w = torch.randn(8, 256, 3, 3, generator=g, dtype=torch.float64)
    ys = {a: O.conv2d(x, w, 1, 1, a) for a in O.ACC_F32}
    assert not torch.equal(ys["f32"], ys["f32c"])
    assert not torch.equal(ys["f32"], ys["f32r"])


# ------------------------------------------------------ the LSTM decoder ----

def test_naive_lstm_cell_is_the_library_cell():
    # the independent reference's cell equations and gate order against
    # torch.nn.LSTMCell (float64, bias_hh zero): W = [W_hh | W_ih]
    g = torch.Generator().manual_seed(8)
    H, E = 6, 4
    cell = torch.nn.LSTMCell(E, H).double()
    with torch.no_grad():
        for p in cell.parameters():
            p.copy_(torch.randn(p.shape, generator=g, dtype=torch.float64))
        cell.bias_hh.zero_()
    h = torch.randn(H, generator=g, dtype=torch.float64)
    c = torch.randn(H, generator=g, dtype=torch.float64)
    e = torch.randn(E, generator=g, dtype=torch.float64)
    hl, cl = cell(e[None], (h[None], c[None]))
    Wl = torch.cat([cell.weight_hh, cell.weight_ih], dim=1).detach().numpy()
    hn, cn = N.lstm_step(Wl, cell.bias_ih.detach().numpy(), h.numpy(), e.numpy(), c.numpy())
    np.testing.assert_allclose(hn, hl[0].detach().numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(cn, cl[0].detach().numpy(), rtol=1e-12, atol=1e-14)


def _tiny_decoder(eos_shift):
    arch = configs.arch_decoder(d_in=6, hidden=4, embed=3, vocab=5, max_len=4, out_gain=8.0)
    wl = configs.raw_workload("tiny_dec", arch)
    W = wl.weights_f32()
    W["out.b"] = W["out.b"].copy()
    W["out.b"][arch["eos"]] += np.float32(eos_shift)
    return arch, wl, W


@pytest.mark.parametrize("eos_shift", [0.0, -0.3])
def test_tiny_decoder_paths(eos_shift):
    # every token sequence of length <= max_len is evaluated as a static
    # network along that sequence; exactly one is self-consistent (each
    # token is its step's argmax, lowest index on ties; the end token or the
    # length bound ends it) and the oracle emits it, with that path's last
    # logits and its gaps as the decision trail
    arch, wl, W = _tiny_decoder(eos_shift)
    V, L, eos = arch["vocab"], arch["max_len"], arch["eos"]
    x, _ = wl.inputs_f32(12)
    res = O.Oracle(arch, W).run(x)
    lengths = set()
    for i in range(12):
        consistent = []
        for n in range(1, L + 1):
            for seq in itertools.product(range(V), repeat=n):
                if any(t == eos for t in seq[:-1]) or (n < L and seq[-1] != eos):
                    continue
                zs = N.decoder_path(arch, W, x[i], seq)
                if all(int(np.argmax(z)) == t for z, t in zip(zs, seq)):
                    consistent.append((seq, zs))
        assert len(consistent) == 1
        seq, zs = consistent[0]
        n = len(seq)
        assert res["iterations"][i] == n and res["exit_index"][i] == -1 and res["skip_mask"][i] == 0
        assert list(res["tokens"][i][:n]) == list(seq) and (res["tokens"][i][n:] == -1).all()
        np.testing.assert_allclose(res["logits"][i], zs[-1], rtol=1e-6, atol=1e-6)
        gaps = [float(np.sort(z)[-1] - np.sort(z)[-2]) for z in zs]
        _check_trail(res, i, gaps, 0.0)
        lengths.add(n)
    assert len(lengths) >= 2


def test_decoder_special_cases():
    arch, wl, W = _tiny_decoder(0.0)
    x, _ = wl.inputs_f32(6)
    # the end token always wins: every sequence is that token alone
    Wb = dict(W, **{"out.b": W["out.b"] + np.where(np.arange(arch["vocab"]) == arch["eos"], 1e4, 0.0)
                    .astype(np.float32)})
    r = O.Oracle(arch, Wb).run(x)
    assert (r["iterations"] == 1).all() and (r["tokens"][:, 0] == arch["eos"]).all()
    # the end token never wins: every sequence runs to the length bound
    Wn = dict(W, **{"out.b": W["out.b"] - np.where(np.arange(arch["vocab"]) == arch["eos"], 1e4, 0.0)
                    .astype(np.float32)})
    r = O.Oracle(arch, Wn).run(x)
    assert (r["iterations"] == arch["max_len"]).all() and (r["tokens"] != arch["eos"]).all()
    # a bound of one step: one token, the argmax of the first step's logits
    a1 = dict(arch, max_len=1)
    r = O.Oracle(a1, W).run(x)
    for i in range(6):
        z = N.decoder_path(a1, W, x[i], [0])[0]
        assert r["iterations"][i] == 1 and r["tokens"][i][0] == int(np.argmax(z))
        np.testing.assert_allclose(r["logits"][i], z, rtol=1e-6, atol=1e-6)


def test_decoder_workload_invariants():
    wl = configs.build("lstm_decoder")
    a = wl.arch
    x, _ = wl.inputs_f32(24)
    r = O.from_workload(wl).run(x)
    L = a["max_len"]
    for i in range(24):
        n = r["iterations"][i]
        assert 1 <= n <= L
        assert (r["tokens"][i][:n] >= 0).all() and (r["tokens"][i][n:] == -1).all()
        if n < L:
            assert r["tokens"][i][n - 1] == a["eos"]      # only the end token stops early
        assert not (r["tokens"][i][:n - 1] == a["eos"]).any()
    # batch-split invariance
    r2 = O.from_workload(wl).run(x, indices=range(10, 24))
    np.testing.assert_array_equal(r2["tokens"], r["tokens"][10:])
    np.testing.assert_array_equal(r2["logits"], r["logits"][10:])
