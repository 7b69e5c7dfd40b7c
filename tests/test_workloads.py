"""The shared seeded generator: determinism, per-sample independence, the
distributions the workload descriptions ask for, and the stored constants."""

import json
import math
import os

import numpy as np
import pytest

from workloads import configs, rng

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_splitmix64_reference_values():
    # SplitMix64 with state 0: the first outputs of the published generator
    k = np.uint64(0)
    out = rng.bits64(k, 0, 3)
    assert [hex(int(v)) for v in out] == ["0xe220a8397b1dcdaf", "0x6e789e6aa1b965f4", "0x6c45d188009454f"]


def test_uniform_normal_moments():
    k = rng.stream_key(7, "moments")
    u = rng.uniform(k, 0, 200000)
    assert u.min() >= 0.0 and u.max() < 1.0
    assert abs(u.mean() - 0.5) < 5e-3 and abs(u.var() - 1 / 12) < 2e-3
    z = rng.normal(k, 0, 200000)
    assert abs(z.mean()) < 1e-2 and abs(z.std() - 1.0) < 1e-2
    # counter mode: a window of the stream is the same numbers
    np.testing.assert_array_equal(rng.normal(k, 1000, 10), z[1000:1010])


@pytest.mark.parametrize("name", configs.NAMES)
def test_inputs_per_sample_and_deterministic(name):
    wl = configs.build(name)
    x1, a1 = wl.inputs(5)
    x2, a2 = wl.inputs(3, start=2)
    np.testing.assert_array_equal(x1[2:], x2)
    if a1 is not None:
        np.testing.assert_array_equal(a1[2:], a2)
        assert abs(wl.inputs(4096)[1].mean() + 1.0) < 0.1          # b ~ N(-1, 1)
    b1, m1 = wl.blob()
    b2, m2 = configs.build(name).blob()
    assert b1 == b2 and m1 == m2
    for e in m1.values():
        assert e["offset"] % 256 == 0


def test_kaiming_bounds_and_bf16_bytes():
    wl = configs.build("resnet18_exit")
    w = wl.tensors["s2.b0.c1.w"].value
    bound = math.sqrt(6.0 / (3 * 3 * 64))
    assert np.abs(w).max() <= bound and np.abs(w).max() > 0.95 * bound
    bits = configs.to_bf16_bits(np.array([1.0, 1.0 + 2 ** -8, -2.0], dtype=np.float32))
    assert list(bits) == [0x3F80, 0x3F80, 0xC000]


def test_stored_calibration_and_floor_files():
    for name in ("mlp_exit", "resnet18_exit", "skipnet38", "resnet50_exit", "lstm_decoder"):
        assert configs.build(name).calibrated
    with open(os.path.join(ROOT, "tests", "golden", "decision_floor.json")) as f:
        fl = json.load(f)
    for name in ("mlp_exit", "resnet18_exit", "skipnet38", "resnet50_exit", "act_loop"):
        assert fl[name]["routing_diverged"] == 0
        assert all(v >= 0 for v in fl[name]["floor"])
