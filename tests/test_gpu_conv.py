"""Sub-network convolution kernels through dycl_op_conv, element by element
against the oracle's convolution (float64, bf16 inputs), at every geometry
the launcher distinguishes: the halo-tiled kernel with register-resident
weights (64 -> 64 channels, 3x3, stride 1: row tiles, partial row tiles,
whole-image tiles with a ragged last tile, several tiles per workgroup), the
direct-to-LDS implicit GEMM (1x1, 3x3, strided; with the K range of each
tile split over workgroups for deep K on few pixels, and without), the
RGB stem kernel (3-channel input read directly: 7x7 stride 2, ragged units
and pixel blocks), the narrow halo kernel (16 or 32 channels, weights in
registers) and the element-gathering kernel (other 3-channel stems, Cout
not a multiple of 8).

Bound per element: the fp32 accumulation error (K terms, gamma_K * sum |x w|)
scaled by |scale|, the fp32 epilogue roundings, and half a bf16 ulp of the
final rounding."""

import numpy as np
import pytest
import torch

from oracle import dycl_oracle as O
from workloads.configs import bf16_bits_to_f32, to_bf16_bits

pytestmark = pytest.mark.gpu

CASES = [
    # n, H, W, cin, cout, k, stride, pad, residual, act
    (3, 32, 32, 64, 64, 3, 1, 1, True, 1),      # row tiles (4 rows of 32)
    (80, 32, 32, 64, 64, 3, 1, 1, True, 1),     # 640 tiles: several per workgroup
    (5, 8, 8, 64, 64, 3, 1, 1, False, 1),       # two images per tile, ragged last tile
    (1500, 8, 8, 64, 64, 3, 1, 1, True, 0),     # 750 image tiles
    (3, 56, 56, 64, 64, 3, 1, 1, True, 1),      # 112-row tiles (2 rows of 56)
    (9, 4, 4, 64, 64, 3, 1, 1, False, 2),       # eight images per tile, GELU
    (40, 14, 14, 64, 64, 3, 1, 1, True, 1),     # 9-row tiles, 5-row remainder
    (2, 9, 9, 64, 64, 3, 1, 1, False, 0),       # one 81-pixel image per tile
    (3, 7, 7, 64, 64, 3, 1, 1, True, 1),
    (4, 16, 16, 128, 128, 3, 1, 1, True, 1),    # halo tiles, streamed weights
    (300, 16, 16, 128, 128, 3, 1, 1, True, 1),  # 600 units: several per workgroup
    (9, 4, 4, 512, 512, 3, 1, 1, True, 1),      # 7 images per tile (patch capacity)
    (3, 7, 7, 512, 512, 3, 1, 1, False, 0),
    (2, 14, 14, 256, 256, 3, 1, 1, True, 1),    # 9-row tiles, 5-row remainder
    (2, 28, 28, 128, 128, 3, 1, 1, False, 2),
    (5, 8, 8, 128, 64, 3, 1, 1, True, 1),       # 64-channel output tiles
    (40, 8, 8, 256, 256, 3, 1, 1, False, 1),
    (4, 16, 16, 64, 128, 3, 2, 1, False, 1),    # strided
    (4, 16, 16, 128, 256, 1, 1, 0, False, 0),   # 1x1
    (5, 15, 15, 128, 256, 1, 1, 0, True, 1),    # 1x1, two K steps requested together, ragged last tile
    (7, 14, 14, 128, 512, 1, 2, 0, False, 1),   # strided 1x1, two K steps
    (60, 14, 14, 64, 256, 1, 1, 0, True, 1),    # 1x1, one K step, ragged last tile
    (6, 8, 8, 256, 512, 3, 1, 1, True, 1),
    (3, 32, 32, 8, 64, 3, 1, 1, False, 1),      # 8-channel stem, weights in registers
    (300, 32, 32, 8, 64, 3, 1, 1, True, 1),     # several tiles per workgroup
    (5, 8, 8, 8, 64, 3, 1, 1, False, 2),        # image tiles, ragged
    (3, 20, 20, 3, 64, 7, 2, 3, False, 1),      # 3-channel stem, W % 8 != 0: element gathers
    (3, 224, 224, 3, 64, 7, 2, 3, False, 1),    # RGB stem kernel: 7x7 / 2, 112-pixel rows
    (2, 42, 40, 3, 64, 7, 2, 3, False, 2),      # 21 x 20 output: ragged last unit, 2 pixel blocks, GELU
    (3, 20, 104, 3, 64, 7, 2, 3, False, 0),     # 52-pixel rows: ragged pixel block
    (2, 64, 64, 3, 64, 7, 2, 2, False, 1),      # pad 2 (even: no column offset)
    (2, 224, 224, 3, 64, 7, 2, 3, True, 1),     # with a residual: element gathers
    (7, 32, 32, 3, 64, 3, 1, 1, False, 1),      # 3x3 CIFAR stem on 3 channels: element gathers
    (5, 12, 12, 16, 32, 3, 1, 1, False, 1),
    (5, 32, 32, 16, 16, 3, 1, 1, True, 1),      # narrow halo kernel: 16 channels, 4-row units
    (7, 32, 32, 16, 16, 3, 1, 1, False, 0),
    (300, 32, 32, 16, 16, 3, 1, 1, True, 1),    # several units per workgroup
    (3, 9, 16, 16, 16, 3, 1, 1, True, 1),       # 16-pixel rows: 8-row units, ragged last unit
    (3, 16, 16, 32, 32, 3, 1, 1, True, 1),      # 32 channels
    (4, 13, 32, 32, 32, 3, 1, 1, False, 2),     # 13 rows: ragged last unit, GELU
    (5, 32, 32, 8, 16, 3, 1, 1, False, 1),      # 8-channel stem to 16: four taps per K step
    (3, 16, 16, 8, 16, 3, 1, 1, True, 2),
    (6, 11, 16, 8, 64, 3, 1, 1, True, 0),       # 8 -> 64 stays on the register-weight halo kernel
    (5, 12, 12, 64, 24, 3, 1, 1, True, 2),      # Cout not a multiple of 8
    (37, 4, 4, 512, 512, 3, 1, 1, False, 1),    # K split in 4, ragged last row tile
    (37, 8, 8, 512, 512, 3, 2, 1, True, 1),     # strided, K split in 4
    (5, 4, 4, 512, 384, 3, 1, 1, True, 2),      # three 128-channel tiles, GELU
    (11, 7, 7, 512, 256, 3, 2, 1, False, 0),    # 7x7 -> 4x4, K split in 4
    (6, 4, 4, 4608, 256, 1, 1, 0, False, 1),    # 1x1 with K = 4608, split in 4
    (37, 14, 14, 512, 512, 3, 2, 1, True, 1),   # strided 14x14 -> 7x7, K split in 4
    (11, 12, 12, 512, 256, 3, 2, 1, False, 0),  # 12x12 -> 6x6, K split in 4
    (6, 6, 6, 4608, 256, 1, 1, 0, False, 1),    # 1x1 with K = 4608 on 36 pixels, split in 4
    # deep K without a split: strided, deep 1x1, ragged channel tiles, many tiles
    (7, 9, 9, 64, 96, 3, 2, 1, True, 1),        # half-used second channel tile
    (3, 16, 16, 1024, 256, 1, 1, 0, True, 0),   # deep 1x1 with residual
    (2, 14, 14, 256, 512, 3, 2, 1, False, 2),   # strided, GELU
    (2000, 8, 8, 128, 256, 3, 2, 1, False, 1),  # 128-pixel tiles, several units per workgroup
    (2500, 8, 8, 128, 256, 3, 2, 1, True, 1),   # 256-pixel tiles, several units per workgroup
    (3, 6, 6, 600, 64, 1, 1, 0, False, 1),      # K = 600: the last step is partly padding
    (24, 56, 56, 64, 256, 1, 1, 0, True, 1),    # one stage, 128 x 256 tiles (588 of them), residual
    (24, 56, 56, 128, 256, 1, 1, 0, False, 2),  # one stage, 128 x 256 tiles, two K steps in turn, GELU
    (48, 28, 28, 384, 512, 1, 1, 0, True, 1),   # one stage, 128 x 256 tiles, six K steps, residual
    (40, 28, 28, 512, 128, 1, 1, 0, False, 1),  # one stage, 128 x 64 tiles, eight K steps
    (42, 56, 56, 128, 128, 3, 2, 1, False, 1),  # strided 3x3, 516 tiles of 128 x 64: 64 x 128 tiles
    (107, 14, 14, 1024, 256, 1, 1, 0, False, 1),  # 656 tiles: 64 x 128, rounds of two K steps
    (107, 28, 28, 256, 256, 3, 2, 1, True, 1),    # strided 3x3 on 64 x 128 tiles, residual
    (30, 14, 14, 1024, 256, 1, 1, 0, True, 2),    # 184 tiles: 64 x 64, GELU
]


def _bits(a):
    return torch.from_numpy(to_bf16_bits(np.asarray(a, np.float32)).view(np.int16).copy())


def _case(n, H, W, cin, cout, k, stride, pad, residual, act, seed, workspace="auto"):
    from paper_2307_04963_amd import runtime
    rng = np.random.default_rng(seed)
    x = bf16_bits_to_f32(to_bf16_bits(rng.standard_normal((n, H, W, cin)).astype(np.float32)))
    bound = np.sqrt(6.0 / (k * k * cin))
    w = bf16_bits_to_f32(to_bf16_bits(rng.uniform(-bound, bound, (cout, k, k, cin)).astype(np.float32)))
    sc = rng.uniform(0.5, 1.5, cout).astype(np.float32)
    sh = rng.uniform(-0.3, 0.3, cout).astype(np.float32)
    Ho, Wo = (H + 2 * pad - k) // stride + 1, (W + 2 * pad - k) // stride + 1
    r = bf16_bits_to_f32(to_bf16_bits(rng.standard_normal((n, Ho, Wo, cout)).astype(np.float32))) if residual else None
    packed = torch.from_numpy(runtime.pack_conv_weights(to_bf16_bits(w)).view(np.int16)).cuda()
    xt = _bits(x).cuda().view(torch.bfloat16)
    rt = _bits(r).cuda().view(torch.bfloat16) if residual else None
    y = runtime.conv(xt, packed, cout, k, stride, pad, torch.from_numpy(sc).cuda(), torch.from_numpy(sh).cuda(), rt, act,
                     workspace=workspace)
    torch.cuda.synchronize()
    got = bf16_bits_to_f32(y.cpu().view(torch.int16).numpy().view(np.uint16)).astype(np.float64)

    # reference on every image of small batches, on 8 spread images of large ones
    imgs = np.arange(n) if n <= 16 else np.unique(np.linspace(0, n - 1, 8).astype(int))
    wt = torch.from_numpy(w.astype(np.float64)).permute(0, 3, 1, 2)
    K = k * k * cin
    gamma = K * 2.0 ** -24 / (1 - K * 2.0 ** -24)
    lip = 1.13 if act == 2 else 1.0
    for i in imgs:
        xi = torch.from_numpy(x[i].astype(np.float64)).permute(2, 0, 1)
        acc = O.conv2d(xi, wt, stride, pad).permute(1, 2, 0).numpy()
        mag = O.conv2d(xi.abs(), wt.abs(), stride, pad).permute(1, 2, 0).numpy()
        v = acc * sc + sh + (r[i] if residual else 0.0)
        if act == 1:
            v = np.maximum(v, 0.0)
        elif act == 2:
            v = O.gelu(torch.from_numpy(v)).numpy()
        tol = (2.0 ** -8 * 1.001 * np.abs(v) +
               lip * (gamma * mag * np.abs(sc) + 2.0 ** -22 * (np.abs(acc * sc) + np.abs(sh) + (np.abs(r[i]) if residual else 0))))
        err = np.abs(got[i] - v)
        bad = np.argwhere(err > tol)
        assert bad.size == 0, (f"image {i}: {len(bad)} elements out of bound, first {tuple(bad[0])}: "
                               f"got {got[i][tuple(bad[0])]} ref {v[tuple(bad[0])]}")
    return got


@pytest.mark.parametrize("case", CASES, ids=lambda c: "n{}_{}x{}_{}to{}_k{}s{}".format(*c[:7]))
def test_conv_op(case):
    _case(*case, seed=hash(case) % (2 ** 31))


def _split(c):
    """Cases whose layer dycl_op_conv splits over K (deep K on at most 64
    output pixels per image, on the implicit GEMM)."""
    n, H, W, cin, cout, k, stride, pad = c[:8]
    Ho, Wo = (H + 2 * pad - k) // stride + 1, (W + 2 * pad - k) // stride + 1
    halo = k == 3 and stride == 1 and not (H * W <= 128 and 2 * H * W < (H + 2) * (W + 2))
    return cout >= 256 and cout % 64 == 0 and k * k * cin >= 4608 and Ho * Wo <= 64 and not halo


@pytest.mark.parametrize("case", [c for c in CASES if _split(c)], ids=str)
def test_conv_op_unsplit_without_workspace(case):
    # the same layers without a workspace: one K range per tile
    _case(*case, seed=hash(case) % (2 ** 31), workspace=None)


def test_conv_op_split_rows_are_independent():
    # the first rows of a K-split batch alone give the same bits (the split
    # depends on the layer shape, not on n)
    from paper_2307_04963_amd import runtime
    rng = np.random.default_rng(11)
    x = _bits(rng.standard_normal((100, 14, 14, 512))).cuda().view(torch.bfloat16)
    w = to_bf16_bits(rng.uniform(-0.02, 0.02, (512, 3, 3, 512)).astype(np.float32))
    packed = torch.from_numpy(runtime.pack_conv_weights(w).view(np.int16)).cuda()
    assert runtime.conv_workspace_bytes(100, 14, 14, 512, 512, 3, 2, 1) > 0   # split over K
    a = runtime.conv(x, packed, 512, 3, 2, 1, None, None, None, 1)
    b = runtime.conv(x[:13].contiguous(), packed, 512, 3, 2, 1, None, None, None, 1)
    torch.cuda.synchronize()
    assert torch.equal(a[:13].view(torch.int16), b.view(torch.int16))


def test_conv_op_full_rgb_stem_shape():
    """The 7x7 / 2 stem of the ResNet-50 early-exit network at its benchmark
    batch (256 x 224 x 224 x 3 -> 112 x 112 x 64, ReLU), 8 images checked
    element by element."""
    _case(256, 224, 224, 3, 64, 7, 2, 3, False, 1, seed=5)


def _maxpool3s2(v):
    """3x3 / stride-2 / pad-1 max-pool of [H, W, C] by its definition: the
    maximum over the window's pixels inside the input."""
    H, W, C = v.shape
    Hp, Wp = (H - 1) // 2 + 1, (W - 1) // 2 + 1
    out = np.empty((Hp, Wp, C), v.dtype)
    for ph in range(Hp):
        for pw in range(Wp):
            r0, r1 = max(2 * ph - 1, 0), min(2 * ph + 2, H)
            c0, c1 = max(2 * pw - 1, 0), min(2 * pw + 2, W)
            out[ph, pw] = v[r0:r1, c0:c1].reshape(-1, C).max(axis=0)
    return out


@pytest.mark.parametrize("case", [(3, 224, 224, 3), (2, 42, 40, 3), (3, 20, 104, 3), (2, 64, 64, 2), (5, 8, 8, 3),
                                  (2, 30, 16, 1)], ids=str)
def test_conv_maxpool_op(case):
    """The RGB stem with its max-pool fused in (n, H, W, pad; 7x7 / 2, 3 -> 64,
    ReLU): bit for bit the max-pool of the unfused stem's bf16 output, and
    within the convolution's bound of the oracle's float64 convolution and
    max-pool (a maximum moves by at most the largest error in its window)."""
    from paper_2307_04963_amd import runtime
    n, H, W, pad = case
    cin, cout, k = 3, 64, 7
    rng = np.random.default_rng(hash(case) % (2 ** 31))
    x = bf16_bits_to_f32(to_bf16_bits(rng.standard_normal((n, H, W, cin)).astype(np.float32)))
    bound = np.sqrt(6.0 / (k * k * cin))
    w = bf16_bits_to_f32(to_bf16_bits(rng.uniform(-bound, bound, (cout, k, k, cin)).astype(np.float32)))
    sc = rng.uniform(0.5, 1.5, cout).astype(np.float32)
    sh = rng.uniform(-0.3, 0.3, cout).astype(np.float32)
    packed = torch.from_numpy(runtime.pack_conv_weights(to_bf16_bits(w)).view(np.int16)).cuda()
    xt = _bits(x).cuda().view(torch.bfloat16)
    sct, sht = torch.from_numpy(sc).cuda(), torch.from_numpy(sh).cuda()
    yp = runtime.conv_maxpool(xt, packed, cout, k, 2, pad, sct, sht)
    yc = runtime.conv(xt, packed, cout, k, 2, pad, sct, sht, None, 1)
    torch.cuda.synchronize()
    got = bf16_bits_to_f32(yp.cpu().view(torch.int16).numpy().view(np.uint16)).astype(np.float64)
    conv = bf16_bits_to_f32(yc.cpu().view(torch.int16).numpy().view(np.uint16)).astype(np.float64)
    wt = torch.from_numpy(w.astype(np.float64)).permute(0, 3, 1, 2)
    K = k * k * cin
    gamma = K * 2.0 ** -24 / (1 - K * 2.0 ** -24)
    for i in range(n):
        assert np.array_equal(got[i], _maxpool3s2(conv[i])), f"image {i}: fused and unfused pooling differ"
        xi = torch.from_numpy(x[i].astype(np.float64)).permute(2, 0, 1)
        acc = O.conv2d(xi, wt, 2, pad).permute(1, 2, 0).numpy()
        mag = O.conv2d(xi.abs(), wt.abs(), 2, pad).permute(1, 2, 0).numpy()
        v = np.maximum(acc * sc + sh, 0.0)
        tol = 2.0 ** -8 * 1.001 * np.abs(v) + gamma * mag * np.abs(sc) + 2.0 ** -22 * (np.abs(acc * sc) + np.abs(sh))
        ref, tp = _maxpool3s2(v), _maxpool3s2(tol)
        bad = np.argwhere(np.abs(got[i] - ref) > tp)
        assert bad.size == 0, f"image {i}: {len(bad)} pooled elements out of bound, first {tuple(bad[0])}"


def test_conv_op_full_stage1_shape():
    """The first-stage layer of the ResNet-18 early-exit network at the
    benchmark batch (1024 x 32 x 32 x 64 -> 64, residual, ReLU), 8 images
    checked element by element."""
    _case(1024, 32, 32, 64, 64, 3, 1, 1, True, 1, seed=7)


def test_conv_op_full_stage2_shape():
    """A second-stage layer of the ResNet-18 early-exit network at the rows
    that reach it in the benchmark (774 x 16 x 16 x 128 -> 128, residual,
    ReLU), 8 images checked element by element."""
    _case(774, 16, 16, 128, 128, 3, 1, 1, True, 1, seed=8)


def test_conv_op_repeat_is_deterministic():
    """Two launches on the same inputs give the same bits (no race between
    the deferred writes and the next tile's staging)."""
    from paper_2307_04963_amd import runtime
    rng = np.random.default_rng(3)
    n, H, W = 300, 32, 32
    x = _bits(rng.standard_normal((n, H, W, 64))).cuda().view(torch.bfloat16)
    w = to_bf16_bits(rng.uniform(-0.06, 0.06, (64, 3, 3, 64)).astype(np.float32))
    packed = torch.from_numpy(runtime.pack_conv_weights(w).view(np.int16)).cuda()
    res = _bits(rng.standard_normal((n, H, W, 64))).cuda().view(torch.bfloat16)
    a = runtime.conv(x, packed, 64, 3, 1, 1, None, None, res, 1)
    b = runtime.conv(x, packed, 64, 3, 1, 1, None, None, res, 1)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
