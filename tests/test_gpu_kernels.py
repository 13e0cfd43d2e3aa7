"""Bit-exact checks of every convolution loader and tile shape on the GPU.

With small-integer images, weights and biases every partial sum is an integer
far below 2^24, so the kernels' fp32 accumulation is exact in any order and the
only rounding is the single round-to-nearest-even of the output to the model
dtype.  The GPU output must therefore equal the oracle's exact result rounded
once, bit for bit.  Max pooling is exact for any values.
"""
import numpy as np
import pytest
import torch

import paper_2210_08650_amd as H
from paper_2210_08650_amd import models as PM
import synth
from oracle import layers as L
from tests.hip_harness import Runner, bf16_round, images_for

pytestmark = pytest.mark.gpu


def _int_conv_case(seed, dtype, pre_pool, C, N, k, s, p, HW, batch, relu=True, lo=-1, hi=1):
    layers = ([PM.maxpool(1, 1)] if pre_pool else []) + [PM.conv(C, N, k, s, p, bias=True, relu=relu)]
    w = synth.small_ints(seed, (N, C, k, k), lo, hi)
    b = synth.small_ints(seed + 1, (N,), -3, 3)
    x = synth.small_ints(seed + 2, (batch, C, HW, HW), -2, 2)
    r = Runner(layers, dtype, [w, b], (C, HW, HW))
    xd, xv = images_for(dtype, x)
    got = r.extract_np(xd, len(layers))
    ref = L.conv2d(xv, w, b, s, p)
    if relu:
        ref = np.maximum(ref, 0)
    ref = ref.astype(np.float32)
    if dtype == H.HAPI_BF16:
        ref = bf16_round(ref)
    print(f"case seed={seed} C={C} N={N} k={k} s={s} p={p} HW={HW} B={batch}", flush=True)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref), np.abs(got - ref).max()


# (pre_pool, C, N, k, s, p, HW, batch): pre_pool routes the conv through the
# NHWC loaders (a 1x1 identity pool first); otherwise it reads NCHW images.
BF16_CASES = [
    (False, 3, 64, 3, 1, 1, 23, 3),      # first-layer kernel (8-slot NHWC, weights in registers), ragged row
    (False, 3, 64, 3, 1, 1, 224, 2),     # VGG's first layer at full resolution
    (False, 3, 64, 3, 2, 1, 31, 3),      # first-layer kernel, stride 2
    (False, 8, 64, 4, 1, 2, 19, 2),      # first-layer kernel, 16 taps (eight k-steps), 8 channels
    (False, 1, 128, 3, 2, 1, 31, 3),     # 8-slot NHWC on the implicit GEMM, one channel, stride 2
    (False, 8, 40, 4, 1, 2, 19, 2),      # 8-slot NHWC on the implicit GEMM, 16 taps, ragged N tile
    (False, 3, 64, 5, 1, 2, 23, 3),      # NCHW gather, K = 75 padded to 128, ragged M
    (False, 3, 64, 7, 2, 3, 37, 2),      # stem geometry on space-to-depth cells
    (False, 3, 64, 7, 2, 3, 224, 2),     # the ResNet stem at full resolution
    (False, 4, 32, 8, 2, 3, 29, 3),      # space-to-depth with 4 channels, k = 8, N = 32
    (False, 3, 64, 7, 3, 3, 37, 2),      # stride 3: NCHW gather, K = 147
    (False, 3, 96, 11, 4, 2, 63, 2),     # 11x11 / 4, K = 363, ragged N tile
    (False, 3, 128, 16, 16, 0, 64, 3),   # patch loader (16-byte NCHW rows)
    (True, 64, 128, 3, 1, 1, 15, 3),     # NHWC 3x3
    (True, 128, 192, 3, 2, 1, 17, 2),    # NHWC 3x3 / 2, N = 192
    (True, 64, 256, 1, 2, 0, 14, 3),     # 1x1 / 2 shortcut geometry
    (True, 128, 64, 1, 1, 0, 21, 2),     # GEMM loader, N = 64 tile
    (True, 512, 128, 1, 1, 0, 14, 2),    # 1x1, K = 512: three workgroups per CU, two stages
    (True, 64, 256, 1, 1, 0, 128, 4),    # M = 65536: 256 x 128 tiles
    (True, 64, 64, 3, 1, 1, 56, 2),      # row-streaming 3x3, 64 -> 64 (ResNet stage 1)
    (True, 64, 64, 3, 1, 1, 17, 3),      # row-streaming 3x3, ragged rows and bands
    (True, 64, 64, 3, 1, 1, 64, 1),      # row-streaming 3x3: one full 64-column strip
    (True, 64, 64, 3, 1, 1, 130, 2),     # row-streaming 3x3: three strips, the last 2 columns wide
    (True, 64, 64, 3, 1, 1, 224, 1),     # VGG's second layer: four 64-column strips
    (True, 128, 32, 3, 1, 1, 15, 3),     # 32 output channels, few rows: 128 x 32 tiles, ragged M
    (True, 128, 32, 3, 1, 1, 256, 2),    # 32 output channels, M = 131072: 128 x 32 tiles
    (True, 128, 24, 3, 1, 1, 256, 2),    # 24 output channels in a 32-column tile
    (True, 256, 256, 3, 1, 1, 7, 3),     # K = 2304, few rows: 32 x 64 tiles, ragged M
    (True, 512, 512, 3, 1, 1, 7, 2),     # K = 4608 (72 k-tiles) on 32 x 64 tiles
    (True, 256, 256, 3, 1, 1, 14, 16),   # K = 2304, more rows: 64 x 64 tiles, four stages
]


@pytest.mark.parametrize("case", BF16_CASES)
def test_conv_bf16_integer_exact(case):
    _int_conv_case(100 + BF16_CASES.index(case) * 10, H.HAPI_BF16, *case)


F32_CASES = [
    (False, 3, 64, 11, 4, 2, 47, 2),     # AlexNet conv1 geometry
    (False, 3, 32, 3, 1, 1, 19, 3),
    (True, 64, 192, 5, 1, 2, 13, 2),     # AlexNet conv2 geometry
    (True, 192, 96, 3, 1, 1, 13, 2),
    (True, 32, 48, 1, 1, 0, 9, 3),       # GEMM loader
    (True, 384, 64, 3, 1, 1, 7, 2),      # K = 3456: 13 reduction slices (AlexNet conv4 shape)
    (True, 512, 32, 3, 1, 1, 5, 2),      # K = 4608: 16 slices (the cap)
]


@pytest.mark.parametrize("case", F32_CASES)
def test_conv_f32_integer_exact(case):
    _int_conv_case(300 + F32_CASES.index(case) * 10, H.HAPI_F32, *case, lo=-3, hi=3)


@pytest.mark.parametrize("dtype", [H.HAPI_BF16, H.HAPI_F32])
@pytest.mark.parametrize("k,s,p", [(3, 2, 0), (3, 2, 1), (2, 2, 0)])
def test_maxpool_exact(dtype, k, s, p):
    x = synth.images(7, 3, 64, 29, 29)
    xd, xv = images_for(dtype, x)
    r = Runner([PM.maxpool(k, s, p)], dtype, [], (64, 29, 29))
    got = r.extract_np(xd, 1)
    ref = L.maxpool2d(xv, k, s, p).astype(np.float32)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("dtype", [H.HAPI_BF16, H.HAPI_F32])
def test_global_avgpool(dtype):
    x = synth.images(8, 3, 256, 7, 7)
    xd, xv = images_for(dtype, x)
    r = Runner([PM.avgpool()], dtype, [], (256, 7, 7))
    got = r.extract_np(xd, 1)
    ref = L.avgpool_global(xv)
    # fp32 summation of 49 terms: |error| <= 49 * 2^-24 * mean|x|; bf16 adds
    # one round-to-nearest of the output, at most 2^-8 relative.
    scale = np.abs(xv).mean(axis=(2, 3), keepdims=True)
    tol = 49 * 2.0 ** -24 * scale + (2.0 ** -8 * np.abs(ref) if dtype == H.HAPI_BF16 else 0)
    assert np.all(np.abs(got - ref) <= tol), np.abs(got - ref).max()


def test_identity_kernel_conv_is_exact_on_random_values():
    # W = delta(o, c) at the kernel centre: y = x exactly, in bf16 and fp32.
    for dtype in (H.HAPI_BF16, H.HAPI_F32):
        C = 64
        w = np.zeros((C, C, 3, 3), np.float32)
        for c in range(C):
            w[c, c, 1, 1] = 1.0
        x = synth.images(9, 2, C, 11, 11)
        xd, xv = images_for(dtype, x)
        r = Runner([PM.maxpool(1, 1), PM.conv(C, C, 3, 1, 1, bias=True, relu=False)], dtype,
                   [w, np.zeros(C, np.float32)], (C, 11, 11))
        assert np.array_equal(r.extract_np(xd, 2), xv)
        r2 = Runner([PM.maxpool(1, 1), PM.conv(C, C, 3, 2, 1, bias=True, relu=False)], dtype,
                    [w, np.zeros(C, np.float32)], (C, 11, 11))
        assert np.array_equal(r2.extract_np(xd, 2), xv[:, :, ::2, ::2])


@pytest.mark.parametrize("hw,batch", [(20, 3), (56, 2), (9, 2), (70, 1)])
def test_fused_bottleneck_block_exact(hw, batch):
    """A stage-1 bottleneck with an identity shortcut runs its 3x3 and its
    expanding 1x1 convolution as one kernel (the 3x3 result stays on chip,
    rounded once to bf16, as the expansion's operand).  With small-integer
    data and batch-norm scales of exactly one, every sum is exact and the
    only roundings are the three bf16 roundings of the block, which the
    reference applies at the same points: the output must match bit for bit."""
    cin, w = 256, 64
    var = np.float32(1.0) - np.float32(1e-5)   # var + 1e-5 == 1 in float32
    assert var + np.float32(1e-5) == np.float32(1.0)

    def bn(seed, c):
        return [np.ones(c, np.float32), synth.small_ints(seed, (c,), -2, 2),
                np.zeros(c, np.float32), np.full(c, var, np.float32)]
    w1 = synth.small_ints(300, (w, cin, 1, 1), -1, 1)
    w2 = synth.small_ints(301, (w, w, 3, 3), -1, 1)
    w3 = synth.small_ints(302, (4 * w, w, 1, 1), -1, 1)
    b1, b2, b3 = bn(303, w), bn(304, w), bn(305, 4 * w)
    params = [w1] + b1 + [w2] + b2 + [w3] + b3
    layers = [PM.maxpool(1, 1), dict(kind=H.HAPI_BOTTLENECK, cin=cin, width=w, cout=4 * w, stride=1)]
    r = Runner(layers, H.HAPI_BF16, params, (cin, hw, hw))
    x = synth.small_ints(306, (batch, cin, hw, hw), -2, 2)
    xd, xv = images_for(H.HAPI_BF16, x)
    H.hapi_stats_enable(True)
    got = r.extract_np(xd, 2)
    st = {s["name"]: s for s in H.hapi_stats_collect()}
    H.hapi_stats_enable(False)
    assert st["conv_bf16"]["launches"] == 2     # c1, then 3x3 + expansion together
    h1 = bf16_round(np.maximum(L.conv2d(xv, w1, b1[1], 1, 0), 0))
    h2 = bf16_round(np.maximum(L.conv2d(h1, w2, b2[1], 1, 1), 0))
    ref = bf16_round(np.maximum(L.conv2d(h2, w3, b3[1], 1, 0) + xv, 0))
    print(f"fused bottleneck {hw}x{hw} batch {batch}: max |h2| {np.abs(h2).max():.0f}, "
          f"max |y| {np.abs(ref).max():.0f}", flush=True)
    assert np.array_equal(got, ref), np.abs(got - ref).max()
