"""Layer descriptors of the frozen feature extractors the paper splits.

The paper evaluates TorchVision image models (Evaluation, Methodology and
Table 2).  Each factory returns the ``hapi_layer`` list (as dicts) in the
library's block-granular numbering: a residual / encoder block is one layer,
ReLU and inference batch-norm belong to their convolution.  ``raw_manifest``
lists the raw float32 tensors the library expects, in order, with the
distribution each synthetic stand-in for pre-trained weights is drawn from.
"""
from __future__ import annotations

from .binding import (HAPI_AVGPOOL, HAPI_BASIC_BLOCK, HAPI_BATCHNORM, HAPI_BF16, HAPI_BOTTLENECK,
                      HAPI_CONV, HAPI_DENSE_BLOCK, HAPI_F32, HAPI_LAYERNORM, HAPI_MAXPOOL,
                      HAPI_PATCH_EMBED, HAPI_PREACT_CONV, HAPI_TOKENS, HAPI_VIT_BLOCK)


def conv(cin, cout, k, stride=1, pad=0, bias=False, bn=False, relu=True):
    return dict(kind=HAPI_CONV, cin=cin, cout=cout, k=k, stride=stride, pad=pad,
                relu=int(relu), has_bias=int(bias), has_bn=int(bn))


def maxpool(k, stride, pad=0):
    return dict(kind=HAPI_MAXPOOL, k=k, stride=stride, pad=pad)


def avgpool(k=0, stride=0):
    return dict(kind=HAPI_AVGPOOL, k=k, stride=stride)


def alexnet():
    return [conv(3, 64, 11, 4, 2, bias=True), maxpool(3, 2),
            conv(64, 192, 5, 1, 2, bias=True), maxpool(3, 2),
            conv(192, 384, 3, 1, 1, bias=True), conv(384, 256, 3, 1, 1, bias=True),
            conv(256, 256, 3, 1, 1, bias=True), maxpool(3, 2)]


def vgg16():
    layers, c = [], 3
    for v in (64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M",
              512, 512, 512, "M"):
        if v == "M":
            layers.append(maxpool(2, 2))
        else:
            layers.append(conv(c, v, 3, 1, 1, bias=True))
            c = v
    return layers


def _resnet(bottleneck, counts):
    layers = [conv(3, 64, 7, 2, 3, bn=True), maxpool(3, 2, 1)]
    c = 64
    for stage, (n, width) in enumerate(zip(counts, (64, 128, 256, 512))):
        for i in range(n):
            stride = 2 if stage > 0 and i == 0 else 1
            if bottleneck:
                layers.append(dict(kind=HAPI_BOTTLENECK, cin=c, width=width, cout=4 * width,
                                   stride=stride))
                c = 4 * width
            else:
                layers.append(dict(kind=HAPI_BASIC_BLOCK, cin=c, cout=width, stride=stride))
                c = width
    layers.append(avgpool())
    return layers


def resnet18():
    return _resnet(False, (2, 2, 2, 2))


def resnet50():
    return _resnet(True, (3, 4, 6, 3))


def dense_block(cin, n_layers, growth=32, bottleneck=128):
    return dict(kind=HAPI_DENSE_BLOCK, cin=cin, cout=cin + n_layers * growth, width=growth,
                mlp_dim=bottleneck)


def dense_block_net(n_layers=4, growth=32, bottleneck=128):
    """DenseNet-121 stem and one dense block at 56 x 56 (channel concatenation)."""
    return [conv(3, 64, 7, 2, 3, bn=True), maxpool(3, 2, 1),
            dense_block(64, n_layers, growth, bottleneck)]


def preact_conv(cin, cout, k=1, stride=1, pad=0):
    return dict(kind=HAPI_PREACT_CONV, cin=cin, cout=cout, k=k, stride=stride, pad=pad)


def batchnorm(c, relu=False):
    return dict(kind=HAPI_BATCHNORM, cout=c, relu=int(relu))


def densenet121(growth=32, bottleneck=128, blocks=(6, 12, 24, 16)):
    """DenseNet-121 features: stem and pooling, four dense blocks with a
    transition (pre-activation 1x1 convolution halving the channels, then 2x2
    average pooling) between them, and the closing batch-norm.  13 layers;
    the paper's freeze layer (after the fourth dense block) is layer 12."""
    layers = [conv(3, 64, 7, 2, 3, bn=True), maxpool(3, 2, 1)]
    c = 64
    for i, n in enumerate(blocks):
        layers.append(dense_block(c, n, growth, bottleneck))
        c += n * growth
        if i + 1 < len(blocks):
            layers += [preact_conv(c, c // 2), avgpool(2, 2)]
            c //= 2
    layers.append(batchnorm(c))
    return layers


def vit(image=224, patch=16, dim=768, heads=12, mlp=3072, depth=12):
    layers = [dict(kind=HAPI_PATCH_EMBED, cin=3, cout=dim, k=patch, stride=patch),
              dict(kind=HAPI_TOKENS, cout=dim)]
    layers += [dict(kind=HAPI_VIT_BLOCK, cout=dim, heads=heads, mlp_dim=mlp)
               for _ in range(depth)]
    layers.append(dict(kind=HAPI_LAYERNORM, cout=dim))
    return layers


def vit_b16():
    return vit()


FACTORIES = {"alexnet": alexnet, "resnet18": resnet18, "resnet50": resnet50,
             "vgg16": vgg16, "vit_b16": vit_b16, "densenet_block": dense_block_net,
             "densenet121": densenet121}

# The five benchmark workloads.  ``seed`` selects the synthetic input stream.
WORKLOADS = {
    "alexnet_f32_b4": dict(seed=0, model="alexnet", dtype=HAPI_F32, batch=4, split=8),
    "resnet18_bf16_b64": dict(seed=1, model="resnet18", dtype=HAPI_BF16, batch=64, split=8),
    "vgg16_bf16_b128": dict(seed=2, model="vgg16", dtype=HAPI_BF16, batch=128, split=18),
    "resnet50_bf16_b256": dict(seed=3, model="resnet50", dtype=HAPI_BF16, batch=256, split=18),
    "vit_b16_bf16_b128": dict(seed=4, model="vit_b16", dtype=HAPI_BF16, batch=128, split=10),
    # synthetic 4-layer dense block (growth 32, 56 x 56) for the channel-concat path
    "densenet_block_bf16_b64": dict(seed=5, model="densenet_block", dtype=HAPI_BF16, batch=64,
                                    split=3),
    # DenseNet-121 to its freeze layer (after the fourth dense block)
    "densenet121_bf16_b256": dict(seed=6, model="densenet121", dtype=HAPI_BF16, batch=256,
                                  split=12),
}


def _bn(c):
    return [((c,), "bn_gamma"), ((c,), "bn_beta"), ((c,), "bn_mean"), ((c,), "bn_var")]


def raw_manifest(layers, in_shape=(3, 224, 224)):
    """[(shape, kind), ...] of the raw float32 weights, in the library's order."""
    m = []
    c, h, w = in_shape
    t = None
    for L in layers:
        kind = L["kind"]
        if kind == HAPI_CONV:
            m.append(((L["cout"], L["cin"], L["k"], L["k"]), "he"))
            if L.get("has_bias"):
                m.append(((L["cout"],), "bias"))
            if L.get("has_bn"):
                m += _bn(L["cout"])
            k, s, p = L["k"], L.get("stride", 1), L.get("pad", 0)
            c, h, w = L["cout"], (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
        elif kind in (HAPI_MAXPOOL, HAPI_AVGPOOL):
            k, s, p = L.get("k", 0), L.get("stride", 1), L.get("pad", 0)
            if k == 0:
                h = w = 1
            else:
                h, w = (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
        elif kind in (HAPI_BASIC_BLOCK, HAPI_BOTTLENECK):
            cin, s = L["cin"], L["stride"]
            if kind == HAPI_BASIC_BLOCK:
                cout = L["cout"]
                m += [((cout, cin, 3, 3), "he")] + _bn(cout) + [((cout, cout, 3, 3), "he")] + _bn(cout)
            else:
                wd = L["width"]
                cout = 4 * wd
                m += ([((wd, cin, 1, 1), "he")] + _bn(wd) + [((wd, wd, 3, 3), "he")] + _bn(wd)
                      + [((cout, wd, 1, 1), "he")] + _bn(cout))
            if s != 1 or cin != cout:
                m += [((cout, cin, 1, 1), "he")] + _bn(cout)
            c, h, w = cout, (h + 2 - 3) // s + 1, (w + 2 - 3) // s + 1
        elif kind == HAPI_PATCH_EMBED:
            D, p = L["cout"], L["k"]
            m += [((D, L["cin"], p, p), "tn02"), ((D,), "tn02")]
            c, h, w = D, h // p, w // p
        elif kind == HAPI_TOKENS:
            D = L["cout"]
            t = 1 + h * w
            m += [((D,), "tn02"), ((t, D), "tn02")]
        elif kind == HAPI_VIT_BLOCK:
            D, F = L["cout"], L["mlp_dim"]
            m += [((D,), "ln_gamma"), ((D,), "ln_beta"), ((3 * D, D), "tn02"), ((3 * D,), "tn02"),
                  ((D, D), "tn02"), ((D,), "tn02"), ((D,), "ln_gamma"), ((D,), "ln_beta"),
                  ((F, D), "tn02"), ((F,), "tn02"), ((D, F), "tn02"), ((D,), "tn02")]
        elif kind == HAPI_LAYERNORM:
            m += [((L["cout"],), "ln_gamma"), ((L["cout"],), "ln_beta")]
        elif kind == HAPI_PREACT_CONV:
            m += _bn(L["cin"]) + [((L["cout"], L["cin"], L["k"], L["k"]), "he")]
            k, s, p = L["k"], L.get("stride", 1), L.get("pad", 0)
            c, h, w = L["cout"], (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
        elif kind == HAPI_BATCHNORM:
            m += _bn(L["cout"])
        elif kind == HAPI_DENSE_BLOCK:
            g, bt = L["width"], L["mlp_dim"]
            for ch in range(L["cin"], L["cout"], g):
                m += _bn(ch) + [((bt, ch, 1, 1), "he")] + _bn(bt) + [((g, bt, 3, 3), "he")]
            c = L["cout"]
        else:
            raise ValueError(f"unknown layer kind {kind}")
    return m
