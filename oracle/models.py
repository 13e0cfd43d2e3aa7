"""Oracle model definitions: the frozen feature extractors the paper splits.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper evaluates TorchVision image models (Evaluation, Methodology and
Table 2: AlexNet, ResNet18, ResNet50, DenseNet, Vgg11/19 and the TorchVision
Vision Transformer).  Blocks of block-structured networks count as one layer,
and split points fall only on block boundaries (Measurement study; Evaluation,
Methodology).  Layer numbering used here: layer k (1-based) is the k-th entry
of ``Model.layers``; ReLU is part of its producing layer and inference
batch-norm part of its convolution; split 0 is the input itself (Algorithm 1
ranges potential splits over [0, freeze index]; split 0 sends the raw input).

Parameters follow one canonical order per layer (the raw-weight layout):
  conv           weight [O, C, k, k], bias [O] if any, then BN gamma, beta,
                 running mean, running var [O] each if any
  basic block    conv1, bn1, conv2, bn2, [shortcut conv 1x1, shortcut bn]
  bottleneck     conv1 1x1, bn1, conv2 3x3, bn2, conv3 1x1, bn3, [shortcut]
  patch embed    weight [D, C, p, p], bias [D]
  tokens         class token [D], position embedding [T, D]
  encoder block  ln1 gamma, beta; in-projection weight [3D, D], bias [3D];
                 out-projection weight [D, D], bias [D]; ln2 gamma, beta;
                 fc1 weight [F, D], bias [F]; fc2 weight [D, F], bias [D]
  layernorm      gamma [D], beta [D]
  dense block    per dense layer l (input channels c = cin + l * growth):
                 bn1 gamma, beta, mean, var [c]; conv1 weight [bottleneck, c, 1, 1];
                 bn2 gamma, beta, mean, var [bottleneck]; conv2 weight [growth, bottleneck, 3, 3]
Convolutions in blocks carry no bias; batch-norm eps is 1e-5, layernorm eps 1e-6.
"""
from __future__ import annotations

import numpy as np

from . import layers as L

BN_EPS = 1e-5
LN_EPS = 1e-6


def _bn_manifest(c):
    return [((c,), "bn_gamma"), ((c,), "bn_beta"), ((c,), "bn_mean"), ((c,), "bn_var")]


class Conv:
    """Convolution [+ bias] [+ inference BN] [+ ReLU] as one layer."""

    def __init__(self, cin, cout, k, stride=1, pad=0, bias=False, bn=False, relu=True,
                 weight_kind="he"):
        self.cin, self.cout, self.k, self.stride, self.pad = cin, cout, k, stride, pad
        self.bias, self.bn, self.relu, self.weight_kind = bias, bn, relu, weight_kind

    def manifest(self):
        m = [((self.cout, self.cin, self.k, self.k), self.weight_kind)]
        if self.bias:
            m.append(((self.cout,), "bias"))
        if self.bn:
            m += _bn_manifest(self.cout)
        return m

    def out_shape(self, s):
        c, h, w = s
        assert c == self.cin, (c, self.cin)
        return (self.cout, (h + 2 * self.pad - self.k) // self.stride + 1,
                (w + 2 * self.pad - self.k) // self.stride + 1)

    def forward(self, x, p, relu=None):
        w = next(p)
        b = next(p) if self.bias else None
        y = L.conv2d(x, w, b, self.stride, self.pad)
        if self.bn:
            g, be, mu, var = next(p), next(p), next(p), next(p)
            y = L.batchnorm(y, g, be, mu, var, BN_EPS)
        if self.relu if relu is None else relu:
            y = L.relu(y)
        return y


class MaxPool:
    def __init__(self, k, stride, pad=0):
        self.k, self.stride, self.pad = k, stride, pad

    def manifest(self):
        return []

    def out_shape(self, s):
        c, h, w = s
        return (c, (h + 2 * self.pad - self.k) // self.stride + 1,
                (w + 2 * self.pad - self.k) // self.stride + 1)

    def forward(self, x, p):
        return L.maxpool2d(x, self.k, self.stride, self.pad)


class AvgPool:
    """k x k window mean with stride, no padding (DenseNet transition pooling)."""

    def __init__(self, k, stride):
        self.k, self.stride = k, stride

    def manifest(self):
        return []

    def out_shape(self, s):
        c, h, w = s
        return (c, (h - self.k) // self.stride + 1, (w - self.k) // self.stride + 1)

    def forward(self, x, p):
        return L.avgpool2d(x, self.k, self.stride)


class PreActConv:
    """Pre-activation convolution y = conv(ReLU(BN(x))), no bias: the DenseNet
    transition's batch-norm and ReLU act on its input."""

    def __init__(self, cin, cout, k=1, stride=1, pad=0):
        self.cin, self.cout, self.k, self.stride, self.pad = cin, cout, k, stride, pad

    def manifest(self):
        return _bn_manifest(self.cin) + [((self.cout, self.cin, self.k, self.k), "he")]

    def out_shape(self, s):
        c, h, w = s
        assert c == self.cin
        return (self.cout, (h + 2 * self.pad - self.k) // self.stride + 1,
                (w + 2 * self.pad - self.k) // self.stride + 1)

    def forward(self, x, p):
        g, b, m, v = next(p), next(p), next(p), next(p)
        w = next(p)
        h = L.relu(L.batchnorm(x, g, b, m, v, BN_EPS))
        return L.conv2d(h, w, None, self.stride, self.pad)


class BatchNorm:
    """Inference batch-norm over channels, optionally followed by ReLU."""

    def __init__(self, c, relu=False):
        self.c, self.relu = c, relu

    def manifest(self):
        return _bn_manifest(self.c)

    def out_shape(self, s):
        assert s[0] == self.c
        return s

    def forward(self, x, p):
        g, b, m, v = next(p), next(p), next(p), next(p)
        y = L.batchnorm(x, g, b, m, v, BN_EPS)
        return L.relu(y) if self.relu else y


class GlobalAvgPool:
    def manifest(self):
        return []

    def out_shape(self, s):
        return (s[0], 1, 1)

    def forward(self, x, p):
        return L.avgpool_global(x)


class BasicBlock:
    """out = ReLU(bn2(conv2(ReLU(bn1(conv1(x))))) + shortcut(x)); stride on conv1."""

    def __init__(self, cin, cout, stride):
        self.c1 = Conv(cin, cout, 3, stride, 1, bn=True, relu=True)
        self.c2 = Conv(cout, cout, 3, 1, 1, bn=True, relu=False)
        self.sc = Conv(cin, cout, 1, stride, 0, bn=True, relu=False) \
            if (stride != 1 or cin != cout) else None

    def manifest(self):
        return self.c1.manifest() + self.c2.manifest() + (self.sc.manifest() if self.sc else [])

    def out_shape(self, s):
        return self.c2.out_shape(self.c1.out_shape(s))

    def forward(self, x, p):
        y = self.c2.forward(self.c1.forward(x, p), p)
        r = self.sc.forward(x, p) if self.sc else x
        return L.relu(L.add(y, r))


class Bottleneck:
    """out = ReLU(c3(c2(c1(x))) + shortcut(x)); 1x1 -> 3x3 (stride here) -> 1x1 x4."""

    def __init__(self, cin, width, stride):
        cout = 4 * width
        self.c1 = Conv(cin, width, 1, 1, 0, bn=True, relu=True)
        self.c2 = Conv(width, width, 3, stride, 1, bn=True, relu=True)
        self.c3 = Conv(width, cout, 1, 1, 0, bn=True, relu=False)
        self.sc = Conv(cin, cout, 1, stride, 0, bn=True, relu=False) \
            if (stride != 1 or cin != cout) else None

    def manifest(self):
        return (self.c1.manifest() + self.c2.manifest() + self.c3.manifest()
                + (self.sc.manifest() if self.sc else []))

    def out_shape(self, s):
        return self.c3.out_shape(self.c2.out_shape(self.c1.out_shape(s)))

    def forward(self, x, p):
        y = self.c3.forward(self.c2.forward(self.c1.forward(x, p), p), p)
        r = self.sc.forward(x, p) if self.sc else x
        return L.relu(L.add(y, r))


class DenseBlock:
    """DenseNet dense block: each layer appends growth channels computed from
    all channels so far, x <- concat(x, conv3x3(ReLU(BN2(conv1x1(ReLU(BN1(x))))))),
    with pre-activation batch-norm (BN1 acts on the concatenated input)."""

    def __init__(self, cin, n_layers, growth, bottleneck):
        self.cin, self.n, self.growth, self.bottleneck = cin, n_layers, growth, bottleneck

    def manifest(self):
        m = []
        for l in range(self.n):
            c = self.cin + l * self.growth
            m += _bn_manifest(c) + [((self.bottleneck, c, 1, 1), "he")]
            m += _bn_manifest(self.bottleneck) + [((self.growth, self.bottleneck, 3, 3), "he")]
        return m

    def out_shape(self, s):
        c, h, w = s
        assert c == self.cin
        return (self.cin + self.n * self.growth, h, w)

    def forward(self, x, p):
        feats = np.asarray(x, np.float64)
        for _ in range(self.n):
            g1, b1, m1, v1 = next(p), next(p), next(p), next(p)
            w1 = next(p)
            g2, b2, m2, v2 = next(p), next(p), next(p), next(p)
            w2 = next(p)
            h = L.relu(L.batchnorm(feats, g1, b1, m1, v1, BN_EPS))
            t = L.relu(L.batchnorm(L.conv2d(h, w1, None, 1, 0), g2, b2, m2, v2, BN_EPS))
            new = L.conv2d(t, w2, None, 1, 1)
            feats = np.concatenate([feats, new], axis=1)
        return feats


class PatchEmbed:
    """Non-overlapping p x p patches projected to D channels (a stride-p convolution)."""

    def __init__(self, cin, dim, patch):
        self.conv = Conv(cin, dim, patch, patch, 0, bias=True, relu=False, weight_kind="tn02")

    def manifest(self):
        w, b = self.conv.manifest()
        return [w, (b[0], "tn02")]

    def out_shape(self, s):
        return self.conv.out_shape(s)

    def forward(self, x, p):
        return self.conv.forward(x, p)


class Tokens:
    """[N, D, h, w] -> [N, 1 + h*w, D]: patch t = row*w + col becomes token 1 + t,
    a learned class token is token 0, and the position embedding is added."""

    def __init__(self, dim, n_tokens):
        self.dim, self.n_tokens = dim, n_tokens

    def manifest(self):
        return [((self.dim,), "tn02"), ((self.n_tokens, self.dim), "tn02")]

    def out_shape(self, s):
        d, h, w = s
        assert d == self.dim and 1 + h * w == self.n_tokens
        return (self.n_tokens, self.dim)

    def forward(self, x, p):
        cls, pos = next(p), next(p)
        N, D, h, w = x.shape
        patches = np.transpose(x.reshape(N, D, h * w), (0, 2, 1))
        clsrow = np.broadcast_to(np.asarray(cls, np.float64).reshape(1, 1, D), (N, 1, D))
        seq = np.concatenate([clsrow, patches], axis=1)
        return L.add(seq, np.broadcast_to(np.asarray(pos, np.float64)[None], seq.shape))


class EncoderBlock:
    """Pre-norm transformer encoder block:
    x = x + out_proj(MHA(LN1(x)));  x = x + fc2(GELU(fc1(LN2(x))))."""

    def __init__(self, dim, heads, mlp):
        self.dim, self.heads, self.mlp = dim, heads, mlp

    def manifest(self):
        D, F = self.dim, self.mlp
        return [((D,), "ln_gamma"), ((D,), "ln_beta"),
                ((3 * D, D), "tn02"), ((3 * D,), "tn02"),
                ((D, D), "tn02"), ((D,), "tn02"),
                ((D,), "ln_gamma"), ((D,), "ln_beta"),
                ((F, D), "tn02"), ((F,), "tn02"),
                ((D, F), "tn02"), ((D,), "tn02")]

    def out_shape(self, s):
        return s

    def branches(self, x, p):
        """Returns (attention-branch output, MLP-branch output, block output)."""
        g1, b1, wi, bi, wo, bo, g2, b2, w1, c1, w2, c2 = (next(p) for _ in range(12))
        h = L.layernorm(x, g1, b1, LN_EPS)
        a = L.linear(L.attention(L.linear(h, wi, bi), self.heads), wo, bo)
        x1 = L.add(x, a)
        m = L.linear(L.gelu(L.linear(L.layernorm(x1, g2, b2, LN_EPS), w1, c1)), w2, c2)
        return a, m, L.add(x1, m)

    def forward(self, x, p):
        return self.branches(x, p)[2]


class LayerNorm:
    def __init__(self, dim):
        self.dim = dim

    def manifest(self):
        return [((self.dim,), "ln_gamma"), ((self.dim,), "ln_beta")]

    def out_shape(self, s):
        return s

    def forward(self, x, p):
        g, b = next(p), next(p)
        return L.layernorm(x, g, b, LN_EPS)


class Model:
    def __init__(self, name, layers, in_shape=(3, 224, 224)):
        self.name, self.layers, self.in_shape = name, layers, tuple(in_shape)

    @property
    def n_layers(self):
        return len(self.layers)

    def manifest(self):
        m = []
        for layer in self.layers:
            m += layer.manifest()
        return m

    def param_counts(self):
        """Number of parameter tensors of each layer, in order."""
        return [len(layer.manifest()) for layer in self.layers]

    def shapes(self):
        """Per-image output shape of every layer; index 0 is the input."""
        s = [self.in_shape]
        for layer in self.layers:
            s.append(layer.out_shape(s[-1]))
        return s

    def out_elems(self):
        return [int(np.prod(s)) for s in self.shapes()]

    def forward(self, params, x, split, collect=False):
        """Run layers 1..split on x [N, C, H, W]; returns the split activation
        (NCHW for convolutional layers, [N, T, D] for token layers), or the list
        of all boundary activations 0..split when ``collect``."""
        if not 0 <= split <= self.n_layers:
            raise ValueError(f"split {split} outside [0, {self.n_layers}]")
        counts = self.param_counts()
        start = sum(counts[:split])
        p = iter(params[:start])
        y = np.asarray(x, np.float64)
        outs = [y]
        for layer in self.layers[:split]:
            y = layer.forward(y, p)
            if collect:
                outs.append(y)
        return outs if collect else y

    def forward_range(self, params, x, start, end):
        """Run layers start+1..end on x, the layer-``start`` activation in the
        layout ``forward`` returns (System implementation: the forward pass
        between arbitrary layers; the compute tier resumes from the split)."""
        if not 0 <= start <= end <= self.n_layers:
            raise ValueError(f"range {start}..{end} outside [0, {self.n_layers}]")
        counts = self.param_counts()
        p = iter(params[sum(counts[:start]):sum(counts[:end])])
        y = np.asarray(x, np.float64)
        for layer in self.layers[start:end]:
            y = layer.forward(y, p)
        return y


def alexnet():
    """AlexNet feature layers: conv11/4(64)-pool-conv5(192)-pool-conv3(384)-conv3(256)-conv3(256)-pool."""
    return Model("alexnet", [
        Conv(3, 64, 11, 4, 2, bias=True), MaxPool(3, 2),
        Conv(64, 192, 5, 1, 2, bias=True), MaxPool(3, 2),
        Conv(192, 384, 3, 1, 1, bias=True), Conv(384, 256, 3, 1, 1, bias=True),
        Conv(256, 256, 3, 1, 1, bias=True), MaxPool(3, 2)])


def vgg16():
    """VGG-16 features: 13 conv3x3 (+bias, ReLU) and 5 maxpool 2x2/2."""
    cfg = [64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M",
           512, 512, 512, "M"]
    layers, c = [], 3
    for v in cfg:
        if v == "M":
            layers.append(MaxPool(2, 2))
        else:
            layers.append(Conv(c, v, 3, 1, 1, bias=True))
            c = v
    return Model("vgg16", layers)


def _resnet(name, block, counts, in_hw=224):
    layers = [Conv(3, 64, 7, 2, 3, bn=True), MaxPool(3, 2, 1)]
    c = 64
    for stage, (n, width) in enumerate(zip(counts, (64, 128, 256, 512))):
        for i in range(n):
            stride = 2 if (stage > 0 and i == 0) else 1
            if block is BasicBlock:
                layers.append(BasicBlock(c, width, stride))
                c = width
            else:
                layers.append(Bottleneck(c, width, stride))
                c = 4 * width
    layers.append(GlobalAvgPool())
    return Model(name, layers, (3, in_hw, in_hw))


def resnet18(in_hw=224):
    return _resnet("resnet18", BasicBlock, (2, 2, 2, 2), in_hw)


def resnet50(in_hw=224):
    return _resnet("resnet50", Bottleneck, (3, 4, 6, 3), in_hw)


def dense_block_net(in_hw=224, n_layers=4, growth=32, bottleneck=128):
    """DenseNet-121 stem (conv 7x7/2 + BN + ReLU, maxpool 3x3/2) and one dense
    block of n_layers at 56 x 56."""
    return Model("densenet_block", [Conv(3, 64, 7, 2, 3, bn=True), MaxPool(3, 2, 1),
                                    DenseBlock(64, n_layers, growth, bottleneck)], (3, in_hw, in_hw))


def densenet121(in_hw=224, growth=32, bottleneck=128, blocks=(6, 12, 24, 16)):
    """DenseNet-121 features (TorchVision layout): conv 7x7/2 + BN + ReLU,
    maxpool 3x3/2, four dense blocks; between blocks a transition of BN, ReLU,
    1x1 convolution halving the channels and 2x2/2 average pooling (here two
    layers: the pre-activation convolution and the pooling); a closing BN."""
    layers = [Conv(3, 64, 7, 2, 3, bn=True), MaxPool(3, 2, 1)]
    c = 64
    for i, n in enumerate(blocks):
        layers.append(DenseBlock(c, n, growth, bottleneck))
        c += n * growth
        if i + 1 < len(blocks):
            layers += [PreActConv(c, c // 2), AvgPool(2, 2)]
            c //= 2
    layers.append(BatchNorm(c))
    return Model("densenet121", layers, (3, in_hw, in_hw))


def vit(image=224, patch=16, dim=768, heads=12, mlp=3072, depth=12, name="vit_b16"):
    """Vision Transformer encoder: patch embed, tokens, ``depth`` blocks, final LN."""
    g = image // patch
    layers = [PatchEmbed(3, dim, patch), Tokens(dim, 1 + g * g)]
    layers += [EncoderBlock(dim, heads, mlp) for _ in range(depth)]
    layers.append(LayerNorm(dim))
    return Model(name, layers, (3, image, image))


def vit_b16():
    return vit()


# The five benchmark workloads: (model factory, dtype, batch, split layer).
WORKLOADS = {
    0: ("alexnet", "f32", 4, 8),
    1: ("resnet18", "bf16", 64, 8),
    2: ("vgg16", "bf16", 128, 18),
    3: ("resnet50", "bf16", 256, 18),
    4: ("vit_b16", "bf16", 128, 10),
}

FACTORIES = {"alexnet": alexnet, "resnet18": resnet18, "resnet50": resnet50,
             "vgg16": vgg16, "vit_b16": vit_b16, "densenet_block": dense_block_net,
             "densenet121": densenet121}


def build(name):
    return FACTORIES[name]()
