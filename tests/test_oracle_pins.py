"""Pins of the CPU oracle against things other than itself.

Each test checks an oracle routine against a closed form, an exact-integer
brute force, an independent library implementation (torch / scipy / numpy in
float64, or the HF ``transformers`` ResNet and ViT modules), a special case
with a known answer, or a fact the paper prints.  None retypes the oracle's
own formula.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import layers as L
from oracle import models as M

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
torch.set_num_threads(min(8, os.cpu_count() or 1))


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float64))


# ---------------------------------------------------------------- convolution

@pytest.mark.parametrize("k,s,p", [(1, 1, 0), (2, 2, 0), (3, 1, 1), (3, 2, 1), (5, 1, 2),
                                   (7, 2, 3), (5, 3, 0), (3, 4, 3), (11, 4, 2)])
def test_conv_small_integers_exact_vs_torch(k, s, p):
    # Small-integer operands: every partial sum is an integer far below 2^53,
    # so any summation order gives the same float64 result bit for bit.
    H = W = max(k, 9) + 2
    x = synth.small_ints(10 + k + s, (2, 4, H, W))
    w = synth.small_ints(20 + k + s, (3, 4, k, k))
    b = synth.small_ints(30 + k, (3,))
    y = L.conv2d(x, w, b, s, p)
    yt = F.conv2d(_t(x), _t(w), _t(b), stride=s, padding=p).numpy()
    assert y.shape == yt.shape
    assert np.array_equal(y, yt)


def test_conv_matches_scipy_correlate():
    from scipy.signal import correlate2d
    rng = np.random.default_rng(1)
    x = rng.standard_normal((1, 3, 12, 10))
    w = rng.standard_normal((2, 3, 5, 5))
    y = L.conv2d(x, w, None, 1, 2)
    xp = np.pad(x, ((0, 0), (0, 0), (2, 2), (2, 2)))
    for o in range(2):
        ref = sum(correlate2d(xp[0, c], w[o, c], mode="valid") for c in range(3))
        np.testing.assert_allclose(y[0, o], ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("k", [1, 3, 5, 7])
def test_conv_identity_kernel_exact(k):
    x = np.random.default_rng(k).standard_normal((2, 5, 9, 8))
    w = np.zeros((5, 5, k, k))
    for c in range(5):
        w[c, c, k // 2, k // 2] = 1.0
    assert np.array_equal(L.conv2d(x, w, None, 1, k // 2), x)
    # strided identity picks every s-th pixel
    assert np.array_equal(L.conv2d(x, w, None, 2, k // 2), x[:, :, ::2, ::2])


def test_conv1x1_is_matmul():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 16, 7, 5))
    w = rng.standard_normal((24, 16, 1, 1))
    b = rng.standard_normal(24)
    y = L.conv2d(x, w, b)
    ref = np.einsum("nchw,oc->nohw", x, w[:, :, 0, 0]) + b[None, :, None, None]
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_patch_embed_is_matmul():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 3, 32, 48))
    w = rng.standard_normal((10, 3, 16, 16))
    y = L.conv2d(x, w, None, 16, 0)
    patches = x.reshape(2, 3, 2, 16, 3, 16).transpose(0, 2, 4, 1, 3, 5).reshape(2, 6, 768)
    ref = (patches @ w.reshape(10, 768).T).reshape(2, 2, 3, 10).transpose(0, 3, 1, 2)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_conv_random_vs_torch_float64():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((2, 6, 15, 13))
    w = rng.standard_normal((5, 6, 3, 3))
    b = rng.standard_normal(5)
    np.testing.assert_allclose(L.conv2d(x, w, b, 2, 1),
                               F.conv2d(_t(x), _t(w), _t(b), stride=2, padding=1).numpy(),
                               rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------- normalisation

def test_batchnorm_identity_params_exact():
    x = np.random.default_rng(5).standard_normal((2, 4, 3, 3))
    c = 4
    y = L.batchnorm(x, np.ones(c), np.zeros(c), np.zeros(c), np.full(c, 1.0 - 1e-5), 1e-5)
    np.testing.assert_allclose(y, x, rtol=0, atol=1e-15)


def test_batchnorm_vs_torch():
    rng = np.random.default_rng(6)
    x = rng.standard_normal((2, 4, 5, 5))
    g, b, mu, var = (rng.uniform(0.5, 1.5, 4), rng.uniform(-.1, .1, 4),
                     rng.uniform(-.1, .1, 4), rng.uniform(0.5, 1.5, 4))
    ref = F.batch_norm(_t(x), _t(mu), _t(var), _t(g), _t(b), training=False, eps=1e-5).numpy()
    np.testing.assert_allclose(L.batchnorm(x, g, b, mu, var), ref, rtol=1e-12, atol=1e-12)


def test_layernorm_constant_row_gives_beta_and_vs_torch():
    beta = np.arange(8.0)
    y = L.layernorm(np.full((3, 8), 2.5), np.full(8, 3.0), beta)
    np.testing.assert_allclose(y, np.broadcast_to(beta, (3, 8)), atol=1e-12)
    x = np.random.default_rng(7).standard_normal((5, 768)) * 3 + 1
    g, b = np.random.default_rng(8).standard_normal((2, 768))
    ref = F.layer_norm(_t(x), (768,), _t(g), _t(b), eps=1e-6).numpy()
    np.testing.assert_allclose(L.layernorm(x, g, b, 1e-6), ref, rtol=1e-10, atol=1e-10)
    z = L.layernorm(x, np.ones(768), np.zeros(768), 1e-6)
    np.testing.assert_allclose(z.mean(-1), 0, atol=1e-12)
    np.testing.assert_allclose(z.var(-1), 1, atol=1e-5)


def test_gelu_vs_math_erf():
    xs = np.linspace(-6, 6, 97)
    ref = np.array([0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in xs])
    np.testing.assert_allclose(L.gelu(xs), ref, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(L.gelu(xs), F.gelu(_t(xs)).numpy(), rtol=1e-12, atol=1e-15)


# ------------------------------------------------------------------- pooling

def test_pools_special_cases():
    x = np.random.default_rng(9).standard_normal((2, 3, 7, 6))
    assert np.array_equal(L.maxpool2d(x, 1, 1, 0), x)
    c = np.full((1, 2, 9, 9), 4.25)
    assert np.array_equal(L.maxpool2d(c, 3, 2, 1), np.full((1, 2, 5, 5), 4.25))
    assert np.array_equal(L.avgpool_global(c), np.full((1, 2, 1, 1), 4.25))
    xi = synth.small_ints(40, (2, 3, 13, 13), -50, 50)
    for k, s, p in [(3, 2, 0), (3, 2, 1), (2, 2, 0)]:
        assert np.array_equal(L.maxpool2d(xi, k, s, p),
                              F.max_pool2d(_t(xi), k, s, p).numpy())
    np.testing.assert_allclose(L.avgpool_global(x)[:, :, 0, 0], x.mean((2, 3)), rtol=1e-14)
    np.testing.assert_allclose(L.avgpool2d(x[:, :, :6, :6], 2, 2),
                               F.avg_pool2d(_t(x[:, :, :6, :6]), 2, 2).numpy(), rtol=1e-14)


# ----------------------------------------------------------------- attention

def test_attention_vs_torch_sdpa():
    rng = np.random.default_rng(10)
    N, T, D, H = 2, 13, 48, 4
    qkv = rng.standard_normal((N, T, 3 * D))
    y = L.attention(qkv, H)
    q, k, v = (_t(qkv[..., i * D:(i + 1) * D]).reshape(N, T, H, D // H).transpose(1, 2)
               for i in range(3))
    ref = F.scaled_dot_product_attention(q, k, v).transpose(1, 2).reshape(N, T, D).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_attention_zero_query_is_mean_of_values():
    rng = np.random.default_rng(11)
    N, T, D = 1, 9, 16
    qkv = rng.standard_normal((N, T, 3 * D))
    qkv[..., :D] = 0.0
    y = L.attention(qkv, 2)
    np.testing.assert_allclose(y, np.broadcast_to(qkv[..., 2 * D:].mean(1, keepdims=True), y.shape),
                               rtol=1e-13, atol=1e-14)


def test_linear_vs_numpy():
    rng = np.random.default_rng(12)
    x, w, b = rng.standard_normal((7, 33)), rng.standard_normal((5, 33)), rng.standard_normal(5)
    np.testing.assert_allclose(L.linear(x, w, b), x @ w.T + b, rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------------- blocks

def _zero_branch_params(model_layer):
    out = []
    for shape, kind in model_layer.manifest():
        if kind == "he":
            out.append(np.zeros(shape))
        elif kind in ("bn_beta", "bn_mean"):
            out.append(np.zeros(shape))
        else:
            out.append(synth.param(0, len(out) + 1, shape, kind))
    return out


@pytest.mark.parametrize("block", [M.BasicBlock(8, 8, 1), M.Bottleneck(16, 4, 1)])
def test_residual_block_with_zero_branch_is_relu(block):
    x = np.random.default_rng(13).standard_normal((2, block.c1.cin, 6, 6))
    y = block.forward(x, iter(_zero_branch_params(block)))
    assert np.array_equal(y, np.maximum(x, 0.0))


def test_encoder_block_with_zero_outputs_is_identity():
    blk = M.EncoderBlock(32, 4, 64)
    ps = synth.params(0, blk.manifest())
    for i in (4, 5, 10, 11):          # out-projection and fc2 weight/bias
        ps[i] = np.zeros_like(ps[i])
    x = np.random.default_rng(14).standard_normal((2, 5, 32))
    assert np.array_equal(blk.forward(x, iter(ps)), x)


# ----------------------------------------------- whole models vs HF modules

def _hf_resnet(kind):
    from transformers import ResNetConfig, ResNetModel
    if kind == "resnet18":
        cfg = ResNetConfig(layer_type="basic", depths=[2, 2, 2, 2],
                           hidden_sizes=[64, 128, 256, 512], embedding_size=64)
    else:
        cfg = ResNetConfig(layer_type="bottleneck", depths=[3, 4, 6, 3],
                           hidden_sizes=[256, 512, 1024, 2048], embedding_size=64)
    return ResNetModel(cfg).double().eval()


def _load_hf_resnet(hf, params):
    """Assign our canonical parameter list to the HF module, conv by conv."""
    convs = [hf.embedder.embedder]
    for stage in hf.encoder.stages:
        for layer in stage.layers:
            seq = list(layer.layer)
            convs += seq
            if hasattr(layer.shortcut, "convolution"):
                convs.append(layer.shortcut)
    it = iter(params)
    with torch.no_grad():
        for cl in convs:
            cl.convolution.weight.copy_(_t(next(it)))
            n = cl.normalization
            for t in (n.weight, n.bias, n.running_mean, n.running_var):
                t.copy_(_t(next(it)))
    assert next(it, None) is None


@pytest.mark.parametrize("name", ["resnet18", "resnet50"])
def test_resnet_oracle_vs_hf_transformers(name):
    model = M.build(name)
    params = synth.params(50, model.manifest())
    x = synth.images(50, 1, height=64, width=64).astype(np.float64)
    small = (M.resnet18 if name == "resnet18" else M.resnet50)(in_hw=64)
    outs = small.forward(params, x, small.n_layers, collect=True)
    hf = _hf_resnet(name)
    _load_hf_resnet(hf, params)
    with torch.no_grad():
        r = hf(_t(x), output_hidden_states=True)
    hs = r.hidden_states
    # hidden_states[0] = after stem + maxpool (our layer 2); then one per stage.
    ends = [2]
    depths = (2, 2, 2, 2) if name == "resnet18" else (3, 4, 6, 3)
    for d in depths:
        ends.append(ends[-1] + d)
    for h, e in zip(hs, ends):
        ref = h.numpy()
        np.testing.assert_allclose(outs[e], ref, rtol=1e-9, atol=1e-9 * np.abs(ref).max())
    np.testing.assert_allclose(outs[-1], r.pooler_output.numpy(), rtol=1e-9,
                               atol=1e-9 * np.abs(outs[-1]).max())


def test_vit_oracle_vs_hf_transformers():
    from transformers import ViTConfig, ViTModel
    D, H, Fm, depth, img = 64, 4, 128, 3, 48
    model = M.vit(image=img, patch=16, dim=D, heads=H, mlp=Fm, depth=depth, name="vit_small")
    params = synth.params(51, model.manifest())
    x = synth.images(51, 2, height=img, width=img).astype(np.float64)
    outs = model.forward(params, x, model.n_layers, collect=True)
    cfg = ViTConfig(hidden_size=D, num_hidden_layers=depth, num_attention_heads=H,
                    intermediate_size=Fm, image_size=img, patch_size=16, layer_norm_eps=1e-6,
                    hidden_act="gelu", qkv_bias=True, hidden_dropout_prob=0.0,
                    attention_probs_dropout_prob=0.0)
    hf = ViTModel(cfg, add_pooling_layer=False).double().eval()
    it = iter(params)
    with torch.no_grad():
        e = hf.embeddings
        e.patch_embeddings.projection.weight.copy_(_t(next(it)))
        e.patch_embeddings.projection.bias.copy_(_t(next(it)))
        e.cls_token.copy_(_t(next(it)).reshape(1, 1, D))
        e.position_embeddings.copy_(_t(next(it))[None])
        for lyr in hf.layers:
            g1, b1, wi, bi, wo, bo, g2, b2, w1, c1, w2, c2 = (next(it) for _ in range(12))
            lyr.layernorm_before.weight.copy_(_t(g1)); lyr.layernorm_before.bias.copy_(_t(b1))
            att = lyr.attention
            for j, lin in enumerate((att.q_proj, att.k_proj, att.v_proj)):
                lin.weight.copy_(_t(wi[j * D:(j + 1) * D])); lin.bias.copy_(_t(bi[j * D:(j + 1) * D]))
            att.o_proj.weight.copy_(_t(wo)); att.o_proj.bias.copy_(_t(bo))
            lyr.layernorm_after.weight.copy_(_t(g2)); lyr.layernorm_after.bias.copy_(_t(b2))
            lyr.mlp.fc1.weight.copy_(_t(w1)); lyr.mlp.fc1.bias.copy_(_t(c1))
            lyr.mlp.fc2.weight.copy_(_t(w2)); lyr.mlp.fc2.bias.copy_(_t(c2))
        hf.layernorm.weight.copy_(_t(next(it))); hf.layernorm.bias.copy_(_t(next(it)))
        r = hf(_t(x), output_hidden_states=True)
    # hidden_states[0] = embeddings (our layer 2); [i] = after block i (our 2 + i)
    for i, h in enumerate(r.hidden_states):
        np.testing.assert_allclose(outs[2 + i], h.numpy(), rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(outs[-1], r.last_hidden_state.numpy(), rtol=1e-9, atol=1e-10)


def _torch_sequential(layers_cfg, x, params):
    it = iter(params)
    y = _t(x)
    for kind, *a in layers_cfg:
        if kind == "C":
            k, s, p = a
            y = F.relu(F.conv2d(y, _t(next(it)), _t(next(it)), stride=s, padding=p))
        else:
            k, s = a
            y = F.max_pool2d(y, k, s)
    return y.numpy()


def test_alexnet_and_vgg_vs_torch_sequential():
    # AlexNet features, restated from the workload description as torch ops.
    alex = [("C", 11, 4, 2), ("M", 3, 2), ("C", 5, 1, 2), ("M", 3, 2), ("C", 3, 1, 1),
            ("C", 3, 1, 1), ("C", 3, 1, 1), ("M", 3, 2)]
    m = M.alexnet()
    ps = synth.params(52, m.manifest())
    x = synth.images(52, 1).astype(np.float64)
    np.testing.assert_allclose(m.forward(ps, x, 8), _torch_sequential(alex, x, ps), rtol=1e-9, atol=1e-9)
    vgg = []
    for v in [2, "M", 2, "M", 3, "M", 3, "M", 3, "M"]:
        vgg += [("M", 2, 2)] if v == "M" else [("C", 3, 1, 1)] * v
    m = M.vgg16()
    ps = synth.params(53, m.manifest())
    x = synth.images(53, 1, height=64, width=64).astype(np.float64)
    m.in_shape = (3, 64, 64)
    np.testing.assert_allclose(m.forward(ps, x, 18), _torch_sequential(vgg, x, ps), rtol=1e-9, atol=1e-9)


# ----------------------------------------------------- shapes and paper facts

# Per-image output shapes: closed form floor((H + 2p - k)/s) + 1 applied by hand
# to each layer of the workload descriptions.
EXPECTED_SHAPES = {
    "alexnet": [(3, 224, 224), (64, 55, 55), (64, 27, 27), (192, 27, 27), (192, 13, 13),
                (384, 13, 13), (256, 13, 13), (256, 13, 13), (256, 6, 6)],
    "resnet18": [(3, 224, 224), (64, 112, 112), (64, 56, 56)] + [(64, 56, 56)] * 2
    + [(128, 28, 28)] * 2 + [(256, 14, 14)] * 2 + [(512, 7, 7)] * 2 + [(512, 1, 1)],
    "resnet50": [(3, 224, 224), (64, 112, 112), (64, 56, 56)] + [(256, 56, 56)] * 3
    + [(512, 28, 28)] * 4 + [(1024, 14, 14)] * 6 + [(2048, 7, 7)] * 3 + [(2048, 1, 1)],
    "vgg16": [(3, 224, 224)] + [(64, 224, 224)] * 2 + [(64, 112, 112)] + [(128, 112, 112)] * 2
    + [(128, 56, 56)] + [(256, 56, 56)] * 3 + [(256, 28, 28)] + [(512, 28, 28)] * 3
    + [(512, 14, 14)] * 4 + [(512, 7, 7)],
    "vit_b16": [(3, 224, 224), (768, 14, 14)] + [(197, 768)] * 14,
}


@pytest.mark.parametrize("name", sorted(EXPECTED_SHAPES))
def test_layer_shapes_closed_form(name):
    assert M.build(name).shapes() == EXPECTED_SHAPES[name]


def test_paper_facts():
    facts = json.load(open(os.path.join(GOLDEN, "paper_facts.json")))
    t2 = facts["table2_layer_counts"]
    # Paper totals count stem conv, bn and relu separately and add the classifier;
    # ours fuse bn/relu into the stem and stop before the classifier.
    assert M.resnet18().n_layers + 2 + 1 == t2["ResNet18"]["total"]
    assert M.resnet50().n_layers + 2 + 1 == t2["ResNet50"]["total"]
    # AlexNet: 5 ReLUs counted separately in the features, then avgpool, flatten
    # and the 7 classifier modules.
    assert M.alexnet().n_layers + 5 + 1 + 1 + 7 == t2["AlexNet"]["total"]
    # Small early outputs: paper AlexNet layers 3 and 6 are our pools 2 and 4;
    # paper ResNet layer 4 is our maxpool 2 (ResNet50: 64x56x56 before 256x56x56).
    # Each is smaller than both neighbours.
    for name, ours in (("alexnet", (2, 4)), ("resnet50", (2,))):
        e = M.build(name).out_elems()
        for k in ours:
            assert e[k] < e[k + 1] and e[k] < e[k - 1]
    # DenseNet: stem conv, bn, relu and pool; four dense blocks; three
    # transitions of bn, relu, conv and pool; the closing bn; the classifier.
    # Ours: stem (bn, relu fused), pool, blocks, 2 layers per transition,
    # the closing bn; the paper's freeze layer 20 ends the fourth block.
    dn = M.densenet121()
    assert dn.n_layers + 2 + 3 * 2 + 1 == t2["DenseNet"]["total"]
    blocks = [i + 1 for i, layer in enumerate(dn.layers) if isinstance(layer, M.DenseBlock)]
    assert blocks[-1] + 2 + 3 * 2 == t2["DenseNet"]["freeze"]
    # @Min over layers 1..freeze of the Transformer is layer 1 (earliest on ties).
    e = M.vit_b16().out_elems()
    assert e[1] == e[0]                      # patch embedding output = input size
    assert int(np.argmin(e[1:])) + 1 == facts["transformer_min_split"]["layer"]


def test_batch_independence_of_oracle():
    m = M.resnet18(in_hw=64)
    ps = synth.params(54, m.manifest())
    x = synth.images(54, 3, height=64, width=64)
    whole = m.forward(ps, x, 8)
    for i in range(3):
        assert np.array_equal(m.forward(ps, x[i:i + 1], 8)[0], whole[i])


def test_split_zero_is_input():
    m = M.alexnet()
    x = synth.images(0, 2)
    assert np.array_equal(m.forward(synth.params(0, m.manifest()), x, 0), x.astype(np.float64))


@pytest.mark.parametrize("name", ["resnet18", "vit_small"])
def test_forward_range_composes_to_forward(name):
    # Resuming from any split reproduces the single pass exactly (same float64
    # operations in the same order); a wrong parameter offset breaks it.
    m = M.resnet18(in_hw=64) if name == "resnet18" else \
        M.vit(image=64, patch=16, dim=128, heads=2, mlp=256, depth=2, name="vit_small")
    ps = synth.params(56, m.manifest())
    x = synth.images(56, 2, height=64, width=64)
    outs = m.forward(ps, x, m.n_layers, collect=True)
    for s in range(m.n_layers + 1):
        for e in range(s, m.n_layers + 1):
            assert np.array_equal(m.forward_range(ps, outs[s], s, e), outs[e]), (s, e)
    with pytest.raises(ValueError):
        m.forward_range(ps, x, 2, 1)


# ----------------------------------------------------------- dense block

def _torch_dense_block(x, params, n, growth):
    """DenseNet dense layers restated with torch.nn.functional (float64)."""
    it = iter(params)
    feats = _t(x)
    for _ in range(n):
        g1, b1, m1, v1, w1, g2, b2, m2, v2, w2 = (_t(next(it)) for _ in range(10))
        h = F.relu(F.batch_norm(feats, m1, v1, g1, b1, training=False, eps=1e-5))
        t = F.relu(F.batch_norm(F.conv2d(h, w1), m2, v2, g2, b2, training=False, eps=1e-5))
        feats = torch.cat([feats, F.conv2d(t, w2, padding=1)], 1)
    return feats.numpy()


def test_dense_block_vs_torch_and_concat_prefix():
    blk = M.DenseBlock(16, 3, 8, 32)
    ps = synth.params(55, blk.manifest())
    x = np.random.default_rng(15).standard_normal((2, 16, 9, 9))
    y = blk.forward(x, iter(ps))
    assert y.shape == (2, 16 + 3 * 8, 9, 9)
    np.testing.assert_allclose(y, _torch_dense_block(x, ps, 3, 8), rtol=1e-10, atol=1e-10)
    # concatenation keeps the block input verbatim in the first channels
    assert np.array_equal(y[:, :16], x)


def test_dense_block_with_zero_growth_convs_appends_zeros():
    blk = M.DenseBlock(8, 2, 4, 16)
    ps = synth.params(56, blk.manifest())
    for i in (9, 19):          # conv2 weights of both layers
        ps[i] = np.zeros_like(ps[i])
    x = np.random.default_rng(16).standard_normal((1, 8, 5, 5))
    y = blk.forward(x, iter(ps))
    assert np.array_equal(y[:, :8], x) and not y[:, 8:].any()


def _torch_densenet121(x, params, blocks=(6, 12, 24, 16), growth=32):
    """DenseNet-121 features restated with torch.nn.functional (float64),
    returning every layer boundary the oracle exposes."""
    it = iter(params)
    nxt = lambda: _t(next(it))
    bn = lambda v, g, b, m, var: F.batch_norm(v, m, var, g, b, training=False, eps=1e-5)
    outs = [_t(x)]
    w = nxt(); g, b, m, v = nxt(), nxt(), nxt(), nxt()
    y = F.relu(bn(F.conv2d(outs[0], w, stride=2, padding=3), g, b, m, v))
    outs.append(y)
    outs.append(F.max_pool2d(y, 3, 2, 1))
    c = 64
    for i, n in enumerate(blocks):
        blk = list(next(it) for _ in range(10 * n))
        outs.append(_t(_torch_dense_block(outs[-1].numpy(), blk, n, growth)))
        c += n * growth
        if i + 1 < len(blocks):
            g, b, m, v = nxt(), nxt(), nxt(), nxt()
            w = nxt()
            outs.append(F.conv2d(F.relu(bn(outs[-1], g, b, m, v)), w))
            outs.append(F.avg_pool2d(outs[-1], 2, 2))
            c //= 2
    g, b, m, v = nxt(), nxt(), nxt(), nxt()
    outs.append(bn(outs[-1], g, b, m, v))
    return [o.numpy() for o in outs]


def test_densenet121_vs_torch_functional():
    m = M.densenet121(in_hw=64)
    ps = synth.params(57, m.manifest())
    x = synth.images(57, 2, height=64, width=64)
    ours = m.forward(ps, x, m.n_layers, collect=True)
    ref = _torch_densenet121(x, ps)
    assert len(ours) == len(ref) == 14
    for k, (a, r) in enumerate(zip(ours, ref)):
        assert a.shape == r.shape, k
        np.testing.assert_allclose(a, r, rtol=1e-9, atol=1e-9 * np.abs(r).max(), err_msg=str(k))
    assert ours[12].shape == (2, 1024, 2, 2)


def test_dense_block_net_shapes():
    m = M.dense_block_net()
    assert m.shapes() == [(3, 224, 224), (64, 112, 112), (64, 56, 56), (192, 56, 56)]


# Total learnable parameters of the TorchVision models the paper uses (as
# TorchVision documents them for alexnet, vgg16, resnet18, resnet50,
# densenet121 and vit_b_16), and the size of the classifier head each adds
# after the feature extractor the oracle assembles (closed forms).
TORCHVISION_TOTALS = {
    "alexnet": (61_100_840, (9216 * 4096 + 4096) + (4096 * 4096 + 4096) + (4096 * 1000 + 1000)),
    "vgg16": (138_357_544, (25088 * 4096 + 4096) + (4096 * 4096 + 4096) + (4096 * 1000 + 1000)),
    "resnet18": (11_689_512, 512 * 1000 + 1000),
    "resnet50": (25_557_032, 2048 * 1000 + 1000),
    "densenet121": (7_978_856, 1024 * 1000 + 1000),
    "vit_b16": (86_567_656, 768 * 1000 + 1000),
}


@pytest.mark.parametrize("name", sorted(TORCHVISION_TOTALS))
def test_feature_extractor_parameter_counts(name):
    """Structural pin: the oracle's learnable parameters (weights, biases,
    batch-norm and layer-norm scale and shift, class token, position
    embedding; not the batch-norm running statistics) number exactly the
    TorchVision model's total less its classifier head.  A misread width,
    kernel size, block count or a missing normalisation changes the count."""
    total, head = TORCHVISION_TOTALS[name]
    m = M.build(name)
    n = sum(int(np.prod(shape)) for shape, kind in m.manifest() if kind not in ("bn_mean", "bn_var"))
    assert n == total - head, (name, n, total - head)
