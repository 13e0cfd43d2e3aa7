"""Host-side checks of libhapi through its C ABI (no GPU needed).

The library's shape calculus, byte profile and raw-weight layout are checked
bit-exactly against the oracle's independent model definitions; the error
paths are checked to fail during validation, before any device access.
"""
import os
import re

import numpy as np
import pytest

import paper_2210_08650_amd as H
from paper_2210_08650_amd import models as PM
from oracle import models as OM

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NAMES = ["alexnet", "resnet18", "resnet50", "vgg16", "vit_b16", "densenet_block", "densenet121"]


def _desc(name, **kw):
    dt = H.HAPI_F32 if name == "alexnet" else H.HAPI_BF16
    return H.Desc(PM.FACTORIES[name](), dt, **kw)


def test_library_exports_every_declared_symbol():
    import ctypes
    header = open(os.path.join(ROOT, "include", "hapi.h")).read()
    declared = set(re.findall(r"^\s*(?:[\w\s\*]+?)\b(hapi_\w+)\s*\(", header, re.M))
    assert declared == set(H.EXPORTED)
    lib = ctypes.CDLL(H.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name


@pytest.mark.parametrize("name", NAMES)
def test_layer_shapes_match_oracle(name):
    d = _desc(name)
    om = OM.build(name)
    assert d.n_layers == om.n_layers
    for k, shp in enumerate(om.shapes()):
        assert H.hapi_layer_shape(d, k) == tuple(shp), k


@pytest.mark.parametrize("name", NAMES)
def test_profile_bytes_bit_exact_and_linear_in_batch(name):
    d = _desc(name)
    esz = 4 if name == "alexnet" else 2
    elems = OM.build(name).out_elems()
    one, us = H.hapi_profile_layers(d, 1)
    assert us is None
    assert one == [e * esz for e in elems]
    for b in (8, 64, 256, 512):
        many, _ = H.hapi_profile_layers(d, b)
        assert many == [b * v for v in one]


@pytest.mark.parametrize("name", NAMES)
def test_raw_manifest_matches_oracle_and_library(name):
    layers = PM.FACTORIES[name]()
    ours = PM.raw_manifest(layers)
    theirs = OM.build(name).manifest()
    assert [(tuple(s), k) for s, k in ours] == [(tuple(s), k) for s, k in theirs]
    assert H.hapi_raw_weight_count(_desc(name)) == sum(int(np.prod(s)) for s, _ in ours)


def test_appendix_byte_tables():
    # Per-layer bytes at the benchmark batches (closed form, bf16 = 2 bytes).
    b, _ = H.hapi_profile_layers(_desc("resnet50"), 256)
    assert b[0] == 77_070_336 and b[1] == 411_041_792 and b[2] == 102_760_448
    assert b[18] == 51_380_224 and b[19] == 1_048_576
    b, _ = H.hapi_profile_layers(_desc("alexnet"), 4)
    assert b == [2_408_448, 3_097_600, 746_496, 2_239_488, 519_168, 1_038_336, 692_224,
                 692_224, 147_456]
    b, _ = H.hapi_profile_layers(_desc("vit_b16"), 128)
    assert b[1] == b[0] == 38_535_168 and b[10] == 38_731_776


def test_min_split_of_transformer_is_layer_one():
    # @Min: smallest output over layers 1..freeze, earliest on ties.
    b, _ = H.hapi_profile_layers(_desc("vit_b16"), 1)
    assert int(np.argmin(b[1:])) + 1 == 1


def test_chunk_plan_matches_paper_example():
    # 1000 objects with a storage-side batch of 200 -> 5 sequential partitions.
    d = _desc("resnet18", chunk=200)
    assert H.hapi_chunk_count(d, 1000) == 5
    d.set(chunk=16)
    assert H.hapi_chunk_count(d, 128) == 8
    assert H.hapi_chunk_count(d, 130) == 9       # short tail partition
    d.set(chunk=0)
    assert H.hapi_chunk_count(d, 64) == 1
    # automatic partitioning: two halves in flight from 128 images on
    assert H.hapi_chunk_count(d, 256) == 2 and H.hapi_chunk_count(d, 127) == 1
    assert H.hapi_chunk_count(d, 1000) == 4                 # 500 per lane, capped at 256
    assert H.hapi_chunk_count(d.set(inflight=1), 256) == 1
    assert H.hapi_chunk_count(d.set(inflight=4), 256) == 4
    d.set(inflight=0)


@pytest.mark.parametrize("name", NAMES)
def test_workspace_covers_memory_estimate(name):
    # The paper's estimate: the largest input + output of any layer.
    d = _desc(name, chunk=16)
    om = OM.build(name)
    e = om.out_elems()
    esz = 4 if name == "alexnet" else 2
    for split in range(1, om.n_layers + 1):
        est = max(e[k - 1] + e[k] for k in range(1, split + 1)) * 16 * esz
        assert H.hapi_workspace_bytes(d, 128, split) >= est
    assert H.hapi_workspace_bytes(d, 128, 0) == 0
    assert H.hapi_workspace_bytes(d, 128, om.n_layers, True) > H.hapi_workspace_bytes(d, 128, om.n_layers)


@pytest.mark.parametrize("name", NAMES)
def test_memory_profile_is_every_buffer_of_an_extraction(name):
    layers = PM.FACTORIES[name]()
    dt = H.HAPI_F32 if name == "alexnet" else H.HAPI_BF16
    d = H.Desc(layers, dt, chunk=16)
    mem = H.hapi_profile_memory(d, 128)
    out, _ = H.hapi_profile_layers(d, 128)
    for k in range(d.n_layers + 1):
        weights = H.hapi_packed_weight_bytes(H.Desc(layers[:k], dt)) if k else 0
        assert mem[k] == weights + out[0] + out[k] + H.hapi_workspace_bytes(d, 128, k), k
        if k:  # at least the paper's estimate for the partition batch
            assert mem[k] - weights - out[0] - out[k] >= max(
                out[j - 1] + out[j] for j in range(1, k + 1)) // 8


def test_workspace_holds_one_slot_set_per_partition_in_flight():
    d = _desc("resnet50", chunk=16)
    one = H.hapi_workspace_bytes(d, 128, 18)
    for k in (2, 3, 4):
        assert H.hapi_workspace_bytes(d.set(inflight=k), 128, 18) == k * one
    assert H.hapi_workspace_bytes(d.set(inflight=4), 32, 18) == 2 * one  # only 2 partitions
    # automatic: 2 x 128-image partitions need what 1 x 256 needs, plus the
    # second partition's four guard gaps
    auto = _desc("resnet50")
    seq = _desc("resnet50", chunk=256)
    assert H.hapi_workspace_bytes(auto, 256, 18) == H.hapi_workspace_bytes(seq, 256, 18) + 4 * H.HAPI_GUARD_BYTES
    _raises(H.HAPI_E_INVAL, H.hapi_workspace_bytes, d.set(inflight=5), 128, 18)
    _raises(H.HAPI_E_INVAL, H.hapi_workspace_bytes, d.set(inflight=-1), 128, 18)


@pytest.mark.parametrize("name,batch,chunk,inflight", [("resnet50", 256, 0, 0), ("resnet50", 40, 16, 0),
                                                       ("resnet18", 64, 0, 3), ("vit_b16", 5, 0, 0)])
def test_workspace_guard_gaps(name, batch, chunk, inflight):
    """Four gaps per partition in flight, each after one of the lane's
    regions: ordered, disjoint and inside the workspace."""
    d = _desc(name, chunk=chunk, inflight=inflight)
    n = d.n_layers
    ws = H.hapi_workspace_bytes(d, batch, n)
    g = H.hapi_workspace_guards(d, batch, n)
    parts = H.hapi_chunk_count(d, batch)
    lanes = min(inflight or (2 if chunk == 0 and batch >= 128 else 1), parts)
    assert len(g) == 4 * lanes
    assert all(b - a >= H.HAPI_GUARD_BYTES for a, b in zip(g, g[1:]))
    assert g[-1] + H.HAPI_GUARD_BYTES == ws
    assert H.hapi_workspace_guards(d, batch, 0) == []


def _raises(code, fn, *a):
    with pytest.raises(H.HapiError) as e:
        fn(*a)
    assert e.value.code == code, str(e.value)
    return str(e.value)


def test_validation_errors_before_any_launch():
    d = _desc("resnet18")
    fake = 1 << 40  # never dereferenced: every call below fails validation first
    _raises(H.HAPI_E_INVAL, H.hapi_extract, d, fake, fake, 0, 8, fake)
    _raises(H.HAPI_E_INVAL, H.hapi_extract, d, fake, fake, 4, 12, fake)
    _raises(H.HAPI_E_INVAL, H.hapi_extract, d, fake, fake, 4, -1, fake)
    _raises(H.HAPI_E_INVAL, H.hapi_extract, d, fake, None, 4, 8, fake)
    _raises(H.HAPI_E_INVAL, H.hapi_layer_shape, d, 12)
    msg = _raises(H.HAPI_E_NOMEM, H.hapi_extract, d.set(workspace=fake, workspace_bytes=1),
                  fake, fake, 4, 8, fake)
    assert "workspace" in msg
    need = H.hapi_workspace_bytes(d, 4, 8)
    d.set(workspace_bytes=need - 1)
    _raises(H.HAPI_E_NOMEM, H.hapi_extract, d, fake, fake, 4, 8, fake)


def test_resume_validation_before_any_launch():
    d = _desc("resnet18")
    fake = 1 << 40
    _raises(H.HAPI_E_INVAL, H.hapi_extract_range, d, fake, fake, 4, 5, 4, fake)
    _raises(H.HAPI_E_INVAL, H.hapi_extract_range, d, fake, fake, 4, -1, 4, fake)
    _raises(H.HAPI_E_INVAL, H.hapi_extract_range, d, fake, fake, 4, 2, 12, fake)
    _raises(H.HAPI_E_INVAL, H.hapi_extract_range, d, fake, None, 4, 2, 8, fake)
    _raises(H.HAPI_E_NOMEM, H.hapi_extract_range, d.set(workspace=fake, workspace_bytes=1),
            fake, fake, 4, 2, 8, fake)


def test_unsupported_and_invalid_descriptors():
    bad_head = PM.vit(dim=768, heads=8)          # head dim 96 is not built
    _raises(H.HAPI_E_UNSUPPORTED, H.hapi_raw_weight_count, H.Desc(bad_head, H.HAPI_BF16))
    _raises(H.HAPI_E_UNSUPPORTED, H.hapi_raw_weight_count, H.Desc(PM.vit_b16(), H.HAPI_F32))
    wrong_cin = PM.alexnet()
    wrong_cin[2] = dict(wrong_cin[2], cin=65)
    _raises(H.HAPI_E_INVAL, H.hapi_raw_weight_count, H.Desc(wrong_cin, H.HAPI_F32))
    _raises(H.HAPI_E_INVAL, H.hapi_raw_weight_count, H.Desc(PM.alexnet(), 7))
    reserved = PM.alexnet()
    d = H.Desc(reserved, H.HAPI_F32)
    d._layers[0].reserved[1] = 3
    _raises(H.HAPI_E_INVAL, H.hapi_raw_weight_count, d)
    too_long = PM.vit(image=272)                  # 290 tokens > attention limit
    _raises(H.HAPI_E_UNSUPPORTED, H.hapi_raw_weight_count, H.Desc(too_long, H.HAPI_BF16, (3, 272, 272)))


def test_profile_timing_needs_workspace():
    d = _desc("resnet18")
    _raises(H.HAPI_E_NOMEM, H.hapi_profile_layers, d, 8, True)
