"""The five benchmark workloads at full batch, in the benchmark's launch
configuration (automatic partitioning), checked on sampled images.

Images are independent through the whole pass, so image i's activation can be
recomputed alone by the oracle; the samples always include the first and the
last image of the batch.
"""
import numpy as np
import pytest

import paper_2210_08650_amd as H
from paper_2210_08650_amd import models as PM
import synth
from oracle import models as OM
from tests.hip_harness import Runner, images_for, rel_l2

pytestmark = pytest.mark.gpu

SAMPLES = {"alexnet_f32_b4": [0, 1, 2, 3], "resnet18_bf16_b64": [0, 17, 63],
           "vgg16_bf16_b128": [0, 127], "resnet50_bf16_b256": [0, 97, 255],
           "vit_b16_bf16_b128": [0, 64, 127], "densenet_block_bf16_b64": [0, 31, 63],
           "densenet121_bf16_b256": [0, 255]}


@pytest.mark.parametrize("wl", list(PM.WORKLOADS))
def test_workload_full_batch_sampled(wl):
    cfg = PM.WORKLOADS[wl]
    om = OM.build(cfg["model"])
    ps = synth.params(cfg["seed"], om.manifest())
    imgs = synth.images(cfg["seed"], cfg["batch"])
    xd, xv = images_for(cfg["dtype"], imgs)
    r = Runner(PM.FACTORIES[cfg["model"]](), cfg["dtype"], ps)
    got = r.extract_np(xd, cfg["split"])
    assert got.shape == (cfg["batch"],) + om.shapes()[cfg["split"]]
    assert np.isfinite(got).all()
    tol = 1e-4 if cfg["dtype"] == H.HAPI_F32 else 2e-2
    idx = SAMPLES[wl]
    ref = om.forward(ps, xv[idx], cfg["split"])
    for j, i in enumerate(idx):
        err = rel_l2(got[i], ref[j])
        print(f"{wl} image {i}: rel_l2 {err:.3e}", flush=True)
        assert err <= tol
    # run-to-run determinism and partition independence, bit for bit
    again = r.extract_np(xd, cfg["split"], chunk=max(1, cfg["batch"] // 3 + 1))
    assert np.array_equal(again, got)


def test_resnet50_batch_512_two_full_partitions():
    """The largest benchmarked batch: two 256-image partitions in flight on two
    streams (the partition size cap), sampled at both ends and in the middle
    of the second partition."""
    cfg = PM.WORKLOADS["resnet50_bf16_b256"]
    om = OM.build("resnet50")
    ps = synth.params(cfg["seed"], om.manifest())
    imgs = synth.images(cfg["seed"], 512)
    xd, xv = images_for(H.HAPI_BF16, imgs)
    r = Runner(PM.resnet50(), H.HAPI_BF16, ps)
    assert H.hapi_chunk_count(r.desc.set(chunk=0, inflight=0), 512) == 2
    got = r.extract_np(xd, 18)
    idx = [0, 300, 511]
    ref = om.forward(ps, xv[idx], 18)
    for j, i in enumerate(idx):
        err = rel_l2(got[i], ref[j])
        print(f"resnet50 b512 image {i}: rel_l2 {err:.3e}", flush=True)
        assert err <= 2e-2
    # image 0 of a batch of 256 is computed by the same kernels with other partners
    assert np.array_equal(r.extract_np(xd[:256].contiguous(), 18), got[:256])
