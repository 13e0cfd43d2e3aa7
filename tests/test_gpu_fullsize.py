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

def samples(batch, n=8):
    """n images spread over the batch, always the first and the last (every
    image when the batch has at most n)."""
    if batch <= n:
        return list(range(batch))
    return sorted({round(i * (batch - 1) / (n - 1)) for i in range(n)})


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
    idx = samples(cfg["batch"])
    ref = om.forward(ps, xv[idx], cfg["split"])
    for j, i in enumerate(idx):
        err = rel_l2(got[i], ref[j])
        print(f"PARITY {wl} split {cfg['split']} image {i}: rel_l2 {err:.3e}", flush=True)
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
    idx = samples(512)
    ref = om.forward(ps, xv[idx], 18)
    for j, i in enumerate(idx):
        err = rel_l2(got[i], ref[j])
        print(f"PARITY resnet50_bf16_b512 split 18 image {i}: rel_l2 {err:.3e}", flush=True)
        assert err <= 2e-2
    # image 0 of a batch of 256 is computed by the same kernels with other partners
    assert np.array_equal(r.extract_np(xd[:256].contiguous(), 18), got[:256])


@pytest.mark.parametrize("batch", [8, 16, 32, 128])
def test_resnet50_sweep_sampled(batch):
    """The rest of the ResNet-50 batch sweep, each batch in the benchmark's
    launch configuration (automatic partitions; tile choice depends on the
    rows of each layer and on the partitions in flight: one at 8, 16 and 32, two
    64-image partitions at 128), against the oracle on images 0, B/2 and B-1.
    Storage-side batch adaptation must not change the result, so image 0 also
    equals its value in a batch of 256 bit for bit."""
    cfg = PM.WORKLOADS["resnet50_bf16_b256"]
    om = OM.build("resnet50")
    ps = synth.params(cfg["seed"], om.manifest())
    imgs = synth.images(cfg["seed"], 256)
    xd, xv = images_for(H.HAPI_BF16, imgs)
    r = Runner(PM.resnet50(), H.HAPI_BF16, ps)
    got = r.extract_np(xd[:batch].contiguous(), 18)
    idx = [0, batch // 2, batch - 1]
    ref = om.forward(ps, xv[idx], 18)
    for j, i in enumerate(idx):
        err = rel_l2(got[i], ref[j])
        print(f"PARITY resnet50_bf16_b{batch} split 18 image {i}: rel_l2 {err:.3e}", flush=True)
        assert err <= 2e-2
    full = r.extract_np(xd, 18)
    assert np.array_equal(full[:batch], got)
