"""hapi_extract_noalloc (the library's static device scratch instead of a
caller workspace) against hapi_extract, bit for bit, through the C ABI: two
calls in a row, the second with a smaller input, so the second call runs on
the scratch contents the first one left."""
import numpy as np
import pytest
import torch

import paper_2210_08650_amd as H
from paper_2210_08650_amd import models as PM
import synth
from oracle import models as OM
from tests.hip_harness import Guarded, images_for

pytestmark = pytest.mark.gpu


def _reference(d, packed, x, split):
    """hapi_extract with a guarded caller workspace."""
    b = x.shape[0]
    need = H.hapi_workspace_bytes(d, b, split)
    ws = Guarded(need, H.hapi_workspace_guards(d, b, split))
    d.set(workspace=ws.body, workspace_bytes=need)
    out = torch.empty((b,) + H.hapi_layer_shape(d, split), dtype=x.dtype, device="cuda")
    H.hapi_extract(d, packed, x, b, split, out)
    torch.cuda.synchronize()
    ws.check()
    return out


@pytest.mark.parametrize("name,split,batches", [("resnet50", 18, (24, 5)), ("vit_b16", 10, (12, 3)),
                                               ("densenet121", 12, (6, 2))])
def test_noalloc_matches_extract(name, split, batches):
    om = OM.build(name)
    ps = synth.params(31, om.manifest())
    layers = PM.FACTORIES[name]()
    d = H.Desc(layers, H.HAPI_BF16, stream=torch.cuda.current_stream())
    raw = torch.from_numpy(synth.flatten(ps)).cuda()
    packed = torch.zeros(H.hapi_packed_weight_bytes(d), dtype=torch.uint8, device="cuda")
    H.hapi_pack_weights(d, raw, packed)
    imgs = synth.images(32, max(batches))
    xd, _ = images_for(H.HAPI_BF16, imgs)
    for b in batches:   # the second call is smaller than the first
        x = xd[:b].contiguous()
        ref = _reference(d, packed, x, split)
        nd = H.Desc(layers, H.HAPI_BF16, stream=torch.cuda.current_stream())  # no workspace at all
        g = Guarded(ref.numel() * 2)
        out = g.view(torch.bfloat16, tuple(ref.shape))
        H.hapi_extract_noalloc(nd, packed, x, b, split, out)
        torch.cuda.synchronize()
        g.check()
        print(f"noalloc {name} b{b} split {split}: max |diff| "
              f"{float((out.float() - ref.float()).abs().max()):.3g}", flush=True)
        assert torch.equal(out, ref), (name, b)


def test_noalloc_rejects_what_the_scratch_cannot_hold():
    d = H.Desc(PM.vgg16(), H.HAPI_BF16, stream=torch.cuda.current_stream())
    need = H.hapi_workspace_bytes(d.set(inflight=1), 64, 18)
    assert need > H.HAPI_NOALLOC_SCRATCH_BYTES
    packed = torch.zeros(H.hapi_packed_weight_bytes(d), dtype=torch.uint8, device="cuda")
    x = torch.zeros((64, 3, 224, 224), dtype=torch.bfloat16, device="cuda")
    out = torch.full((64, 512, 7, 7), 3.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(H.HapiError) as e:
        H.hapi_extract_noalloc(d, packed, x, 64, 18, out)
    assert e.value.code == H.HAPI_E_NOMEM
    torch.cuda.synchronize()
    assert bool((out == 3.0).all())
