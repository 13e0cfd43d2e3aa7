"""Helpers that drive libhapi on the GPU through its C ABI for the tests.

Torch only allocates device memory and provides the stream; every step of the
forward pass runs in the library.  Inputs come from ``synth``; expected values
come from the oracle, computed on the CPU from the same synthetic arrays.
"""
from __future__ import annotations

import numpy as np
import torch

import paper_2210_08650_amd as H
import synth


def rel_l2(y, ref) -> float:
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref.ravel())
    return float(np.linalg.norm((y - ref).ravel()) / (den if den > 0 else 1.0))


def bf16_round(x) -> np.ndarray:
    """Round to bfloat16 (nearest even) and widen back to float32."""
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).float().numpy()


def images_for(dtype: int, imgs_f32: np.ndarray):
    """(device tensor in the model dtype, float32 values the oracle should see)."""
    if dtype == H.HAPI_BF16:
        t = torch.from_numpy(np.ascontiguousarray(imgs_f32, np.float32)).to(torch.bfloat16)
        return t.cuda(), t.float().numpy()
    t = torch.from_numpy(np.ascontiguousarray(imgs_f32, np.float32))
    return t.cuda(), imgs_f32.astype(np.float32)


class Runner:
    """A packed model resident on the GPU, ready for repeated extraction."""

    def __init__(self, layers, dtype, params, in_shape=(3, 224, 224)):
        self.layers, self.dtype, self.in_shape = layers, dtype, tuple(in_shape)
        self.stream = torch.cuda.current_stream()
        self.desc = H.Desc(layers, dtype, in_shape, stream=self.stream)
        raw = torch.from_numpy(synth.flatten(params)).cuda()
        assert raw.numel() == H.hapi_raw_weight_count(self.desc)
        # zeroed, so that the alignment gaps the packer skips compare equal
        self.packed = torch.zeros(max(H.hapi_packed_weight_bytes(self.desc), 256),
                                  dtype=torch.uint8, device="cuda")
        H.hapi_pack_weights(self.desc, raw if raw.numel() else None, self.packed)
        torch.cuda.synchronize()
        del raw
        self.tdtype = torch.bfloat16 if dtype == H.HAPI_BF16 else torch.float32

    def out_shape(self, split):
        return H.hapi_layer_shape(self.desc, split)

    def extract(self, images_dev, split, chunk=0, workspace_pad=0, out=None, inflight=0):
        batch = images_dev.shape[0]
        self.desc.set(chunk=chunk, inflight=inflight)
        need = H.hapi_workspace_bytes(self.desc, batch, split)
        ws = torch.empty(max(need + workspace_pad, 256), dtype=torch.uint8, device="cuda")
        self.desc.set(workspace=ws, workspace_bytes=need + workspace_pad)
        if out is None:
            out = torch.empty((batch,) + self.out_shape(split), dtype=self.tdtype, device="cuda")
        H.hapi_extract(self.desc, self.packed, images_dev, batch, split, out)
        torch.cuda.synchronize()
        return out

    def resume(self, input_dev, start, end, chunk=0, inflight=0):
        """Layers start+1..end on the layer-``start`` tensor (caller layout)."""
        batch = input_dev.shape[0]
        self.desc.set(chunk=chunk, inflight=inflight)
        need = H.hapi_workspace_bytes(self.desc, batch, end)
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device="cuda")
        self.desc.set(workspace=ws, workspace_bytes=need)
        out = torch.empty((batch,) + self.out_shape(end), dtype=self.tdtype, device="cuda")
        H.hapi_extract_range(self.desc, self.packed, input_dev, batch, start, end, out)
        torch.cuda.synchronize()
        return out

    def extract_np(self, images_dev, split, chunk=0, inflight=0):
        return self.extract(images_dev, split, chunk, inflight=inflight).float().cpu().numpy()
