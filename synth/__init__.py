"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle.

This module holds random draws only: input images and parameter tensors drawn
from fixed distributions with counter-based seeds.  It holds none of the
feature-extraction arithmetic, so the HIP path and the oracle can both consume
its arrays without sharing any part of the computation.

Workloads (the paper evaluates ImageNet-sized 3x224x224 pre-processed tensors,
Evaluation / Methodology, "Training input"): images are N(0, 1) stand-ins for
those tensors; weights stand in for pre-trained ones.

Seeding: tensor ``index`` of workload ``w`` is drawn from
``numpy.random.Generator(PCG64(2210086500 + 1000 * w + index))``.
Index 0 is the image batch; parameter tensor ``i`` of a model's manifest uses
index ``1 + i``.  Image batches are prefix-consistent: the first ``b`` images of
a batch of ``B > b`` equal the batch of ``b``.
"""
from __future__ import annotations

import numpy as np

SEED_BASE = 2210086500

# Parameter distributions.  A manifest entry is ``(shape, kind)``.
#   he        N(0, 2 / fan_in), fan_in = prod(shape[1:])   (Kaiming-normal, ReLU gain)
#   bias      U(-0.1, 0.1)
#   bn_gamma  U(0.5, 1.5)      bn_beta  U(-0.1, 0.1)
#   bn_mean   U(-0.1, 0.1)     bn_var   U(0.5, 1.5)
#   tn02      N(0, 0.02^2) truncated at +-2 sigma
#   ln_gamma  1 + tn02         ln_beta  tn02
#   zeros / ones               constant tensors (degenerate-case tests)
KINDS = ("he", "bias", "bn_gamma", "bn_beta", "bn_mean", "bn_var",
         "tn02", "ln_gamma", "ln_beta", "zeros", "ones")


def seed_for(workload: int, index: int) -> int:
    return SEED_BASE + 1000 * int(workload) + int(index)


def _rng(workload: int, index: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed_for(workload, index)))


def images(workload: int, batch: int, channels: int = 3, height: int = 224,
           width: int = 224) -> np.ndarray:
    """float32 [batch, channels, height, width] drawn from N(0, 1), NCHW."""
    rng = _rng(workload, 0)
    return rng.standard_normal((batch, channels, height, width), dtype=np.float32)


def _trunc_normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    n = int(np.prod(shape)) if len(shape) else 1
    z = rng.standard_normal(n)
    bad = np.abs(z) > 2.0
    while bad.any():
        z[bad] = rng.standard_normal(int(bad.sum()))
        bad = np.abs(z) > 2.0
    return (z * std).astype(np.float32).reshape(shape)


def param(workload: int, index: int, shape, kind: str) -> np.ndarray:
    """One float32 parameter tensor of ``shape`` drawn from distribution ``kind``."""
    shape = tuple(int(s) for s in shape)
    rng = _rng(workload, index)
    if kind == "he":
        fan_in = int(np.prod(shape[1:])) if len(shape) > 1 else 1
        return (rng.standard_normal(shape) * np.sqrt(2.0 / fan_in)).astype(np.float32)
    if kind in ("bias", "bn_beta", "bn_mean"):
        return rng.uniform(-0.1, 0.1, shape).astype(np.float32)
    if kind in ("bn_gamma", "bn_var"):
        return rng.uniform(0.5, 1.5, shape).astype(np.float32)
    if kind in ("tn02", "ln_beta"):
        return _trunc_normal(rng, shape, 0.02)
    if kind == "ln_gamma":
        return (1.0 + _trunc_normal(rng, shape, 0.02)).astype(np.float32)
    if kind == "zeros":
        return np.zeros(shape, np.float32)
    if kind == "ones":
        return np.ones(shape, np.float32)
    raise ValueError(f"unknown parameter kind {kind!r}")


def params(workload: int, manifest) -> list:
    """All parameter tensors of a manifest ``[(shape, kind), ...]``, in order."""
    return [param(workload, 1 + i, shape, kind) for i, (shape, kind) in enumerate(manifest)]


def flatten(arrays) -> np.ndarray:
    """Concatenate float32 tensors into one flat float32 buffer, in order."""
    if not arrays:
        return np.zeros(0, np.float32)
    return np.concatenate([np.asarray(a, np.float32).ravel() for a in arrays])


def small_ints(seed: int, shape, lo: int = -3, hi: int = 3) -> np.ndarray:
    """float32 tensor of integers uniform in [lo, hi] (exact-arithmetic tests)."""
    rng = np.random.Generator(np.random.PCG64(SEED_BASE + 7_000_000 + int(seed)))
    return rng.integers(lo, hi + 1, size=tuple(shape)).astype(np.float32)


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round-to-nearest-even), returning uint16 bit patterns."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns (uint16) to the float32 values they encode."""
    b = np.ascontiguousarray(bits, np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def split_job(workload: int, image_bytes, freeze_idx: int, train_batch: int = 512,
              request_images: int = 128, server_slots: int = 4,
              images_per_epoch: int = 30720) -> dict:
    """Random split-choice job (field names of the library's split-job record).

    Stand-in measurements for the paper's setting (Evaluation, Methodology):
    requests of 128 objects, at most 4 run at once, an epoch of 30720 images
    and a 12 Gbps network, with every time and throughput drawn uniformly
    around plausible values: per-layer forward times of 0.2-5 ms per request
    on the server and 0.5-20 ms per training batch on the client, reading a
    request 20-80 ms, loading the model 50-300 ms, copies at 10-25 GB/s,
    (un)pickling at 1-4 GB/s, data loading at 2-8 GB/s, the bandwidth scaled
    by 0.25-4x.  ``image_bytes`` (the per-image output sizes) is passed in.
    """
    rng = _rng(workload, 900)
    n = len(image_bytes) - 1
    layer = lambda lo, hi: [0.0] + [float(v) for v in rng.uniform(lo, hi, n)]
    return {
        "n_layers": n, "freeze_idx": int(freeze_idx), "train_batch": int(train_batch),
        "request_images": int(request_images), "server_slots": int(server_slots),
        "iterations": max(1, int(images_per_epoch) // int(train_batch)),
        "image_bytes": [int(v) for v in image_bytes],
        "srv_layer_s": layer(0.2e-3, 5e-3), "cli_layer_s": layer(0.5e-3, 20e-3),
        "srv_read_data_s": float(rng.uniform(0.02, 0.08)),
        "srv_read_model_s": float(rng.uniform(0.05, 0.3)),
        "srv_to_gpu_s": float(rng.uniform(1e-3, 10e-3)),
        "cli_rest_s": float(rng.uniform(0.05, 0.5)),
        "srv_from_gpu_s_per_byte": 1.0 / float(rng.uniform(10e9, 25e9)),
        "srv_pickle_s_per_byte": 1.0 / float(rng.uniform(1e9, 4e9)),
        "cli_unpickle_s_per_byte": 1.0 / float(rng.uniform(1e9, 4e9)),
        "cli_loader_s_per_byte": 1.0 / float(rng.uniform(2e9, 8e9)),
        "cli_to_gpu_s_per_byte": 1.0 / float(rng.uniform(10e9, 25e9)),
        "net_bytes_per_s": 1.5e9 * float(np.exp(rng.uniform(np.log(0.25), np.log(4.0)))),
        "cli_mem_bytes": 0, "cli_fixed_mem_bytes": 0, "nosplit_iter_s": 0.0,
    }
