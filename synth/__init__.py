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
