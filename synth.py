"""Seeded synthetic inputs shared by the oracle-side tests and the HIP path.

This module holds no arithmetic of the training method: it only draws
numbers.  Both sides receive identical arrays from here, so input
generation can never hide a disagreement between them.

Workload recipe (stand-ins for CIFAR-10/100 and ImageNet, which are not
used): images are i.i.d. N(0, 1) per element, i.e. the first two moments of
per-channel-normalised natural images; labels are uniform over the classes.
"""
from __future__ import annotations

import numpy as np


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(int(seed)))


def images(seed: int, n: int, c: int, h: int, w: int) -> np.ndarray:
    """float32 NCHW batch, elements i.i.d. N(0, 1)."""
    return _rng(seed).standard_normal((n, c, h, w), dtype=np.float32)


def labels(seed: int, n: int, n_classes: int) -> np.ndarray:
    """int32 labels, uniform in [0, n_classes)."""
    return _rng(seed + 7_777_777).integers(0, n_classes, size=n, dtype=np.int64).astype(np.int32)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """float32 values rounded to the nearest bfloat16 (ties to even), returned
    as float32.  Used to pre-round images for the bf16 workloads so both sides
    see the same quantised input."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).reshape(a.shape)


def init_params(specs, seed: int) -> np.ndarray:
    """Initial parameter vector (float32) from a list of tensor specs.

    Each spec is (kind, numel, fan_in), in parameter order:
      'conv_w'   -> N(0, 2 / fan_in)            (He normal)
      'linear_w' -> U(-1/sqrt(fan_in), +1/sqrt(fan_in))
      'bias'     -> 0
      'bn_gamma' -> 1
      'bn_beta'  -> 0
    """
    rng = _rng(seed + 1_000_003)
    parts = []
    for kind, numel, fan_in in specs:
        if kind == "conv_w":
            parts.append(rng.standard_normal(numel, dtype=np.float32) * np.float32(np.sqrt(2.0 / fan_in)))
        elif kind == "linear_w":
            b = np.float32(1.0 / np.sqrt(fan_in))
            parts.append(rng.uniform(-b, b, size=numel).astype(np.float32))
        elif kind in ("bias", "bn_beta"):
            parts.append(np.zeros(numel, np.float32))
        elif kind == "bn_gamma":
            parts.append(np.ones(numel, np.float32))
        else:
            raise ValueError(kind)
    return np.concatenate(parts).astype(np.float32) if parts else np.zeros(0, np.float32)


def perturb(x: np.ndarray, seed: int, scale: float) -> np.ndarray:
    """x plus i.i.d. N(0, scale^2) noise (float32); used to move BN affine
    parameters and biases off their trivial initial values in tests."""
    return (x + _rng(seed + 31).standard_normal(x.shape, dtype=np.float32) * np.float32(scale)).astype(np.float32)


def grid_values(seed: int, shape, step: float, bound: float) -> np.ndarray:
    """float32 values drawn uniformly from the grid {k * step : |k*step| <=
    bound} (step a power of two).  Sums of products of a few such values are
    exact in float32, so two evaluations of a small convolution in any order
    and precision produce identical values."""
    k = int(round(bound / step))
    return (_rng(seed + 4242).integers(-k, k + 1, size=shape).astype(np.float32) * np.float32(step))
