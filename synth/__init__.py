"""Seeded synthetic inputs shared by the product path and the oracle.

This module draws random numbers and nothing else: it holds none of the
arithmetic of the scheduling method or of the CNN it trains.  Both the
oracle (under ``oracle/``) and the product binding consume the arrays it
returns, so that both sides see bit-identical inputs.

Draw order for one CNN workload (one ``numpy.random.default_rng(seed)``,
PCG64):

1. ``x``: batch of images, standard normal, drawn as float64 in NHWC order
   and cast to float32;
2. ``y``: integer labels, uniform in ``[0, classes)``;
3. parameters, in parameter-server order: every tensor whose spec is
   ``("he", n, fan_in)`` is drawn from N(0, sqrt(2 / fan_in)) as float64
   and cast to float32; ``("zeros", n)`` tensors are 0 and ``("ones", n)``
   tensors are 1 and consume no random numbers.

Images stand in for ImageNet-shaped (3x224x224, 1000 classes) and
CIFAR-shaped (3x32x32, 10 classes) data; no dataset item is used.
"""
from __future__ import annotations

import numpy as np


def cnn_inputs(seed: int, batch: int, hwc: tuple, classes: int, param_specs: list):
    """Return ``(x, y, params)`` for one seeded CNN workload.

    ``x`` is float32 ``[batch, H, W, C]`` (NHWC), ``y`` int32 ``[batch]``,
    ``params`` one flat float32 vector holding every tensor of
    ``param_specs`` back to back.
    """
    rng = np.random.default_rng(seed)
    h, w, c = hwc
    x = rng.standard_normal(size=(batch, h, w, c)).astype(np.float32)
    y = rng.integers(0, classes, size=batch).astype(np.int32)
    total = sum(int(s[1]) for s in param_specs)
    params = np.empty(total, dtype=np.float32)
    off = 0
    for spec in param_specs:
        kind, n = spec[0], int(spec[1])
        if kind == "he":
            fan_in = int(spec[2])
            params[off:off + n] = rng.normal(0.0, np.sqrt(2.0 / fan_in), size=n).astype(np.float32)
        elif kind == "zeros":
            params[off:off + n] = 0.0
        elif kind == "ones":
            params[off:off + n] = 1.0
        else:
            raise ValueError(f"unknown parameter spec kind {kind!r}")
        off += n
    return x, y, params


def random_profile(seed: int, L: int, hi: int = 1000, dt_hi: int = 50):
    """Integer per-layer cost vectors ``(pt, fc, bc, gt, dt)`` for planner tests.

    Every entry is uniform in ``[0, hi]``; ``dt`` is uniform in ``[0, dt_hi]``.
    The values are plain random integers (nanoseconds), nothing more.
    """
    rng = np.random.default_rng(seed)
    pt, fc, bc, gt = (rng.integers(0, hi + 1, size=L).astype(np.int64) for _ in range(4))
    dt = int(rng.integers(0, dt_hi + 1))
    return [int(v) for v in pt], [int(v) for v in fc], [int(v) for v in bc], [int(v) for v in gt], dt


def random_tensor(seed: int, shape, scale: float = 1.0):
    """A float32 standard-normal tensor (times ``scale``) for kernel tests."""
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(size=shape) * scale).astype(np.float32)
