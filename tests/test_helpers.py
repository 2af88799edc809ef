"""The comparison helpers the GPU tests measure parity with, on the CPU."""
import numpy as np

from tests.gpu_helpers import rel_err, update_err


def test_update_err_forgives_only_the_stored_weights_rounding():
    rng = np.random.default_rng(0)
    g = rng.standard_normal(512) * 3e-3
    p = np.ones(512, np.float32)
    exact = (p - 0.01 * g).astype(np.float32)  # w - lr g rounded once to float32
    # the plain relative error of p_new - p is dominated by that rounding ...
    assert rel_err(exact.astype(np.float64) - p, -0.01 * g) > 3e-4
    # ... which update_err does not count
    assert update_err(exact, p, -0.01 * g) == 0.0
    # a 1% wrong learning rate still shows, less at most two half ulps of 1 (the one
    # forgiven and the rounding of the wrong weight itself)
    off = (p - 0.0101 * g).astype(np.float32)
    ulp = np.spacing(np.float32(1.0)) / np.abs(0.01 * g).max()
    assert update_err(off, p, -0.01 * g) >= 1e-2 - ulp
    # large weights: the half ulp scales with each weight
    big = np.full(512, 1024.0, np.float32)
    assert update_err((big - 0.01 * g).astype(np.float32), big, -0.01 * g) == 0.0
    assert update_err(big, big, -0.01 * g) < 1.0  # an update below the weights' resolution
    assert update_err((big - 2.0 * g).astype(np.float32), big, -0.01 * g) > 10.0


def test_update_err_degenerate_cases():
    z = np.zeros(4, np.float32)
    assert update_err(z, z, np.zeros(4)) == 0.0
    assert update_err(np.ones(4, np.float32), z, np.zeros(4)) == np.inf
    assert update_err(np.zeros(0, np.float32), np.zeros(0), np.zeros(0)) == 0.0
