"""dc_conv2d_forward_noalloc (scratch in a static device array) against dc_conv2d_forward.

Two calls in a row on one stream, the second on a smaller input, each checked
element by element against dc_conv2d_forward on the same inputs under the
same launch plan (bit-identical: the same kernels add in the same order).
The first shape runs a split-K plan, so its partial sums live in the static
scratch; the second has C % 4 != 0, so its channel-padded input copy does.
"""
import ctypes

import numpy as np
import pytest

from paper_2101_07968_amd import _lib as D
from tests.gpu_helpers import dev, host, scratch, stream, zeros

pytestmark = pytest.mark.gpu

SHAPES = [(32, 1, 1, 4096, 1000, 1, 1, 1, 0, 0), (3, 17, 13, 3, 16, 3, 3, 1, 1, 1)]


def _forward_both(shape, relu, seed):
    sh = D.ConvShape(*shape)
    n, h, w, c, k, r, s, st, pad, pad_w = shape
    p, q = (h + 2 * pad - r) // st + 1, (w + 2 * pad_w - s) // st + 1
    rng = np.random.default_rng(seed)
    x = dev(rng.standard_normal((n, h, w, c)).astype(np.float32))
    wt = dev((rng.standard_normal((k, r, s, c)) * np.sqrt(2.0 / (r * s * c))).astype(np.float32))
    b = dev(rng.standard_normal(k).astype(np.float32))
    _ws_t, ws, wsb = scratch(D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh)))
    y_ref, y_na = zeros((n, p, q, k)), zeros((n, p, q, k))
    y_na.fill_(float("nan"))
    st_ = stream()
    print(f"no-alloc forward {shape} relu {relu}", flush=True)
    D.call("dc_conv2d_forward", ctypes.byref(sh), x.data_ptr(), wt.data_ptr(), b.data_ptr(), relu,
           y_ref.data_ptr(), ws, wsb, st_)
    D.call("dc_conv2d_forward_noalloc", ctypes.byref(sh), x.data_ptr(), wt.data_ptr(), b.data_ptr(), relu,
           y_na.data_ptr(), st_)
    return host(y_ref), host(y_na)


def test_noalloc_forward_matches_workspace_forward():
    fwd = [D.conv_plan_info(s, 0) for s in SHAPES]
    assert fwd[0][2] > 1                 # split-K: partial sums in the scratch
    assert SHAPES[1][3] % 4 != 0         # padded channels: the padded copy in the scratch
    assert SHAPES[1][0] * SHAPES[1][1] * SHAPES[1][2] < SHAPES[0][0] * SHAPES[0][3]
    for i, (shape, relu) in enumerate(zip(SHAPES, (0, 1))):
        y_ref, y_na = _forward_both(shape, relu, seed=71 + i)
        assert np.isfinite(y_ref).all()
        np.testing.assert_array_equal(y_na, y_ref)
    # the first shape again after the smaller call: nothing left over changes it
    y_ref, y_na = _forward_both(SHAPES[0], 1, seed=73)
    np.testing.assert_array_equal(y_na, y_ref)
