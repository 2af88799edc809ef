"""GPU parity of the gfx950 kernels against the oracle, through the C ABI.

Tolerances (per tensor, max |gpu - oracle| / max |oracle|): the kernels add
float32 products, so a sum of K terms carries a relative rounding error of
order sqrt(number of sequential fp32 additions) * 2^-24.  The bars below are
1e-5 * max(1, sqrt(K / 256)), capped at 2e-4 for the longest reductions (up to
1.6 M terms), well inside the 1e-3 the full iteration must meet.  Max-pool
forward picks values, so it must be bit-exact; its argmax is decided in
float32 on both sides.  Average pooling sums at most a window's taps, so its
bar is 1e-6.
"""
import ctypes
import math

import numpy as np
import pytest

import synth
from oracle import cnn as OC
from oracle import nets as ON
from paper_2101_07968_amd import _lib as D
from tests.gpu_helpers import dev, host, rel_err, scratch, stream, zeros

pytestmark = pytest.mark.gpu


def tol(k_terms):
    return min(2e-4, 1e-5 * max(1.0, math.sqrt(k_terms / 256.0)))


def geom10(shape):
    """(n, h, w, c, k, r, s, stride, pad, pad_w) from a square 8-tuple
    (n, h, w, c, k, r, stride, pad) or a full 10-tuple."""
    if len(shape) == 8:
        n, h, w, c, k, r, st, pad = shape
        return (n, h, w, c, k, r, r, st, pad, pad)
    return tuple(shape)


def conv_shape(*shape):
    return D.ConvShape(*geom10(shape))


def out_hw(h, r, st, pad):
    return (h + 2 * pad - r) // st + 1


def run_conv(shape, x, w, b, dy, relu, acc_init):
    """All three passes on the GPU; returns (y, dx, dw, db) as numpy."""
    sh = conv_shape(*shape)
    n, h, wd, c, k, r, s, st, pad, pad_w = geom10(shape)
    P, Q = out_hw(h, r, st, pad), out_hw(wd, s, st, pad_w)
    ws_t, ws, wsb = scratch(D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh)))
    xd, wd_, bd, dyd = dev(x), dev(w), dev(b), dev(dy)
    y = zeros((n, P, Q, k))
    D.call("dc_conv2d_forward", ctypes.byref(sh), xd.data_ptr(), wd_.data_ptr(), bd.data_ptr(), relu,
           y.data_ptr(), ws, wsb, stream())
    dx = dev(acc_init) if acc_init is not None else zeros((n, h, wd, c))
    D.call("dc_conv2d_backward_data", ctypes.byref(sh), dyd.data_ptr(), wd_.data_ptr(),
           1 if acc_init is not None else 0, dx.data_ptr(), ws, wsb, stream())
    dw = zeros((k, r, s, c))
    db = zeros((k,))
    D.call("dc_conv2d_backward_filter", ctypes.byref(sh), xd.data_ptr(), dyd.data_ptr(), dw.data_ptr(),
           db.data_ptr(), ws, wsb, stream())
    return host(y), host(dx), host(dw), host(db)


SMALL = [
    # n, h, w, c, k, r, stride, pad
    (2, 13, 11, 8, 20, 3, 1, 1),
    (2, 9, 9, 3, 70, 3, 1, 1),
    (3, 15, 15, 16, 33, 3, 2, 1),
    (2, 12, 12, 12, 24, 1, 2, 0),
    (1, 31, 31, 3, 16, 11, 4, 2),
    (2, 14, 14, 3, 8, 7, 2, 3),
    (2, 7, 7, 64, 130, 3, 1, 1),
    (2, 28, 28, 64, 64, 3, 1, 1),
    (4, 1, 1, 1024, 64, 1, 1, 0),
    (4, 1, 1, 64, 10, 1, 1, 0),
    (3, 1, 1, 300, 130, 1, 1, 0),
    (2, 5, 5, 6, 5, 5, 1, 2),
    (2, 6, 6, 4, 4, 3, 3, 1),
    (5, 17, 17, 40, 136, 3, 1, 1),
    # lean address modes: wgrad pixel carry with row and image wraps and a
    # ragged last stage (Q >= 16), strided; dgrad / forward tap-uniform stages
    (3, 17, 19, 8, 12, 3, 1, 1),
    (2, 35, 33, 4, 8, 3, 2, 1),
    (2, 9, 10, 32, 48, 3, 2, 1),
    (3, 20, 18, 16, 32, 5, 1, 2),
    # a single output pixel; a stride larger than the filter (dgrad phases with no tap)
    (2, 3, 3, 8, 16, 3, 1, 0),
    (2, 9, 9, 4, 8, 1, 3, 0),
    # rectangular filters, row and column padding apart (n, h, w, c, k, r, s, stride, pad, pad_w):
    # the 1 x 7 / 7 x 1 / 1 x 3 / 3 x 1 convs and an unpadded strided 3 x 3
    (2, 17, 17, 32, 48, 1, 7, 1, 0, 3),
    (2, 17, 17, 32, 40, 7, 1, 1, 3, 0),
    (2, 8, 8, 64, 32, 1, 3, 1, 0, 1),
    (2, 8, 8, 48, 64, 3, 1, 1, 1, 0),
    (2, 11, 13, 6, 10, 1, 7, 1, 0, 3),
    (3, 9, 10, 5, 7, 7, 1, 1, 3, 0),
    (2, 19, 18, 16, 24, 3, 5, 2, 1, 2),
    (2, 15, 15, 16, 24, 3, 3, 2, 0, 0),
    (3, 21, 20, 16, 32, 1, 3, 1, 0, 1),
]


@pytest.mark.parametrize("shape", SMALL, ids=[str(s) for s in SMALL])
@pytest.mark.parametrize("variant", ["plain", "relu_acc"])
def test_conv_small(shape, variant):
    n, h, w, c, k, r, s, st, pad, pad_w = geom10(shape)
    P, Q = out_hw(h, r, st, pad), out_hw(w, s, st, pad_w)
    seed = sum(shape) * 7 + (variant == "relu_acc")
    x = synth.random_tensor(seed, (n, h, w, c))
    wt = synth.random_tensor(seed + 1, (k, r, s, c))
    b = synth.random_tensor(seed + 2, (k,))
    dy = synth.random_tensor(seed + 3, (n, P, Q, k))
    relu = 1 if variant == "relu_acc" else 0
    acc0 = synth.random_tensor(seed + 4, (n, h, w, c)) if variant == "relu_acc" else None
    y, dx, dw, db = run_conv(shape, x, wt, b, dy, relu, acc0)
    y_ref = OC.conv2d_forward(x, wt, b, st, (pad, pad_w))
    if relu:
        y_ref = np.maximum(y_ref, 0)
    dx_ref = OC.conv2d_backward_data(dy, wt, (h, w), st, (pad, pad_w))
    if acc0 is not None:
        dx_ref = dx_ref + acc0
    dw_ref = OC.conv2d_backward_filter(x, dy, (r, s), st, (pad, pad_w))
    db_ref = dy.astype(np.float64).sum(axis=(0, 1, 2))
    assert rel_err(y, y_ref) <= tol(r * s * c)
    assert rel_err(dx, dx_ref) <= tol(r * s * k)
    assert rel_err(dw, dw_ref) <= tol(n * P * Q)
    assert rel_err(db, db_ref) <= tol(n * P * Q)


RGB_SHAPES = [(2, 13, 11, 3, 64, 3, 1, 1), (3, 15, 15, 3, 32, 3, 2, 0), (2, 9, 10, 3, 96, 3, 1, 1),
              (1, 7, 5, 3, 128, 3, 1, 1), (2, 33, 35, 3, 32, 3, 2, 1), (5, 4, 4, 3, 64, 3, 1, 2),
              (4, 40, 36, 3, 64, 3, 1, 1)]


@pytest.mark.parametrize("shape", RGB_SHAPES, ids=[str(s) for s in RGB_SHAPES])
def test_conv_rgb_direct(shape):
    """C = 3 with a 3 x 3 filter: the forward pass and the filter gradient (with the bias
    gradient) run on the direct kernels (plan source 4), the data gradient on the implicit
    GEMM; against the oracle, with bias + ReLU, for 1 to 4 blocks of 32 output channels,
    strides 1 and 2, paddings 0 to 2 and ragged last tiles.  An output that is not 16-byte aligned falls back to
    the implicit GEMM, within the same bar."""
    n, h, w, c, k, r, st, pad = shape
    g10 = geom10(shape)
    assert [D.conv_plan_info(g10, p)[7] for p in range(3)][0::2] == [4, 4]
    assert D.conv_plan_info(g10, 1)[7] != 4
    P, Q = out_hw(h, r, st, pad), out_hw(w, r, st, pad)
    seed = sum(shape) * 11
    x = synth.random_tensor(seed, (n, h, w, c))
    wt = synth.random_tensor(seed + 1, (k, r, r, c))
    b = synth.random_tensor(seed + 2, (k,))
    dy = synth.random_tensor(seed + 3, (n, P, Q, k))
    y, dx, dw, db = run_conv(shape, x, wt, b, dy, 1, None)
    y_ref = np.maximum(OC.conv2d_forward(x, wt, b, st, pad), 0)
    assert rel_err(y, y_ref) <= tol(r * r * c)
    assert rel_err(dx, OC.conv2d_backward_data(dy, wt, (h, w), st, pad)) <= tol(r * r * k)
    assert rel_err(dw, OC.conv2d_backward_filter(x, dy, (r, r), st, pad)) <= tol(n * P * Q)
    assert rel_err(db, dy.astype(np.float64).sum(axis=(0, 1, 2))) <= tol(n * P * Q)
    # a misaligned output takes the implicit GEMM
    sh = conv_shape(*shape)
    ws_t, ws, wsb = scratch(D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh)))
    xd, wd, bd = dev(x), dev(wt), dev(b)
    yb = zeros((n * P * Q * k + 4,))
    D.call("dc_conv2d_forward", ctypes.byref(sh), xd.data_ptr(), wd.data_ptr(), bd.data_ptr(), 1,
           yb.data_ptr() + 4, ws, wsb, stream())
    assert rel_err(host(yb)[1:1 + n * P * Q * k].reshape(y.shape), y_ref) <= tol(r * r * c)


FC_SHAPES = [(1, 4000, 1003), (5, 1004, 3999), (31, 2052, 2001), (32, 4096, 1000), (32, 25088, 4096),
             (33, 4096, 1000), (32, 3996, 1000), (4, 1024, 64), (3, 300, 130), (7, 4100, 4000),
             (32, 16000, 1004), (1, 9216, 4096)]


@pytest.mark.parametrize("n,fin,fout", FC_SHAPES, ids=[f"{n}x{i}->{o}" for n, i, o in FC_SHAPES])
def test_fc_streaming(n, fin, fout):
    """FC layers of at most 32 rows run on the FC kernels (plan source 3): the forward from 16 M
    weights (outputs a multiple of 4), the data gradient from 4 M weights; the filter gradient
    and smaller layers on the implicit GEMM.  Ragged rows, features and
    outputs, bias + ReLU, an accumulating data gradient and the ReLU-masked data gradient,
    against the oracle."""
    shape = (n, 1, 1, fin, fout, 1, 1, 1, 0, 0)
    src = [D.conv_plan_info(shape, p)[7] for p in range(3)]
    small = n <= 32 and fin % 4 == 0
    want = [small and fout % 4 == 0 and fin * fout >= 16000000, small and fin * fout >= 4000000, False]
    assert [s == 3 for s in src] == want, (src, want)
    seed = n * 1000 + fin + fout
    x = synth.random_tensor(seed, (n, 1, 1, fin))
    wt = synth.random_tensor(seed + 1, (fout, 1, 1, fin), scale=math.sqrt(2.0 / fin))
    b = synth.random_tensor(seed + 2, (fout,))
    dy = synth.random_tensor(seed + 3, (n, 1, 1, fout))
    acc0 = synth.random_tensor(seed + 4, (n, 1, 1, fin))
    y, dx, dw, db = run_conv(shape, x, wt, b, dy, 1, acc0)
    assert rel_err(y, np.maximum(OC.conv2d_forward(x, wt, b, 1, 0), 0)) <= tol(fin)
    dx_ref = OC.conv2d_backward_data(dy, wt, (1, 1), 1, 0)
    assert rel_err(dx, dx_ref + acc0) <= tol(fout)
    assert rel_err(dw, OC.conv2d_backward_filter(x, dy, (1, 1), 1, 0)) <= tol(n)
    assert rel_err(db, dy.astype(np.float64).sum(axis=(0, 1, 2))) <= tol(n)
    # the data gradient through a ReLU whose output is x (the model's folded launch)
    sh = conv_shape(*shape)
    ws_t, ws, wsb = scratch(D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh)))
    relu_y = np.maximum(x, 0)
    dxm = zeros((n, 1, 1, fin))
    dyd, wd, yd = dev(dy), dev(wt), dev(relu_y)   # held: a freed tensor's memory is reused at once
    D.call("dc_conv2d_backward_data_relu", ctypes.byref(sh), dyd.data_ptr(), wd.data_ptr(), yd.data_ptr(), 0,
           dxm.data_ptr(), ws, wsb, stream())
    exp = np.where(relu_y.astype(np.float32) > 0, dx_ref, 0.0)
    assert rel_err(host(dxm), exp) <= tol(fout)
    assert (host(dxm)[relu_y <= 0] == 0).all()


PLAN_SHAPES = [
    (4, 14, 14, 64, 96, 3, 3, 1, 1, 1),    # K = 576: split-K up to 8 in forward and dgrad
    (3, 15, 15, 32, 48, 3, 3, 2, 1, 1),    # strided: four dgrad phases
    (2, 17, 17, 32, 48, 1, 7, 1, 0, 3),    # 1 x 7 filter, columns padded only
    (2, 20, 20, 3, 16, 3, 3, 1, 1, 1),     # C = 3: channel-padded forward and wgrad
]


@pytest.mark.parametrize("shape", PLAN_SHAPES, ids=[str(s) for s in PLAN_SHAPES])
def test_every_plan_matches_oracle(shape):
    """Each (tile, split-K) plan the planner may pick, pinned in turn, gives the
    oracle's result to the pass's bar: the table of measured plans can choose
    any of them."""
    n, h, w, c, k, r, s, st, pad, pad_w = shape
    P, Q = out_hw(h, r, st, pad), out_hw(w, s, st, pad_w)
    seed = sum(shape)
    x = synth.random_tensor(seed, (n, h, w, c))
    wt = synth.random_tensor(seed + 1, (k, r, s, c))
    b = synth.random_tensor(seed + 2, (k,))
    dy = synth.random_tensor(seed + 3, (n, P, Q, k))
    refs = [OC.conv2d_forward(x, wt, b, st, (pad, pad_w)),
            OC.conv2d_backward_data(dy, wt, (h, w), st, (pad, pad_w)),
            OC.conv2d_backward_filter(x, dy, (r, s), st, (pad, pad_w))]
    bars = [tol(r * s * c), tol(r * s * k), tol(n * P * Q)]
    sh = conv_shape(*shape)
    xd, wd_, bd, dyd = dev(x), dev(wt), dev(b), dev(dy)
    tried = 0
    for pas in range(3):
        for plan in D.conv_plan_candidates(shape, pas):
            D.conv_set_plan(shape, pas, *plan)
            try:
                assert D.conv_plan_info(shape, pas)[:3] == plan
                ws_t, ws, wsb = scratch(D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh)))
                if pas == 0:
                    out = zeros((n, P, Q, k))
                    D.call("dc_conv2d_forward", ctypes.byref(sh), xd.data_ptr(), wd_.data_ptr(), bd.data_ptr(), 0,
                           out.data_ptr(), ws, wsb, stream())
                elif pas == 1:
                    out = zeros((n, h, w, c))
                    D.call("dc_conv2d_backward_data", ctypes.byref(sh), dyd.data_ptr(), wd_.data_ptr(), 0,
                           out.data_ptr(), ws, wsb, stream())
                else:
                    out = zeros((k, r, s, c))
                    D.call("dc_conv2d_backward_filter", ctypes.byref(sh), xd.data_ptr(), dyd.data_ptr(),
                           out.data_ptr(), None, ws, wsb, stream())
                err = rel_err(host(out), refs[pas])
                assert err <= bars[pas], (pas, plan, err)
                tried += 1
            finally:
                D.conv_set_plan(shape, pas, 0)
    assert tried >= 3 * 4


def _full_size_geoms():
    """Every distinct conv / FC geometry of the workloads at their own batch."""
    seen, out = set(), []
    for name, batch in (("tiny", 4), ("alexnet", 32), ("resnet18", 128), ("vgg16", 32), ("resnet50", 64),
                        ("googlenet", 32), ("vgg19", 32), ("resnet152", 32), ("inception_v4", 32)):
        net = OC.Net(ON.get(name), batch)
        for i, op in enumerate(net.ops):
            if op["op"] not in ("conv", "fc"):
                continue
            n, h, w, c = net.shapes[op["in"]]
            if op["op"] == "conv":
                g = (n, h, w, c, op["k"], op["r"], op["s"], op["stride"], op["pad"], op.get("pad_w", op["pad"]))
            else:
                g = (n, 1, 1, h * w * c, op["out"], 1, 1, 1, 0, 0)
            if g not in seen:
                seen.add(g)
                out.append((name, g))
    return out


FULL = _full_size_geoms()


def _sample(rng, shape, count):
    idx = [np.zeros(len(shape), dtype=int), np.array(shape) - 1]
    for _ in range(count):
        idx.append(np.array([rng.integers(0, s) for s in shape]))
    return np.stack(idx)


@pytest.mark.parametrize("case", FULL, ids=[f"{n}-{g}" for n, g in FULL])
def test_conv_full_size_sampled(case):
    name, shape = case
    n, h, w, c, k, r, s, st, pad, pad_w = shape
    P, Q = out_hw(h, r, st, pad), out_hw(w, s, st, pad_w)
    seed = sum((i + 1) * v for i, v in enumerate(shape)) % 10000
    x = synth.random_tensor(seed, (n, h, w, c))
    wt = synth.random_tensor(seed + 1, (k, r, s, c), scale=math.sqrt(2.0 / (r * s * c)))
    b = synth.random_tensor(seed + 2, (k,))
    dy = synth.random_tensor(seed + 3, (n, P, Q, k), scale=1e-3)
    print(f"conv {name} {shape}", flush=True)
    y, dx, dw, db = run_conv(shape, x, wt, b, dy, 0, None)
    rng = np.random.default_rng(seed)
    geom = shape
    i = _sample(rng, y.shape, 48)
    ref = OC.conv2d_samples("fwd", geom, x, wt, i, b)
    got = y[tuple(i.T)]
    assert np.abs(got - ref).max() <= tol(r * s * c) * np.abs(y).max()
    i = _sample(rng, dx.shape, 48)
    ref = OC.conv2d_samples("dgrad", geom, dy, wt, i)
    got = dx[tuple(i.T)]
    assert np.abs(got - ref).max() <= tol(r * s * k) * np.abs(dx).max()
    i = _sample(rng, dw.shape, 32)
    ref = OC.conv2d_samples("wgrad", geom, x, dy, i)
    got = dw[tuple(i.T)]
    assert np.abs(got - ref).max() <= tol(n * P * Q) * np.abs(dw).max()
    db_ref = dy.astype(np.float64).sum(axis=(0, 1, 2))
    assert rel_err(db, db_ref) <= tol(n * P * Q)


def test_conv_operand_over_2gb_sampled():
    """A 2.2 GB input (553,648,128 floats): past the lean mode's 2 GB limit, so
    every pass runs on 64-bit element offsets that cross the 2^31-byte mark.
    Sampled outputs, including the first and last element of each result,
    against the oracle."""
    shape = (66, 256, 256, 128, 16, 1, 1, 1, 0, 0)
    n, h, w, c, k, r, s, st, pad, pad_w = shape
    assert 4 * n * h * w * c >= 2 ** 31
    print("conv over 2 GB: generating inputs", flush=True)
    x = synth.random_tensor(90, (n, h, w, c))
    wt = synth.random_tensor(91, (k, r, s, c), scale=math.sqrt(2.0 / (r * s * c)))
    b = synth.random_tensor(92, (k,))
    dy = synth.random_tensor(93, (n, h, w, k), scale=1e-3)
    print("conv over 2 GB: running the three passes", flush=True)
    y, dx, dw, db = run_conv(shape, x, wt, b, dy, 0, None)
    print("conv over 2 GB: checking samples", flush=True)
    rng = np.random.default_rng(94)
    i = _sample(rng, y.shape, 48)
    assert np.abs(y[tuple(i.T)] - OC.conv2d_samples("fwd", shape, x, wt, i, b)).max() <= tol(c) * np.abs(y).max()
    i = _sample(rng, dx.shape, 48)
    assert np.abs(dx[tuple(i.T)] - OC.conv2d_samples("dgrad", shape, dy, wt, i)).max() <= tol(k) * np.abs(dx).max()
    i = _sample(rng, dw.shape, 32)
    assert np.abs(dw[tuple(i.T)] - OC.conv2d_samples("wgrad", shape, x, dy, i)).max() <= tol(n * h * w) * np.abs(dw).max()


def test_conv_rejects_bad_shapes_and_accepts_empty():
    sh = conv_shape(2, 4, 4, 3, 5, 3, 1, 3)  # pad >= r
    assert D.lib().dc_conv2d_forward(ctypes.byref(sh), 1, 1, None, 0, 1, None, 0, None) == D.DC_EINVAL
    sh = conv_shape(0, 4, 4, 3, 5, 3, 1, 1)  # empty batch: nothing to do
    assert D.lib().dc_conv2d_forward(ctypes.byref(sh), None, None, None, 0, None, None, 0, stream()) == D.DC_OK
    # the bias gradient needs scratch: a missing workspace is an error, not a fault
    sh = conv_shape(2, 40, 40, 64, 64, 3, 1, 1)
    assert D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh)) > 0
    x, dy, dw, db = zeros((2, 40, 40, 64)), zeros((2, 40, 40, 64)), zeros((64, 3, 3, 64)), zeros((64,))
    assert D.lib().dc_conv2d_backward_filter(ctypes.byref(sh), x.data_ptr(), dy.data_ptr(), dw.data_ptr(),
                                             db.data_ptr(), None, 0, stream()) == D.DC_EINVAL


# ---------------------------------------------------------------- elementwise

@pytest.mark.parametrize("n,offset", [(1000, 0), (1003, 1), (4 * 1024 * 1024 + 3, 0)])
def test_relu_add_copy(n, offset):
    a = synth.random_tensor(1, (n + offset,))
    b = synth.random_tensor(2, (n + offset,))
    g = synth.random_tensor(3, (n + offset,))
    ad, bd, gd = dev(a), dev(b), dev(g)
    y = zeros((n + offset,))
    D.call("dc_relu_forward", ad.data_ptr() + 4 * offset, y.data_ptr() + 4 * offset, n, stream())
    yh = host(y)[offset:]
    np.testing.assert_array_equal(yh, np.maximum(a[offset:], 0))
    dx = dev(b)
    D.call("dc_relu_backward", gd.data_ptr() + 4 * offset, y.data_ptr() + 4 * offset, 1,
           dx.data_ptr() + 4 * offset, n, stream())
    ref = b[offset:] + np.where(yh > 0, g[offset:], 0)
    np.testing.assert_array_equal(host(dx)[offset:], ref.astype(np.float32))
    z = zeros((n + offset,))
    D.call("dc_add_forward", ad.data_ptr() + 4 * offset, bd.data_ptr() + 4 * offset, 1, z.data_ptr() + 4 * offset,
           n, stream())
    np.testing.assert_array_equal(host(z)[offset:], np.maximum(a[offset:] + b[offset:], 0))
    D.call("dc_copy_grad", gd.data_ptr(), 1, ad.data_ptr(), n + offset, stream())
    np.testing.assert_array_equal(host(ad), (a + g).astype(np.float32))


POOLS = [(2, 8, 8, 5, 2, 2, 0), (3, 13, 13, 16, 3, 2, 0), (2, 12, 12, 7, 3, 2, 1), (32, 55, 55, 64, 3, 2, 0),
         (64, 112, 112, 64, 3, 2, 1), (32, 224, 224, 64, 2, 2, 0), (2, 9, 9, 12, 3, 1, 1), (3, 14, 14, 4, 3, 2, 1),
         # windows that tile the input (r = stride, no padding): the per-window backward kernel, also with
         # c / 4 = 1 and 3 x 3 windows; an odd extent leaves a row uncovered and takes the gather kernel
         (2, 12, 12, 8, 3, 3, 0), (4, 16, 16, 4, 2, 2, 0), (2, 9, 10, 8, 2, 2, 0)]


@pytest.mark.parametrize("cfg", POOLS, ids=[str(p) for p in POOLS])
def test_maxpool(cfg):
    n, h, w, c, r, st, pad = cfg
    x = synth.random_tensor(11, (n, h, w, c))
    P, Q = out_hw(h, r, st, pad), out_hw(w, r, st, pad)
    dy = synth.random_tensor(12, (n, P, Q, c))
    sh = D.PoolShape(n, h, w, c, r, r, st, pad)
    xd, dyd = dev(x), dev(dy)
    y = zeros((n, P, Q, c))
    arg = zeros((n, P, Q, c), "uint8")
    D.call("dc_maxpool_forward", ctypes.byref(sh), xd.data_ptr(), y.data_ptr(), arg.data_ptr(), stream())
    dx = zeros((n, h, w, c))
    D.call("dc_maxpool_backward", ctypes.byref(sh), dyd.data_ptr(), arg.data_ptr(), 0, dx.data_ptr(), stream())
    y_ref, arg_ref = OC.maxpool_forward(x, r, r, st, pad)
    np.testing.assert_array_equal(host(y), y_ref.astype(np.float32))
    np.testing.assert_array_equal(host(arg).astype(np.int32), arg_ref)
    dx_ref = OC.maxpool_backward(dy, arg_ref, x.shape, r, r, st, pad)
    assert rel_err(host(dx), dx_ref) <= 1e-7
    # accumulating into an existing gradient
    acc0 = synth.random_tensor(13, (n, h, w, c))
    dxa = dev(acc0)
    D.call("dc_maxpool_backward", ctypes.byref(sh), dyd.data_ptr(), arg.data_ptr(), 1, dxa.data_ptr(), stream())
    assert rel_err(host(dxa), dx_ref + acc0) <= 1e-6


POOLS_RELU = [p for p in POOLS if p[0] * p[1] * p[2] * p[3] < 100000]


@pytest.mark.parametrize("cfg", POOLS_RELU, ids=[str(p) for p in POOLS_RELU])
def test_maxpool_backward_relu(cfg):
    """Max-pool backward with the ReLU before it folded in (dc_maxpool_backward_relu):
    a window adds its dy only where its maximum, the pool's output, is positive.
    Against the oracle's backward of dy masked by y > 0, plain and accumulating, on the
    scalar, gather and per-window kernels; inputs shifted by -1 so that about a third
    of the windows have a negative maximum."""
    n, h, w, c, r, st, pad = cfg
    x = (synth.random_tensor(21, (n, h, w, c)) - 1.0).astype(np.float32)
    P, Q = out_hw(h, r, st, pad), out_hw(w, r, st, pad)
    dy = synth.random_tensor(22, (n, P, Q, c))
    sh = D.PoolShape(n, h, w, c, r, r, st, pad)
    xd, dyd = dev(x), dev(dy)
    y = zeros((n, P, Q, c))
    arg = zeros((n, P, Q, c), "uint8")
    D.call("dc_maxpool_forward", ctypes.byref(sh), xd.data_ptr(), y.data_ptr(), arg.data_ptr(), stream())
    y_ref, arg_ref = OC.maxpool_forward(x, r, r, st, pad)
    neg = float((y_ref <= 0).mean())
    assert 0.05 < neg < 0.95, neg
    dx_ref = OC.maxpool_backward(np.where(y_ref > 0, dy, 0.0), arg_ref, x.shape, r, r, st, pad)
    dx = zeros((n, h, w, c))
    D.call("dc_maxpool_backward_relu", ctypes.byref(sh), dyd.data_ptr(), arg.data_ptr(), y.data_ptr(), 0,
           dx.data_ptr(), stream())
    assert rel_err(host(dx), dx_ref) <= 1e-7
    acc0 = synth.random_tensor(23, (n, h, w, c))
    dxa = dev(acc0)
    D.call("dc_maxpool_backward_relu", ctypes.byref(sh), dyd.data_ptr(), arg.data_ptr(), y.data_ptr(), 1,
           dxa.data_ptr(), stream())
    assert rel_err(host(dxa), dx_ref + acc0) <= 1e-6


AVGPOOLS = [(2, 8, 8, 5, 3, 1, 1), (2, 9, 7, 12, 3, 1, 1), (3, 13, 13, 16, 3, 2, 1), (2, 12, 12, 7, 2, 2, 0),
            (32, 35, 35, 384, 3, 1, 1), (32, 17, 17, 1024, 3, 1, 1), (32, 8, 8, 1536, 3, 1, 1),
            (2, 11, 10, 6, 5, 3, 2), (1, 1, 1, 4, 3, 1, 1)]


@pytest.mark.parametrize("cfg", AVGPOOLS, ids=[str(p) for p in AVGPOOLS])
def test_avgpool(cfg):
    """Average pooling over the in-image taps, forward and backward (also accumulating)."""
    n, h, w, c, r, st, pad = cfg
    x = synth.random_tensor(15, (n, h, w, c))
    P, Q = out_hw(h, r, st, pad), out_hw(w, r, st, pad)
    dy = synth.random_tensor(16, (n, P, Q, c))
    sh = D.PoolShape(n, h, w, c, r, r, st, pad)
    xd, dyd = dev(x), dev(dy)
    y = zeros((n, P, Q, c))
    D.call("dc_avgpool_forward", ctypes.byref(sh), xd.data_ptr(), y.data_ptr(), stream())
    assert rel_err(host(y), OC.avgpool_forward(x, r, r, st, pad)) <= 1e-6
    dx_ref = OC.avgpool_backward(dy, x.shape, r, r, st, pad)
    dx = zeros((n, h, w, c))
    D.call("dc_avgpool_backward", ctypes.byref(sh), dyd.data_ptr(), 0, dx.data_ptr(), stream())
    assert rel_err(host(dx), dx_ref) <= 1e-6
    acc0 = synth.random_tensor(17, (n, h, w, c))
    dxa = dev(acc0)
    D.call("dc_avgpool_backward", ctypes.byref(sh), dyd.data_ptr(), 1, dxa.data_ptr(), stream())
    assert rel_err(host(dxa), dx_ref + acc0) <= 1e-6


def test_avgpool_rejects_bad_shapes():
    sh = D.PoolShape(2, 4, 4, 3, 3, 3, 1, 3)    # pad >= window
    assert D.lib().dc_avgpool_forward(ctypes.byref(sh), 1, 1, None) == D.DC_EINVAL
    sh = D.PoolShape(0, 4, 4, 3, 3, 3, 1, 1)    # empty batch: nothing to do
    assert D.lib().dc_avgpool_forward(ctypes.byref(sh), None, None, stream()) == D.DC_OK


def test_pooling_near_2g_elements():
    """Largest pooling sizes: 1,996,920,000 elements (below the 2^31 limit, past
    2^31 - 2^28, where a 32-bit grid-stride step would wrap), c = 3 so the
    per-channel kernels run.  With 1 x 1 windows at stride 1 each output is its
    one input tap divided by a count of 1, so average and max pooling are the
    identity both ways, bit for bit: y = x, dx = dy, every argmax 0."""
    t = __import__("torch")
    n, h, w, c = 1, 25800, 25800, 3
    total = n * h * w * c
    assert 2 ** 31 - 2 ** 28 < total < 2 ** 31 - 1
    print(f"pooling near 2^31: {total} elements", flush=True)
    g = t.Generator(device="cuda").manual_seed(95)
    x = t.rand(total, device="cuda", generator=g)
    y = t.full((total,), float("nan"), device="cuda")
    sh = D.PoolShape(n, h, w, c, 1, 1, 1, 0)
    D.call("dc_avgpool_forward", ctypes.byref(sh), x.data_ptr(), y.data_ptr(), stream())
    t.cuda.synchronize()
    assert t.equal(x, y)
    y.fill_(float("nan"))
    D.call("dc_avgpool_backward", ctypes.byref(sh), x.data_ptr(), 0, y.data_ptr(), stream())
    t.cuda.synchronize()
    assert t.equal(x, y)
    y.fill_(float("nan"))
    arg = t.full((total,), 7, dtype=t.uint8, device="cuda")
    D.call("dc_maxpool_forward", ctypes.byref(sh), x.data_ptr(), y.data_ptr(), arg.data_ptr(), stream())
    t.cuda.synchronize()
    assert t.equal(x, y) and int(arg.max()) == 0
    y.fill_(float("nan"))
    D.call("dc_maxpool_backward", ctypes.byref(sh), x.data_ptr(), arg.data_ptr(), 0, y.data_ptr(), stream())
    t.cuda.synchronize()
    assert t.equal(x, y)


@pytest.mark.parametrize("cfg", [(3, 4, 4, 10), (128, 4, 4, 512), (64, 7, 7, 2048)])
def test_gap(cfg):
    n, h, w, c = cfg
    x = synth.random_tensor(13, (n, h, w, c))
    dy = synth.random_tensor(14, (n, 1, 1, c))
    y = zeros((n, 1, 1, c))
    xd, dyd = dev(x), dev(dy)
    D.call("dc_gap_forward", n, h * w, c, xd.data_ptr(), y.data_ptr(), stream())
    assert rel_err(host(y), x.astype(np.float64).mean(axis=(1, 2), keepdims=True)) <= 1e-6
    dx = zeros((n, h, w, c))
    D.call("dc_gap_backward", n, h * w, c, dyd.data_ptr(), 0, dx.data_ptr(), stream())
    assert rel_err(host(dx), np.broadcast_to(dy.astype(np.float64) / (h * w), x.shape)) <= 1e-7


BNS = [(2, 5, 5, 64, 0.5), (4, 9, 9, 130, 0.5), (128, 32, 32, 64, 0.5), (64, 112, 112, 64, 0.5),
       (64, 7, 7, 2048, 0.5), (1, 7, 7, 512, 0.5), (3, 5, 5, 4, 0.5), (2, 11, 13, 12, 0.5), (5, 7, 7, 208, 0.5),
       (32, 28, 28, 96, 300.0), (16, 56, 56, 64, -1000.0), (64, 56, 56, 64, -1000.0), (32, 17, 17, 224, 0.5),
       (32, 8, 8, 448, 0.5), (8, 17, 17, 64, 300.0), (4, 8, 8, 68, -1000.0), (10, 32, 32, 16, 0.5)]


@pytest.mark.parametrize("cfg", BNS, ids=[str(b) for b in BNS])
def test_batchnorm(cfg):
    """Includes channel counts off the float4 path (130) and inputs whose mean is far
    larger than their spread (the one-pass statistics must not cancel)."""
    n, h, w, c, mu = cfg
    rows = n * h * w
    x = (synth.random_tensor(15, (n, h, w, c)) * 2 + mu).astype(np.float32)
    gamma = synth.random_tensor(16, (c,))
    beta = synth.random_tensor(17, (c,))
    dy = synth.random_tensor(18, (n, h, w, c))
    acc0 = synth.random_tensor(19, (n, h, w, c))
    ws_t, ws, wsb = scratch(D.lib().dc_batchnorm_workspace_bytes(rows, c))
    xd, gd, bd, dyd = dev(x), dev(gamma), dev(beta), dev(dy)
    y, mean, invstd = zeros((n, h, w, c)), zeros((c,)), zeros((c,))
    D.call("dc_batchnorm_forward", rows, c, xd.data_ptr(), gd.data_ptr(), bd.data_ptr(), ctypes.c_float(1e-5),
           y.data_ptr(), mean.data_ptr(), invstd.data_ptr(), ws, wsb, stream())
    dx = dev(acc0)
    dg, db = zeros((c,)), zeros((c,))
    D.call("dc_batchnorm_backward", rows, c, dyd.data_ptr(), xd.data_ptr(), gd.data_ptr(), mean.data_ptr(),
           invstd.data_ptr(), 1, dx.data_ptr(), dg.data_ptr(), db.data_ptr(), ws, wsb, stream())
    y_ref, xhat, inv_ref = OC.batchnorm_forward(x.astype(np.float64), gamma.astype(np.float64),
                                                beta.astype(np.float64))
    dx_ref, dg_ref, db_ref = OC.batchnorm_backward(dy.astype(np.float64), xhat, inv_ref, gamma.astype(np.float64))
    # the normalisation subtracts the float32 mean: its rounding, up to half an
    # ulp of |mu|, shifts every xhat by that much over the spread (2), a
    # relative error of |mu| 2^-24 / 2 in y, dgamma and dx beside the sums' own
    t = tol(rows) + 4 * abs(mu) * 2.0 ** -24 / 2
    assert rel_err(host(y), y_ref) <= t
    assert rel_err(host(invstd), inv_ref) <= t
    assert rel_err(host(dg), dg_ref) <= t
    assert rel_err(host(db), db_ref) <= t
    assert rel_err(host(dx), dx_ref + acc0) <= 10 * t
    # without a data gradient the parameter gradients are the same, bit for bit
    dg2, db2 = zeros((c,)), zeros((c,))
    D.call("dc_batchnorm_backward", rows, c, dyd.data_ptr(), xd.data_ptr(), gd.data_ptr(), mean.data_ptr(),
           invstd.data_ptr(), 0, None, dg2.data_ptr(), db2.data_ptr(), ws, wsb, stream())
    np.testing.assert_array_equal(host(dg2), host(dg))
    np.testing.assert_array_equal(host(db2), host(db))
    # through a ReLU on the output: the same as the plain backward on the masked gradient, bit for bit
    relu_y = dev(np.maximum(host(y), 0))
    dym = dev(np.where(host(y) > 0, dy, 0).astype(np.float32))
    dx_r, dx_m = zeros((n, h, w, c)), zeros((n, h, w, c))
    dg_r, db_r, dg_m, db_m = zeros((c,)), zeros((c,)), zeros((c,)), zeros((c,))
    D.call("dc_batchnorm_backward_relu", rows, c, dyd.data_ptr(), relu_y.data_ptr(), xd.data_ptr(), gd.data_ptr(),
           mean.data_ptr(), invstd.data_ptr(), 0, dx_r.data_ptr(), dg_r.data_ptr(), db_r.data_ptr(), ws, wsb,
           stream())
    D.call("dc_batchnorm_backward", rows, c, dym.data_ptr(), xd.data_ptr(), gd.data_ptr(), mean.data_ptr(),
           invstd.data_ptr(), 0, dx_m.data_ptr(), dg_m.data_ptr(), db_m.data_ptr(), ws, wsb, stream())
    np.testing.assert_array_equal(host(dx_r), host(dx_m))
    np.testing.assert_array_equal(host(dg_r), host(dg_m))
    np.testing.assert_array_equal(host(db_r), host(db_m))


@pytest.mark.parametrize("n,classes", [(4, 10), (32, 1000), (128, 10), (3, 257)])
def test_softmax_xent(n, classes):
    z = synth.random_tensor(20, (n, classes)) * 3
    y = np.random.default_rng(n).integers(0, classes, n).astype(np.int32)
    ws_t, ws, wsb = scratch(D.lib().dc_softmax_xent_workspace_bytes(n))
    loss = zeros((1,))
    dz = zeros((n, classes))
    zd, yd = dev(z), dev(y)  # keep the inputs alive until the kernel has run
    D.call("dc_softmax_xent", n, classes, zd.data_ptr(), yd.data_ptr(), loss.data_ptr(), dz.data_ptr(),
           ws, wsb, stream())
    l_ref, dz_ref = OC.softmax_xent(z.astype(np.float64), y)
    assert abs(host(loss)[0] - l_ref) <= 1e-6 * abs(l_ref)
    assert rel_err(host(dz), dz_ref) <= 1e-6


@pytest.mark.parametrize("cfg", [(10, (4, 8, 12, 4)), (7, (3, 5, 2)), (32 * 28 * 28, (64, 128, 32, 32))])
def test_concat(cfg):
    rows, parts = cfg
    cout = sum(parts)
    xs = [synth.random_tensor(30 + i, (rows, c)) for i, c in enumerate(parts)]
    xds = [dev(x) for x in xs]
    y = zeros((rows, cout))
    off = 0
    for c, xd in zip(parts, xds):
        D.call("dc_concat_forward", rows, c, cout, off, xd.data_ptr(), y.data_ptr(), stream())
        off += c
    np.testing.assert_array_equal(host(y), np.concatenate(xs, axis=1))
    dy = synth.random_tensor(40, (rows, cout))
    dyd = dev(dy)
    off = 0
    for i, c in enumerate(parts):
        acc0 = synth.random_tensor(50 + i, (rows, c))
        dx = dev(acc0)
        D.call("dc_concat_backward", rows, c, cout, off, dyd.data_ptr(), 1, dx.data_ptr(), stream())
        np.testing.assert_array_equal(host(dx), (acc0 + dy[:, off:off + c]).astype(np.float32))
        off += c
    assert D.lib().dc_concat_forward(rows, parts[0], cout, cout, None, None, None) == D.DC_EINVAL


@pytest.mark.parametrize("cfg", [(10, (4, 8, 12, 4)), (7, (3, 5, 2)), (32 * 28 * 28, (64, 128, 32, 32))])
def test_concat_backward_relu(cfg):
    """The concatenation's backward with the ReLU that produced a part folded in:
    dx (+)= dy's slice where the ReLU's output is positive, bit for bit, written and
    accumulated, on the float4 and per-channel kernels."""
    rows, parts = cfg
    cout = sum(parts)
    dy = synth.random_tensor(60, (rows, cout))
    dyd = dev(dy)
    off = 0
    for i, c in enumerate(parts):
        relu_y = np.maximum(synth.random_tensor(61 + i, (rows, c)), 0.0).astype(np.float32)
        g = np.where(relu_y > 0, dy[:, off:off + c], np.float32(0.0)).astype(np.float32)
        yd = dev(relu_y)
        dx = zeros((rows, c))
        D.call("dc_concat_backward_relu", rows, c, cout, off, dyd.data_ptr(), yd.data_ptr(), 0, dx.data_ptr(),
               stream())
        np.testing.assert_array_equal(host(dx), g)
        acc0 = synth.random_tensor(70 + i, (rows, c))
        dxa = dev(acc0)
        D.call("dc_concat_backward_relu", rows, c, cout, off, dyd.data_ptr(), yd.data_ptr(), 1, dxa.data_ptr(),
               stream())
        np.testing.assert_array_equal(host(dxa), (acc0 + g).astype(np.float32))
        off += c


@pytest.mark.parametrize("n", [1, 7, 4096 + 3, 32 * 56 * 56 * 64])
def test_add_relu_backward(n):
    """Backward of relu(a + b): m = dy where y > 0, written to one input's gradient
    and accumulated into the other's (and the reverse), or to one of them alone,
    bit for bit, on the float4 body and the scalar tail."""
    dy = synth.random_tensor(80, (n,))
    y = np.maximum(synth.random_tensor(81, (n,)), 0.0).astype(np.float32)
    m = np.where(y > 0, dy, np.float32(0.0)).astype(np.float32)
    acc = synth.random_tensor(82, (n,))
    dyd, yd = dev(dy), dev(y)
    for acc0, acc1 in ((0, 1), (1, 0)):
        d0 = dev(acc) if acc0 else zeros((n,))
        d1 = dev(acc) if acc1 else zeros((n,))
        D.call("dc_add_relu_backward", dyd.data_ptr(), yd.data_ptr(), acc0, d0.data_ptr(), acc1, d1.data_ptr(), n,
               stream())
        np.testing.assert_array_equal(host(d0), (acc + m).astype(np.float32) if acc0 else m)
        np.testing.assert_array_equal(host(d1), (acc + m).astype(np.float32) if acc1 else m)
    d0 = dev(acc)
    D.call("dc_add_relu_backward", dyd.data_ptr(), yd.data_ptr(), 1, d0.data_ptr(), 0, None, n, stream())
    np.testing.assert_array_equal(host(d0), (acc + m).astype(np.float32))
