"""Pins for the oracle CNN iteration.

* Forward operators against torch's CPU float64 library routines (conv2d with
  stride and padding, max_pool2d with padding, batch_norm in training mode,
  adaptive average pooling) - special cases that reduce to a library routine.
* Backward operators against torch autograd in float64 on the same inputs.
* Whole-network gradients against central finite differences in float64, on
  the tiny workload and on a small residual network that has every operator
  (BN, stride-2 conv, 1x1 projection, residual add, padded 3x3/2 max-pool,
  global average pooling).
* Closed forms: with the last FC zeroed the loss is exactly ln(classes) and
  the last bias gradient is (1/classes - onehot) averaged over the batch; the
  server update is w - 0.01 g.
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import cnn, nets


def _nchw(a):
    return torch.from_numpy(np.ascontiguousarray(a.transpose(0, 3, 1, 2)))


def _nhwc(t):
    return t.detach().numpy().transpose(0, 2, 3, 1)


@pytest.mark.parametrize("shape", [
    # N, H, W, C, K, R, stride, pad
    (2, 9, 7, 3, 5, 3, 1, 1),
    (2, 11, 11, 4, 6, 3, 2, 1),
    (1, 23, 23, 3, 4, 11, 4, 2),
    (3, 8, 8, 6, 7, 1, 2, 0),
    (2, 14, 14, 3, 8, 7, 2, 3),
    (2, 6, 6, 5, 3, 5, 1, 2),
])
def test_conv_against_torch(shape):
    N, H, W, C, K, R, st, pad = shape
    x = synth.random_tensor(1, (N, H, W, C)).astype(np.float64)
    w = synth.random_tensor(2, (K, R, R, C)).astype(np.float64)
    b = synth.random_tensor(3, (K,)).astype(np.float64)
    y = cnn.conv2d_forward(x, w, b, st, pad)
    xt = _nchw(x).requires_grad_(True)
    wt = torch.from_numpy(np.ascontiguousarray(w.transpose(0, 3, 1, 2))).requires_grad_(True)
    yt = torch.nn.functional.conv2d(xt, wt, torch.from_numpy(b), stride=st, padding=pad)
    np.testing.assert_allclose(y, _nhwc(yt), rtol=1e-12, atol=1e-12)
    dy = synth.random_tensor(4, y.shape).astype(np.float64)
    yt.backward(_nchw(dy))
    dx = cnn.conv2d_backward_data(dy, w, (H, W), st, pad)
    dw = cnn.conv2d_backward_filter(x, dy, (R, R), st, pad)
    np.testing.assert_allclose(dx, _nhwc(xt.grad), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, wt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("shape", [
    # N, H, W, C, K, R, S, stride, pad rows, pad columns
    (2, 9, 8, 3, 5, 1, 7, 1, 0, 3),
    (2, 9, 8, 4, 3, 7, 1, 1, 3, 0),
    (2, 11, 10, 3, 4, 1, 3, 2, 0, 1),
    (1, 8, 9, 2, 3, 3, 1, 1, 1, 0),
    (2, 7, 7, 3, 2, 3, 5, 2, 1, 2),
    (1, 7, 9, 2, 3, 3, 3, 2, 0, 0),
])
def test_conv_asymmetric_against_torch(shape):
    """Rectangular filters with separate row and column padding (the 1 x n / n x 1 convs)."""
    N, H, W, C, K, R, S, st, ph, pw = shape
    x = synth.random_tensor(21, (N, H, W, C)).astype(np.float64)
    w = synth.random_tensor(22, (K, R, S, C)).astype(np.float64)
    b = synth.random_tensor(23, (K,)).astype(np.float64)
    y = cnn.conv2d_forward(x, w, b, st, (ph, pw))
    xt = _nchw(x).requires_grad_(True)
    wt = torch.from_numpy(np.ascontiguousarray(w.transpose(0, 3, 1, 2))).requires_grad_(True)
    yt = torch.nn.functional.conv2d(xt, wt, torch.from_numpy(b), stride=st, padding=(ph, pw))
    np.testing.assert_allclose(y, _nhwc(yt), rtol=1e-12, atol=1e-12)
    dy = synth.random_tensor(24, y.shape).astype(np.float64)
    yt.backward(_nchw(dy))
    dx = cnn.conv2d_backward_data(dy, w, (H, W), st, (ph, pw))
    dw = cnn.conv2d_backward_filter(x, dy, (R, S), st, (ph, pw))
    np.testing.assert_allclose(dx, _nhwc(xt.grad), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, wt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-11, atol=1e-11)
    # the sampled evaluations follow the same geometry
    geom = (N, H, W, C, K, R, S, st, ph, pw)
    idx = np.array([[n, p, q, k] for n in range(N) for p in range(y.shape[1]) for q in range(y.shape[2])
                    for k in range(K)][::3])
    got = cnn.conv2d_samples("fwd", geom, x.astype(np.float32), w.astype(np.float32), idx,
                             bias=b.astype(np.float32))
    ref = cnn.conv2d_forward(x.astype(np.float32), w.astype(np.float32), b.astype(np.float32), st, (ph, pw))
    np.testing.assert_allclose(got, ref[tuple(idx.T)], rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("cfg", [(3, 1, 1, 7, 7), (3, 1, 1, 5, 8), (2, 2, 0, 8, 6), (3, 2, 1, 9, 9), (5, 3, 2, 11, 10)])
def test_avgpool_against_torch(cfg):
    """Average pooling, padded taps left out of the count."""
    r, st, pad, H, W = cfg
    x = synth.random_tensor(25, (2, H, W, 3)).astype(np.float64)
    y = cnn.avgpool_forward(x, r, r, st, pad)
    xt = _nchw(x).requires_grad_(True)
    yt = torch.nn.functional.avg_pool2d(xt, r, st, pad, count_include_pad=False)
    np.testing.assert_allclose(y, _nhwc(yt), rtol=1e-13, atol=1e-13)
    dy = synth.random_tensor(26, y.shape).astype(np.float64)
    yt.backward(_nchw(dy))
    dx = cnn.avgpool_backward(dy, x.shape, r, r, st, pad)
    np.testing.assert_allclose(dx, _nhwc(xt.grad), rtol=1e-13, atol=1e-13)


def test_avgpool_closed_forms():
    """A constant image pools to itself (corners included, since padding is not
    counted); each window spreads its gradient with weights summing to one, so
    the input gradient sums to the output gradient's sum; with a 1 x 1 window
    the pool is the identity."""
    x = np.full((2, 6, 5, 3), 2.5)
    np.testing.assert_array_equal(cnn.avgpool_forward(x, 3, 3, 1, 1), x)
    dy = synth.random_tensor(27, (2, 6, 5, 3)).astype(np.float64)
    dx = cnn.avgpool_backward(dy, x.shape, 3, 3, 1, 1)
    np.testing.assert_allclose(dx.sum(axis=(1, 2)), dy.sum(axis=(1, 2)), rtol=1e-13)
    # the corner input is covered by 4 windows of 4, 6, 6 and 9 in-image taps
    w = dy[0, 0, 0, 0] / 4 + dy[0, 0, 1, 0] / 6 + dy[0, 1, 0, 0] / 6 + dy[0, 1, 1, 0] / 9
    assert dx[0, 0, 0, 0] == pytest.approx(w, rel=1e-14)
    x = synth.random_tensor(28, (1, 4, 4, 2)).astype(np.float64)
    np.testing.assert_array_equal(cnn.avgpool_forward(x, 1, 1, 1, 0), x)


@pytest.mark.parametrize("cfg", [(2, 2, 0, 8), (3, 2, 0, 13), (3, 2, 1, 12), (3, 2, 0, 55)])
def test_maxpool_against_torch(cfg):
    r, st, pad, H = cfg
    x = synth.random_tensor(5, (2, H, H, 3)).astype(np.float64)
    y, arg = cnn.maxpool_forward(x, r, r, st, pad)
    xt = _nchw(x).requires_grad_(True)
    yt = torch.nn.functional.max_pool2d(xt, r, st, pad)
    np.testing.assert_array_equal(y, _nhwc(yt))
    dy = synth.random_tensor(6, y.shape).astype(np.float64)
    yt.backward(_nchw(dy))
    dx = cnn.maxpool_backward(dy, arg, x.shape, r, r, st, pad)
    np.testing.assert_allclose(dx, _nhwc(xt.grad), rtol=1e-13, atol=1e-13)


def test_maxpool_ties_pick_first():
    x = np.zeros((1, 4, 4, 1))
    x[0, 1, 1, 0] = 0.0
    y, arg = cnn.maxpool_forward(x, 2, 2, 2, 0)
    assert (arg == 0).all()
    # values that only differ below float32 resolution count as a tie
    x = np.zeros((1, 2, 2, 1))
    x[0, 0, 1, 0] = 1e-60
    y, arg = cnn.maxpool_forward(x, 2, 2, 2, 0)
    assert arg[0, 0, 0, 0] == 0


def test_batchnorm_against_torch():
    x = (synth.random_tensor(7, (3, 5, 4, 6)) * 3 + 1).astype(np.float64)
    gamma = synth.random_tensor(8, (6,)).astype(np.float64)
    beta = synth.random_tensor(9, (6,)).astype(np.float64)
    y, xhat, invstd = cnn.batchnorm_forward(x, gamma, beta)
    xt = _nchw(x).requires_grad_(True)
    gt = torch.from_numpy(gamma).requires_grad_(True)
    bt = torch.from_numpy(beta).requires_grad_(True)
    yt = torch.nn.functional.batch_norm(xt, None, None, gt, bt, training=True, eps=cnn.BN_EPS)
    np.testing.assert_allclose(y, _nhwc(yt), rtol=1e-12, atol=1e-12)
    dy = synth.random_tensor(10, y.shape).astype(np.float64)
    yt.backward(_nchw(dy))
    dx, dg, db = cnn.batchnorm_backward(dy, xhat, invstd, gamma)
    np.testing.assert_allclose(dx, _nhwc(xt.grad), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_softmax_xent_against_torch():
    z = synth.random_tensor(11, (5, 7)).astype(np.float64) * 4
    y = np.array([0, 6, 3, 3, 1])
    loss, dz = cnn.softmax_xent(z, y)
    zt = torch.from_numpy(z).requires_grad_(True)
    lt = torch.nn.functional.cross_entropy(zt, torch.from_numpy(y))
    lt.backward()
    assert abs(loss - lt.item()) < 1e-13
    np.testing.assert_allclose(dz, zt.grad.numpy(), rtol=1e-12, atol=1e-14)


def _mini_resnet():
    """Small network with every operator kind, for finite differences."""
    ops = []

    def add(kind, inp, layer, **kw):
        d = {"op": kind, "in": inp, "layer": layer}
        d.update(kw)
        ops.append(d)
        return len(ops)

    t = add("conv", 0, 1, k=4, r=3, s=3, stride=1, pad=1, bias=False)
    t = add("bn", t, 1)
    t = add("relu", t, 1)
    t = add("maxpool", t, 1, r=3, s=3, stride=2, pad=1)
    x = t
    u = add("conv", x, 2, k=6, r=3, s=3, stride=2, pad=1, bias=False)
    u = add("bn", u, 2)
    u = add("relu", u, 2)
    sc = add("conv", x, 2, k=6, r=1, s=1, stride=2, pad=0, bias=False)
    sc = add("bn", sc, 2)
    u = add("conv", u, 3, k=6, r=3, s=3, stride=1, pad=1, bias=True)
    u = add("bn", u, 3)
    u = add("add", u, 3, other=sc)
    u = add("relu", u, 3)
    u = add("gap", u, 3)
    add("fc", u, 4, out=5, bias=True)
    return {"name": "mini", "ops": ops, "hwc": (10, 10, 3), "classes": 5}


def _mini_inception():
    """Two Inception-style modules (four branches, concat) at small size."""
    ops = []

    def add(kind, inp, layer, **kw):
        d = {"op": kind, "in": inp, "layer": layer}
        d.update(kw)
        ops.append(d)
        return len(ops)

    t = add("relu", add("conv", 0, 1, k=6, r=3, s=3, stride=1, pad=1, bias=True), 1)
    layer = 1
    for c1, r3, c3, r5, c5, pp in ((3, 2, 4, 2, 3, 2), (2, 3, 3, 1, 2, 3)):
        layer += 1
        b1 = add("relu", add("conv", t, layer, k=c1, r=1, s=1, stride=1, pad=0, bias=True), layer)
        b3 = add("relu", add("conv", t, layer, k=r3, r=1, s=1, stride=1, pad=0, bias=True), layer)
        b5 = add("relu", add("conv", t, layer, k=r5, r=1, s=1, stride=1, pad=0, bias=True), layer)
        bp = add("maxpool", t, layer, r=3, s=3, stride=1, pad=1)
        bp = add("relu", add("conv", bp, layer, k=pp, r=1, s=1, stride=1, pad=0, bias=True), layer)
        layer += 1
        b3 = add("relu", add("conv", b3, layer, k=c3, r=3, s=3, stride=1, pad=1, bias=True), layer)
        b5 = add("relu", add("conv", b5, layer, k=c5, r=5, s=5, stride=1, pad=2, bias=True), layer)
        t = add("concat", b1, layer, others=[b3, b5, bp])
    t = add("gap", t, layer)
    add("fc", t, layer + 1, out=4, bias=True)
    return {"name": "mini_inception", "ops": ops, "hwc": (7, 7, 3), "classes": 4}


def _mini_inception_v4():
    """Inception-v4 operators at small size: unpadded stride-2 conv and max-pool
    reduction, 1 x 3 / 3 x 1 and 1 x 7 / 7 x 1 convs with one-sided padding, an
    average-pool branch, a split into parallel convs, BN + ReLU after every
    conv, concatenation, global average pooling."""
    ops = []

    def add(kind, inp, layer, **kw):
        d = {"op": kind, "in": inp, "layer": layer}
        d.update(kw)
        ops.append(d)
        return len(ops)

    def cbr(inp, layer, k, r, s, stride, ph, pw):
        t = add("conv", inp, layer, k=k, r=r, s=s, stride=stride, pad=ph, pad_w=pw, bias=False)
        return add("relu", add("bn", t, layer), layer)

    t = cbr(0, 1, 5, 3, 3, 2, 0, 0)                        # 11x11 -> 5x5
    a = add("avgpool", t, 2, r=3, s=3, stride=1, pad=1)
    a = cbr(a, 2, 3, 1, 1, 1, 0, 0)
    u = cbr(t, 2, 4, 1, 1, 1, 0, 0)
    v = cbr(t, 2, 3, 1, 1, 1, 0, 0)
    u = cbr(u, 3, 4, 1, 7, 1, 0, 3)
    v1 = cbr(v, 3, 2, 1, 3, 1, 0, 1)
    v2 = cbr(v, 3, 2, 3, 1, 1, 1, 0)
    u = cbr(u, 4, 3, 7, 1, 1, 3, 0)
    t = add("concat", a, 4, others=[u, v1, v2])
    m = add("maxpool", t, 5, r=3, s=3, stride=2, pad=0)     # 5x5 -> 2x2
    c = cbr(t, 5, 4, 3, 3, 2, 0, 0)
    t = add("concat", m, 5, others=[c])
    t = add("gap", t, 5)
    add("fc", t, 6, out=4, bias=True)
    return {"name": "mini_inception_v4", "ops": ops, "hwc": (11, 11, 3), "classes": 4}


def test_finite_differences_inception_v4_ops():
    _fd_check(_mini_inception_v4(), 2, 9, 100, 1e-6)


def test_inception_v4_ops_against_torch():
    spec = _mini_inception_v4()
    net = cnn.Net(spec, 3)
    x, y, p = synth.cnn_inputs(10, 3, spec["hwc"], spec["classes"], net.param_specs)
    loss, g = net.loss_and_grads(x, y, p)
    lt, gt = _torch_loss(spec, net, x, y, p)
    assert abs(loss - lt) <= 1e-12 * max(1.0, abs(lt))
    np.testing.assert_allclose(g, gt, rtol=1e-9, atol=1e-12 * np.abs(gt).max())


def test_finite_differences_inception():
    _fd_check(_mini_inception(), 2, 4, 80, 1e-6)


def test_inception_against_torch():
    spec = _mini_inception()
    net = cnn.Net(spec, 3)
    x, y, p = synth.cnn_inputs(5, 3, spec["hwc"], spec["classes"], net.param_specs)
    loss, g = net.loss_and_grads(x, y, p)
    lt, gt = _torch_loss(spec, net, x, y, p)
    assert abs(loss - lt) <= 1e-12 * max(1.0, abs(lt))
    np.testing.assert_allclose(g, gt, rtol=1e-9, atol=1e-12 * np.abs(gt).max())


def _fd_check(spec, batch, seed, n_probe, rel):
    net = cnn.Net(spec, batch)
    x, y, p = synth.cnn_inputs(seed, batch, spec["hwc"], spec["classes"], net.param_specs)
    p = p.astype(np.float64)
    loss, g = net.loss_and_grads(x, y, p)
    rng = np.random.default_rng(seed + 100)
    idx = set(rng.choice(net.n_params, size=n_probe, replace=False).tolist())
    for l in range(1, net.L + 1):   # probe every layer's first and last parameter too
        lo, cnt = net.layer_ranges[l]
        idx.update((lo, lo + cnt - 1))
    gmax = np.abs(g).max()
    for i in sorted(idx):
        h = 1e-6 * max(1.0, abs(p[i]))
        pp, pm = p.copy(), p.copy()
        pp[i] += h
        pm[i] -= h
        fd = (net.loss(x, y, pp) - net.loss(x, y, pm)) / (2 * h)
        assert abs(fd - g[i]) <= rel * gmax + 1e-7 * abs(g[i]), (i, fd, g[i])
    return loss


def test_finite_differences_tiny():
    _fd_check(nets.tiny(), 2, 0, 60, 1e-6)


def test_finite_differences_all_operators():
    _fd_check(_mini_resnet(), 3, 1, 120, 1e-6)


def test_zero_last_fc_gives_ln_classes():
    spec = nets.tiny()
    net = cnn.Net(spec, 4)
    x, y, p = synth.cnn_inputs(0, 4, spec["hwc"], spec["classes"], net.param_specs)
    lo, cnt = net.layer_ranges[net.L]
    p = p.astype(np.float64)
    p[lo:lo + cnt] = 0.0
    loss, g = net.loss_and_grads(x, y, p)
    assert loss == pytest.approx(math.log(10), abs=1e-15)
    onehot = np.zeros((4, 10))
    onehot[np.arange(4), y] = 1
    db = (1.0 / 10 - onehot).mean(axis=0)
    np.testing.assert_allclose(g[lo + cnt - 10:lo + cnt], db, rtol=0, atol=1e-15)


def test_sgd_closed_form():
    w = synth.random_tensor(12, (100,))
    g = synth.random_tensor(13, (100,))
    np.testing.assert_array_equal(cnn.sgd(w, g), w.astype(np.float64) - 0.01 * g.astype(np.float64))


@pytest.mark.parametrize("name,count", [("tiny", 67642), ("alexnet", 61100840), ("resnet18", 11173962),
                                        ("vgg16", 138357544), ("resnet50", 25557032), ("googlenet", 6998552),
                                        ("vgg19", 143667240), ("resnet152", 60192808),
                                        ("inception_v4", 42679816)])
def test_parameter_counts(name, count):
    net = cnn.Net(nets.get(name), 1)
    assert net.n_params == count
    assert sum(c for _, c in net.layer_ranges.values()) == count
    assert {"tiny": 4, "alexnet": 8, "resnet18": 18, "vgg16": 16, "resnet50": 50, "googlenet": 22, "vgg19": 19,
            "resnet152": 152, "inception_v4": 76}[name] == net.L


def _torch_loss(spec, net, x, y, p):
    """The same network evaluated with torch float64 library routines."""
    from tests import torch_ref
    return torch_ref.loss_and_grads(spec, net, x, y, p, torch.float64)


@pytest.mark.parametrize("which", ["tiny", "mini"])
def test_network_against_torch(which):
    spec = nets.tiny() if which == "tiny" else _mini_resnet()
    batch = 3
    net = cnn.Net(spec, batch)
    x, y, p = synth.cnn_inputs(3, batch, spec["hwc"], spec["classes"], net.param_specs)
    loss, g = net.loss_and_grads(x, y, p)
    lt, gt = _torch_loss(spec, net, x, y, p)
    assert abs(loss - lt) <= 1e-12 * max(1.0, abs(lt))
    np.testing.assert_allclose(g, gt, rtol=1e-9, atol=1e-12 * np.abs(gt).max())


@pytest.mark.slow
def test_resnet18_against_torch():
    spec = nets.resnet18_small()
    net = cnn.Net(spec, 2)
    x, y, p = synth.cnn_inputs(2, 2, spec["hwc"], spec["classes"], net.param_specs)
    loss, g = net.loss_and_grads(x, y, p)
    lt, gt = _torch_loss(spec, net, x, y, p)
    assert abs(loss - lt) <= 1e-11 * max(1.0, abs(lt))
    np.testing.assert_allclose(g, gt, rtol=1e-8, atol=1e-11 * np.abs(gt).max())


@pytest.mark.parametrize("shape", [(2, 9, 7, 3, 5, 3, 1, 1), (2, 11, 11, 4, 6, 3, 2, 1), (1, 23, 23, 3, 4, 11, 4, 2),
                                   (3, 8, 8, 6, 7, 1, 2, 0)])
def test_conv_samples_match_whole_tensors(shape):
    """The one-output-at-a-time sums equal the whole-tensor ones at every index."""
    N, H, W, C, K, R, st, pad = shape
    x = synth.random_tensor(21, (N, H, W, C))
    w = synth.random_tensor(22, (K, R, R, C))
    b = synth.random_tensor(23, (K,))
    y = cnn.conv2d_forward(x, w, b, st, pad)
    dy = synth.random_tensor(24, y.shape)
    geom = (N, H, W, C, K, R, R, st, pad)
    idx = np.argwhere(np.ones(y.shape, dtype=bool))
    np.testing.assert_allclose(cnn.conv2d_samples("fwd", geom, x, w, idx, b), y.reshape(-1), rtol=1e-14, atol=1e-13)
    dx = cnn.conv2d_backward_data(dy, w, (H, W), st, pad)
    idx = np.argwhere(np.ones(dx.shape, dtype=bool))
    np.testing.assert_allclose(cnn.conv2d_samples("dgrad", geom, dy, w, idx), dx.reshape(-1), rtol=1e-14, atol=1e-13)
    dw = cnn.conv2d_backward_filter(x, dy, (R, R), st, pad)
    idx = np.argwhere(np.ones(dw.shape, dtype=bool))
    np.testing.assert_allclose(cnn.conv2d_samples("wgrad", geom, x, dy, idx), dw.reshape(-1), rtol=1e-14, atol=1e-13)


# ---------------------------------------------------------------- given decisions
# The oracle can take the ReLU masks and max-pool window taps as given (the
# GPU's, in the test that compares arithmetic apart from decision flips).


def test_maxpool_at_takes_the_given_taps():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 9, 7, 3))
    for r, st, pad in ((3, 2, 1), (2, 2, 0), (3, 1, 1)):
        y, arg = cnn.maxpool_forward(x, r, r, st, pad)
        np.testing.assert_array_equal(cnn.maxpool_at(x, arg, r, r, st, pad), y)
    # tap 4 of a 3x3 window at stride 2 with padding 1 is the pixel (2p, 2q)
    y = cnn.maxpool_at(x, np.full((2, 5, 4, 3), 4), 3, 3, 2, 1)
    np.testing.assert_array_equal(y, x[:, ::2, ::2, :])
    with pytest.raises(AssertionError):
        cnn.maxpool_at(x, np.zeros((2, 5, 4, 3), dtype=int), 3, 3, 2, 1)  # tap 0 of window (0, 0) is padding


def test_given_decisions_equal_to_its_own_reproduce_the_iteration():
    spec = _mini_resnet()
    net = cnn.Net(spec, 3)
    x, y, p = synth.cnn_inputs(8, 3, spec["hwc"], spec["classes"], net.param_specs)
    loss, g, t, cache, _ = net.loss_and_grads(x, y, p, keep=True)
    dec = {i: cache[i] for i, op in enumerate(net.ops) if op["op"] in ("relu", "maxpool")}
    assert len(dec) == sum(op["op"] in ("relu", "maxpool") for op in net.ops)
    loss2, g2 = net.loss_and_grads(x, y, p, decisions=dec)
    assert loss2 == loss
    np.testing.assert_array_equal(g2, g)
    from tests import torch_ref
    lt, gt = torch_ref.loss_and_grads(spec, net, x, y, p, torch.float64, decisions=dec)
    assert abs(loss - lt) <= 1e-12 * max(1.0, abs(lt))
    np.testing.assert_allclose(g, gt, rtol=1e-9, atol=1e-12 * np.abs(gt).max())


def test_given_decisions_against_a_network_without_them():
    """Every ReLU told to pass everything and every 2x2/2 max-pool told to take tap 0 is the
    same network with those ops replaced by identity (1x1 average pooling, stride 1) and by
    stride-2 subsampling (1x1 average pooling, stride 2): bit for bit."""
    spec = nets.tiny()
    lin = dict(spec, ops=[dict(op) for op in spec["ops"]])
    for op in lin["ops"]:
        if op["op"] == "relu":
            op.update(op="avgpool", r=1, s=1, stride=1, pad=0)
        elif op["op"] == "maxpool":
            assert (op["r"], op["s"], op["stride"], op["pad"]) == (2, 2, 2, 0)
            op.update(op="avgpool", r=1, s=1, stride=2, pad=0)
    batch = 3
    a, b = cnn.Net(spec, batch), cnn.Net(lin, batch)
    x, y, p = synth.cnn_inputs(9, batch, spec["hwc"], spec["classes"], a.param_specs)
    dec = {}
    for i, op in enumerate(a.ops):
        if op["op"] == "relu":
            dec[i] = np.ones(a.shapes[op["in"]], dtype=bool)
        elif op["op"] == "maxpool":
            dec[i] = np.zeros(a.shapes[i + 1], dtype=np.int32)
    la, ga = a.loss_and_grads(x, y, p, decisions=dec)
    lb, gb = b.loss_and_grads(x, y, p)
    assert la == lb
    np.testing.assert_array_equal(ga, gb)
    # torch's float64 routines with the same decisions given (the float32 yardstick's path)
    from tests import torch_ref
    lt, gt = torch_ref.loss_and_grads(spec, a, x, y, p, torch.float64, decisions=dec)
    assert abs(la - lt) <= 1e-12 * abs(lt)
    np.testing.assert_allclose(ga, gt, rtol=1e-9, atol=1e-12 * np.abs(gt).max())
    # and the decisions matter: the network's own ones give another iteration
    assert a.loss_and_grads(x, y, p)[0] != la
