"""Oracle CNN training iteration (test infrastructure only).

A plain CPU implementation of what one worker computes between pulling the
parameters and pushing the gradients in the parameter-server iteration of
Sec. III-A (pull, forward, backward, push), and of the server's update:

* forward: convolution (its row and column padding may differ), FC,
  BatchNorm (training mode, batch statistics), ReLU, max-pooling, average
  pooling (padded taps excluded from the count), global average pooling,
  residual add, channel concatenation;
* loss: mean over the batch of the softmax cross-entropy;
* backward by the chain rule, giving the gradient of every parameter;
* the server's SGD update w <- w - lr * g.

Everything is float64.  Convolutions and max-pooling run in the C loops of
``cnn.c`` (built by ``oracle/build.py``); the rest are numpy expressions of
the definitions.  Decisions that floating point takes (the ReLU sign, the
max-pool argmax) are taken on the values rounded to float32, or, when the
caller passes them (``decisions``), taken as given: a parity check can then
hand the oracle another implementation's decisions and compare the arithmetic
alone, apart from the decisions that float32 rounding flips near a tie.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may use this module.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle_cnn.so")
_lib = None

BN_EPS = 1e-5
LR = 0.01


def lib():
    """Load the compiled oracle loops (build them with ``python -m oracle.build``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"oracle library missing: {LIB_PATH}; run `python -m oracle.build`")
        L = ctypes.CDLL(LIB_PATH)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int)
        i = ctypes.c_int
        L.or_conv2d_forward.argtypes = [i] * 12 + [dp, dp, dp, dp]
        L.or_conv2d_backward_data.argtypes = [i] * 12 + [dp, dp, dp]
        L.or_conv2d_backward_filter.argtypes = [i] * 12 + [dp, dp, dp]
        L.or_maxpool_forward.argtypes = [i] * 10 + [dp, dp, ip]
        L.or_maxpool_backward.argtypes = [i] * 10 + [dp, ip, dp]
        fp = ctypes.POINTER(ctypes.c_float)
        L.or_conv2d_forward_samples.argtypes = [i] * 12 + [fp, fp, fp, i, ip, dp]
        L.or_conv2d_backward_data_samples.argtypes = [i] * 12 + [fp, fp, i, ip, dp]
        L.or_conv2d_backward_filter_samples.argtypes = [i] * 12 + [fp, fp, i, ip, dp]
        for f in ("or_conv2d_forward", "or_conv2d_backward_data", "or_conv2d_backward_filter",
                  "or_maxpool_forward", "or_maxpool_backward", "or_conv2d_forward_samples",
                  "or_conv2d_backward_data_samples", "or_conv2d_backward_filter_samples"):
            getattr(L, f).restype = None
        _lib = L
    return _lib


def _dp(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double)) if a is not None else None


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def conv_out(h, r, st, pad):
    return (h + 2 * pad - r) // st + 1


def _pads(pad):
    """Padding given as one int (rows and columns alike) or as (rows, columns)."""
    if isinstance(pad, (tuple, list)):
        return int(pad[0]), int(pad[1])
    return int(pad), int(pad)


# ---------------------------------------------------------------- primitives

def conv2d_forward(x, w, b, st, pad):
    """y[n,p,q,k] = b[k] + sum_{r,s,c} x[n,p*st+r-ph,q*st+s-pw,c] w[k,r,s,c], (ph, pw) = pad."""
    x, w = _f64(x), _f64(w)
    N, H, W, C = x.shape
    K, R, S, C2 = w.shape
    assert C == C2
    ph, pw = _pads(pad)
    P, Q = conv_out(H, R, st, ph), conv_out(W, S, st, pw)
    y = np.empty((N, P, Q, K))
    bb = _f64(b) if b is not None else None
    lib().or_conv2d_forward(N, H, W, C, K, R, S, st, ph, pw, P, Q, _dp(x), _dp(w), _dp(bb), _dp(y))
    return y


def conv2d_backward_data(dy, w, in_hw, st, pad):
    dy, w = _f64(dy), _f64(w)
    N, P, Q, K = dy.shape
    K2, R, S, C = w.shape
    assert K == K2
    H, W = in_hw
    dx = np.empty((N, H, W, C))
    ph, pw = _pads(pad)
    lib().or_conv2d_backward_data(N, H, W, C, K, R, S, st, ph, pw, P, Q, _dp(dy), _dp(w), _dp(dx))
    return dx


def conv2d_backward_filter(x, dy, rs, st, pad):
    x, dy = _f64(x), _f64(dy)
    N, H, W, C = x.shape
    N2, P, Q, K = dy.shape
    R, S = rs
    dw = np.empty((K, R, S, C))
    ph, pw = _pads(pad)
    lib().or_conv2d_backward_filter(N, H, W, C, K, R, S, st, ph, pw, P, Q, _dp(x), _dp(dy), _dp(dw))
    return dw


def maxpool_forward(x, r, s, st, pad):
    x = _f64(x)
    N, H, W, C = x.shape
    P, Q = conv_out(H, r, st, pad), conv_out(W, s, st, pad)
    y = np.empty((N, P, Q, C))
    arg = np.empty((N, P, Q, C), dtype=np.int32)
    lib().or_maxpool_forward(N, H, W, C, r, s, st, pad, P, Q, _dp(x), _dp(y),
                             arg.ctypes.data_as(ctypes.POINTER(ctypes.c_int)))
    return y, arg


def maxpool_at(x, arg, r, s, st, pad):
    """The max-pool forward with given window taps: y[n,p,q,c] = x at tap arg = r' * s + s' of the
    window at (p*st - pad, q*st - pad); every tap must lie inside the image."""
    x = _f64(x)
    N, H, W, C = x.shape
    P, Q = conv_out(H, r, st, pad), conv_out(W, s, st, pad)
    arg = np.asarray(arg).reshape(N, P, Q, C)
    h = np.arange(P)[None, :, None, None] * st + arg // s - pad
    w = np.arange(Q)[None, None, :, None] * st + arg % s - pad
    assert (h >= 0).all() and (h < H).all() and (w >= 0).all() and (w < W).all(), "a tap outside the image"
    n = np.arange(N)[:, None, None, None]
    c = np.arange(C)[None, None, None, :]
    return x[n, h, w, c]


def maxpool_backward(dy, arg, in_shape, r, s, st, pad):
    dy = _f64(dy)
    N, P, Q, C = dy.shape
    _, H, W, _ = in_shape
    dx = np.empty((N, H, W, C))
    arg = np.ascontiguousarray(arg, dtype=np.int32)
    lib().or_maxpool_backward(N, H, W, C, r, s, st, pad, P, Q, _dp(dy),
                              arg.ctypes.data_as(ctypes.POINTER(ctypes.c_int)), _dp(dx))
    return dx


def _avg_counts(H, W, r, s, st, pad, P, Q):
    """Number of in-image taps of each R x S window (padded taps do not count)."""
    hs = np.arange(P)[:, None] * st + np.arange(r)[None, :] - pad
    ws = np.arange(Q)[:, None] * st + np.arange(s)[None, :] - pad
    rows = ((hs >= 0) & (hs < H)).sum(axis=1)
    cols = ((ws >= 0) & (ws < W)).sum(axis=1)
    return rows[:, None] * cols[None, :]


def avgpool_forward(x, r, s, st, pad):
    """y[n,p,q,c] = mean of x over the in-image taps of the window at (p*st-pad, q*st-pad)."""
    x = _f64(x)
    N, H, W, C = x.shape
    P, Q = conv_out(H, r, st, pad), conv_out(W, s, st, pad)
    y = np.zeros((N, P, Q, C))
    for p in range(P):
        for q in range(Q):
            h0, w0 = p * st - pad, q * st - pad
            win = x[:, max(h0, 0):min(h0 + r, H), max(w0, 0):min(w0 + s, W), :]
            y[:, p, q, :] = win.sum(axis=(1, 2)) / (win.shape[1] * win.shape[2])
    return y


def avgpool_backward(dy, in_shape, r, s, st, pad):
    """dx[n,h,w,c] = sum over the windows holding (h, w) of dy[n,p,q,c] / count(p, q)."""
    dy = _f64(dy)
    N, P, Q, C = dy.shape
    _, H, W, _ = in_shape
    cnt = _avg_counts(H, W, r, s, st, pad, P, Q)
    dx = np.zeros((N, H, W, C))
    for p in range(P):
        for q in range(Q):
            h0, w0 = p * st - pad, q * st - pad
            dx[:, max(h0, 0):min(h0 + r, H), max(w0, 0):min(w0 + s, W), :] += \
                (dy[:, p, q, :] / cnt[p, q])[:, None, None, :]
    return dx


def _fp(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if a is not None else None


def conv2d_samples(which, geom, a, b, idx, bias=None):
    """Selected outputs of a conv pass, each from its definition, on float32 inputs.

    geom = (N, H, W, C, K, R, S, stride, pad[, pad_w]) (pad_w defaults to pad);
    which = "fwd" (a = x, b = w,
    idx rows (n, p, q, k)), "dgrad" (a = dy, b = w, rows (n, h, w, c)) or
    "wgrad" (a = x, b = dy, rows (k, r, s, c)).  Returns float64 values.
    """
    N, H, W, C, K, R, S, st, pad = geom[:9]
    pad_w = geom[9] if len(geom) > 9 else pad
    P, Q = conv_out(H, R, st, pad), conv_out(W, S, st, pad_w)
    a = np.ascontiguousarray(a, dtype=np.float32)
    b = np.ascontiguousarray(b, dtype=np.float32)
    idx = np.ascontiguousarray(idx, dtype=np.int32).reshape(-1, 4)
    out = np.empty(len(idx))
    args = (N, H, W, C, K, R, S, st, pad, pad_w, P, Q)
    ip = idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int))
    if which == "fwd":
        bb = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        lib().or_conv2d_forward_samples(*args, _fp(a), _fp(b), _fp(bb), len(idx), ip, _dp(out))
    elif which == "dgrad":
        lib().or_conv2d_backward_data_samples(*args, _fp(a), _fp(b), len(idx), ip, _dp(out))
    elif which == "wgrad":
        lib().or_conv2d_backward_filter_samples(*args, _fp(a), _fp(b), len(idx), ip, _dp(out))
    else:
        raise ValueError(which)
    return out


def relu_mask(x):
    """ReLU's decision, taken in float32: x > 0 (so relu'(0) = 0)."""
    return x.astype(np.float32) > 0


def batchnorm_forward(x, gamma, beta, eps=BN_EPS):
    """Training-mode BatchNorm over (n, h, w) per channel with the biased variance."""
    mu = x.mean(axis=(0, 1, 2))
    var = ((x - mu) ** 2).mean(axis=(0, 1, 2))
    invstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mu) * invstd
    return gamma * xhat + beta, xhat, invstd


def batchnorm_backward(dy, xhat, invstd, gamma):
    """Chain rule through the batch statistics: returns (dx, dgamma, dbeta)."""
    M = dy.shape[0] * dy.shape[1] * dy.shape[2]
    dbeta = dy.sum(axis=(0, 1, 2))
    dgamma = (dy * xhat).sum(axis=(0, 1, 2))
    dx = gamma * invstd * (dy - dbeta / M - xhat * dgamma / M)
    return dx, dgamma, dbeta


def softmax_xent(z, y):
    """Mean over the batch of -log softmax(z)_y, and its gradient (softmax - onehot) / N."""
    N, K = z.shape
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    s = e.sum(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(s[:, 0])
    loss = float(np.mean(lse - z[np.arange(N), y]))
    dz = e / s
    dz[np.arange(N), y] -= 1.0
    return loss, dz / N


def sgd(params, grads, lr=LR):
    """The server's update w <- w - lr * g."""
    return np.asarray(params, dtype=np.float64) - lr * np.asarray(grads, dtype=np.float64)


# ---------------------------------------------------------------- network

class Net:
    """Shapes, parameter layout and the training iteration of one oracle network."""

    # Test hook: when set, perturb(i, y) replaces the output y of every conv,
    # FC and BN op i in the forward pass.  None (the default) leaves the
    # arithmetic untouched; tests use it to emulate float32 storage error.
    perturb = None

    def __init__(self, spec, batch):
        self.spec = spec
        self.ops = spec["ops"]
        self.classes = spec["classes"]
        self.batch = batch
        H, W, C = spec["hwc"]
        shapes = [(batch, H, W, C)]
        self.pslots = []   # per op: dict name -> (offset, shape)
        self.param_specs = []
        self.layer_ranges = {}
        off = 0

        def take(name, shape, kind, fan_in=None):
            nonlocal off
            n = int(np.prod(shape))
            slots[name] = (off, shape)
            self.param_specs.append((kind, n, fan_in) if kind == "he" else (kind, n))
            off += n

        for op in self.ops:
            n, h, w, c = shapes[op["in"]]
            slots = {}
            start = off
            kind = op["op"]
            if kind == "conv":
                ph, pw = _op_pads(op)
                P, Q = conv_out(h, op["r"], op["stride"], ph), conv_out(w, op["s"], op["stride"], pw)
                take("w", (op["k"], op["r"], op["s"], c), "he", op["r"] * op["s"] * c)
                if op["bias"]:
                    take("b", (op["k"],), "zeros")
                out = (n, P, Q, op["k"])
            elif kind == "fc":
                fin = h * w * c
                take("w", (op["out"], fin), "he", fin)
                if op["bias"]:
                    take("b", (op["out"],), "zeros")
                out = (n, 1, 1, op["out"])
            elif kind == "bn":
                take("gamma", (c,), "ones")
                take("beta", (c,), "zeros")
                out = (n, h, w, c)
            elif kind in ("relu", "add"):
                if kind == "add":
                    assert shapes[op["other"]] == (n, h, w, c)
                out = (n, h, w, c)
            elif kind == "concat":
                cs = c
                for o in op["others"]:
                    assert shapes[o][:3] == (n, h, w)
                    cs += shapes[o][3]
                out = (n, h, w, cs)
            elif kind in ("maxpool", "avgpool"):
                out = (n, conv_out(h, op["r"], op["stride"], op["pad"]),
                       conv_out(w, op["s"], op["stride"], op["pad"]), c)
            elif kind == "gap":
                out = (n, 1, 1, c)
            else:
                raise ValueError(kind)
            l = op["layer"]
            lo, cnt = self.layer_ranges.get(l, (start, 0))
            self.layer_ranges[l] = (lo, cnt + (off - start))
            self.pslots.append(slots)
            shapes.append(out)
        self.shapes = shapes
        self.n_params = off
        self.L = max(op["layer"] for op in self.ops)
        assert shapes[-1][1:] == (1, 1, self.classes)

    def layer_bytes(self):
        return [4 * self.layer_ranges[l][1] for l in range(1, self.L + 1)]

    def _p(self, params, i, name):
        off, shape = self.pslots[i][name]
        return params[off:off + int(np.prod(shape))].reshape(shape)

    def forward(self, x, params, decisions=None):
        """Returns (tensors, caches); tensors[0] is the input, tensors[-1] the logits.
        decisions: optional {op index: ReLU mask (bool, the op's input shape) or max-pool window
        tap r * S + s (int, the op's output shape)} taken instead of deciding."""
        decisions = decisions or {}
        params = np.asarray(params, dtype=np.float64)
        t = [np.asarray(x, dtype=np.float64)]
        cache = {}
        for i, op in enumerate(self.ops):
            a = t[op["in"]]
            kind = op["op"]
            if kind == "conv":
                b = self._p(params, i, "b") if op["bias"] else None
                y = conv2d_forward(a, self._p(params, i, "w"), b, op["stride"], _op_pads(op))
            elif kind == "fc":
                a2 = a.reshape(a.shape[0], -1)
                y = a2 @ self._p(params, i, "w").T
                if op["bias"]:
                    y = y + self._p(params, i, "b")
                y = y.reshape(a.shape[0], 1, 1, -1)
            elif kind == "bn":
                y, xhat, invstd = batchnorm_forward(a, self._p(params, i, "gamma"), self._p(params, i, "beta"))
                cache[i] = (xhat, invstd)
            elif kind == "relu":
                mask = np.asarray(decisions[i], dtype=bool) if i in decisions else relu_mask(a)
                y = np.where(mask, a, 0.0)
                cache[i] = mask
            elif kind == "maxpool":
                if i in decisions:
                    arg = np.asarray(decisions[i], dtype=np.int32)
                    y = maxpool_at(a, arg, op["r"], op["s"], op["stride"], op["pad"])
                else:
                    y, arg = maxpool_forward(a, op["r"], op["s"], op["stride"], op["pad"])
                cache[i] = arg
            elif kind == "avgpool":
                y = avgpool_forward(a, op["r"], op["s"], op["stride"], op["pad"])
            elif kind == "gap":
                y = a.mean(axis=(1, 2), keepdims=True)
            elif kind == "add":
                y = a + t[op["other"]]
            elif kind == "concat":
                y = np.concatenate([a] + [t[o] for o in op["others"]], axis=3)
            if self.perturb is not None and kind in ("conv", "fc", "bn"):
                y = self.perturb(i, y)
            t.append(y)
        return t, cache

    def loss_and_grads(self, x, y, params, keep=False, decisions=None):
        """One forward and backward pass: returns (loss, flat float64 gradient), and
        with keep=True also (tensors, caches, tensor gradients) of the pass."""
        params = np.asarray(params, dtype=np.float64)
        t, cache = self.forward(x, params, decisions)
        N = self.batch
        loss, dz = softmax_xent(t[-1].reshape(N, self.classes), np.asarray(y))
        g = [None] * len(t)
        g[-1] = dz.reshape(t[-1].shape)
        grads = np.zeros(self.n_params)

        def acc(tid, d):
            if g[tid] is None:
                g[tid] = np.array(d, dtype=np.float64, copy=True)
            else:
                g[tid] += d

        def put(i, name, d):
            off, shape = self.pslots[i][name]
            grads[off:off + int(np.prod(shape))] = np.asarray(d).reshape(-1)

        for i in range(len(self.ops) - 1, -1, -1):
            op = self.ops[i]
            dy = g[i + 1]
            if dy is None:
                raise RuntimeError(f"tensor {i + 1} has no consumer")
            a = t[op["in"]]
            kind = op["op"]
            if kind == "conv":
                put(i, "w", conv2d_backward_filter(a, dy, (op["r"], op["s"]), op["stride"], _op_pads(op)))
                if op["bias"]:
                    put(i, "b", dy.sum(axis=(0, 1, 2)))
                if op["in"] != 0:  # the input batch needs no gradient
                    acc(op["in"], conv2d_backward_data(dy, self._p(params, i, "w"), a.shape[1:3],
                                                       op["stride"], _op_pads(op)))
            elif kind == "fc":
                a2 = a.reshape(a.shape[0], -1)
                dy2 = dy.reshape(dy.shape[0], -1)
                put(i, "w", dy2.T @ a2)
                if op["bias"]:
                    put(i, "b", dy2.sum(axis=0))
                if op["in"] != 0:
                    acc(op["in"], (dy2 @ self._p(params, i, "w")).reshape(a.shape))
            elif kind == "bn":
                xhat, invstd = cache[i]
                dx, dgamma, dbeta = batchnorm_backward(dy, xhat, invstd, self._p(params, i, "gamma"))
                put(i, "gamma", dgamma)
                put(i, "beta", dbeta)
                acc(op["in"], dx)
            elif kind == "relu":
                acc(op["in"], np.where(cache[i], dy, 0.0))
            elif kind == "maxpool":
                acc(op["in"], maxpool_backward(dy, cache[i], a.shape, op["r"], op["s"], op["stride"], op["pad"]))
            elif kind == "avgpool":
                acc(op["in"], avgpool_backward(dy, a.shape, op["r"], op["s"], op["stride"], op["pad"]))
            elif kind == "gap":
                hw = a.shape[1] * a.shape[2]
                acc(op["in"], np.broadcast_to(dy / hw, a.shape))
            elif kind == "add":
                acc(op["in"], dy)
                acc(op["other"], dy)
            elif kind == "concat":
                lo = 0
                for tid in [op["in"]] + list(op["others"]):
                    ci = t[tid].shape[3]
                    acc(tid, dy[..., lo:lo + ci])
                    lo += ci
        if keep:
            return loss, grads, t, cache, g
        return loss, grads

    def loss(self, x, y, params):
        t, _ = self.forward(x, params)
        l, _ = softmax_xent(t[-1].reshape(self.batch, self.classes), np.asarray(y))
        return l

    def step(self, x, y, params, lr=LR):
        """One full iteration: (loss, gradient, updated parameters)."""
        loss, grads = self.loss_and_grads(x, y, params)
        return loss, grads, sgd(params, grads, lr)


def _op_pads(op):
    """(row, column) padding of a conv op; "pad_w" defaults to "pad"."""
    return op["pad"], op.get("pad_w", op["pad"])


def flops_per_image(net):
    """Multiply-add FLOPs (2 per MAC) of forward + both backward GEMM passes, per image."""
    f = 0
    for i, op in enumerate(net.ops):
        if op["op"] == "conv":
            n, P, Q, K = net.shapes[i + 1]
            C = net.shapes[op["in"]][3]
            mac = P * Q * K * op["r"] * op["s"] * C
            f += 2 * mac * (2 if op["in"] == 0 else 3)
        elif op["op"] == "fc":
            n, h, w, c = net.shapes[op["in"]]
            mac = h * w * c * op["out"]
            f += 2 * mac * (2 if op["in"] == 0 else 3)
    return f


def ln_classes(classes):
    return math.log(classes)
