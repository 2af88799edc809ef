"""Each op's GPU kernels on the oracle's own tensors (helper of the GPU tests).

The oracle runs the whole float64 iteration; then each op's kernel is called
through the C ABI on the oracle's input tensors (forward) and on the oracle's
gradient of the op's output (backward), rounded to float32, and its output is
compared with the oracle's output of that op at the kernel-level bars of
test_gpu_kernels.py.  Nothing flows from the GPU into the oracle.

Two sets of launches are checked:
* the plain entry points of every op;
* the launches a model makes in their place where it folds a ReLU's backward
  into a neighbouring op (dc_backward_schedule names them): the masked data
  gradient of a conv / FC, the masked max-pool and concatenation backward,
  BatchNorm backward through a ReLU and the backward of relu(a + b).

Bars per tensor (max |gpu - oracle| / max |oracle|): conv / FC passes
tol(sum length); BatchNorm tol(rows), 10x for its data gradient; pooling,
GAP and residual add 1e-6; ReLU, max-pool forward, concatenation and the
masked copies bit-exact against the oracle's value rounded to float32 (their
decisions are taken in float32 on both sides); loss 1e-6 relative.
"""
import ctypes
import math

import numpy as np

from oracle import cnn as OC
from paper_2101_07968_amd import _lib as D
from paper_2101_07968_amd import nets as PN
from tests.gpu_helpers import dev, host, rel_err, scratch, stream, zeros


def tol(k_terms):
    return min(2e-4, 1e-5 * max(1.0, math.sqrt(k_terms / 256.0)))


def f32(a):
    return dev(np.ascontiguousarray(np.asarray(a, dtype=np.float32)))


def exact(got, ref):
    np.testing.assert_array_equal(got, np.asarray(ref, dtype=np.float32))


def _conv_geom(op, a, out_shape):
    n, h, w, c = a.shape
    if op["op"] == "conv":
        return (n, h, w, c, op["k"], op["r"], op["s"], op["stride"], op["pad"], op.get("pad_w", op["pad"]))
    return (n, 1, 1, h * w * c, op["out"], 1, 1, 1, 0, 0)


def check_ops(name, net, y, params, res):
    """Run every op's kernels on the oracle's tensors; res = (loss, grads, t, cache, g)
    from net.loss_and_grads(..., keep=True).  Returns the worst error / bar per kind."""
    loss_ref, grads_ref, t, cache, g = res
    batch = net.batch
    p64 = np.asarray(params, dtype=np.float64)
    worst = {}
    readers = {}
    for op in net.ops:
        for tid in [op["in"]] + ([op["other"]] if op["op"] == "add" else []) + list(op.get("others", [])):
            readers[tid] = readers.get(tid, 0) + 1

    def check(kind, err, bar):
        assert err <= bar, (kind, err, bar)
        worst[kind] = max(worst.get(kind, 0.0), err / bar)

    def prm(i, key):
        off, shape = net.pslots[i][key]
        return p64[off:off + int(np.prod(shape))].reshape(shape)

    def weight(i):
        op = net.ops[i]
        wt = prm(i, "w")
        if op["op"] == "fc":
            wt = wt.reshape(op["out"], 1, 1, -1)
        return wt

    def dgrad_ref(i):
        """The data gradient of op i alone: the oracle's input gradient when op i is its
        input's only reader, else recomputed from the definition."""
        op = net.ops[i]
        a, dy = t[op["in"]], g[i + 1]
        if readers[op["in"]] == 1:
            return g[op["in"]]
        if op["op"] == "conv":
            return OC.conv2d_backward_data(dy, prm(i, "w"), a.shape[1:3], op["stride"],
                                           (op["pad"], op.get("pad_w", op["pad"])))
        return (dy.reshape(batch, -1) @ prm(i, "w")).reshape(a.shape)

    s = stream()
    for i, op in enumerate(net.ops):
        if i % 25 == 0:
            print(f"  layer-wise {name}: op {i} of {len(net.ops)}", flush=True)
        kind = op["op"]
        a = t[op["in"]]
        out_ref = t[i + 1]
        dy = g[i + 1]
        n, h, w, c = a.shape
        if kind in ("conv", "fc"):
            geom = _conv_geom(op, a, out_ref.shape)
            r, ss, K = geom[5], geom[6], geom[4]
            wt = weight(i)
            sh = D.ConvShape(*geom)
            P, Q = out_ref.shape[1], out_ref.shape[2]
            _ws_t, ws, wsb = scratch(D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh)))
            xd, wd, dyd = f32(a), f32(wt), f32(dy)
            bias = f32(prm(i, "b")) if op["bias"] else None
            yo = zeros((n, P, Q, K))
            D.call("dc_conv2d_forward", ctypes.byref(sh), xd.data_ptr(), wd.data_ptr(),
                   bias.data_ptr() if bias is not None else None, 0, yo.data_ptr(), ws, wsb, s)
            check(kind + " fwd", rel_err(host(yo).reshape(out_ref.shape), out_ref), tol(r * ss * geom[3]))
            del yo
            dw = zeros(wt.shape)
            db = zeros((K,))
            D.call("dc_conv2d_backward_filter", ctypes.byref(sh), xd.data_ptr(), dyd.data_ptr(), dw.data_ptr(),
                   db.data_ptr() if op["bias"] else None, ws, wsb, s)
            off, shape = net.pslots[i]["w"]
            check(kind + " wgrad", rel_err(host(dw).reshape(-1), grads_ref[off:off + int(np.prod(shape))]),
                  tol(n * P * Q))
            if op["bias"]:
                off, shape = net.pslots[i]["b"]
                check(kind + " bias grad", rel_err(host(db), grads_ref[off:off + shape[0]]), tol(n * P * Q))
            del dw, db, xd
            if op["in"] != 0:
                dx = zeros(a.shape)
                D.call("dc_conv2d_backward_data", ctypes.byref(sh), dyd.data_ptr(), wd.data_ptr(), 0,
                       dx.data_ptr(), ws, wsb, s)
                check(kind + " dgrad", rel_err(host(dx), dgrad_ref(i)), tol(r * ss * K))
        elif kind == "bn":
            rows = n * h * w
            gamma, beta = prm(i, "gamma"), prm(i, "beta")
            _ws_t, ws, wsb = scratch(D.lib().dc_batchnorm_workspace_bytes(rows, c))
            xd, gd, bd, dyd = f32(a), f32(gamma), f32(beta), f32(dy)
            yo, mean, invstd = zeros(a.shape), zeros((c,)), zeros((c,))
            D.call("dc_batchnorm_forward", rows, c, xd.data_ptr(), gd.data_ptr(), bd.data_ptr(),
                   ctypes.c_float(OC.BN_EPS), yo.data_ptr(), mean.data_ptr(), invstd.data_ptr(), ws, wsb, s)
            check("bn fwd", rel_err(host(yo), out_ref), tol(rows))
            dx, dg, dbeta = zeros(a.shape), zeros((c,)), zeros((c,))
            D.call("dc_batchnorm_backward", rows, c, dyd.data_ptr(), xd.data_ptr(), gd.data_ptr(), mean.data_ptr(),
                   invstd.data_ptr(), 0, dx.data_ptr(), dg.data_ptr(), dbeta.data_ptr(), ws, wsb, s)
            xhat, inv_ref = cache[i]
            dx_ref, dg_ref, db_ref = OC.batchnorm_backward(dy, xhat, inv_ref, gamma)
            check("bn dgamma", rel_err(host(dg), dg_ref), tol(rows))
            check("bn dbeta", rel_err(host(dbeta), db_ref), tol(rows))
            check("bn dgrad", rel_err(host(dx), dx_ref), 10 * tol(rows))
        elif kind == "relu":
            nel = a.size
            xd, dyd = f32(a), f32(dy)
            yo = zeros(a.shape)
            D.call("dc_relu_forward", xd.data_ptr(), yo.data_ptr(), nel, s)
            exact(host(yo), out_ref)
            dx = zeros(a.shape)
            D.call("dc_relu_backward", dyd.data_ptr(), yo.data_ptr(), 0, dx.data_ptr(), nel, s)
            exact(host(dx), np.where(OC.relu_mask(a), dy, 0.0))
            worst["relu"] = 0.0
        elif kind in ("maxpool", "avgpool"):
            r, st, pad = op["r"], op["stride"], op["pad"]
            psh = D.PoolShape(n, h, w, c, r, op["s"], st, pad)
            xd, dyd = f32(a), f32(dy)
            yo = zeros(out_ref.shape)
            dx = zeros(a.shape)
            if kind == "maxpool":
                arg = zeros(out_ref.shape, "uint8")
                D.call("dc_maxpool_forward", ctypes.byref(psh), xd.data_ptr(), yo.data_ptr(), arg.data_ptr(), s)
                exact(host(yo), out_ref)
                np.testing.assert_array_equal(host(arg).astype(np.int32), cache[i])
                D.call("dc_maxpool_backward", ctypes.byref(psh), dyd.data_ptr(), arg.data_ptr(), 0, dx.data_ptr(), s)
                check("maxpool bwd", rel_err(host(dx), OC.maxpool_backward(dy, cache[i], a.shape, r, op["s"], st, pad)),
                      1e-6)
            else:
                D.call("dc_avgpool_forward", ctypes.byref(psh), xd.data_ptr(), yo.data_ptr(), s)
                check("avgpool fwd", rel_err(host(yo), out_ref), 1e-6)
                D.call("dc_avgpool_backward", ctypes.byref(psh), dyd.data_ptr(), 0, dx.data_ptr(), s)
                check("avgpool bwd", rel_err(host(dx), OC.avgpool_backward(dy, a.shape, r, op["s"], st, pad)), 1e-6)
        elif kind == "gap":
            xd, dyd = f32(a), f32(dy)
            yo, dx = zeros(out_ref.shape), zeros(a.shape)
            D.call("dc_gap_forward", n, h * w, c, xd.data_ptr(), yo.data_ptr(), s)
            check("gap fwd", rel_err(host(yo), out_ref), 1e-6)
            D.call("dc_gap_backward", n, h * w, c, dyd.data_ptr(), 0, dx.data_ptr(), s)
            check("gap bwd", rel_err(host(dx), np.broadcast_to(dy / (h * w), a.shape)), 1e-6)
        elif kind == "add":
            ad, bd = f32(a), f32(t[op["other"]])
            yo = zeros(a.shape)
            D.call("dc_add_forward", ad.data_ptr(), bd.data_ptr(), 0, yo.data_ptr(), a.size, s)
            check("add fwd", rel_err(host(yo), out_ref), 1e-6)
        elif kind == "concat":
            parts = [op["in"]] + list(op["others"])
            ct = out_ref.shape[3]
            rows = n * h * w
            yo = zeros(out_ref.shape)
            dyd = f32(dy)
            lo = 0
            for tid in parts:
                ci = t[tid].shape[3]
                xd = f32(t[tid])
                D.call("dc_concat_forward", rows, ci, ct, lo, xd.data_ptr(), yo.data_ptr(), s)
                dx = zeros(t[tid].shape)
                D.call("dc_concat_backward", rows, ci, ct, lo, dyd.data_ptr(), 0, dx.data_ptr(), s)
                exact(host(dx), dy[..., lo:lo + ci])
                lo += ci
            exact(host(yo), out_ref)
            worst["concat"] = 0.0
        else:
            raise AssertionError(kind)
    _check_folds(name, net, t, cache, g, prm, weight, check, worst, s)
    # the loss on the oracle's logits
    z = t[-1].reshape(batch, -1)
    classes = z.shape[1]
    _ws_t, ws, wsb = scratch(D.lib().dc_softmax_xent_workspace_bytes(batch))
    zd, yd = f32(z), dev(np.asarray(y, dtype=np.int32))
    loss, dz = zeros((1,)), zeros((batch, classes))
    D.call("dc_softmax_xent", batch, classes, zd.data_ptr(), yd.data_ptr(), loss.data_ptr(), dz.data_ptr(), ws, wsb, s)
    l_ref, dz_ref = OC.softmax_xent(z, np.asarray(y))
    check("loss", abs(float(host(loss)[0]) - l_ref) / abs(l_ref), 1e-6)
    check("dlogits", rel_err(host(dz), dz_ref), 1e-6)
    return worst


KIND_NAME = {D.DC_OP_CONV: "conv", D.DC_OP_FC: "fc", D.DC_OP_BN: "bn", D.DC_OP_RELU: "relu",
             D.DC_OP_MAXPOOL: "maxpool", D.DC_OP_GAP: "gap", D.DC_OP_ADD: "add", D.DC_OP_CONCAT: "concat",
             D.DC_OP_AVGPOOL: "avgpool"}


def op_map(ops, net):
    """Product op index -> oracle op index.  The two sides describe each network
    separately, in the same order, except that the product nests a concatenation of
    more than four parts (its inner concatenation maps to None)."""
    tmap, parts, out = {0: 0}, {}, {}
    j = 0
    for i, o in enumerate(ops):
        ins = []
        for tid in [o[2]] + ([o[3]] if o[0] in (D.DC_OP_ADD, D.DC_OP_CONCAT) else []) + \
                [x for x in (o[10], o[11]) if o[0] == D.DC_OP_CONCAT and x >= 0]:
            ins += parts[tid] if tid in parts else [tmap[tid]]
        oo = net.ops[j]
        o_ins = [oo["in"]] + ([oo["other"]] if oo["op"] == "add" else []) + list(oo.get("others", []))
        if KIND_NAME[o[0]] == oo["op"] and ins == o_ins:
            out[i], tmap[i + 1] = j, j + 1
            j += 1
        else:
            assert o[0] == D.DC_OP_CONCAT and oo["op"] == "concat" and ins == o_ins[:len(ins)], (i, j)
            out[i], parts[i + 1] = None, ins
    assert j == len(net.ops)
    return out


def _check_folds(name, net, t, cache, g, prm, weight, check, worst, s):
    """The launches that carry a ReLU's backward in a model, on the oracle's tensors.
    A folded ReLU's output has one reader, so its gradient g[r + 1] is that reader's
    term alone, and the expected result is the ReLU's mask applied to it."""
    ops, hwc, classes = PN.build(name)
    sched = D.backward_schedule(ops, net.batch, hwc, classes)
    omap = op_map(ops, net)
    folds = sorted({(omap[e["origin_op"]], omap[e["exec_op"]]) for e in sched
                    if ops[e["origin_op"]][0] == D.DC_OP_RELU and e["exec_op"] != e["origin_op"]})
    assert folds and all(r is not None and j is not None for r, j in folds), (name, folds)
    for r, j in folds:
        r_in = net.ops[r]["in"]
        mask = OC.relu_mask(t[r_in])
        relu_y = t[r + 1]
        masked = np.where(mask, g[r + 1], 0.0)
        op = net.ops[j]
        kind = op["op"]
        if kind in ("conv", "fc"):
            assert op["in"] == r + 1
            a = t[op["in"]]
            geom = _conv_geom(op, a, t[j + 1].shape)
            sh = D.ConvShape(*geom)
            _ws_t, ws, wsb = scratch(D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh)))
            dyd, wd, yd = f32(g[j + 1]), f32(weight(j)), f32(relu_y)
            dx = zeros(a.shape)
            D.call("dc_conv2d_backward_data_relu", ctypes.byref(sh), dyd.data_ptr(), wd.data_ptr(), yd.data_ptr(), 0,
                   dx.data_ptr(), ws, wsb, s)
            check(kind + " dgrad + relu", rel_err(host(dx), masked), tol(geom[5] * geom[6] * geom[4]))
        elif kind == "maxpool":
            a = t[op["in"]]
            n, h, w, c = a.shape
            psh = D.PoolShape(n, h, w, c, op["r"], op["s"], op["stride"], op["pad"])
            dyd, argd, yd = f32(g[j + 1]), dev(np.asarray(cache[j], dtype=np.uint8)), f32(t[j + 1])
            dx = zeros(a.shape)
            D.call("dc_maxpool_backward_relu", ctypes.byref(psh), dyd.data_ptr(), argd.data_ptr(), yd.data_ptr(), 0,
                   dx.data_ptr(), s)
            check("maxpool bwd + relu", rel_err(host(dx), masked), 1e-6)
        elif kind == "concat":
            parts = [op["in"]] + list(op["others"])
            ct = t[j + 1].shape[3]
            rows = int(np.prod(t[j + 1].shape[:3]))
            lo = 0
            dyd = f32(g[j + 1])
            for tid in parts:
                ci = t[tid].shape[3]
                if tid == r + 1:
                    yd = f32(relu_y)
                    dx = zeros(relu_y.shape)
                    D.call("dc_concat_backward_relu", rows, ci, ct, lo, dyd.data_ptr(), yd.data_ptr(), 0,
                           dx.data_ptr(), s)
                    exact(host(dx), np.where(mask, g[j + 1][..., lo:lo + ci], 0.0))
                    worst["concat bwd + relu"] = 0.0
                lo += ci
        elif kind == "bn":
            assert j == r - 1 and r_in == j + 1
            a = t[op["in"]]
            rows = int(np.prod(a.shape[:3]))
            c = a.shape[3]
            gamma, beta = prm(j, "gamma"), prm(j, "beta")
            _ws_t, ws, wsb = scratch(D.lib().dc_batchnorm_workspace_bytes(rows, c))
            xd, gd, bd = f32(a), f32(gamma), f32(beta)
            yo, mean, invstd = zeros(a.shape), zeros((c,)), zeros((c,))
            D.call("dc_batchnorm_forward", rows, c, xd.data_ptr(), gd.data_ptr(), bd.data_ptr(),
                   ctypes.c_float(OC.BN_EPS), yo.data_ptr(), mean.data_ptr(), invstd.data_ptr(), ws, wsb, s)
            del yo
            dyd, yd = f32(g[r + 1]), f32(relu_y)
            dx, dg, dbeta = zeros(a.shape), zeros((c,)), zeros((c,))
            D.call("dc_batchnorm_backward_relu", rows, c, dyd.data_ptr(), yd.data_ptr(), xd.data_ptr(), gd.data_ptr(),
                   mean.data_ptr(), invstd.data_ptr(), 0, dx.data_ptr(), dg.data_ptr(), dbeta.data_ptr(), ws, wsb, s)
            xhat, inv_ref = cache[j]
            dx_ref, dg_ref, db_ref = OC.batchnorm_backward(masked, xhat, inv_ref, gamma)
            check("bn bwd + relu dgamma", rel_err(host(dg), dg_ref), tol(rows))
            check("bn bwd + relu dbeta", rel_err(host(dbeta), db_ref), tol(rows))
            if op["in"] != 0:
                check("bn bwd + relu dgrad", rel_err(host(dx), dx_ref), 10 * tol(rows))
        elif kind == "add":
            assert j == r - 1 and r_in == j + 1
            dyd, yd = f32(g[r + 1]), f32(relu_y)
            d0, d1 = zeros(relu_y.shape), zeros(relu_y.shape)
            D.call("dc_add_relu_backward", dyd.data_ptr(), yd.data_ptr(), 0, d0.data_ptr(), 0, d1.data_ptr(),
                   relu_y.size, s)
            exact(host(d0), masked)
            exact(host(d1), masked)
            worst["add + relu bwd"] = 0.0
        else:
            raise AssertionError((name, r, j, kind))
