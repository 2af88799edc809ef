"""The oracle's network evaluated with torch CPU library routines (test helper).

Used two ways: in float64 as a library cross-check of the oracle's
definitions, and in float32 as a yardstick of how far an ordinary float32
evaluation of the same iteration lands from the float64 oracle.
"""
import numpy as np
import torch


def _nchw(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a).transpose(0, 3, 1, 2))).to(dtype)


def _maxpool_at(a, arg, r, s, st, pad):
    """Max-pool forward (NCHW) taking the window tap arg = r' * s + s' (NHWC array) of each output."""
    N, C, H, W = a.shape
    arg = torch.from_numpy(np.ascontiguousarray(np.asarray(arg).transpose(0, 3, 1, 2))).long()
    P, Q = arg.shape[2], arg.shape[3]
    h = torch.arange(P).view(1, 1, P, 1) * st + torch.div(arg, s, rounding_mode="floor") - pad
    w = torch.arange(Q).view(1, 1, 1, Q) * st + arg % s - pad
    return a.flatten(2).gather(2, (h * W + w).flatten(2)).view(N, C, P, Q)


def loss_and_grads(spec, net, x, y, p, dtype=torch.float64, perturb=None, decisions=None):
    """(loss, flat gradient as float64) of one iteration in the given torch dtype on the CPU.

    perturb(i, o), if given, replaces the output o (NCHW) of every conv, FC and
    BN op i in the forward pass, as the oracle's test hook does.  decisions, if
    given, are taken as the oracle's are: {op index: ReLU mask (NHWC bool) or
    max-pool window tap (NHWC int)}."""
    decisions = decisions or {}
    pt = torch.from_numpy(np.asarray(p, dtype=np.float64)).to(dtype).requires_grad_(True)

    def prm(i, name):
        off, shape = net.pslots[i][name]
        return pt[off:off + int(np.prod(shape))].reshape(shape)

    F = torch.nn.functional
    t = [_nchw(x, dtype)]
    for i, op in enumerate(spec["ops"]):
        a = t[op["in"]]
        k = op["op"]
        if k == "conv":
            w = prm(i, "w").permute(0, 3, 1, 2)
            b = prm(i, "b") if op["bias"] else None
            o = F.conv2d(a, w, b, stride=op["stride"], padding=(op["pad"], op.get("pad_w", op["pad"])))
        elif k == "fc":
            flat = a.permute(0, 2, 3, 1).reshape(a.shape[0], -1)   # NHWC flatten
            o = F.linear(flat, prm(i, "w"), prm(i, "b") if op["bias"] else None)
            o = o.reshape(a.shape[0], -1, 1, 1)
        elif k == "bn":
            o = F.batch_norm(a, None, None, prm(i, "gamma"), prm(i, "beta"), training=True, eps=1e-5)
        elif k == "relu":
            o = a * _nchw(decisions[i], dtype) if i in decisions else F.relu(a)
        elif k == "maxpool":
            o = (_maxpool_at(a, decisions[i], op["r"], op["s"], op["stride"], op["pad"]) if i in decisions
                 else F.max_pool2d(a, op["r"], op["stride"], op["pad"]))
        elif k == "avgpool":
            o = F.avg_pool2d(a, (op["r"], op["s"]), op["stride"], op["pad"], count_include_pad=False)
        elif k == "gap":
            o = F.adaptive_avg_pool2d(a, 1)
        elif k == "add":
            o = a + t[op["other"]]
        elif k == "concat":
            o = torch.cat([a] + [t[j] for j in op["others"]], dim=1)
        if perturb is not None and k in ("conv", "fc", "bn"):
            o = perturb(i, o)
        t.append(o)
    loss = F.cross_entropy(t[-1].reshape(net.batch, -1), torch.from_numpy(np.asarray(y, dtype=np.int64)))
    loss.backward()
    return loss.item(), pt.grad.double().numpy()
