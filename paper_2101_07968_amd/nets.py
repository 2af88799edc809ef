"""The synthetic workloads as dc_op_desc lists for dc_model_create.

Each builder returns ``(ops, hwc, classes)``: ``ops`` is a list of 13-tuples
``(kind, layer, in0, in1, out_ch, r, s, stride, pad, bias, in2, in3, pad_w)`` in forward order
(tensor 0 = input batch, tensor i+1 = output of op i).  A planner layer is one
conv / FC and the parameter-less ops after it, BatchNorm joins its conv, and
a residual projection shares the layer of its block's first conv (the layer
decomposition of Sec. III-A).

Workloads (inputs NHWC; batch and link are chosen by the caller):
  tiny      conv3x3 3->8 +ReLU+pool2, conv3x3 8->16 +ReLU+pool2, FC 1024->64 +ReLU, FC 64->10   (L=4)
  alexnet   conv11x11/4 64, conv5x5 192, conv3x3 384/256/256, pools 3/2, FC 9216->4096->4096->1000 (L=8)
  resnet18  32x32 ResNet-18 with BN and 1x1/2 projections, FC 512->10                         (L=18)
  vgg16     13 conv3x3 + 3 FC, 224x224                                                        (L=16)
  resnet50  bottleneck [3,4,6,3], stride on the 3x3 conv, FC 2048->1000                        (L=50)
  googlenet Inception v1 (5x5 third branch, no LRN / dropout / auxiliary heads), FC 1024->1000  (L=22)
  vgg19     16 conv3x3 + 3 FC, 224x224                                                        (L=19)
  resnet152 bottleneck [3,8,36,3], as resnet50                                                (L=152)
  inception_v4  299x299 Inception-v4: stem, 4xA, reduction A, 7xB, reduction B, 3xC (BN+ReLU
            after every bias-free conv, 3x3/1 average-pool branches), FC 1536->1000       (L=76)
"""
from __future__ import annotations

from ._lib import (DC_OP_ADD, DC_OP_AVGPOOL, DC_OP_BN, DC_OP_CONCAT, DC_OP_CONV, DC_OP_FC, DC_OP_GAP, DC_OP_MAXPOOL,
                   DC_OP_RELU)


class NetBuilder:
    def __init__(self):
        self.ops = []
        self.layer = 0

    def _emit(self, kind, src, other=-1, out_ch=0, r=0, s=0, stride=0, pad=0, bias=0, in2=-1, in3=-1, pad_w=None):
        self.ops.append((kind, self.layer, src, other, out_ch, r, s, stride, pad, bias, in2, in3,
                         pad if pad_w is None else pad_w))
        return len(self.ops)

    def conv(self, src, out_ch, k, stride=1, pad=0, bias=True, new_layer=True):
        """k and pad are an int (square) or (rows, columns)."""
        if new_layer:
            self.layer += 1
        r, s = (k, k) if isinstance(k, int) else k
        ph, pw = (pad, pad) if isinstance(pad, int) else pad
        return self._emit(DC_OP_CONV, src, out_ch=out_ch, r=r, s=s, stride=stride, pad=ph, bias=int(bias),
                          pad_w=pw)

    def fc(self, src, out, bias=True):
        self.layer += 1
        return self._emit(DC_OP_FC, src, out_ch=out, bias=int(bias))

    def bn(self, src):
        return self._emit(DC_OP_BN, src)

    def relu(self, src):
        return self._emit(DC_OP_RELU, src)

    def maxpool(self, src, k, stride, pad=0):
        return self._emit(DC_OP_MAXPOOL, src, r=k, s=k, stride=stride, pad=pad)

    def avgpool(self, src, k, stride, pad=0):
        return self._emit(DC_OP_AVGPOOL, src, r=k, s=k, stride=stride, pad=pad)

    def gap(self, src):
        return self._emit(DC_OP_GAP, src)

    def add(self, a, b):
        return self._emit(DC_OP_ADD, a, other=b)

    def concat(self, a, b, c=-1, d=-1):
        return self._emit(DC_OP_CONCAT, a, other=b, in2=c, in3=d)


def tiny():
    n = NetBuilder()
    t = n.maxpool(n.relu(n.conv(0, 8, 3, pad=1)), 2, 2)
    t = n.maxpool(n.relu(n.conv(t, 16, 3, pad=1)), 2, 2)
    t = n.relu(n.fc(t, 64))
    n.fc(t, 10)
    return n.ops, (32, 32, 3), 10


def alexnet():
    n = NetBuilder()
    t = n.maxpool(n.relu(n.conv(0, 64, 11, stride=4, pad=2)), 3, 2)
    t = n.maxpool(n.relu(n.conv(t, 192, 5, pad=2)), 3, 2)
    t = n.relu(n.conv(t, 384, 3, pad=1))
    t = n.relu(n.conv(t, 256, 3, pad=1))
    t = n.maxpool(n.relu(n.conv(t, 256, 3, pad=1)), 3, 2)
    t = n.relu(n.fc(t, 4096))
    t = n.relu(n.fc(t, 4096))
    n.fc(t, 1000)
    return n.ops, (224, 224, 3), 1000


def _vgg(reps_per_stage):
    n = NetBuilder()
    t = 0
    for width, reps in zip((64, 128, 256, 512, 512), reps_per_stage):
        for _ in range(reps):
            t = n.relu(n.conv(t, width, 3, pad=1))
        t = n.maxpool(t, 2, 2)
    t = n.relu(n.fc(t, 4096))
    t = n.relu(n.fc(t, 4096))
    n.fc(t, 1000)
    return n.ops, (224, 224, 3), 1000


def vgg16():
    return _vgg((2, 2, 3, 3, 3))


def vgg19():
    return _vgg((2, 2, 4, 4, 4))


def _basic_block(n, x, cin, cout, stride):
    u = n.relu(n.bn(n.conv(x, cout, 3, stride=stride, pad=1, bias=False)))
    short = x
    if stride != 1 or cin != cout:  # projection at the depth of the first conv
        short = n.bn(n.conv(x, cout, 1, stride=stride, bias=False, new_layer=False))
    u = n.bn(n.conv(u, cout, 3, pad=1, bias=False))
    return n.relu(n.add(u, short))


def resnet18():
    n = NetBuilder()
    t = n.relu(n.bn(n.conv(0, 64, 3, pad=1, bias=False)))
    cin = 64
    for cout, stride in ((64, 1), (128, 2), (256, 2), (512, 2)):
        t = _basic_block(n, t, cin, cout, stride)
        t = _basic_block(n, t, cout, cout, 1)
        cin = cout
    t = n.gap(t)
    n.fc(t, 10)
    return n.ops, (32, 32, 3), 10


def _bottleneck(n, x, width, stride, project):
    out = 4 * width
    u = n.relu(n.bn(n.conv(x, width, 1, bias=False)))
    short = x
    if project:
        short = n.bn(n.conv(x, out, 1, stride=stride, bias=False, new_layer=False))
    u = n.relu(n.bn(n.conv(u, width, 3, stride=stride, pad=1, bias=False)))
    u = n.bn(n.conv(u, out, 1, bias=False))
    return n.relu(n.add(u, short))


def _resnet_bottleneck(blocks_per_stage):
    n = NetBuilder()
    t = n.relu(n.bn(n.conv(0, 64, 7, stride=2, pad=3, bias=False)))
    t = n.maxpool(t, 3, 2, pad=1)
    for width, blocks, stride in zip((64, 128, 256, 512), blocks_per_stage, (1, 2, 2, 2)):
        for i in range(blocks):
            t = _bottleneck(n, t, width, stride if i == 0 else 1, i == 0)
    t = n.gap(t)
    n.fc(t, 1000)
    return n.ops, (224, 224, 3), 1000


def resnet50():
    return _resnet_bottleneck((3, 4, 6, 3))


def resnet152():
    return _resnet_bottleneck((3, 8, 36, 3))


def _inception(n, x, c1, r3, c3, r5, c5, pool_proj):
    """Four branches; the depth-1 convs form one planner layer, the depth-2 convs and the concat the next."""
    b1 = n.relu(n.conv(x, c1, 1))
    b3 = n.relu(n.conv(x, r3, 1, new_layer=False))
    b5 = n.relu(n.conv(x, r5, 1, new_layer=False))
    bp = n.maxpool(x, 3, 1, pad=1)
    bp = n.relu(n.conv(bp, pool_proj, 1, new_layer=False))
    b3 = n.relu(n.conv(b3, c3, 3, pad=1))
    b5 = n.relu(n.conv(b5, c5, 5, pad=2, new_layer=False))
    return n.concat(b1, b3, b5, bp)


def googlenet():
    n = NetBuilder()
    t = n.maxpool(n.relu(n.conv(0, 64, 7, stride=2, pad=3)), 3, 2, pad=1)
    t = n.relu(n.conv(t, 64, 1))
    t = n.maxpool(n.relu(n.conv(t, 192, 3, pad=1)), 3, 2, pad=1)
    for m in ((64, 96, 128, 16, 32, 32), (128, 128, 192, 32, 96, 64), None,
              (192, 96, 208, 16, 48, 64), (160, 112, 224, 24, 64, 64), (128, 128, 256, 24, 64, 64),
              (112, 144, 288, 32, 64, 64), (256, 160, 320, 32, 128, 128), None,
              (256, 160, 320, 32, 128, 128), (384, 192, 384, 48, 128, 128)):
        t = n.maxpool(t, 3, 2, pad=1) if m is None else _inception(n, t, *m)
    t = n.gap(t)
    n.fc(t, 1000)
    return n.ops, (224, 224, 3), 1000


def _cbr(n, src, ch, k, stride=1, pad=0, first=False):
    """Bias-free conv + BN + ReLU; first=True opens the next planner layer."""
    return n.relu(n.bn(n.conv(src, ch, k, stride=stride, pad=pad, bias=False, new_layer=first)))


# Inception-v4 modules.  Each planner layer holds the convs at one depth from
# the module input, listed in the order of the branches in the concatenation;
# a pool that opens a branch joins the layer before (a layer is a weighted op
# and the parameter-less ops after it);
# 1 x n filters pad (0, n // 2), n x 1 filters (n // 2, 0); "valid" convs and
# the reduction max-pools are unpadded.

def _v4_stem(n):
    t = _cbr(n, 0, 32, 3, stride=2, first=True)                 # 149 x 149
    t = _cbr(n, t, 32, 3, first=True)                           # 147
    t = _cbr(n, t, 64, 3, pad=1, first=True)
    p = n.maxpool(t, 3, 2)                                      # 73
    c = _cbr(n, t, 96, 3, stride=2, first=True)
    t = n.concat(p, c)                                          # 160 channels
    a = _cbr(n, t, 64, 1, first=True)
    b = _cbr(n, t, 64, 1)
    a = _cbr(n, a, 96, 3, first=True)                           # 71
    b = _cbr(n, b, 64, (7, 1), pad=(3, 0))
    b = _cbr(n, b, 64, (1, 7), pad=(0, 3), first=True)
    b = _cbr(n, b, 96, 3, first=True)
    t = n.concat(a, b)                                          # 192
    p = n.maxpool(t, 3, 2)
    c = _cbr(n, t, 192, 3, stride=2, first=True)                # 35
    return n.concat(c, p)                                       # 384


def _v4_a(n, x):
    p = _cbr(n, n.avgpool(x, 3, 1, pad=1), 96, 1, first=True)
    b1 = _cbr(n, x, 96, 1)
    b2 = _cbr(n, x, 64, 1)
    b3 = _cbr(n, x, 64, 1)
    b2 = _cbr(n, b2, 96, 3, pad=1, first=True)
    b3 = _cbr(n, b3, 96, 3, pad=1)
    b3 = _cbr(n, b3, 96, 3, pad=1, first=True)
    return n.concat(p, b1, b2, b3)                              # 384


def _v4_reduction_a(n, x):
    p = n.maxpool(x, 3, 2)                                      # 17
    b1 = _cbr(n, x, 384, 3, stride=2, first=True)
    b2 = _cbr(n, x, 192, 1)
    b2 = _cbr(n, b2, 224, 3, pad=1, first=True)
    b2 = _cbr(n, b2, 256, 3, stride=2, first=True)
    return n.concat(p, b1, b2)                                  # 1024


def _v4_b(n, x):
    p = _cbr(n, n.avgpool(x, 3, 1, pad=1), 128, 1, first=True)
    b1 = _cbr(n, x, 384, 1)
    b2 = _cbr(n, x, 192, 1)
    b3 = _cbr(n, x, 192, 1)
    b2 = _cbr(n, b2, 224, (1, 7), pad=(0, 3), first=True)
    b3 = _cbr(n, b3, 192, (1, 7), pad=(0, 3))
    b2 = _cbr(n, b2, 256, (7, 1), pad=(3, 0), first=True)
    b3 = _cbr(n, b3, 224, (7, 1), pad=(3, 0))
    b3 = _cbr(n, b3, 224, (1, 7), pad=(0, 3), first=True)
    b3 = _cbr(n, b3, 256, (7, 1), pad=(3, 0), first=True)
    return n.concat(p, b1, b2, b3)                              # 1024


def _v4_reduction_b(n, x):
    p = n.maxpool(x, 3, 2)                                      # 8
    b1 = _cbr(n, x, 192, 1, first=True)
    b2 = _cbr(n, x, 256, 1)
    b1 = _cbr(n, b1, 192, 3, stride=2, first=True)
    b2 = _cbr(n, b2, 256, (1, 7), pad=(0, 3))
    b2 = _cbr(n, b2, 320, (7, 1), pad=(3, 0), first=True)
    b2 = _cbr(n, b2, 320, 3, stride=2, first=True)
    return n.concat(p, b1, b2)                                  # 1536


def _v4_c(n, x):
    p = _cbr(n, n.avgpool(x, 3, 1, pad=1), 256, 1, first=True)
    b1 = _cbr(n, x, 256, 1)
    b2 = _cbr(n, x, 384, 1)
    b3 = _cbr(n, x, 384, 1)
    b2a = _cbr(n, b2, 256, (1, 3), pad=(0, 1), first=True)
    b2b = _cbr(n, b2, 256, (3, 1), pad=(1, 0))
    b3 = _cbr(n, b3, 448, (1, 3), pad=(0, 1))
    b3 = _cbr(n, b3, 512, (3, 1), pad=(1, 0), first=True)
    b3a = _cbr(n, b3, 256, (1, 3), pad=(0, 1), first=True)
    b3b = _cbr(n, b3, 256, (3, 1), pad=(1, 0))
    # six parts, concat takes four: the channel order is that of one flat concat
    return n.concat(n.concat(p, b1, b2a, b2b), b3a, b3b)       # 1536


def inception_v4():
    n = NetBuilder()
    t = _v4_stem(n)
    for _ in range(4):
        t = _v4_a(n, t)
    t = _v4_reduction_a(n, t)
    for _ in range(7):
        t = _v4_b(n, t)
    t = _v4_reduction_b(n, t)
    for _ in range(3):
        t = _v4_c(n, t)
    n.fc(n.gap(t), 1000)
    return n.ops, (299, 299, 3), 1000


BUILDERS = {"tiny": tiny, "alexnet": alexnet, "resnet18": resnet18, "vgg16": vgg16, "resnet50": resnet50,
            "googlenet": googlenet, "vgg19": vgg19, "resnet152": resnet152, "inception_v4": inception_v4}

# The workloads' batch size, emulated link rate (bytes/s; 1 Gb/s = 1.25e8 B/s),
# input seed and SGD learning rate (1e-3 for the two networks without
# BatchNorm, whose loss diverges within three steps at 1e-2 from He-normal
# weights on N(0,1) images).
WORKLOADS = {
    "tiny": {"batch": 4, "link": 1e9, "seed": 0, "lr": 1e-2},
    "alexnet": {"batch": 32, "link": 100e6 / 8, "seed": 1, "lr": 1e-3},
    "resnet18": {"batch": 128, "link": 1e9 / 8, "seed": 2, "lr": 1e-2},
    "vgg16": {"batch": 32, "link": 10e9 / 8, "seed": 3, "lr": 1e-3},
    "resnet50": {"batch": 64, "link": 10e9 / 8, "seed": 4, "lr": 1e-2},
    "googlenet": {"batch": 32, "link": 10e9 / 8, "seed": 5, "lr": 1e-2},
    "vgg19": {"batch": 32, "link": 10e9 / 8, "seed": 6, "lr": 1e-3},
    "resnet152": {"batch": 32, "link": 10e9 / 8, "seed": 7, "lr": 1e-2},
    "inception_v4": {"batch": 32, "link": 10e9 / 8, "seed": 8, "lr": 1e-2},
}


def build(name):
    return BUILDERS[name]()


def shapes(ops, hwc):
    """(h, w, c) of every tensor: the input, then each op's output (FC and GAP give 1 x 1)."""
    out = [(hwc[0], hwc[1], hwc[2])]
    for (kind, _layer, src, other, out_ch, r, s, stride, pad, bias, in2, in3, pad_w) in ops:
        h, w, c = out[src]
        if kind == DC_OP_CONCAT:
            out.append((h, w, sum(out[t][2] for t in (src, other, in2, in3) if t >= 0)))
        elif kind in (DC_OP_CONV, DC_OP_MAXPOOL, DC_OP_AVGPOOL):
            out.append(((h + 2 * pad - r) // stride + 1, (w + 2 * pad_w - s) // stride + 1,
                        out_ch if kind == DC_OP_CONV else c))
        elif kind == DC_OP_FC:
            out.append((1, 1, out_ch))
        elif kind == DC_OP_GAP:
            out.append((1, 1, c))
        else:
            out.append((h, w, c))
    return out


def param_specs(ops, hwc):
    """Initialisation kinds of the parameter tensors in parameter-server order.

    He-normal for conv / FC weights (fan-in = r*s*c or in-features), zeros for
    biases and BN beta, ones for BN gamma - the argument list of
    ``synth.cnn_inputs``.
    """
    shp = shapes(ops, hwc)
    specs = []
    for (kind, _layer, src, other, out_ch, r, s, stride, pad, bias, in2, in3, pad_w) in ops:
        h, w, c = shp[src]
        if kind == DC_OP_CONV:
            specs.append(("he", out_ch * r * s * c, r * s * c))
            if bias:
                specs.append(("zeros", out_ch))
        elif kind == DC_OP_FC:
            specs.append(("he", out_ch * h * w * c, h * w * c))
            if bias:
                specs.append(("zeros", out_ch))
        elif kind == DC_OP_BN:
            specs.append(("ones", c))
            specs.append(("zeros", c))
    return specs


def conv_geoms(ops, hwc, batch):
    """(op index, dc_conv_shape fields incl. pad_w, reads_input_batch) of every conv / FC op; FC as a 1x1 conv."""
    shp = shapes(ops, hwc)
    out = []
    for i, (kind, _layer, src, other, out_ch, r, s, stride, pad, bias, in2, in3, pad_w) in enumerate(ops):
        h, w, c = shp[src]
        if kind == DC_OP_CONV:
            out.append((i, (batch, h, w, c, out_ch, r, s, stride, pad, pad_w), src == 0))
        elif kind == DC_OP_FC:
            out.append((i, (batch, 1, 1, h * w * c, out_ch, 1, 1, 1, 0, 0), src == 0))
    return out
