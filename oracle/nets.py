"""Network definitions for the oracle (test infrastructure only).

The synthetic workloads, written independently of the product library's own
definitions.  A network is a list of operations in forward order; tensor 0 is
the input batch and tensor i+1 is the output of operation i.

Each operation carries the planner layer it belongs to.  Following the layer
decomposition of Sec. III-A, one layer is one weighted operation (conv or FC)
together with the parameter-less operations that follow it (ReLU, pooling,
flatten, residual add, global average pooling); BatchNorm's scale and shift
belong to the convolution they normalise, and branches at the same depth form
one layer, so a residual block's 1x1 projection joins the layer of the block's
first convolution.

Parameter-server order: layers in order, and within a layer the operations in
forward order, each contributing conv/FC weight then bias, or BN gamma then
beta.  Conv weights are KRSC, FC weights [out][in] over the NHWC-flattened
input.
"""
from __future__ import annotations


def _op(kind, inp, layer, **kw):
    d = {"op": kind, "in": inp, "layer": layer}
    d.update(kw)
    return d


class _Builder:
    def __init__(self):
        self.ops = []
        self.layer = 0

    def new_layer(self):
        self.layer += 1

    def add(self, kind, inp, **kw):
        self.ops.append(_op(kind, inp, self.layer, **kw))
        return len(self.ops)  # tensor id of the output

    def conv(self, inp, k, r, stride=1, pad=0, bias=True):
        """r: filter size, or (rows, columns); pad: padding, or (rows, columns)."""
        rr, ss = r if isinstance(r, tuple) else (r, r)
        ph, pw = pad if isinstance(pad, tuple) else (pad, pad)
        return self.add("conv", inp, k=k, r=rr, s=ss, stride=stride, pad=ph, pad_w=pw, bias=bias)

    def fc(self, inp, out, bias=True):
        return self.add("fc", inp, out=out, bias=bias)


def tiny():
    """Tiny CNN: conv3x3(3->8)+ReLU+maxpool2, conv3x3(8->16)+ReLU+maxpool2, FC(1024->64)+ReLU, FC(64->10)."""
    b = _Builder()
    t = 0
    for k in (8, 16):
        b.new_layer()
        t = b.conv(t, k, 3, pad=1)
        t = b.add("relu", t)
        t = b.add("maxpool", t, r=2, s=2, stride=2, pad=0)
    b.new_layer()
    t = b.fc(t, 64)
    t = b.add("relu", t)
    b.new_layer()
    b.fc(t, 10)
    return {"name": "tiny", "ops": b.ops, "hwc": (32, 32, 3), "classes": 10}


def alexnet():
    """AlexNet-style 8-layer CNN (no LRN, no dropout; paddings 2, 2, 1, 1, 1)."""
    b = _Builder()
    t = 0
    spec = [(64, 11, 4, 2, True), (192, 5, 1, 2, True), (384, 3, 1, 1, False),
            (256, 3, 1, 1, False), (256, 3, 1, 1, True)]
    for k, r, st, pad, pool in spec:
        b.new_layer()
        t = b.conv(t, k, r, stride=st, pad=pad)
        t = b.add("relu", t)
        if pool:
            t = b.add("maxpool", t, r=3, s=3, stride=2, pad=0)
    for out, relu in ((4096, True), (4096, True), (1000, False)):
        b.new_layer()
        t = b.fc(t, out)
        if relu:
            t = b.add("relu", t)
    return {"name": "alexnet", "ops": b.ops, "hwc": (224, 224, 3), "classes": 1000}


def _vgg(name, cfg):
    b = _Builder()
    t = 0
    for v in cfg:
        if v == "M":
            t = b.add("maxpool", t, r=2, s=2, stride=2, pad=0)
        else:
            b.new_layer()
            t = b.conv(t, v, 3, pad=1)
            t = b.add("relu", t)
    for out, relu in ((4096, True), (4096, True), (1000, False)):
        b.new_layer()
        t = b.fc(t, out)
        if relu:
            t = b.add("relu", t)
    return {"name": name, "ops": b.ops, "hwc": (224, 224, 3), "classes": 1000}


def vgg16():
    """VGG-16 (configuration D): 13 conv3x3 pad 1 with ReLU, five 2x2 max-pools, FC 25088->4096->4096->1000."""
    return _vgg("vgg16", [64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M", 512, 512, 512, "M"])


def vgg19():
    """VGG-19 (configuration E): 16 conv3x3, otherwise as VGG-16."""
    return _vgg("vgg19", [64, 64, "M", 128, 128, "M", 256, 256, 256, 256, "M", 512, 512, 512, 512, "M",
                          512, 512, 512, 512, "M"])


def resnet18_small():
    """ResNet-18 for 32x32 inputs: 3x3 stem, 4 stages of 2 basic blocks, global avg-pool, FC 512->10."""
    b = _Builder()
    b.new_layer()
    t = b.conv(0, 64, 3, pad=1, bias=False)
    t = b.add("bn", t)
    t = b.add("relu", t)
    cin = 64
    for cout, first_stride in ((64, 1), (128, 2), (256, 2), (512, 2)):
        for blk in range(2):
            st = first_stride if blk == 0 else 1
            x = t
            b.new_layer()
            u = b.conv(x, cout, 3, stride=st, pad=1, bias=False)
            u = b.add("bn", u)
            u = b.add("relu", u)
            short = x
            if st != 1 or cin != cout:
                short = b.conv(x, cout, 1, stride=st, pad=0, bias=False)
                short = b.add("bn", short)
            b.new_layer()
            u = b.conv(u, cout, 3, pad=1, bias=False)
            u = b.add("bn", u)
            u = b.add("add", u, other=short)
            t = b.add("relu", u)
            cin = cout
    t = b.add("gap", t)
    b.new_layer()
    b.fc(t, 10)
    return {"name": "resnet18", "ops": b.ops, "hwc": (32, 32, 3), "classes": 10}


def _bottleneck_resnet(name, stages):
    b = _Builder()
    b.new_layer()
    t = b.conv(0, 64, 7, stride=2, pad=3, bias=False)
    t = b.add("bn", t)
    t = b.add("relu", t)
    t = b.add("maxpool", t, r=3, s=3, stride=2, pad=1)
    cin = 64
    for width, blocks, first_stride in zip((64, 128, 256, 512), stages, (1, 2, 2, 2)):
        cout = 4 * width
        for blk in range(blocks):
            st = first_stride if blk == 0 else 1
            x = t
            b.new_layer()
            u = b.conv(x, width, 1, bias=False)
            u = b.add("bn", u)
            u = b.add("relu", u)
            short = x
            if blk == 0:
                short = b.conv(x, cout, 1, stride=st, pad=0, bias=False)
                short = b.add("bn", short)
            b.new_layer()
            u = b.conv(u, width, 3, stride=st, pad=1, bias=False)
            u = b.add("bn", u)
            u = b.add("relu", u)
            b.new_layer()
            u = b.conv(u, cout, 1, bias=False)
            u = b.add("bn", u)
            u = b.add("add", u, other=short)
            t = b.add("relu", u)
            cin = cout
    t = b.add("gap", t)
    b.new_layer()
    b.fc(t, 1000)
    return {"name": name, "ops": b.ops, "hwc": (224, 224, 3), "classes": 1000}


def resnet50():
    """ResNet-50 (stride on the 3x3 conv of a bottleneck, projection in each stage's first block)."""
    return _bottleneck_resnet("resnet50", (3, 4, 6, 3))


def resnet152():
    """ResNet-152: bottleneck stages of 3, 8, 36 and 3 blocks, otherwise as ResNet-50."""
    return _bottleneck_resnet("resnet152", (3, 8, 36, 3))


def googlenet():
    """GoogLeNet (Inception v1, 5x5 convs in the third branch, no LRN / dropout / auxiliary heads).

    Each Inception module is two planner layers (branches at the same depth
    form one layer): its four depth-1 convs (1x1, 3x3-reduce, 5x5-reduce and
    the projection after the 3x3/1 max-pool) and its two depth-2 convs (3x3,
    5x5) followed by the channel concatenation of the four branches.
    """
    b = _Builder()
    b.new_layer()
    t = b.conv(0, 64, 7, stride=2, pad=3)
    t = b.add("relu", t)
    t = b.add("maxpool", t, r=3, s=3, stride=2, pad=1)
    b.new_layer()
    t = b.add("relu", b.conv(t, 64, 1))
    b.new_layer()
    t = b.add("relu", b.conv(t, 192, 3, pad=1))
    t = b.add("maxpool", t, r=3, s=3, stride=2, pad=1)
    spec = [(64, 96, 128, 16, 32, 32), (128, 128, 192, 32, 96, 64), "M",
            (192, 96, 208, 16, 48, 64), (160, 112, 224, 24, 64, 64), (128, 128, 256, 24, 64, 64),
            (112, 144, 288, 32, 64, 64), (256, 160, 320, 32, 128, 128), "M",
            (256, 160, 320, 32, 128, 128), (384, 192, 384, 48, 128, 128)]
    for m in spec:
        if m == "M":
            t = b.add("maxpool", t, r=3, s=3, stride=2, pad=1)
            continue
        c1, r3, c3, r5, c5, pp = m
        b.new_layer()
        b1 = b.add("relu", b.conv(t, c1, 1))
        b3 = b.add("relu", b.conv(t, r3, 1))
        b5 = b.add("relu", b.conv(t, r5, 1))
        bp = b.add("maxpool", t, r=3, s=3, stride=1, pad=1)
        bp = b.add("relu", b.conv(bp, pp, 1))
        b.new_layer()
        b3 = b.add("relu", b.conv(b3, c3, 3, pad=1))
        b5 = b.add("relu", b.conv(b5, c5, 5, pad=2))
        t = b.add("concat", b1, others=[b3, b5, bp])
    t = b.add("gap", t)
    b.new_layer()
    b.fc(t, 1000)
    return {"name": "googlenet", "ops": b.ops, "hwc": (224, 224, 3), "classes": 1000}


def inception_v4():
    """Inception-v4 (stem, 4 x Inception-A, Reduction-A, 7 x Inception-B,
    Reduction-B, 3 x Inception-C, global average pooling, FC 1536 -> 1000) on
    299 x 299 inputs.  Every convolution is bias-free and followed by BN and
    ReLU; "V" convolutions and pools are unpadded, the others keep the size
    (a 1 x 7 filter pads 3 columns, a 7 x 1 filter 3 rows).  The pooling
    branch of modules A, B and C is a 3 x 3 / 1 average pool padded by one,
    averaging the in-image taps only.  No dropout, no auxiliary head.

    Planner layers follow depth: inside a module, the convolutions at the same
    distance from the module input form one layer (in the order of the
    branches in the concatenation), a pool that opens a branch joins the
    layer before it, and the concatenation joins the module's last layer.
    Operations are listed layer by layer.
    """
    b = _Builder()

    def cbr(inp, k, r, stride=1, pad=0):
        return b.add("relu", b.add("bn", b.conv(inp, k, r, stride=stride, pad=pad, bias=False)))

    def module(t, branches, tail=None):
        """branches: per branch a list of steps, each ("conv", k, r, stride, pad) or
        ("avg",) or ("max",); a step may be ("split", [conv, conv]) to end the
        branch in parallel convs."""
        heads = [t] * len(branches)
        outs = [None] * len(branches)
        pos = [0] * len(branches)
        while any(pos[i] < len(br) for i, br in enumerate(branches)):
            # pools are parameter-less: they join the layer that is open
            for i, br in enumerate(branches):
                while pos[i] < len(br) and br[pos[i]][0] in ("avg", "max"):
                    if br[pos[i]][0] == "avg":
                        heads[i] = b.add("avgpool", heads[i], r=3, s=3, stride=1, pad=1)
                    else:
                        heads[i] = b.add("maxpool", heads[i], r=3, s=3, stride=2, pad=0)
                    pos[i] += 1
                    if pos[i] == len(br):
                        outs[i] = [heads[i]]
            if all(pos[i] == len(br) for i, br in enumerate(branches)):
                break
            b.new_layer()
            for i, br in enumerate(branches):
                if pos[i] >= len(br):
                    continue
                step = br[pos[i]]
                if step[0] == "split":
                    outs[i] = [cbr(heads[i], *c) for c in step[1]]
                else:
                    heads[i] = cbr(heads[i], *step[1:])
                    if pos[i] + 1 == len(br):
                        outs[i] = [heads[i]]
                pos[i] += 1
        parts = [o for out in outs for o in out]
        return b.add("concat", parts[0], others=parts[1:])

    b.new_layer()
    t = cbr(0, 32, 3, stride=2)
    b.new_layer()
    t = cbr(t, 32, 3)
    b.new_layer()
    t = cbr(t, 64, 3, pad=1)
    t = module(t, [[("max",)], [("conv", 96, 3, 2, 0)]])
    t = module(t, [[("conv", 64, 1), ("conv", 96, 3)],
                   [("conv", 64, 1), ("conv", 64, (7, 1), 1, (3, 0)), ("conv", 64, (1, 7), 1, (0, 3)),
                    ("conv", 96, 3)]])
    t = module(t, [[("conv", 192, 3, 2, 0)], [("max",)]])
    for _ in range(4):
        t = module(t, [[("avg",), ("conv", 96, 1)],
                       [("conv", 96, 1)],
                       [("conv", 64, 1), ("conv", 96, 3, 1, 1)],
                       [("conv", 64, 1), ("conv", 96, 3, 1, 1), ("conv", 96, 3, 1, 1)]])
    t = module(t, [[("max",)],
                   [("conv", 384, 3, 2, 0)],
                   [("conv", 192, 1), ("conv", 224, 3, 1, 1), ("conv", 256, 3, 2, 0)]])
    for _ in range(7):
        t = module(t, [[("avg",), ("conv", 128, 1)],
                       [("conv", 384, 1)],
                       [("conv", 192, 1), ("conv", 224, (1, 7), 1, (0, 3)), ("conv", 256, (7, 1), 1, (3, 0))],
                       [("conv", 192, 1), ("conv", 192, (1, 7), 1, (0, 3)), ("conv", 224, (7, 1), 1, (3, 0)),
                        ("conv", 224, (1, 7), 1, (0, 3)), ("conv", 256, (7, 1), 1, (3, 0))]])
    t = module(t, [[("max",)],
                   [("conv", 192, 1), ("conv", 192, 3, 2, 0)],
                   [("conv", 256, 1), ("conv", 256, (1, 7), 1, (0, 3)), ("conv", 320, (7, 1), 1, (3, 0)),
                    ("conv", 320, 3, 2, 0)]])
    split = ("split", [(256, (1, 3), 1, (0, 1)), (256, (3, 1), 1, (1, 0))])
    for _ in range(3):
        t = module(t, [[("avg",), ("conv", 256, 1)],
                       [("conv", 256, 1)],
                       [("conv", 384, 1), split],
                       [("conv", 384, 1), ("conv", 448, (1, 3), 1, (0, 1)), ("conv", 512, (3, 1), 1, (1, 0)),
                        split]])
    t = b.add("gap", t)
    b.new_layer()
    b.fc(t, 1000)
    return {"name": "inception_v4", "ops": b.ops, "hwc": (299, 299, 3), "classes": 1000}


NETS = {"tiny": tiny, "alexnet": alexnet, "resnet18": resnet18_small, "vgg16": vgg16, "resnet50": resnet50,
        "googlenet": googlenet, "vgg19": vgg19, "resnet152": resnet152, "inception_v4": inception_v4}


def get(name):
    return NETS[name]()
