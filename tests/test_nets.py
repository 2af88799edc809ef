"""The product's workload definitions against the oracle's (host logic, no GPU).

The two sides describe each network independently; here they must agree on
the parameter tensors in server order, on every layer's byte count and on
the layers' conv / pool geometry, and the product's op lists must obey the
rules dc_model_create enforces (contiguous, non-decreasing layers, each
opened by a CONV or FC op, the pools' row and column padding equal).
"""
from collections import Counter, defaultdict

import pytest

from oracle import cnn as OC
from oracle import nets as ON
from paper_2101_07968_amd import _lib as D
from paper_2101_07968_amd import nets as PN

NAMES = sorted(PN.BUILDERS)
KIND = {"conv": D.DC_OP_CONV, "maxpool": D.DC_OP_MAXPOOL, "avgpool": D.DC_OP_AVGPOOL}


def test_same_workloads():
    assert set(PN.BUILDERS) == set(ON.NETS) == set(PN.WORKLOADS)


@pytest.mark.parametrize("name", NAMES)
def test_product_net_matches_oracle(name):
    ops, hwc, classes = PN.build(name)
    spec = ON.get(name)
    assert tuple(hwc) == tuple(spec["hwc"]) and classes == spec["classes"]
    onet = OC.Net(spec, 1)
    assert PN.param_specs(ops, hwc) == onet.param_specs
    assert max(o[1] for o in ops) == onet.L
    # per layer: the same conv and pool geometries on the same input shapes
    # (the op lists themselves may differ: the product nests concats of more
    # than four parts)
    sh = PN.shapes(ops, hwc)
    mine, theirs = defaultdict(Counter), defaultdict(Counter)
    for o in ops:
        if o[0] in KIND.values():
            mine[o[1]][(o[0], tuple(sh[o[2]]), o[4] if o[0] == D.DC_OP_CONV else 0, o[5], o[6], o[7], o[8],
                        o[12])] += 1
    for o in spec["ops"]:
        if o["op"] in KIND:
            theirs[o["layer"]][(KIND[o["op"]], tuple(onet.shapes[o["in"]][1:]), o.get("k", 0), o["r"], o["s"],
                                o["stride"], o["pad"], o.get("pad_w", o["pad"]))] += 1
    assert mine == theirs
    assert tuple(sh[-1]) == tuple(onet.shapes[-1][1:])


@pytest.mark.parametrize("name", NAMES)
def test_product_ops_follow_model_rules(name):
    ops, _, _ = PN.build(name)
    prev = 0
    for i, o in enumerate(ops):
        kind, layer = o[0], o[1]
        assert layer in (prev, prev + 1), i
        if layer == prev + 1:
            assert kind in (D.DC_OP_CONV, D.DC_OP_FC), i
        if kind in (D.DC_OP_MAXPOOL, D.DC_OP_AVGPOOL):
            assert o[12] == o[8], i
        assert 0 <= o[2] <= i
        prev = layer
    assert ops[0][1] == 1
