"""Launch-plan selection on the host (no GPU): candidates, pins and the table of measured plans.

Which plan runs a conv pass changes how its sums are tiled and split, never
what they are; the GPU parity of every candidate plan is in
test_gpu_kernels.py.  Here: the candidate list holds the cost model's choice,
pins take effect and come off, invalid pins are refused, and every entry of
the compiled-in table is a candidate of its shape and is what the planner
picks for it.
"""
import os
import re

import pytest

from paper_2101_07968_amd import _lib as D
from paper_2101_07968_amd import nets as PN

INC = os.path.join(os.path.dirname(D.__file__), "csrc", "plan_table.inc")


def _table():
    rows = []
    for line in open(INC):
        m = re.match(r"\s*\{([-\d,\s]+)\},", line)
        if m:
            v = [int(t) for t in m.group(1).split(",")]
            assert len(v) == 14, line
            rows.append((v[0], tuple(v[1:11]), tuple(v[11:14])))
    return rows


SHAPES = [(32, 14, 14, 256, 256, 3, 3, 1, 1, 1), (32, 17, 17, 224, 256, 7, 1, 1, 3, 0),
          (32, 224, 224, 3, 64, 3, 3, 1, 1, 1), (32, 1, 1, 4096, 1000, 1, 1, 1, 0, 0),
          (2, 9, 9, 4, 8, 3, 3, 2, 1, 1)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("pas", [0, 1, 2])
def test_candidates_hold_the_model_choice_and_pins_apply(shape, pas):
    D.conv_set_plan(shape, pas, -1)
    try:
        model = D.conv_plan_info(shape, pas)
        cands = D.conv_plan_candidates(shape, pas)
        assert model[:3] in cands and model[7] == 0
        assert len(set(cands)) == len(cands)
        for mt, nt, sp in cands:
            assert (mt, nt) in ((128, 128), (128, 64), (64, 128), (64, 64)) and sp >= 1
        for plan in (cands[0], cands[-1]):
            D.conv_set_plan(shape, pas, *plan)
            info = D.conv_plan_info(shape, pas)
            assert info[:3] == plan and info[7] == 2
            assert info[3:7] == model[3:7]   # the GEMM itself does not change
        with pytest.raises(D.DcError):
            D.conv_set_plan(shape, pas, 96, 64, 1)
        with pytest.raises(D.DcError):
            D.conv_set_plan(shape, pas, 64, 64, 10 ** 6)
    finally:
        D.conv_set_plan(shape, pas, 0)


def test_workspace_follows_the_pinned_plan():
    shape = (32, 14, 14, 512, 512, 3, 3, 1, 1, 1)
    import ctypes
    sh = D.ConvShape(*shape)
    try:
        D.conv_set_plan(shape, 0, 128, 128, 1)
        D.conv_set_plan(shape, 1, 128, 128, 1)
        D.conv_set_plan(shape, 2, 128, 128, 1)
        small = D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh))   # bias-gradient scratch only
        assert small < 32 * 14 * 14 * 512 * 4
        big = max(D.conv_plan_candidates(shape, 0), key=lambda p: p[2])
        D.conv_set_plan(shape, 0, *big)
        assert D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh)) >= big[2] * 32 * 14 * 14 * 512 * 4
    finally:
        for p in range(3):
            D.conv_set_plan(shape, p, 0)


def test_table_entries_are_candidates_and_are_picked():
    rows = _table()
    keys = set()
    for pas, g, plan in rows:
        assert (pas, g) not in keys, (pas, g)
        keys.add((pas, g))
        assert plan in D.conv_plan_candidates(g, pas), (pas, g, plan)
        info = D.conv_plan_info(g, pas)
        assert info[:3] == plan and info[7] == 1, (pas, g, info)
        # pinning the cost model bypasses the table
        D.conv_set_plan(g, pas, -1)
        try:
            assert D.conv_plan_info(g, pas)[7] == 0
        finally:
            D.conv_set_plan(g, pas, 0)


def test_table_covers_only_workload_shapes():
    """Entries are keyed on the workloads' own geometries at their own batch sizes."""
    known = set()
    for name, wl in PN.WORKLOADS.items():
        ops, hwc, _ = PN.build(name)
        for _i, g, _first in PN.conv_geoms(ops, hwc, wl["batch"]):
            known.add(tuple(g))
    for pas, g, _plan in _table():
        assert g in known, g


RGB = [((32, 224, 224, 3, 64, 3, 3, 1, 1, 1), True), ((32, 299, 299, 3, 32, 3, 3, 2, 0, 0), True),
       ((128, 32, 32, 3, 64, 3, 3, 1, 1, 1), True), ((2, 9, 9, 3, 128, 3, 3, 1, 1, 1), True),
       ((2, 9, 9, 3, 70, 3, 3, 1, 1, 1), False), ((2, 9, 9, 3, 160, 3, 3, 1, 1, 1), False),
       ((2, 9, 9, 3, 16, 3, 3, 1, 1, 1), False), ((32, 224, 224, 3, 64, 7, 7, 2, 3, 3), False),
       ((2, 9, 9, 4, 64, 3, 3, 1, 1, 1), False), ((2, 9, 1, 3, 64, 3, 3, 1, 1, 1), False)]


@pytest.mark.parametrize("shape,direct", RGB, ids=[str(s) for s, _ in RGB])
def test_rgb_layer_takes_the_direct_kernels(shape, direct):
    """Three input channels, a 3 x 3 filter and 32 to 128 output channels in blocks of 32
    (and output rows of at least two pixels): forward and filter gradient report plan source 4,
    the data gradient stays on the implicit GEMM; a pinned plan overrides the direct kernels."""
    src = [D.conv_plan_info(shape, p)[7] for p in range(3)]
    assert (src[0] == 4, src[2] == 4) == (direct, direct), src
    assert src[1] != 4
    if direct:
        mt, nt, sp = D.conv_plan_candidates(shape, 0)[0]
        D.conv_set_plan(shape, 0, mt, nt, sp)
        try:
            assert D.conv_plan_info(shape, 0)[7] == 2
        finally:
            D.conv_set_plan(shape, 0, 0)
        assert D.conv_plan_info(shape, 0)[7] == 4
