"""The C-ABI library on the host: exported symbols and the planner.

libdc.so must export every function that include/dc.h and
include/dc_kernels.h declare.  dc_plan is pure host code, so it is checked
here, without a GPU, against the oracle's transcription of Eq. 8 / Algorithm 3
and Eq. 9 / Algorithm 4: the decisions must be bit-identical and the model
times equal, for random profiles, the tiny workload's fixture and deep
networks.  Error paths of the planner and of model validation are exercised
too (validation fails before any HIP call).
"""
import ctypes
import json
import os
import re

import numpy as np
import pytest

import synth
from oracle import plan as OP
from paper_2101_07968_amd import _lib as D

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in ("dc.h", "dc_kernels.h"):
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for m in re.finditer(r"\b(dc_[a-z0-9_]+)\s*\(", text):
            names.add(m.group(1))
    return sorted(names)


def test_library_exports_every_declared_function():
    lib = D.lib()
    names = declared_functions()
    assert len(names) >= 30
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    assert set(D._SIGS) == set(names), set(D._SIGS) ^ set(names)


def test_strerror():
    lib = D.lib()
    assert lib.dc_strerror(0) == b"ok"
    assert lib.dc_strerror(D.DC_ETIMEOUT) == b"watchdog timeout"


def _check_against_oracle(pt, fc, bc, gt, dt):
    prof = D.Profile(pt, fc, bc, gt, dt)
    plan = D.dc_plan(prof)
    p, g = plan.decisions()
    op, tf, _, _ = OP.forward_dp(pt, fc, dt)
    og, tb, _, _ = OP.backward_dp(bc, gt, dt)
    assert p == op and g == og
    assert plan.t_fwd_ns == tf and plan.t_bwd_ns == tb
    return plan


@pytest.mark.parametrize("block", range(20))
def test_plan_bit_exact_random(block):
    for i in range(150):
        seed = block * 1000 + i
        L = 1 + seed % 20
        hi = (10, 60, 1000, 10 ** 6)[seed % 4]
        pt, fc, bc, gt, dt = synth.random_profile(seed, L, hi=hi, dt_hi=hi // 2 + 1)
        _check_against_oracle(pt, fc, bc, gt, dt)


@pytest.mark.parametrize("L", [50, 75, 120])
def test_plan_bit_exact_deep(L):
    for seed in range(3):
        pt, fc, bc, gt, dt = synth.random_profile(50000 + L * 10 + seed, L, hi=10 ** 7, dt_hi=10 ** 6)
        _check_against_oracle(pt, fc, bc, gt, dt)


def test_plan_tiny_fixture():
    d = json.load(open(os.path.join(ROOT, "tests", "golden", "tiny_plan.json")))
    pr = d["profile"]
    plan = _check_against_oracle(pr["pt"], pr["fc"], pr["bc"], pr["gt"], pr["dt"])
    assert plan.decisions() == (d["p"], d["g"])
    seq = D.dc_plan_sequential(D.Profile(pr["pt"], pr["fc"], pr["bc"], pr["gt"], pr["dt"]))
    assert (seq.t_fwd_ns, seq.t_bwd_ns) == (d["T_fwd_sequential"], d["T_bwd_sequential"])
    lbl = D.dc_plan_lbl(D.Profile(pr["pt"], pr["fc"], pr["bc"], pr["gt"], pr["dt"]))
    assert (lbl.t_fwd_ns, lbl.t_bwd_ns) == (d["T_fwd_lbl"], d["T_bwd_lbl"])


@pytest.mark.parametrize("seed", range(50))
def test_plan_eval_matches_fm(seed):
    L = 2 + seed % 12
    pt, fc, bc, gt, dt = synth.random_profile(70000 + seed, L, hi=5000, dt_hi=3000)
    rng = np.random.default_rng(seed)
    p = rng.integers(0, 2, L - 1).tolist()
    g = rng.integers(0, 2, L - 1).tolist()
    plan = D.dc_plan_eval(D.Profile(pt, fc, bc, gt, dt), p, g)
    assert plan.t_fwd_ns == OP.fm_forward(pt, fc, dt, p)
    assert plan.t_bwd_ns == OP.fm_backward(bc, gt, dt, g)


def test_plan_single_layer():
    plan = D.dc_plan(D.Profile([5], [7], [3], [2], 4))
    assert (plan.t_fwd_ns, plan.t_bwd_ns) == (4 + 5 + 7, 3 + 4 + 2)


def test_plan_rejects_bad_input():
    with pytest.raises(D.DcError) as e:
        D.dc_plan(D.Profile([1, -2], [1, 1], [1, 1], [1, 1], 0))
    assert e.value.status == D.DC_EINVAL
    with pytest.raises(D.DcError) as e:
        D.dc_plan(D.Profile([1, 1], [1, 1], [1, 1], [1, 1], -1))
    assert e.value.status == D.DC_EINVAL
    big = 2 ** 62
    with pytest.raises(D.DcError) as e:
        D.dc_plan(D.Profile([big, big], [1, 1], [1, 1], [1, 1], 0))
    assert e.value.status == D.DC_EINVAL
    # L = 0
    prof = D.Profile([], [], [], [], 0)
    pc, plan = prof.c(), D.PlanT(0, None, None, 0, 0)
    assert D.lib().dc_plan(ctypes.byref(pc), ctypes.byref(plan)) == D.DC_EINVAL


def _create(ops, batch=2, hwc=(8, 8, 3), classes=10):
    arr = (D.OpDesc * len(ops))(*[D.OpDesc(*o) for o in ops])
    h = ctypes.c_void_p()
    st = D.lib().dc_model_create(arr, len(ops), batch, hwc[0], hwc[1], hwc[2], classes, ctypes.byref(h))
    return st, h


def test_model_validation_rejects_bad_descriptions():
    conv = (D.DC_OP_CONV, 1, 0, -1, 4, 3, 3, 1, 1, 1)
    # layer must start with a weighted op
    assert _create([(D.DC_OP_RELU, 1, 0, -1, 0, 0, 0, 0, 0, 0)])[0] == D.DC_EINVAL
    # input tensor from the future
    assert _create([conv, (D.DC_OP_RELU, 1, 5, -1, 0, 0, 0, 0, 0, 0)])[0] == D.DC_EINVAL
    # layers skip a number
    assert _create([conv, (D.DC_OP_FC, 3, 1, -1, 10, 0, 0, 0, 0, 1)])[0] == D.DC_EINVAL
    # logits of the wrong width
    assert _create([conv, (D.DC_OP_FC, 2, 1, -1, 7, 0, 0, 0, 0, 1)])[0] == D.DC_EINVAL
    # an output nobody reads
    assert _create([conv, (D.DC_OP_RELU, 1, 1, -1, 0, 0, 0, 0, 0, 0),
                    (D.DC_OP_FC, 2, 1, -1, 10, 0, 0, 0, 0, 1)])[0] == D.DC_EINVAL
    # ADD of different shapes (4 and 6 channels)
    conv6 = (D.DC_OP_CONV, 1, 1, -1, 6, 3, 3, 1, 1, 1)
    assert _create([conv, conv6, (D.DC_OP_ADD, 1, 2, 1, 0, 0, 0, 0, 0, 0)])[0] == D.DC_EINVAL
    assert b"ADD" in D.lib().dc_last_error()
    # only a CONV / FC reads the input batch, which has no gradient buffer:
    # a conv followed by add(conv output, input batch), and a ReLU of the batch
    assert _create([(D.DC_OP_CONV, 1, 0, -1, 3, 3, 3, 1, 1, 1), (D.DC_OP_ADD, 1, 1, 0, 0, 0, 0, 0, 0, 0),
                    (D.DC_OP_FC, 2, 2, -1, 10, 0, 0, 0, 0, 1)])[0] == D.DC_EINVAL
    assert b"input batch" in D.lib().dc_last_error()
    assert _create([conv, (D.DC_OP_RELU, 1, 0, -1, 0, 0, 0, 0, 0, 0), (D.DC_OP_FC, 2, 2, -1, 10, 0, 0, 0, 0, 1)])[0] \
        == D.DC_EINVAL
    assert b"input batch" in D.lib().dc_last_error()
    # column padding as large as the filter's width (1 x 3 filter padded by 3 columns)
    wide = (D.DC_OP_CONV, 1, 0, -1, 4, 1, 3, 1, 0, 1, -1, -1, 3)
    assert _create([wide, (D.DC_OP_FC, 2, 1, -1, 10, 0, 0, 0, 0, 1)])[0] == D.DC_EINVAL
    # pools pad rows and columns alike
    for kind in (D.DC_OP_MAXPOOL, D.DC_OP_AVGPOOL):
        pool = (kind, 1, 1, -1, 0, 3, 3, 1, 1, 0, -1, -1, 0)
        assert _create([conv, pool, (D.DC_OP_FC, 2, 2, -1, 10, 0, 0, 0, 0, 1)])[0] == D.DC_EINVAL
        assert b"pad_w" in D.lib().dc_last_error()


def test_shape_checks_do_not_overflow():
    """Sizes whose 32-bit products or sums would wrap are refused before any launch."""
    lib = D.lib()
    # padded extent past 2^31: h + 2 pad overflows int
    sh = D.ConvShape(1, 2 ** 31 - 10, 1, 1, 1, 101, 1, 1, 100, 0)
    assert lib.dc_conv2d_workspace_bytes(ctypes.byref(sh)) == 0
    out = (ctypes.c_int32 * 8)()
    assert lib.dc_conv2d_plan_info(ctypes.byref(sh), 0, out) == D.DC_EINVAL
    # a pooling window of 65536 x 65536 taps: r * s wraps to 0 in 32 bits
    ps = D.PoolShape(0, 65536, 65536, 1, 65536, 65536, 1, 0)
    assert lib.dc_maxpool_forward(ctypes.byref(ps), None, None, None, None) == D.DC_EINVAL
    assert lib.dc_avgpool_forward(ctypes.byref(ps), None, None, None) == D.DC_EINVAL
    # channel offset + width past 2^31
    for fn in ("dc_concat_forward", "dc_concat_backward"):
        args = [0, 1, 10, 2 ** 31 - 1, None] + ([0] if fn == "dc_concat_backward" else []) + [None, None]
        assert getattr(lib, fn)(*args) == D.DC_EINVAL, fn
    # a concatenation of two 2^30-channel tensors: 2^31 channels
    big = (D.DC_OP_CONV, 1, 0, -1, 2 ** 30, 1, 1, 1, 0, 0)
    st, _ = _create([big, big, (D.DC_OP_CONCAT, 1, 1, 2, 0, 0, 0, 0, 0, 0, -1, -1, 0),
                     (D.DC_OP_FC, 2, 3, -1, 10, 0, 0, 0, 0, 1)], batch=1, hwc=(1, 1, 1))
    assert st == D.DC_EINVAL and b"channels" in lib.dc_last_error()
    # an input batch of 2^31 elements
    assert _create([(D.DC_OP_FC, 1, 0, -1, 10, 0, 0, 0, 0, 1)], batch=2, hwc=(32768, 32768, 1))[0] == D.DC_EINVAL
    assert b"input batch" in lib.dc_last_error()


@pytest.mark.parametrize("block", range(10))
def test_ibatch_bit_exact(block):
    for i in range(100):
        seed = 90000 + block * 1000 + i
        L = 1 + seed % 18
        hi = (10, 80, 1000, 10 ** 6)[seed % 4]
        pt, fc, bc, gt, dt = synth.random_profile(seed, L, hi=hi, dt_hi=hi // 2 + 1)
        plan = D.dc_plan_ibatch(D.Profile(pt, fc, bc, gt, dt))
        p, g = plan.decisions()
        assert p == OP.ibatch_forward(pt, fc, dt)
        og, tb = OP.ibatch_backward(bc, gt, dt)
        assert g == og and plan.t_bwd_ns == tb
        assert plan.t_fwd_ns == OP.fm_forward(pt, fc, dt, p)


def test_ibatch_hand_fixture_through_abi():
    d = json.load(open(os.path.join(ROOT, "tests", "golden", "ibatch_hand.json")))
    f, b = d["forward"], d["backward"]
    plan = D.dc_plan_ibatch(D.Profile(f["pt"], f["fc"], b["bc"], b["gt"], 3))
    assert plan.decisions() == (f["p"], b["g"])
    assert (plan.t_fwd_ns, plan.t_bwd_ns) == (f["T"], b["T"])


def test_ibatch_hand_worked_cases_through_abi():
    d = json.load(open(os.path.join(ROOT, "tests", "golden", "ibatch_cases.json")))
    for f in d["forward"]:
        z = [0] * len(f["pt"])
        plan = D.dc_plan_ibatch(D.Profile(f["pt"], f["fc"], z, z, f["dt"]))
        assert plan.decisions()[0] == f["p"] and plan.t_fwd_ns == f["T"], f["name"]
    for b in d["backward"]:
        z = [0] * len(b["bc"])
        plan = D.dc_plan_ibatch(D.Profile(z, z, b["bc"], b["gt"], b["dt"]))
        assert plan.decisions()[1] == b["g"] and plan.t_bwd_ns == b["T"], b["name"]


def test_noalloc_forward_refuses_shapes_beyond_its_scratch():
    """dc_conv2d_forward_noalloc checks the plan's scratch against its 64 MiB static array
    on the host, before any HIP call: a 128 x 224 x 224 x 3 input (a 103 MB channel-padded
    copy) is refused.  The pointers are never dereferenced on that path."""
    sh = D.ConvShape(128, 224, 224, 3, 64, 3, 3, 1, 1, 1)
    fake = 1 << 20
    st = D.lib().dc_conv2d_forward_noalloc(ctypes.byref(sh), fake, fake, None, 0, fake, None)
    assert st == D.DC_EINVAL
    assert b"static scratch" in D.lib().dc_last_error()
