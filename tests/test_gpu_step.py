"""The whole iteration through dc_step, against the oracle and the paper's invariants.

* Parity (loss within 1e-4 relative; every parameter tensor's gradient and
  post-step weight within 1e-3 max relative error, or within 5x the scatter of
  float32 evaluations of the same iteration where that scatter exceeds 1e-3)
  on every workload: the tiny one at its own batch of 4, the others at
  reduced batches that the oracle finishes in seconds.
* Scheduling leaves the numbers untouched: results are bit-identical for the
  sequential, layer-by-layer, DP and random segmentations, here and at the
  full batch sizes.
* The partial orders Eq. 1-7 hold in the recorded timeline.
* dc_profile -> dc_plan gives the oracle's decisions on the measured profile,
  and the measured iteration time at a paced link is within 10% of f_m.
"""
import ctypes

import numpy as np
import pytest

import synth
from oracle import cnn as OC
from oracle import nets as ON
from oracle import plan as OP
from paper_2101_07968_amd import _lib as D
from paper_2101_07968_amd import nets as PN
from tests.gpu_helpers import dev, rel_err, report, update_err

pytestmark = pytest.mark.gpu

UNPACED = D.link(1e9, 0, paced=False)


def setup_model(name, batch, seed):
    ops, hwc, classes = PN.build(name)
    specs = PN.param_specs(ops, hwc)
    onet = OC.Net(ON.get(name), batch)
    assert specs == onet.param_specs  # same tensors in the same server order
    x, y, params = synth.cnn_inputs(seed, batch, hwc, classes, specs)
    model = D.Model(ops, batch, hwc, classes)
    assert model.L == onet.L
    assert model.layer_bytes() == onet.layer_bytes()
    model.ps_write(params)
    return model, onet, dev(x), dev(y), x, y, params


def plans_for(L, seed=0):
    rng = np.random.default_rng(seed)
    return {
        "sequential": D.Plan(L),
        "lbl": D.Plan(L, np.ones(max(L - 1, 1)), np.ones(max(L - 1, 1))),
        "random": D.Plan(L, rng.integers(0, 2, max(L - 1, 1)), rng.integers(0, 2, max(L - 1, 1))),
    }


PARITY = [("tiny", 4), ("alexnet", 2), ("resnet18", 8), ("resnet50", 2), ("vgg16", 1), ("googlenet", 2),
          ("vgg19", 1), ("resnet152", 2), ("inception_v4", 1), ("tiny", 1), ("resnet18", 1)]


def gpu_decisions(model, onet, name):
    """The discrete decisions of the model's last step, keyed by oracle op, for the
    oracle's forward: every ReLU's mask (its output > 0) and every max-pool's window
    taps (dc_model_read_tensor; the product's op j + 1 output is its tensor j + 1, and
    its op list nests concatenations of more than four parts, so ops are matched by
    layerwise.op_map)."""
    from tests import layerwise
    omap = layerwise.op_map(PN.build(name)[0], onet)
    prod = {i: j for j, i in omap.items() if i is not None}
    dec = {}
    for i, op in enumerate(onet.ops):
        if op["op"] == "relu":
            dec[i] = model.read_tensor(prod[i] + 1, onet.shapes[i + 1]) > 0
        elif op["op"] == "maxpool":
            dec[i] = model.read_tensor(prod[i] + 1, onet.shapes[i + 1], D.DC_READ_ARGMAX).astype(np.int32)
    return dec


def fp32_spread(spec, onet, x, y, params, g_ref, decisions=None):
    """Per tensor, how far float32-grade evaluations of this iteration land from the oracle.

    Members of the yardstick ensemble:
    * torch's CPU float32 (an independent library evaluation of the network);
    * the same with every parameter scaled by (1 + 2^-24 xi), xi ~ N(0, 1);
    * the float64 oracle with every conv / FC / BN output scaled by
      (1 + eps xi), eps = 2^-23 and 2^-21: the relative storage and
      accumulation error of a float32 implementation.
    Deep ReLU / max-pool / BatchNorm stacks turn such nudges into large,
    discrete gradient changes (a decision near its threshold flips), so the
    float64 result is only determined to within this spread.  Returns the
    per-tensor largest distance from the oracle, for gradients and for the
    post-step weights w - 0.01 g.  With `decisions` every member holds those
    ReLU masks and max-pool taps fixed.
    """
    import torch
    from tests import torch_ref
    rng = np.random.default_rng(1234)
    runs_g = [torch_ref.loss_and_grads(spec, onet, x, y, params, torch.float32, decisions=decisions)[1]]
    pp = params.astype(np.float64) * (1.0 + 2.0 ** -24 * rng.standard_normal(params.size))
    runs_g.append(torch_ref.loss_and_grads(spec, onet, x, y, pp, torch.float32, decisions=decisions)[1])
    for eps in (2.0 ** -23, 2.0 ** -21):
        onet.perturb = lambda i, t, eps=eps: t * (1.0 + eps * rng.standard_normal(t.shape))
        try:
            runs_g.append(onet.loss_and_grads(x, y, params, decisions=decisions)[1])
        finally:
            onet.perturb = None
    w_ref = params.astype(np.float64) - 0.01 * g_ref
    runs_w = [params.astype(np.float64) - 0.01 * r for r in runs_g]
    spread, spread_w = {}, {}
    for i, slots in enumerate(onet.pslots):
        for pname, (off, shape) in slots.items():
            sl = slice(off, off + int(np.prod(shape)))
            spread[(i, pname)] = max(rel_err(r[sl], g_ref[sl]) for r in runs_g)
            spread_w[(i, pname)] = max(rel_err(r[sl], w_ref[sl]) for r in runs_w)
    return spread, spread_w


@pytest.mark.parametrize("name,batch", PARITY, ids=[f"{n}-b{b}" for n, b in PARITY])
def test_step_matches_oracle(name, batch):
    """Loss within 1e-4; each gradient and post-step weight tensor within 1e-3 -
    or, for a tensor whose float32 evaluations scatter wider than that, within
    5x the scatter of the float32 yardstick (see fp32_spread).  Then the same
    against the oracle given the GPU's own ReLU and max-pool decisions."""
    model, onet, xd, yd, x, y, params = setup_model(name, batch, seed=10 + batch)
    print(f"step {name} batch {batch}", flush=True)
    st = model.step(xd, yd, plans_for(model.L)["random"], UNPACED)
    p_new, g = model.ps_read()
    loss_ref, g_ref, p_ref = onet.step(x, y, params)
    spread, spread_w = fp32_spread(ON.get(name), onet, x, y, params, g_ref)
    assert np.isfinite(st["loss"])
    assert abs(st["loss"] - loss_ref) <= 1e-4 * abs(loss_ref), (st["loss"], loss_ref)
    widened, worst, rows = 0, 0.0, []
    for i, slots in enumerate(onet.pslots):
        for pname, (off, shape) in slots.items():
            sl = slice(off, off + int(np.prod(shape)))
            bar = max(1e-3, 5.0 * spread[(i, pname)])
            widened += bar > 1e-3
            err = rel_err(g[sl], g_ref[sl])
            rows.append((i, pname, err, spread[(i, pname)]))
            worst = max(worst, err / bar)
            assert err <= bar, (i, pname, err, spread[(i, pname)])
            bar_w = max(1e-3, 5.0 * spread_w[(i, pname)])
            assert rel_err(p_new[sl], p_ref[sl]) <= bar_w, (i, pname, rel_err(p_new[sl], p_ref[sl]))
            # the update itself, not just the weights, follows w - 0.01 g
            assert update_err(p_new[sl], params[sl], -0.01 * g_ref[sl]) <= 1.01 * bar + 1e-6, (i, pname)
    rows.sort(key=lambda r: -r[2])
    print(f"{name}: {len(rows)} tensors, {widened} with a widened bar, worst err/bar {worst:.3f}; "
          f"largest errors (op, tensor, err, fp32 spread): "
          + ", ".join(f"({i},{p},{e:.1e},{s:.1e})" for i, p, e, s in rows[:4]), flush=True)
    # The same iteration with the GPU's own ReLU masks and max-pool taps given to the
    # oracle: no decision near its threshold can flip, so 1e-3 holds unless float32
    # evaluations with those decisions held scatter wider than 2e-4 (then 5x that).
    dec = gpu_decisions(model, onet, name)
    loss_d, g_d = onet.loss_and_grads(x, y, params, decisions=dec)
    assert abs(st["loss"] - loss_d) <= 1e-4 * abs(loss_d)
    errs = {}
    for i, slots in enumerate(onet.pslots):
        for pname, (off, shape) in slots.items():
            sl = slice(off, off + int(np.prod(shape)))
            errs[(i, pname)] = max(rel_err(g[sl], g_d[sl]), rel_err(p_new[sl], params[sl] - 0.01 * g_d[sl]),
                                   update_err(p_new[sl], params[sl], -0.01 * g_d[sl]) / 1.01)
    spread_d = {}
    if max(errs.values()) > 1e-3:
        spread_d, _ = fp32_spread(ON.get(name), onet, x, y, params, g_d, decisions=dec)
    bars = {k: 1e-3 if spread_d.get(k, 0.0) <= 2e-4 else max(1e-3, 5.0 * spread_d[k]) for k in errs}
    worst_k = max(errs, key=lambda k: errs[k] / bars[k])
    report(f"step {name} b{batch} with the GPU's decisions: {len(errs)} tensors, "
           f"{sum(e > 1e-3 for e in errs.values())} above 1e-3, {sum(b > 1e-3 for b in bars.values())} on a "
           f"widened bar, worst err/bar {errs[worst_k] / bars[worst_k]:.3f} at {worst_k} (err {errs[worst_k]:.1e})")
    fails = [(k, errs[k], spread_d.get(k), bars[k]) for k in errs if errs[k] > bars[k]]
    assert not fails, fails[:5]


@pytest.mark.parametrize("name,batch", [("tiny", 4), ("resnet18", 16), ("resnet50", 2), ("googlenet", 2)])
def test_results_do_not_depend_on_segmentation(name, batch):
    model, onet, xd, yd, x, y, params = setup_model(name, batch, seed=3)
    outs = []
    for key, plan in plans_for(model.L, seed=5).items():
        model.ps_write(params)
        st = model.step(xd, yd, plan, UNPACED)
        p, g = model.ps_read()
        outs.append((key, st["loss"], p, g))
    for key, loss, p, g in outs[1:]:
        assert loss == outs[0][1], key
        np.testing.assert_array_equal(p, outs[0][2], err_msg=key)
        np.testing.assert_array_equal(g, outs[0][3], err_msg=key)


FULL = [("tiny", 4, 0), ("alexnet", 32, 1), ("resnet18", 128, 2), ("vgg16", 32, 3), ("resnet50", 64, 4),
        ("googlenet", 32, 5), ("vgg19", 32, 6), ("resnet152", 32, 7), ("inception_v4", 32, 8)]


@pytest.mark.parametrize("name,batch,seed", FULL, ids=[f"{n}-b{b}" for n, b, _ in FULL])
def test_full_size_invariance(name, batch, seed):
    """At the benchmark's sizes: finite loss, nonzero update, identical results for three segmentations."""
    ops, hwc, classes = PN.build(name)
    specs = PN.param_specs(ops, hwc)
    x, y, params = synth.cnn_inputs(seed, batch, hwc, classes, specs)
    model = D.Model(ops, batch, hwc, classes)
    xd, yd = dev(x), dev(y)
    ref = None
    print(f"full-size {name} batch {batch}", flush=True)
    for key, plan in plans_for(model.L, seed=seed).items():
        model.ps_write(params)
        st = model.step(xd, yd, plan, UNPACED)
        p, g = model.ps_read()
        assert np.isfinite(st["loss"]) and np.isfinite(g).all()
        assert np.abs(g).max() > 0
        if ref is None:
            ref = (st["loss"], p, g)
        else:
            assert st["loss"] == ref[0], key
            np.testing.assert_array_equal(g, ref[2], err_msg=key)
            np.testing.assert_array_equal(p, ref[1], err_msg=key)
    # the last layer's bias gradient sums to zero: softmax minus one-hot over each sample
    lo, cnt = model.layer_range(model.L)
    assert abs(float(ref[2][lo + cnt - classes:lo + cnt].astype(np.float64).sum())) <= 1e-5


def _check_partial_orders(tl, eps):
    L = tl.shape[0]
    pull_s, pull_e, f_s, f_e, b_s, b_e, push_s, push_e = (tl[:, i] for i in range(8))
    for l in range(L):
        assert pull_e[l] <= f_s[l] + eps                           # Eq. 1
        assert b_e[l] <= push_s[l] + eps                           # Eq. 2
        assert f_e[l] <= b_s[l] + eps                              # Eq. 3
    for m in range(L):
        for n in range(m + 1, L):
            assert pull_e[m] <= pull_s[n] + eps or pull_s[m] == pull_s[n]   # Eq. 4
            assert f_e[m] <= f_s[n] + eps                                    # Eq. 5
            assert b_e[n] <= b_s[m] + eps                                    # Eq. 6
            assert push_e[n] <= push_s[m] + eps or push_s[m] == push_s[n]   # Eq. 7


@pytest.mark.parametrize("name,batch,rate", [("tiny", 4, 2e8), ("resnet18", 32, 2e9)])
def test_profile_plan_timeline_and_model(name, batch, rate):
    model, onet, xd, yd, x, y, params = setup_model(name, batch, seed=7)
    lnk = D.link(rate, 0, paced=True)
    prof = model.profile(xd, yd, lnk, reps=3)
    assert (prof.fc > 0).all() and (prof.bc > 0).all()
    bytes_ = np.array(model.layer_bytes())
    np.testing.assert_allclose(prof.pt, np.round(bytes_ / rate * 1e9), atol=1)
    plan = D.dc_plan(prof)
    p_ref, tf, _, _ = OP.forward_dp(prof.pt.tolist(), prof.fc.tolist(), prof.dt)
    g_ref, tb, _, _ = OP.backward_dp(prof.bc.tolist(), prof.gt.tolist(), prof.dt)
    assert plan.decisions() == (p_ref, g_ref) and (plan.t_fwd_ns, plan.t_bwd_ns) == (tf, tb)
    model.set_option(D.DC_OPT_TIMELINE, 1)
    for key, pl in {"dp": plan, "sequential": D.Plan(model.L), "lbl": plans_for(model.L)["lbl"]}.items():
        pl = D.dc_plan_eval(prof, *pl.decisions()) if key != "dp" else pl
        model.step(xd, yd, pl, lnk)  # warm
        st = model.step(xd, yd, pl, lnk)
        tl = model.timeline()
        _check_partial_orders(tl, eps=2000)
        t_model = pl.t_fwd_ns + pl.t_bwd_ns
        assert abs(st["t_iter_ns"] - t_model) <= 0.10 * t_model, (key, st["t_iter_ns"], t_model)


CONFIG_RATES = [("vgg16", 32, 3, 100e9 / 8), ("vgg16", 32, 3, 10e9 / 8), ("vgg16", 32, 3, 1e9 / 8),
                ("vgg16", 32, 3, None), ("resnet50", 64, 4, 10e9 / 8), ("resnet50", 64, 4, None),
                ("resnet18", 128, 2, 1e9 / 8)]


@pytest.mark.parametrize("name,batch,seed,rate", CONFIG_RATES,
                         ids=[f"{n}-b{b}-" + (f"{r * 8 / 1e9:g}Gbps" if r else "unpaced") for n, b, _, r in CONFIG_RATES])
def test_time_model_at_config_rates(name, batch, seed, rate):
    """The benchmark configurations at their own link rates, paced, and on the
    unpaced host interface (rate None): the plan is the oracle DP's on the
    measured profile, and the measured iteration time of the DP and of the
    sequential plan is within 10% of f_m (Eq. 8 / 9).  AlexNet's own 0.1 Gb/s has a
    test of its own below (one iteration, 39 s); VGG-16 at 0.1 Gb/s takes 89 s per
    iteration and is left to the report."""
    ops, hwc, classes = PN.build(name)
    specs = PN.param_specs(ops, hwc)
    x, y, params = synth.cnn_inputs(seed, batch, hwc, classes, specs)
    model = D.Model(ops, batch, hwc, classes)
    model.set_option(D.DC_OPT_LR, PN.WORKLOADS[name]["lr"])  # the workload's own rate: VGG diverges at 1e-2
    model.ps_write(params)
    xd, yd = dev(x), dev(y)
    lnk = D.link(rate, 0, paced=True) if rate else UNPACED
    label = f"{rate * 8 / 1e9:g} Gb/s" if rate else "unpaced"
    print(f"time model {name} batch {batch} at {label}", flush=True)
    prof = model.profile(xd, yd, lnk, reps=3)
    plan = D.dc_plan(prof)
    p_ref, tf, _, _ = OP.forward_dp(prof.pt.tolist(), prof.fc.tolist(), prof.dt)
    g_ref, tb, _, _ = OP.backward_dp(prof.bc.tolist(), prof.gt.tolist(), prof.dt)
    assert plan.decisions() == (p_ref, g_ref) and (plan.t_fwd_ns, plan.t_bwd_ns) == (tf, tb)
    errs = {}
    for key, pl in {"dp": plan, "sequential": D.dc_plan_eval(prof, *D.Plan(model.L).decisions())}.items():
        model.step(xd, yd, pl, lnk)  # warm
        st = model.step(xd, yd, pl, lnk)
        t_model = pl.t_fwd_ns + pl.t_bwd_ns
        errs[key] = (st["t_iter_ns"] - t_model) / t_model
        assert abs(st["t_iter_ns"] - t_model) <= 0.10 * t_model, (key, st["t_iter_ns"], t_model)
        assert np.isfinite(st["loss"])
    report(f"time model {name} b{batch} {label}: (measured - f_m) / f_m = DP {errs['dp']:+.2%}, "
           f"sequential {errs['sequential']:+.2%}; DP p={p_ref} g={g_ref}")


def test_time_model_alexnet_at_its_link():
    """AlexNet at batch 32 on its configuration's 0.1 Gb/s link: the DP plan is the
    oracle DP's on the measured profile and one measured iteration (about 39 s, the
    two transfers of 244 MB at 12.5 MB/s) is within 10% of f_m.  No warm-up step:
    start-up costs are milliseconds against tens of seconds."""
    ops, hwc, classes = PN.build("alexnet")
    specs = PN.param_specs(ops, hwc)
    x, y, params = synth.cnn_inputs(1, 32, hwc, classes, specs)
    model = D.Model(ops, 32, hwc, classes)
    model.set_option(D.DC_OPT_LR, PN.WORKLOADS["alexnet"]["lr"])
    model.ps_write(params)
    xd, yd = dev(x), dev(y)
    lnk = D.link(0.1e9 / 8, 0, paced=True)
    print("time model alexnet batch 32 at 0.1 Gb/s: profiling", flush=True)
    prof = model.profile(xd, yd, lnk, reps=3)
    plan = D.dc_plan(prof)
    p_ref, tf, _, _ = OP.forward_dp(prof.pt.tolist(), prof.fc.tolist(), prof.dt)
    g_ref, tb, _, _ = OP.backward_dp(prof.bc.tolist(), prof.gt.tolist(), prof.dt)
    assert plan.decisions() == (p_ref, g_ref) and (plan.t_fwd_ns, plan.t_bwd_ns) == (tf, tb)
    t_model = plan.t_fwd_ns + plan.t_bwd_ns
    print(f"time model alexnet: one DP iteration, f_m = {t_model / 1e9:.1f} s", flush=True)
    st = model.step(xd, yd, plan, lnk)
    err = (st["t_iter_ns"] - t_model) / t_model
    assert abs(err) <= 0.10, (st["t_iter_ns"], t_model)
    assert np.isfinite(st["loss"])
    report(f"time model alexnet b32 0.1 Gb/s: (measured - f_m) / f_m = DP {err:+.2%}; DP p={p_ref} g={g_ref}")


def test_argument_errors():
    model, onet, xd, yd, x, y, params = setup_model("tiny", 4, seed=0)
    with pytest.raises(D.DcError) as e:
        model.step(xd, yd, D.Plan(3), UNPACED)
    assert e.value.status == D.DC_EINVAL
    with pytest.raises(D.DcError) as e:
        model.step(xd[:2], yd[:2], D.Plan(4), UNPACED)
    assert e.value.status == D.DC_EINVAL
    with pytest.raises(D.DcError) as e:
        model.step(xd, yd, D.Plan(4), D.link(0, 0, paced=True))
    assert e.value.status == D.DC_EINVAL
    # the binding rejects inputs the library would misread: wrong dtype, host memory, strided views
    for bad_x, bad_y in ((xd.double(), yd), (xd, yd.long()), (xd.cpu(), yd), (xd.transpose(1, 2), yd)):
        with pytest.raises(D.DcError) as e:
            model.step(bad_x, bad_y, D.Plan(4), UNPACED)
        assert e.value.status == D.DC_EINVAL
    with pytest.raises(D.DcError) as e:
        model.set_option(D.DC_OPT_TIMEOUT_S, -1)
    assert e.value.status == D.DC_EINVAL
    with pytest.raises(D.DcError) as e:
        model.timeline()
    assert e.value.status == D.DC_ESTATE


def test_read_tensor_returns_the_steps_tensors():
    """dc_model_read_tensor after a step: every kept activation equals the oracle's
    forward (taken with the GPU's max-pool taps), and the reads it cannot serve fail."""
    model, onet, xd, yd, x, y, params = setup_model("tiny", 4, seed=5)
    model.step(xd, yd, D.Plan(model.L), UNPACED)
    t, _ = onet.forward(x, params)
    read, refused = 0, 0
    for i, op in enumerate(onet.ops):
        try:
            a = model.read_tensor(i + 1, onet.shapes[i + 1])
        except D.DcError as e:
            # only a producer whose ReLU is folded into it keeps no output
            assert e.status == D.DC_EINVAL
            assert onet.ops[i + 1]["op"] == "relu" and onet.ops[i + 1]["in"] == i + 1, i
            refused += 1
            continue
        read += 1
        if op["op"] == "maxpool":
            arg = model.read_tensor(i + 1, onet.shapes[i + 1], D.DC_READ_ARGMAX)
            assert arg.max() < op["r"] * op["s"]
            ref = OC.maxpool_at(t[op["in"]], arg.astype(np.int32), op["r"], op["s"], op["stride"], op["pad"])
            assert rel_err(ref, t[i + 1]) <= 1e-6, i  # the GPU took a maximum of each window
            assert rel_err(a, ref) <= 1e-5, i
        else:
            assert rel_err(a, t[i + 1]) <= 1e-5, i
    assert read and refused
    bad = [(0, D.DC_READ_ACT, onet.shapes[0]), (len(onet.ops) + 1, D.DC_READ_ACT, (1,)),
           (-1, D.DC_READ_ACT, (1,)), (2, D.DC_READ_ARGMAX, onet.shapes[2]),
           (2, D.DC_READ_ACT, (onet.shapes[2][0] - 1,) + onet.shapes[2][1:]), (3, 7, onet.shapes[3])]
    for tensor, what, shape in bad:
        with pytest.raises(D.DcError) as e:
            model.read_tensor(tensor, shape, what)
        assert e.value.status == D.DC_EINVAL, (tensor, what, shape)
    model.close()


def test_watchdog_times_out_and_gpu_drains():
    import torch
    model, onet, xd, yd, x, y, params = setup_model("tiny", 4, seed=0)
    model.set_option(D.DC_OPT_TIMEOUT_S, 0.02)
    slow = D.link(2e6, 0, paced=True)  # ~135 ms per direction, bounded spin
    with pytest.raises(D.DcError) as e:
        model.step(xd, yd, D.Plan(4), slow)
    assert e.value.status == D.DC_ETIMEOUT
    torch.cuda.synchronize()  # every kernel ends on its own
    model.set_option(D.DC_OPT_TIMEOUT_S, 60)
    st = model.step(xd, yd, D.Plan(4), UNPACED)
    assert np.isfinite(st["loss"])


def test_destroy_right_after_watchdog():
    """A step that ends on the watchdog leaves pulls, pushes and the loss
    copy in flight; destroying the model at once must wait for the library's
    own work before it frees the pinned buffers, and a new model then runs."""
    import torch
    model, onet, xd, yd, x, y, params = setup_model("tiny", 4, seed=0)
    model.set_option(D.DC_OPT_TIMEOUT_S, 0.02)
    with pytest.raises(D.DcError) as e:
        model.step(xd, yd, D.Plan(4), D.link(2e6, 0, paced=True))
    assert e.value.status == D.DC_ETIMEOUT
    model.close()
    torch.cuda.synchronize()
    model2, onet, xd, yd, x, y, params = setup_model("tiny", 4, seed=0)
    st = model2.step(xd, yd, D.Plan(4), UNPACED)
    loss_ref, _, _ = onet.step(x, y, params)
    assert abs(st["loss"] - loss_ref) <= 1e-4 * abs(loss_ref)


@pytest.mark.parametrize("name,batch", [("tiny", 4), ("resnet18", 8)])
def test_checkpoint_resume_is_bit_exact(name, batch):
    """The parameter server holds the whole training state (BatchNorm keeps no
    running statistics): two steps equal one step, a dc_ps_read checkpoint
    written into a fresh model with dc_ps_write, and a second step there."""
    model, onet, xd, yd, x, y, params = setup_model(name, batch, seed=11)
    x2, y2, _ = synth.cnn_inputs(12, batch, onet.spec["hwc"], onet.classes, onet.param_specs)
    x2d, y2d = dev(x2), dev(y2)
    plan = plans_for(model.L, seed=2)["random"]
    model.step(xd, yd, plan, UNPACED)
    ckpt, _ = model.ps_read()
    st_a = model.step(x2d, y2d, plan, UNPACED)
    p_a, g_a = model.ps_read()
    model.close()
    ops, hwc, classes = PN.build(name)
    fresh = D.Model(ops, batch, hwc, classes)
    fresh.ps_write(ckpt)
    st_b = fresh.step(x2d, y2d, plan, UNPACED)
    p_b, g_b = fresh.ps_read()
    assert st_b["loss"] == st_a["loss"]
    np.testing.assert_array_equal(g_b, g_a)
    np.testing.assert_array_equal(p_b, p_a)
    fresh.close()


@pytest.mark.parametrize("name,batch", [("tiny", 4), ("resnet18", 8), ("googlenet", 2)])
def test_layer_graphs_replay_the_eager_iteration(name, batch):
    """DC_OPT_GRAPHS: each layer's kernels replayed from a captured HIP graph give
    bit-identical steps to launching them one by one, over several replays with
    the other model's eager work in between, and after a new batch address
    forces a recapture."""
    g_model, onet, xd, yd, x, y, params = setup_model(name, batch, seed=13)
    g_model.set_option(D.DC_OPT_GRAPHS, 1)
    ops, hwc, classes = PN.build(name)
    e_model = D.Model(ops, batch, hwc, classes)
    e_model.set_option(D.DC_OPT_GRAPHS, 0)
    e_model.ps_write(params)
    plan = plans_for(g_model.L, seed=4)["random"]
    x2, y2, _ = synth.cnn_inputs(14, batch, hwc, classes, onet.param_specs)
    batches = [(xd, yd), (xd, yd), (dev(x2), dev(y2)), (xd, yd)]
    for i, (bx, by) in enumerate(batches):
        st_g = g_model.step(bx, by, plan, UNPACED)
        st_e = e_model.step(bx, by, plan, UNPACED)
        p_g, g_g = g_model.ps_read()
        p_e, g_e = e_model.ps_read()
        assert st_g["loss"] == st_e["loss"], i
        np.testing.assert_array_equal(g_g, g_e, err_msg=str(i))
        np.testing.assert_array_equal(p_g, p_e, err_msg=str(i))
    # profiles come from the same (graph) launches the steps use
    prof = g_model.profile(xd, yd, UNPACED, reps=1)
    assert (prof.fc > 0).all() and (prof.bc > 0).all()
    g_model.close()
    e_model.close()


def test_dynamic_step_plans_in_idle_windows():
    """dc_step_dynamic (idle-event trigger, Sec. IV-C) against the oracle: the
    backward decision it plans on the fly and the forward decision it plans for
    the next call are the oracle DP's (Eq. 8 / 9, Algorithms 3 / 4) on the
    profile it was given, with the same f_m; its loss, gradients and post-step
    weights are the oracle iteration's (the bars of test_step_matches_oracle);
    planning finished while a transfer was in flight.  A second call runs on the
    forward decision the first one planned, from the same parameters, and gives
    bit-identical results; both equal a plain dc_step under the oracle's plan."""
    model, onet, xd, yd, x, y, params = setup_model("resnet18", 16, seed=5)
    lnk = D.link(5e8, 0, paced=True)
    prof = model.profile(xd, yd, lnk, reps=2)
    p_or, tf, _, _ = OP.forward_dp(prof.pt.tolist(), prof.fc.tolist(), prof.dt)
    g_or, tb, _, _ = OP.backward_dp(prof.bc.tolist(), prof.gt.tolist(), prof.dt)
    loss_ref, g_ref, w_ref = onet.step(x, y, params)
    spread, spread_w = fp32_spread(ON.get("resnet18"), onet, x, y, params, g_ref)
    plan = D.Plan(model.L)
    plan.p[:] = p_or            # first call: the forward decision given, the backward one planned on the fly
    outs = []
    for call in range(2):
        model.ps_write(params)
        st = model.step_dynamic(xd, yd, prof, plan, lnk)
        p_new, g = model.ps_read()
        outs.append((st["loss"], p_new, g))
        assert plan.decisions() == (p_or, g_or), call
        assert (plan.t_fwd_ns, plan.t_bwd_ns) == (tf, tb), call
        assert st["plan_hidden"] == 3, st
        assert 0 < st["t_plan_bwd_ns"] and 0 < st["t_plan_fwd_ns"]
        assert abs(st["loss"] - loss_ref) <= 1e-4 * abs(loss_ref)
        for i, slots in enumerate(onet.pslots):
            for pname, (off, shape) in slots.items():
                sl = slice(off, off + int(np.prod(shape)))
                assert rel_err(g[sl], g_ref[sl]) <= max(1e-3, 5.0 * spread[(i, pname)]), (call, i, pname)
                assert rel_err(p_new[sl], w_ref[sl]) <= max(1e-3, 5.0 * spread_w[(i, pname)]), (call, i, pname)
    assert outs[1][0] == outs[0][0]
    np.testing.assert_array_equal(outs[1][1], outs[0][1])
    np.testing.assert_array_equal(outs[1][2], outs[0][2])
    # the same numbers as dc_step under the oracle's decisions
    model.ps_write(params)
    st_ref = model.step(xd, yd, D.dc_plan_eval(prof, p_or, g_or), lnk)
    p_s, g_s = model.ps_read()
    assert st_ref["loss"] == outs[0][0]
    np.testing.assert_array_equal(g_s, outs[0][2])
    np.testing.assert_array_equal(p_s, outs[0][1])


def test_replanning_follows_the_link():
    """Re-profiling after the link changes (once-per-epoch cadence, Sec. IV-C) re-plans
    exactly as the oracle does on the new profile."""
    model, onet, xd, yd, x, y, params = setup_model("resnet18", 32, seed=6)
    plans, profs = {}, {}
    for rate in (1.25e10 / 8 * 8, 1.25e8):
        lnk = D.link(rate, 0, paced=True)
        prof = model.profile(xd, yd, lnk, reps=2)
        plan = D.dc_plan(prof)
        p_ref, _, _, _ = OP.forward_dp(prof.pt.tolist(), prof.fc.tolist(), prof.dt)
        g_ref, _, _, _ = OP.backward_dp(prof.bc.tolist(), prof.gt.tolist(), prof.dt)
        assert plan.decisions() == (p_ref, g_ref)
        ratio = prof.pt.sum() / np.array(model.layer_bytes()).sum()
        assert abs(ratio * rate / 1e9 - 1) < 1e-3
        plans[rate] = plan.decisions()
        profs[rate] = (prof.pt.tolist(), prof.fc.tolist(), prof.bc.tolist(), prof.gt.tolist(), prof.dt)
    # on each link's profile, its own plan is at least as good under f_m as the
    # plan made for the other link: re-planning never loses (Sec. IV-B-3)
    for rate, other in ((1.25e10, 1.25e8), (1.25e8, 1.25e10)):
        pr = profs[rate]
        own = OP.fm(*pr, *plans[rate])
        stale = OP.fm(*pr, *plans[other])
        assert own <= stale, (rate, own, stale)


def test_relu_folds_on_odd_graphs():
    """The ReLU backward folds on graphs the workloads do not contain, against the oracle:
    * a conv output read by a ReLU -> max-pool and twice by add(t, t) -> ReLU: the masked pool
      accumulates into a gradient the fused add-ReLU wrote through two aliased outputs;
    * a ReLU whose only consumer is a concatenation three ops later (non-adjacent fold);
    * a ReLU -> conv whose input is also read by a residual add: the masked data-gradient
      epilogue accumulates;
    * concat(relu(t), t) and concat(t, relu(t)): a concatenation that reads a ReLU's input
      as well as its output (the ReLU's backward is then not folded into it)."""
    C, R, MP, A, CAT, F = D.DC_OP_CONV, D.DC_OP_RELU, D.DC_OP_MAXPOOL, D.DC_OP_ADD, D.DC_OP_CONCAT, D.DC_OP_FC
    conv = lambda i, l, k, r, pad: {"op": "conv", "in": i, "layer": l, "k": k, "r": r, "s": r, "stride": 1,
                                    "pad": pad, "bias": True}
    relu = lambda i, l: {"op": "relu", "in": i, "layer": l}
    pool = lambda i, l: {"op": "maxpool", "in": i, "layer": l, "r": 2, "s": 2, "stride": 2, "pad": 0}
    cases = [
        ({"name": "folds1", "hwc": (8, 8, 4), "classes": 5, "ops": [
            conv(0, 1, 8, 3, 1), relu(1, 1), pool(2, 1),
            {"op": "add", "in": 1, "other": 1, "layer": 1}, relu(4, 1), pool(5, 1),
            {"op": "concat", "in": 3, "others": [6], "layer": 1},
            conv(7, 2, 8, 3, 1), relu(8, 2), conv(7, 2, 4, 1, 0), relu(10, 2),
            {"op": "concat", "in": 9, "others": [11], "layer": 2},
            {"op": "fc", "in": 12, "layer": 3, "out": 5, "bias": True}]},
         [(C, 1, 0, -1, 8, 3, 3, 1, 1, 1, -1, -1, 1), (R, 1, 1, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0),
          (MP, 1, 2, -1, 0, 2, 2, 2, 0, 0, -1, -1, 0), (A, 1, 1, 1, 0, 0, 0, 0, 0, 0, -1, -1, 0),
          (R, 1, 4, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0), (MP, 1, 5, -1, 0, 2, 2, 2, 0, 0, -1, -1, 0),
          (CAT, 1, 3, 6, 0, 0, 0, 0, 0, 0, -1, -1, 0),
          (C, 2, 7, -1, 8, 3, 3, 1, 1, 1, -1, -1, 1), (R, 2, 8, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0),
          (C, 2, 7, -1, 4, 1, 1, 1, 0, 1, -1, -1, 0), (R, 2, 10, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0),
          (CAT, 2, 9, 11, 0, 0, 0, 0, 0, 0, -1, -1, 0), (F, 3, 12, -1, 5, 0, 0, 0, 0, 1, -1, -1, 0)]),
        ({"name": "folds2", "hwc": (6, 6, 4), "classes": 5, "ops": [
            conv(0, 1, 8, 3, 1), relu(1, 1), conv(2, 2, 8, 3, 1),
            {"op": "add", "in": 3, "other": 1, "layer": 2}, relu(4, 2),
            {"op": "fc", "in": 5, "layer": 3, "out": 5, "bias": True}]},
         [(C, 1, 0, -1, 8, 3, 3, 1, 1, 1, -1, -1, 1), (R, 1, 1, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0),
          (C, 2, 2, -1, 8, 3, 3, 1, 1, 1, -1, -1, 1), (A, 2, 3, 1, 0, 0, 0, 0, 0, 0, -1, -1, 0),
          (R, 2, 4, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0), (F, 3, 5, -1, 5, 0, 0, 0, 0, 1, -1, -1, 0)]),
        ({"name": "folds3", "hwc": (6, 6, 4), "classes": 5, "ops": [
            conv(0, 1, 8, 3, 1), relu(1, 1), {"op": "concat", "in": 2, "others": [1], "layer": 1},
            conv(3, 2, 8, 3, 1), relu(4, 2), {"op": "concat", "in": 4, "others": [5], "layer": 2},
            {"op": "fc", "in": 6, "layer": 3, "out": 5, "bias": True}]},
         [(C, 1, 0, -1, 8, 3, 3, 1, 1, 1, -1, -1, 1), (R, 1, 1, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0),
          (CAT, 1, 2, 1, 0, 0, 0, 0, 0, 0, -1, -1, 0),
          (C, 2, 3, -1, 8, 3, 3, 1, 1, 1, -1, -1, 1), (R, 2, 4, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0),
          (CAT, 2, 4, 5, 0, 0, 0, 0, 0, 0, -1, -1, 0), (F, 3, 6, -1, 5, 0, 0, 0, 0, 1, -1, -1, 0)]),
    ]
    for spec, ops in cases:
        for batch in (1, 3):
            print(f"folds {spec['name']} batch {batch}", flush=True)
            hwc, classes = spec["hwc"], spec["classes"]
            specs = PN.param_specs(ops, hwc)
            onet = OC.Net(spec, batch)
            assert specs == onet.param_specs
            x, y, params = synth.cnn_inputs(31 + batch, batch, hwc, classes, specs)
            model = D.Model(ops, batch, hwc, classes)
            model.ps_write(params)
            st = model.step(dev(x), dev(y), plans_for(model.L, seed=batch)["random"], UNPACED)
            p_new, g = model.ps_read()
            loss_ref, g_ref, p_ref = onet.step(x, y, params)
            assert abs(st["loss"] - loss_ref) <= 1e-4 * abs(loss_ref)
            assert rel_err(g, g_ref) <= 1e-3
            assert rel_err(p_new, p_ref) <= 1e-3
            model.close()


def test_degenerate_models():
    """L = 1 (one FC layer: no segment decision to make) at batch 1, and a two-layer
    conv net whose conv output is a single pixel, each against the oracle."""
    cases = [
        ({"name": "fc1", "ops": [{"op": "fc", "in": 0, "layer": 1, "out": 10, "bias": True}],
          "hwc": (4, 4, 3), "classes": 10},
         [(D.DC_OP_FC, 1, 0, -1, 10, 0, 0, 0, 0, 1, -1, -1, 0)], 1),
        ({"name": "pix1", "ops": [
            {"op": "conv", "in": 0, "layer": 1, "k": 8, "r": 3, "s": 3, "stride": 1, "pad": 0, "bias": True},
            {"op": "relu", "in": 1, "layer": 1},
            {"op": "fc", "in": 2, "layer": 2, "out": 5, "bias": True}],
          "hwc": (3, 3, 4), "classes": 5},
         [(D.DC_OP_CONV, 1, 0, -1, 8, 3, 3, 1, 0, 1, -1, -1, 0),
          (D.DC_OP_RELU, 1, 1, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0),
          (D.DC_OP_FC, 2, 2, -1, 5, 0, 0, 0, 0, 1, -1, -1, 0)], 3),
    ]
    for spec, ops, batch in cases:
        print(f"degenerate {spec['name']} batch {batch}", flush=True)
        hwc, classes = spec["hwc"], spec["classes"]
        specs = PN.param_specs(ops, hwc)
        onet = OC.Net(spec, batch)
        assert specs == onet.param_specs
        x, y, params = synth.cnn_inputs(21, batch, hwc, classes, specs)
        model = D.Model(ops, batch, hwc, classes)
        model.ps_write(params)
        xd, yd = dev(x), dev(y)
        prof = model.profile(xd, yd, D.link(1e9, 0, paced=True), reps=1)
        plan = D.dc_plan(prof)
        p_ref, _, _, _ = OP.forward_dp(prof.pt.tolist(), prof.fc.tolist(), prof.dt)
        assert list(plan.decisions()[0]) == list(p_ref)
        model.ps_write(params)
        st = model.step(xd, yd, plan, UNPACED)
        p_new, g = model.ps_read()
        loss_ref, g_ref, p_ref = onet.step(x, y, params)
        assert abs(st["loss"] - loss_ref) <= 1e-4 * abs(loss_ref)
        assert rel_err(g, g_ref) <= 1e-3
        assert rel_err(p_new, p_ref) <= 1e-3
        model.close()


def test_gemm_timing_counts_every_pass():
    """DC_OPT_GEMM_TIMING: every conv / FC pass of the step is timed (forward, filter gradient,
    and data gradient unless the op reads the input batch), with its algorithmic FLOPs; the
    events change no number."""
    model, onet, xd, yd, x, y, params = setup_model("resnet18", 4, seed=9)
    plan = plans_for(model.L, seed=3)["random"]
    st0 = model.step(xd, yd, plan, UNPACED)
    p0, g0 = model.ps_read()
    assert st0["n_gemm"] == 0 and st0["t_gemm_ns"] == 0
    n_exp, flop_exp = 0, 0.0
    for i, op in enumerate(onet.ops):
        if op["op"] in ("conv", "fc"):
            n, P, Q, K = onet.shapes[i + 1]
            _, h, w, c = onet.shapes[op["in"]]
            mac = n * P * Q * K * (op["r"] * op["s"] * c if op["op"] == "conv" else h * w * c)
            passes = 2 if op["in"] == 0 else 3
            n_exp += passes
            flop_exp += passes * 2.0 * mac
    model.set_option(D.DC_OPT_GEMM_TIMING, 1)
    for _ in range(2):
        model.ps_write(params)
        st = model.step(xd, yd, plan, UNPACED)
        p1, g1 = model.ps_read()
        assert st["n_gemm"] == n_exp and st["gemm_flop"] == flop_exp
        assert 0 < st["t_gemm_ns"] < st["t_iter_ns"]
        assert st["loss"] == st0["loss"]
        np.testing.assert_array_equal(g1, g0)
        np.testing.assert_array_equal(p1, p0)
    # a profile in between neither times passes nor disturbs the next step's count
    model.profile(xd, yd, UNPACED, reps=1)
    model.ps_write(params)
    assert model.step(xd, yd, plan, UNPACED)["n_gemm"] == n_exp
