"""Pins for the oracle scheduler: exhaustive search, closed forms, hand-worked cases.

The oracle's dynamic programs (Eq. 8 / Algorithm 3, Eq. 9 / Algorithm 4) are
checked against things that do not share their recurrences:

* exhaustive search over every decision (Sec. III-B), valued by f_m;
* f_m itself against an event simulation of the mini-procedures under the
  partial orders Eq. 1-7 and against the max-plus closed form of the
  back-to-back link / in-order compute pipeline;
* hand-worked examples (tests/golden/hand_plan.json);
* the special cases of Sec. III-B: one segment is the sequential default PS,
  and with no per-transmission overhead layer-by-layer is never worse than it.
"""
import inspect
import itertools
import json
import os

import pytest

import synth
from oracle import plan as P

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def closed_form_forward(pt, fc, dt, p):
    """max over segments j of (j*dt + pt_1..e_j + fc_lo_j..L): the critical path of the pipeline."""
    segs = P.pull_segments(p)
    best = 0
    for j, (lo, hi) in enumerate(segs, 1):
        best = max(best, j * dt + sum(pt[:hi]) + sum(fc[lo - 1:]))
    return best


def closed_form_backward(bc, gt, dt, g):
    """max over push segments j of (ready_j + durations of segments j..n)."""
    segs = P.push_segments(g)
    L = len(bc)
    best = 0
    for j, (lo, hi) in enumerate(segs):
        ready = sum(bc[lo - 1:L])
        tail = sum(dt + sum(gt[a - 1:b]) for a, b in segs[j:])
        best = max(best, ready + tail)
    return best


def test_hand_worked_forward():
    d = _load("hand_plan.json")["forward"]
    for key, (val, _why) in d["all"].items():
        p = [int(v) for v in key.split(",")]
        assert P.fm_forward(d["pt"], d["fc"], d["dt"], p) == val, key
    p, t, _, _ = P.forward_dp(d["pt"], d["fc"], d["dt"])
    assert p == d["best"] and t == d["T"]


def test_hand_worked_backward():
    d = _load("hand_plan.json")["backward"]
    for key, (val, _why) in d["all"].items():
        g = [int(v) for v in key.split(",")]
        assert P.fm_backward(d["bc"], d["gt"], d["dt"], g) == val, key
    g, t, _, _ = P.backward_dp(d["bc"], d["gt"], d["dt"])
    assert g == d["best"] and t == d["T"]


def test_overhead_makes_lbl_lose():
    d = _load("hand_plan.json")["two_layer_overhead"]
    assert P.fm_forward(d["pt"], d["fc"], d["dt"], P.sequential(2)) == d["sequential"]
    assert P.fm_forward(d["pt"], d["fc"], d["dt"], P.layer_by_layer(2)) == d["lbl"]
    p, t, _, _ = P.forward_dp(d["pt"], d["fc"], d["dt"])
    assert p == [0] and t == d["sequential"]


def test_segments_decode():
    # p_l = 1: layer l+1 starts a new pull; g_k = 1: boundary between L-k+1 and L-k
    assert P.pull_segments([0, 1, 0]) == [(1, 2), (3, 4)]
    assert P.pull_segments([1, 1, 1]) == [(1, 1), (2, 2), (3, 3), (4, 4)]
    assert P.push_segments([0, 1, 1]) == [(3, 4), (2, 2), (1, 1)]
    assert P.push_segments([1, 0, 0]) == [(4, 4), (1, 3)]
    assert P.push_segments([0, 0, 0]) == [(1, 4)]


@pytest.mark.parametrize("seed", range(400))
def test_dp_matches_brute_force(seed):
    L = 1 + seed % 9
    pt, fc, bc, gt, dt = synth.random_profile(seed, L, hi=60 if seed % 3 else 1000, dt_hi=50)
    p, tf, _, _ = P.forward_dp(pt, fc, dt)
    best, arg = P.brute_force_forward(pt, fc, dt)
    assert tf == best
    assert tuple(p) in arg
    assert P.fm_forward(pt, fc, dt, p) == tf
    g, tb, _, _ = P.backward_dp(bc, gt, dt)
    best, arg = P.brute_force_backward(bc, gt, dt)
    assert tb == best
    assert tuple(g) in arg
    assert P.fm_backward(bc, gt, dt, g) == tb


@pytest.mark.parametrize("seed", range(6))
def test_dp_matches_brute_force_deeper(seed):
    L = 12 + seed
    pt, fc, bc, gt, dt = synth.random_profile(1000 + seed, L, hi=500, dt_hi=200)
    p, tf, _, _ = P.forward_dp(pt, fc, dt)
    best, arg = P.brute_force_forward(pt, fc, dt)
    assert tf == best and tuple(p) in arg
    g, tb, _, _ = P.backward_dp(bc, gt, dt)
    best, arg = P.brute_force_backward(bc, gt, dt)
    assert tb == best and tuple(g) in arg


def test_tie_breaks_fewest_segments():
    # all-zero compute: every decision with one segment costs dt + sum(pt); more
    # segments cost more overhead, so the single segment must be chosen
    pt, fc = [5, 5, 5], [0, 0, 0]
    p, t, _, _ = P.forward_dp(pt, fc, 0)
    # with dt = 0 every decision ties at 15: fewest segments wins
    assert p == [0, 0] and t == 15
    g, t, _, _ = P.backward_dp([0, 0, 0], [5, 5, 5], 0)
    assert g == [0, 0] and t == 15


@pytest.mark.parametrize("seed", range(200))
def test_fm_against_simulation_and_closed_form(seed):
    L = 1 + seed % 12
    pt, fc, bc, gt, dt = synth.random_profile(5000 + seed, L, hi=100, dt_hi=40)
    rng = synth.random_profile(9000 + seed, max(L - 1, 1), hi=1)  # random bits
    p = [int(v > 0) for v in rng[0][:L - 1]]
    g = [int(v > 0) for v in rng[1][:L - 1]]
    sim = P.simulate(pt, fc, bc, gt, dt, p, g)
    assert sim["T_fwd"] == P.fm_forward(pt, fc, dt, p) == closed_form_forward(pt, fc, dt, p)
    assert sim["T_bwd"] == P.fm_backward(bc, gt, dt, g) == closed_form_backward(bc, gt, dt, g)
    # the simulated timeline obeys the partial orders of Eq. 1-7
    for l in range(1, L + 1):
        assert sim["pt"][l][1] <= sim["fc"][l][0]          # Eq. 1
        assert sim["bc"][l][1] <= sim["gt"][l][0]          # Eq. 2
    for m in range(1, L + 1):
        for n in range(m + 1, L + 1):
            assert sim["pt"][m][1] <= sim["pt"][n][0] or sim["pt"][m] == sim["pt"][n]   # Eq. 4
            assert sim["fc"][m][1] <= sim["fc"][n][0]      # Eq. 5
            assert sim["bc"][n][1] <= sim["bc"][m][0]      # Eq. 6
            assert sim["gt"][n][1] <= sim["gt"][m][0] or sim["gt"][m] == sim["gt"][n]   # Eq. 7


@pytest.mark.parametrize("seed", range(100))
def test_one_segment_is_no_overlap(seed):
    L = 1 + seed % 15
    pt, fc, bc, gt, dt = synth.random_profile(7000 + seed, L)
    assert P.fm_forward(pt, fc, dt, P.sequential(L)) == dt + sum(pt) + sum(fc)
    assert P.fm_backward(bc, gt, dt, P.sequential(L)) == sum(bc) + dt + sum(gt)


@pytest.mark.parametrize("seed", range(100))
def test_lbl_never_worse_without_overhead(seed):
    L = 1 + seed % 15
    pt, fc, bc, gt, _ = synth.random_profile(8000 + seed, L)
    assert P.fm_forward(pt, fc, 0, P.layer_by_layer(L)) <= P.fm_forward(pt, fc, 0, P.sequential(L))
    assert P.fm_backward(bc, gt, 0, P.layer_by_layer(L)) <= P.fm_backward(bc, gt, 0, P.sequential(L))
    # and the dynamic program is never worse than either, at any overhead
    for dt in (0, 7, 300):
        p, tf, _, _ = P.forward_dp(pt, fc, dt)
        g, tb, _, _ = P.backward_dp(bc, gt, dt)
        assert tf <= min(P.fm_forward(pt, fc, dt, P.sequential(L)), P.fm_forward(pt, fc, dt, P.layer_by_layer(L)))
        assert tb <= min(P.fm_backward(bc, gt, dt, P.sequential(L)), P.fm_backward(bc, gt, dt, P.layer_by_layer(L)))


def test_tiny_workload_fixture():
    d = _load("tiny_plan.json")
    pr = d["profile"]
    p, tf, _, _ = P.forward_dp(pr["pt"], pr["fc"], pr["dt"])
    g, tb, _, _ = P.backward_dp(pr["bc"], pr["gt"], pr["dt"])
    assert (p, tf, g, tb) == (d["p"], d["T_fwd"], d["g"], d["T_bwd"])
    best, arg = P.brute_force_forward(pr["pt"], pr["fc"], pr["dt"])
    assert best == tf and tuple(p) in arg
    best, arg = P.brute_force_backward(pr["bc"], pr["gt"], pr["dt"])
    assert best == tb and tuple(g) in arg
    L = 4
    assert P.fm_forward(pr["pt"], pr["fc"], pr["dt"], P.sequential(L)) == d["T_fwd_sequential"]
    assert d["T_fwd_sequential"] == pr["dt"] + sum(pr["pt"]) + sum(pr["fc"])


def test_planted_mistakes_are_caught():
    """A dropped overhead term or an off-by-one prefix in f_m breaks the pins above."""
    pt, fc, dt = [2, 1, 4], [3, 5, 1], 3

    def fm_no_dt(pt, fc, dt, p):
        return P.fm_forward(pt, fc, 0, p)

    def fm_off_by_one(pt, fc, dt, p):
        link = done = 0
        for lo, hi in P.pull_segments(p):
            link += dt + sum(pt[lo - 1:hi - 1])
            done = max(done, link) + sum(fc[lo - 1:hi])
        return done

    for bad in (fm_no_dt, fm_off_by_one):
        assert any(bad(pt, fc, dt, list(b)) != closed_form_forward(pt, fc, dt, list(b))
                   for b in itertools.product((0, 1), repeat=2))


def test_ibatch_hand_worked():
    d = _load("ibatch_hand.json")
    f = d["forward"]
    p = P.ibatch_forward(f["pt"], f["fc"], f["dt"])
    assert p == f["p"] and P.fm_forward(f["pt"], f["fc"], f["dt"], p) == f["T"]
    assert P.forward_dp(f["pt"], f["fc"], f["dt"])[1] == f["dp_T"]
    b = d["backward"]
    g, t = P.ibatch_backward(b["bc"], b["gt"], b["dt"])
    assert g == b["g"] and t == b["T"]


def test_ibatch_hand_worked_cases():
    """Algorithm 1's loop choosing among several positions in three iterations, and
    finding none; Algorithm 2's winning candidate running to k = 3 with k * dt
    deciding a step (tests/golden/ibatch_cases.json, derived by hand)."""
    d = _load("ibatch_cases.json")
    for f in d["forward"]:
        p = P.ibatch_forward(f["pt"], f["fc"], f["dt"])
        assert p == f["p"] and P.fm_forward(f["pt"], f["fc"], f["dt"], p) == f["T"], f["name"]
        assert P.forward_dp(f["pt"], f["fc"], f["dt"])[1] <= f["T"]
    for b in d["backward"]:
        g, t = P.ibatch_backward(b["bc"], b["gt"], b["dt"])
        assert g == b["g"] and t == b["T"], b["name"]
        assert P.backward_dp(b["bc"], b["gt"], b["dt"])[1] <= b["T"]


def _mutant(fn, old, new):
    """fn with one source fragment replaced: a plausible slip, planted in a copy on the CPU."""
    src = inspect.getsource(fn)
    assert old in src, old
    ns = dict(vars(P))
    exec(src.replace(old, new), ns)
    return ns[fn.__name__]


SLIPS = [
    ("forward", P.ibatch_forward, "j = min((dt + (PT[x] - PT[m])", "j = max((dt + (PT[x] - PT[m])"),
    ("forward", P.ibatch_forward, "            j = L\n", "            j = m + 1\n"),
    ("forward", P.ibatch_forward, "d2 = min((dt + (PT[b] - PT[a])", "d2 = max((dt + (PT[b] - PT[a])"),
    ("backward", P.ibatch_backward, "pushed = k * dt +", "pushed = dt +"),
    ("backward", P.ibatch_backward, "j = min((pushed - (BC[m - 1] - BC[x - 1]), x)",
     "j = max((pushed - (BC[m - 1] - BC[x - 1]), x)"),
    ("backward", P.ibatch_backward, "                j = m - 1\n", "                j = 1\n"),
]


@pytest.mark.parametrize("which,fn,old,new", SLIPS, ids=[f"{w}-{i}" for i, (w, *_rest) in enumerate(SLIPS)])
def test_ibatch_fixtures_catch_slips(which, fn, old, new):
    """Each slip, planted in a copy of the oracle, fails one of the hand-worked fixtures."""
    bad = _mutant(fn, old, new)
    cases = _load("ibatch_cases.json")[which] + [_load("ibatch_hand.json")[which]]
    if which == "forward":
        assert any(bad(c["pt"], c["fc"], c["dt"]) != c["p"] for c in cases)
    else:
        assert any(bad(c["bc"], c["gt"], c["dt"]) != (c["g"], c["T"]) for c in cases)


@pytest.mark.parametrize("seed", range(150))
def test_ibatch_never_beats_the_dp(seed):
    """The DP is optimal (Sec. IV-B-3), so a greedy decision can only tie or lose."""
    L = 1 + seed % 14
    pt, fc, bc, gt, dt = synth.random_profile(20000 + seed, L, hi=500, dt_hi=200)
    p = P.ibatch_forward(pt, fc, dt)
    g, tb = P.ibatch_backward(bc, gt, dt)
    assert len(p) == L - 1 and len(g) == L - 1
    assert P.forward_dp(pt, fc, dt)[1] <= P.fm_forward(pt, fc, dt, p)
    assert P.backward_dp(bc, gt, dt)[1] <= tb == P.fm_backward(bc, gt, dt, g)


def test_ibatch_fallbacks():
    # no pair passes step 2 (transfers are free, compute is not): one segment
    assert P.ibatch_forward([0, 0, 0], [5, 5, 5], 0) == [0, 0]
    # a single layer has nothing to decide
    assert P.ibatch_forward([3], [4], 1) == [] and P.ibatch_backward([3], [4], 1) == ([], 8)
