"""Oracle for DynaComm's communication scheduler (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  The product library never calls it.

Everything here is exact integer arithmetic on nanosecond costs (Python ints,
``math.inf`` for the +infinity boundary of the tables), so two correct
implementations of the same recurrence agree bit for bit.

Contents, each following the paper:

* ``forward_dp``  - the forward Bellman equation (Eq. 8) solved and traced
  back as Algorithm 3 describes (Sec. IV-B-2);
* ``backward_dp`` - the backward Bellman equation (Eq. 9) and Algorithm 4;
* ``fm_forward`` / ``fm_backward`` - the O(L) cost function f_m of the
  zero-one program (Sec. III-B) evaluated for a given decision;
* ``brute_force_forward`` / ``brute_force_backward`` - the exhaustive
  O(L 2^L) search the paper names as the impractical alternative (Sec. III-B);
* ``simulate`` - a per-mini-procedure event simulation of one iteration that
  obeys the partial orders Eq. 1-7 (Sec. III-A); it is an independent
  formulation used to pin f_m.

Readings of the paper taken here:

* Ties: the listings only replace a table entry when the candidate is strictly
  smaller, scanning k (and then n) upwards, so the smallest k and the fewest
  segments win a tie.
* Algorithm 4's final argmin reads the forward table F; it is read as the
  backward table B.
* g_k = 1 enables the decomposition position between layer L-k+1 and layer
  L-k, i.e. the k topmost layers are pushed in earlier segments than layer
  L-k (Sec. III-B definition of the backward decision).
* Pulls are issued back to back from time 0 and a segment's computation waits
  for the whole segment (the n*dt + sum(pt) term of Eq. 8); the backward pass
  starts at time 0 of its own clock, right when the forward pass ends (Eq. 3),
  so an iteration takes T_fwd + T_bwd.
"""
from __future__ import annotations

import itertools
import math

INF = math.inf


def _prefix(v):
    """Partial accumulations of a cost vector, 1-based: S[l] = v_1 + ... + v_l (Sec. IV-B-4)."""
    s = [0]
    for x in v:
        s.append(s[-1] + int(x))
    return s


def _check(*vecs):
    L = len(vecs[0])
    if L < 1:
        raise ValueError("need at least one layer")
    for v in vecs:
        if len(v) != L:
            raise ValueError("cost vectors differ in length")
        for x in v:
            if int(x) != x or x < 0:
                raise ValueError("costs must be non-negative integers")
    return L


def forward_dp(pt, fc, dt):
    """Forward scheduling: Eq. 8 and Algorithm 3.

    Returns ``(p, T_forward, F, Path)`` where ``p[l-1]`` is the paper's p_l
    (1 = layer l+1 starts a new pull mini-procedure), for l = 1..L-1.
    """
    L = _check(pt, fc)
    dt = int(dt)
    if dt < 0:
        raise ValueError("dt must be non-negative")
    PT, FC = _prefix(pt), _prefix(fc)
    # F[m][n]: least time to finish the forward computation of the first m
    # layers when their parameters arrive in n pull mini-procedures.
    F = [[INF] * (L + 1) for _ in range(L + 1)]
    Path = [[-1] * (L + 1) for _ in range(L + 1)]
    F[0][0] = 0
    for m in range(1, L + 1):
        for n in range(1, m + 1):
            for k in range(0, m):
                # legal starting time of layers k+1..m: the previous n-1
                # segments are computed and the n-th pull has arrived
                t_lst = max(F[k][n - 1], n * dt + PT[m])
                cand = t_lst + (FC[m] - FC[k])
                if F[m][n] <= cand:
                    continue
                F[m][n] = cand
                Path[m][n] = k
    t_forward, steps = INF, -1
    for k in range(1, L + 1):
        if t_forward <= F[L][k]:
            continue
        t_forward, steps = F[L][k], k
    p = [0] * (L - 1)
    cl = L
    for k in range(1, steps + 1):
        tmp = Path[cl][steps - k + 1]
        if 1 <= tmp <= L - 1:
            p[tmp - 1] = 1
        cl = tmp
    return p, t_forward, F, Path


def backward_dp(bc, gt, dt):
    """Backward scheduling: Eq. 9 and Algorithm 4.

    Returns ``(g, T_backward, B, Path)`` where ``g[k-1]`` is the paper's g_k
    (1 = a push boundary between layer L-k+1 and layer L-k).
    """
    L = _check(bc, gt)
    dt = int(dt)
    if dt < 0:
        raise ValueError("dt must be non-negative")
    BC, GT = _prefix(bc), _prefix(gt)

    def bc_sum(lo, hi):  # bc^lo + ... + bc^hi, 1-based inclusive
        return BC[hi] - BC[lo - 1] if hi >= lo else 0

    def gt_sum(lo, hi):
        return GT[hi] - GT[lo - 1] if hi >= lo else 0

    # B[m][n]: least time to finish pushing the gradients of the last m
    # layers in n push mini-procedures.
    B = [[INF] * (L + 1) for _ in range(L + 1)]
    Path = [[-1] * (L + 1) for _ in range(L + 1)]
    B[0][0] = 0
    for m in range(1, L + 1):
        for n in range(1, m + 1):
            for k in range(0, m):
                # the new segment holds layers L-m+1..L-k; it can start once
                # the link is free and backward has finished layer L-m+1
                t_lst = max(B[k][n - 1], bc_sum(L - m + 1, L))
                cand = t_lst + dt + gt_sum(L - m + 1, L - k)
                if B[m][n] <= cand:
                    continue
                B[m][n] = cand
                Path[m][n] = k
    t_backward, steps = INF, -1
    for k in range(1, L + 1):
        if t_backward <= B[L][k]:
            continue
        t_backward, steps = B[L][k], k
    g = [0] * (L - 1)
    cl = 1
    for k in range(1, steps + 1):
        tmp = Path[L - cl + 1][steps - k + 1]
        if 1 <= tmp <= L - 1:
            g[tmp - 1] = 1
        cl = L - tmp + 1
    return g, t_backward, B, Path


def pull_segments(p):
    """Layer ranges (lo, hi), 1-based inclusive, of the pull mini-procedures of decision p."""
    L = len(p) + 1
    segs, lo = [], 1
    for l in range(1, L):
        if p[l - 1]:
            segs.append((lo, l))
            lo = l + 1
    segs.append((lo, L))
    return segs


def push_segments(g):
    """Layer ranges (lo, hi) of the push mini-procedures of decision g, in push order (top first)."""
    L = len(g) + 1
    segs, hi = [], L
    for k in range(1, L):
        if g[k - 1]:
            segs.append((L - k + 1, hi))
            hi = L - k
    segs.append((1, hi))
    return segs


def fm_forward(pt, fc, dt, p):
    """f_m's forward part: time at which the forward computation of layer L ends (Sec. III-B)."""
    _check(pt, fc)
    link = 0
    done = 0
    for lo, hi in pull_segments(p):
        link += int(dt) + sum(int(v) for v in pt[lo - 1:hi])
        done = max(done, link) + sum(int(v) for v in fc[lo - 1:hi])
    return done


def fm_backward(bc, gt, dt, g):
    """f_m's backward part: time at which the last push ends, counted from the end of forward."""
    L = _check(bc, gt)
    link = 0
    for lo, hi in push_segments(g):
        ready = sum(int(v) for v in bc[lo - 1:L])
        link = max(link, ready) + int(dt) + sum(int(v) for v in gt[lo - 1:hi])
    return link


def fm(pt, fc, bc, gt, dt, p, g):
    """Estimated iteration time f_m(pt, fc, bc, gt, dt, L, p, g) = T_fwd + T_bwd."""
    return fm_forward(pt, fc, dt, p) + fm_backward(bc, gt, dt, g)


def brute_force_forward(pt, fc, dt):
    """Every forward decision p and its f_m value: returns (best value, set of optimal p)."""
    L = _check(pt, fc)
    best, arg = INF, []
    for bits in itertools.product((0, 1), repeat=L - 1):
        t = fm_forward(pt, fc, dt, list(bits))
        if t < best:
            best, arg = t, [bits]
        elif t == best:
            arg.append(bits)
    return best, set(arg)


def brute_force_backward(bc, gt, dt):
    """Every backward decision g and its f_m value: returns (best value, set of optimal g)."""
    L = _check(bc, gt)
    best, arg = INF, []
    for bits in itertools.product((0, 1), repeat=L - 1):
        t = fm_backward(bc, gt, dt, list(bits))
        if t < best:
            best, arg = t, [bits]
        elif t == best:
            arg.append(bits)
    return best, set(arg)


def simulate(pt, fc, bc, gt, dt, p, g):
    """Event simulation of one iteration, one mini-procedure at a time.

    Resources: one link that carries pulls and pushes one message at a time,
    and one compute unit.  Each mini-procedure starts as soon as every partial
    order of Eq. 1-7 that constrains it is met.  Returns a dict with per-layer
    (start, end) pairs for pull ("pt"), forward ("fc"), backward ("bc") and
    push ("gt") plus the totals T_fwd and T_bwd; backward times are counted
    from the end of the forward pass.
    """
    L = _check(pt, fc, bc, gt)
    dt = int(dt)
    tl = {"pt": [None] * (L + 1), "fc": [None] * (L + 1), "bc": [None] * (L + 1), "gt": [None] * (L + 1)}
    # pulls: each segment is one message of dt + sum(pt); its layers' data is
    # usable when the whole message has arrived
    link = 0
    arrive = [0] * (L + 1)
    for lo, hi in pull_segments(p):
        start = link
        link = start + dt + sum(pt[lo - 1:hi])
        for l in range(lo, hi + 1):
            tl["pt"][l] = (start, link)
            arrive[l] = link
    t = 0
    for l in range(1, L + 1):  # Eq. 5: forward in layer order; Eq. 1: after its pull
        start = max(t, arrive[l])
        t = start + fc[l - 1]
        tl["fc"][l] = (start, t)
    t_fwd = t
    t = 0
    bwd_end = [0] * (L + 2)
    for l in range(L, 0, -1):  # Eq. 6: backward in reverse order; Eq. 3 via the reset clock
        tl["bc"][l] = (t, t + bc[l - 1])
        t += bc[l - 1]
        bwd_end[l] = t
    link = 0
    for lo, hi in push_segments(g):  # Eq. 7: pushes top first; Eq. 2: after its backward
        start = max(link, max(bwd_end[l] for l in range(lo, hi + 1)))
        link = start + dt + sum(gt[lo - 1:hi])
        for l in range(lo, hi + 1):
            tl["gt"][l] = (start, link)
    tl["T_fwd"] = t_fwd
    tl["T_bwd"] = link
    return tl


def sequential(L):
    """The default-PS decision [0, L] / [L+1, 1]: one pull and one push mini-procedure."""
    return [0] * (L - 1)


def layer_by_layer(L):
    """The layer-by-layer decision [0, 1, ..., L] / [L+1, L, ..., 1]."""
    return [1] * (L - 1)


# ---------------------------------------------------------------- iBatch (Sec. III-C)
#
# The greedy schedulers DynaComm is compared with.  Readings where the
# listings leave a case open:
# * Algorithm 1 fixes D_f[1] by its steps 3-4 (largest first-segment compute,
#   then cheapest first transfer) but not D_f[2] among the pairs sharing that
#   D_f[1]; it is chosen by the loop's own rule, least slack
#   dt + pt(D_f[1]+1..D_f[2]) - fc(1..D_f[1]), ties to the smaller position.
# * If no pair passes step 2, the whole model is one segment.
# * If no x qualifies inside the forward loop, the rest of the model is one
#   segment (j = L); inside the backward loop, the next segment is the single
#   layer m-1 (its compute is the shortest, so it overruns the least).
# * Ties of the least-slack choice go to the position met first in the scan
#   (the smallest x), and ties between Algorithm 2's candidates to the first.
# * Algorithm 1's reverse twin is not given in the paper; only the printed
#   front-to-back pass is used.

def ibatch_forward(pt, fc, dt):
    """Algorithm 1: greedy forward batching.  Returns the decision p (list of L-1 bits)."""
    L = _check(pt, fc)
    dt = int(dt)
    PT, FC = _prefix(pt), _prefix(fc)
    if L == 1:
        return []
    S2 = []
    for d1 in range(1, L):
        for d2 in range(d1 + 1, L + 1):
            if dt + (PT[d2] - PT[d1]) >= FC[d1] - FC[0]:
                S2.append((d1, d2))
    if not S2:
        return [0] * (L - 1)
    best_fc = max(FC[d1] for d1, _ in S2)
    S3 = [(d1, d2) for d1, d2 in S2 if FC[d1] == best_fc]
    best_pull = min(dt + PT[d1] for d1, _ in S3)
    S4 = [(d1, d2) for d1, d2 in S3 if dt + PT[d1] == best_pull]
    d1 = S4[0][0]
    d2 = min((dt + (PT[b] - PT[a]) - (FC[a] - FC[0]), b) for a, b in S4 if a == d1)[1]
    D = [0, d1, d2]
    n, m = d1, d2
    while m != L:
        opts = [x for x in range(m + 1, L + 1) if dt + (PT[x] - PT[m]) >= FC[m] - FC[n]]
        if opts:
            j = min((dt + (PT[x] - PT[m]) - (FC[m] - FC[n]), x) for x in opts)[1]
        else:
            j = L
        n, m = m, j
        D.append(m)
    p = [0] * (L - 1)
    for d in D[1:-1]:
        p[d - 1] = 1
    return p


def ibatch_backward(bc, gt, dt):
    """Algorithm 2: greedy gradient batching over every second position n.

    Returns (g, T_backward) with the candidate of least f_m backward time.
    """
    L = _check(bc, gt)
    dt = int(dt)
    BC, GT = _prefix(bc), _prefix(gt)
    if L == 1:
        return [], fm_backward(bc, gt, dt, [])
    best = None
    for n in range(2, L + 1):
        D = [L + 1, n]
        k, m = 1, n
        while m != 1:
            pushed = k * dt + (GT[L] - GT[m - 1])          # gt over layers m..L
            opts = [x for x in range(1, m) if pushed >= BC[m - 1] - BC[x - 1]]  # bc over x..m-1
            if opts:
                j = min((pushed - (BC[m - 1] - BC[x - 1]), x) for x in opts)[1]
            else:
                j = m - 1
            D.append(j)
            m = j
            k += 1
        # positions L+1 > d_1 > ... > 1: segment layers d_{i}-1 .. d_{i+1}; a boundary
        # between layer d and d-1 (1 < d <= L) is g_k with L - k = d - 1
        g = [0] * (L - 1)
        for d in D[1:-1]:
            g[L - d] = 1
        t = fm_backward(bc, gt, dt, g)
        if best is None or t < best[1]:
            best = (g, t)
    return best
