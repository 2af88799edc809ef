"""Where the backward pass's gradient terms are carried out, on the host.

Sec. III-A's backward procedure applies the chain rule op by op in reverse
order; a tensor read by several ops receives one term from each reader.  The
library fixes, when a model is built, which term writes a tensor's gradient
and which add to it, and folds a ReLU's term into a neighbouring launch where
it can.  dc_backward_schedule reports the terms in the order the launches make
them, without a GPU.  These tests check, for the nine workloads, for graphs
built to stress the folds and for random graphs, that

* the terms are exactly the chain rule's: one per (reader op, input slot) of
  every tensor but the input batch;
* each tensor receives its terms in reverse op order, the order of the
  unfolded pass, the first writing and the rest adding (so every gradient is
  the same floating-point sum as without folding, bit for bit);
* no term reads an output gradient before every term of that gradient is in.
"""
import numpy as np
import pytest

from paper_2101_07968_amd import _lib as D
from paper_2101_07968_amd import nets as PN

C, FC, BN, R, MP, GAP, A, CAT, AP = (D.DC_OP_CONV, D.DC_OP_FC, D.DC_OP_BN, D.DC_OP_RELU, D.DC_OP_MAXPOOL,
                                      D.DC_OP_GAP, D.DC_OP_ADD, D.DC_OP_CONCAT, D.DC_OP_AVGPOOL)


def inputs(op):
    kind, in0, in1, in2, in3 = op[0], op[2], op[3], op[10], op[11]
    if kind == A:
        return [in0, in1]
    if kind == CAT:
        return [in0, in1] + [t for t in (in2, in3) if t >= 0]
    return [in0]


def chain_rule_terms(ops):
    """The unfolded backward pass: ops last to first, each op's input slots in order;
    (tensor, reader op, accumulate)."""
    seen, out = set(), []
    for i in range(len(ops) - 1, -1, -1):
        for t in inputs(ops[i]):
            if t > 0:
                out.append((t, i, int(t in seen)))
                seen.add(t)
    return out


def check_schedule(ops, batch, hwc, classes):
    sch = D.backward_schedule(ops, batch, hwc, classes)
    ref = chain_rule_terms(ops)
    assert sorted((e["tensor"], e["origin_op"]) for e in sch) == sorted((t, o) for t, o, _ in ref)
    per_ref, per_sch = {}, {}
    for t, o, acc in ref:
        per_ref.setdefault(t, []).append((o, acc))
    for e in sch:
        per_sch.setdefault(e["tensor"], []).append((e["origin_op"], e["accumulate"]))
    for t in per_ref:
        assert per_sch[t] == per_ref[t], (t, per_sch[t], per_ref[t])
    # a term of op o reads the gradient of o's output (tensor o + 1): all of its terms come first
    pos = {}
    for k, e in enumerate(sch):
        pos.setdefault(e["tensor"], []).append(k)
    for k, e in enumerate(sch):
        o = e["origin_op"]
        assert all(j < k for j in pos.get(o + 1, [])), (k, e)
    # launches run layer L..1, each layer's ops last to first
    layer = [op[1] for op in ops]
    execs = [e["exec_op"] for e in sch]
    assert all((layer[b], b) <= (layer[a], a) for a, b in zip(execs, execs[1:]))
    return sch


@pytest.mark.parametrize("name", sorted(PN.WORKLOADS))
def test_workload_schedules_follow_the_chain_rule(name):
    ops, hwc, classes = PN.build(name)
    sch = check_schedule(ops, 2, hwc, classes)
    relus = sum(op[0] == R for op in ops)
    # every ReLU of these workloads has its backward folded into a neighbouring launch
    carried = {e["origin_op"] for e in sch if ops[e["origin_op"]][0] == R and e["exec_op"] != e["origin_op"]}
    assert len(carried) == relus


def conv(i, layer, k=4, r=3, pad=1):
    return (C, layer, i, -1, k, r, r, 1, pad, 1, -1, -1, pad)


def relu(i, layer):
    return (R, layer, i, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0)


def concat(layer, *ts):
    ts = list(ts) + [-1] * (4 - len(ts))
    return (CAT, layer, ts[0], ts[1], 0, 0, 0, 0, 0, 0, ts[2], ts[3], 0)


def head(i, layer, classes=5):
    return [(GAP, layer, i, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0), (FC, layer + 1, i + 1, -1, classes, 0, 0, 0, 0, 1,
                                                                 -1, -1, 0)]


FOLD_CASES = {
    # a concatenation reading a ReLU's output and the ReLU's input directly
    "cat(relu(t),t)": [conv(0, 1), relu(1, 1), concat(1, 2, 1)],
    "cat(t,relu(t))": [conv(0, 1), relu(1, 1), concat(1, 1, 2)],
    "cat(relu(t),t,relu(u))": [conv(0, 1), conv(0, 1), relu(2, 1), relu(1, 1), concat(1, 4, 1, 3)],
    "cat(t,relu(t),t)": [conv(0, 1), relu(1, 1), concat(1, 1, 2, 1)],
    # a conv reading a ReLU whose input another op reads too
    "conv(relu(t))+t": [conv(0, 1), relu(1, 1), conv(2, 2), (A, 2, 3, 1, 0, 0, 0, 0, 0, 0, -1, -1, 0)],
    # a max-pool after a ReLU whose input is also added
    "pool(relu(t)),t": [conv(0, 1), relu(1, 1), (MP, 1, 2, -1, 0, 3, 3, 1, 1, 0, -1, -1, 1), concat(1, 3, 1)],
}


@pytest.mark.parametrize("name", sorted(FOLD_CASES))
def test_fold_cases(name):
    ops = list(FOLD_CASES[name])
    ops += head(len(ops), ops[-1][1])
    check_schedule(ops, 1, (4, 4, 3), 5)


def random_graph(rng):
    """A random valid network on 6 x 6 maps whose every op keeps the map size, so any
    two tensors can meet in an ADD (same channels) or a CONCAT.  Reads of the newest
    tensor are favoured, since the folds look at adjacent ops."""
    ops, ch = [], {0: 3}
    layer = 1
    r = int(rng.choice([1, 3]))
    ops.append(conv(0, 1, k=int(rng.choice([4, 8])), r=r, pad=r // 2))
    ch[1] = ops[-1][4]
    for _ in range(int(rng.integers(4, 18))):
        n = len(ops)
        pick = lambda: n if rng.random() < 0.6 else int(rng.integers(1, n + 1))
        kind = rng.choice(["conv", "conv_same", "relu", "relu", "bn", "pool", "avg", "add", "cat"])
        a = pick()
        if kind in ("conv", "conv_same"):
            if kind == "conv":
                layer += 1
            k = int(rng.choice([4, 8]))
            r = int(rng.choice([1, 3]))
            ops.append((C, layer, a, -1, k, r, r, 1, r // 2, int(rng.integers(0, 2)), -1, -1, r // 2))
            ch[n + 1] = k
        elif kind == "relu":
            ops.append(relu(a, layer))
            ch[n + 1] = ch[a]
        elif kind == "bn":
            ops.append((BN, layer, a, -1, 0, 0, 0, 0, 0, 0, -1, -1, 0))
            ch[n + 1] = ch[a]
        elif kind in ("pool", "avg"):
            ops.append((MP if kind == "pool" else AP, layer, a, -1, 0, 3, 3, 1, 1, 0, -1, -1, 1))
            ch[n + 1] = ch[a]
        elif kind == "add":
            same = [t for t in range(1, n + 1) if ch[t] == ch[a]]
            b = int(rng.choice(same))
            ops.append((A, layer, a, b, 0, 0, 0, 0, 0, 0, -1, -1, 0))
            ch[n + 1] = ch[a]
        else:
            ts = [a] + [pick() for _ in range(int(rng.integers(1, 4)))]
            ops.append(concat(layer, *ts))
            ch[n + 1] = sum(ch[t] for t in ts)
    # every tensor must be read: concatenate the unread ones into the head
    read = {t for op in ops for t in inputs(op)}
    unread = [t for t in range(1, len(ops) + 1) if t not in read and t != len(ops)] + [len(ops)]
    while len(unread) > 1:
        grp, unread = unread[:4], unread[4:]
        ops.append(concat(layer, *grp))
        unread.append(len(ops))
    return ops + head(len(ops), layer)


@pytest.mark.parametrize("block", range(10))
def test_random_graph_schedules(block):
    rng = np.random.default_rng(4242 + block)
    for _ in range(60):
        check_schedule(random_graph(rng), 1, (6, 6, 3), 5)


def test_schedule_rejects_what_model_create_rejects():
    # only a CONV / FC may read the input batch: a ReLU of tensor 0, an ADD with in1 = 0
    bad = [[relu(0, 1)] + head(1, 1),
           [conv(0, 1, k=3), (A, 1, 1, 0, 0, 0, 0, 0, 0, 0, -1, -1, 0)] + head(2, 1),
           [conv(0, 1, k=3), concat(1, 1, 0)] + head(2, 1)]
    for ops in bad:
        with pytest.raises(D.DcError) as e:
            D.backward_schedule(ops, 1, (4, 4, 3), 5)
        assert e.value.status == D.DC_EINVAL
        assert b"input batch" in D.lib().dc_last_error()
