"""Write the planner fixture for the tiny workload from the oracle alone.

The tiny CNN (conv3x3 3->8, conv3x3 8->16, FC 1024->64, FC 64->10) has
per-layer parameter bytes 896, 4672, 262400 and 2600.  Its synthetic profile
prices a transfer at 1 GB/s (1 byte = 1 ns), a forward layer at 10 GFLOP/s of
its forward multiply-adds at batch 4, a backward layer at twice that, and the
per-transmission overhead dt at 100 us.  The expected decisions come from the
oracle's forward (Eq. 8, Algorithm 3) and backward (Eq. 9, Algorithm 4)
dynamic programs; the test that reads this file also checks them against
exhaustive search.

Run: python tests/golden/make_golden.py
"""
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))

from oracle import plan  # noqa: E402


def tiny_profile():
    pt = [896, 4672, 262400, 2600]
    gt = list(pt)
    # forward multiply-adds at batch 4, 2 FLOPs each, at 10 GFLOP/s = 10 FLOP/ns
    macs = [4 * 32 * 32 * 8 * 27, 4 * 16 * 16 * 16 * 72, 4 * 1024 * 64, 4 * 64 * 10]
    fc = [round(2 * m / 10) for m in macs]
    bc = [2 * v for v in fc]
    return pt, fc, bc, gt, 100000


def main():
    pt, fc, bc, gt, dt = tiny_profile()
    p, tf, _, _ = plan.forward_dp(pt, fc, dt)
    g, tb, _, _ = plan.backward_dp(bc, gt, dt)
    L = len(pt)
    out = {
        "source": "written by tests/golden/make_golden.py from oracle.plan",
        "profile": {"pt": pt, "fc": fc, "bc": bc, "gt": gt, "dt": dt},
        "p": p, "T_fwd": tf, "g": g, "T_bwd": tb,
        "T_fwd_sequential": plan.fm_forward(pt, fc, dt, plan.sequential(L)),
        "T_fwd_lbl": plan.fm_forward(pt, fc, dt, plan.layer_by_layer(L)),
        "T_bwd_sequential": plan.fm_backward(bc, gt, dt, plan.sequential(L)),
        "T_bwd_lbl": plan.fm_backward(bc, gt, dt, plan.layer_by_layer(L)),
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_plan.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(path, out)


if __name__ == "__main__":
    main()
