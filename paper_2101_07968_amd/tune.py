"""Measure the best launch plan of every conv pass of the built-in workloads.

Writes the table of measured plans that libdc.so compiles in
(``csrc/plan_table.inc``).  For each distinct conv / FC geometry of the
workloads at their own batch sizes and each of its passes, every candidate
plan (tile M x tile N, split-K factor; dc_conv2d_plan_candidates) is pinned
with dc_conv2d_set_plan and timed through the conv entry point on HIP events.
The three fastest and the cost model's own choice are then timed again in
interleaved rounds; the median decides.  A shape enters the table only when
its winner beats the cost model's choice by more than --margin, so timing
noise does not churn plans.  A pass that runs on the weight-streaming FC
data-gradient kernel (plan source 3) or on the direct RGB-layer kernels (source 4) is
skipped.  Needs a GPU; run from the repository root:

    python -m paper_2101_07968_amd.tune --out plan_table.inc

then copy the output over ``paper_2101_07968_amd/csrc/plan_table.inc`` and
rebuild.
"""
from __future__ import annotations

import argparse
import ctypes
import statistics
import sys
import time

PASS_NAMES = ("fwd", "dgrad", "wgrad")


def _geometries(PN, workloads):
    geoms = {}
    for name in workloads:
        ops, hwc, _ = PN.build(name)
        batch = PN.WORKLOADS[name]["batch"]
        for _i, g, first in PN.conv_geoms(ops, hwc, batch):
            rec = geoms.setdefault(tuple(g), {"first": True, "users": {}})
            rec["first"] = rec["first"] and bool(first)   # dgrad is timed if any use needs it
            rec["users"][name] = rec["users"].get(name, 0) + 1
    return geoms


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", required=True)
    ap.add_argument("--workloads", default="", help="comma list (default: every built-in workload)")
    ap.add_argument("--margin", type=float, default=0.03, help="minimum gain over the cost model's plan")
    ap.add_argument("--rounds", type=int, default=3)
    a = ap.parse_args(argv)

    import torch
    from . import _lib as D
    from . import nets as PN

    names = [w for w in a.workloads.split(",") if w] or sorted(PN.WORKLOADS)
    geoms = _geometries(PN, names)
    s = torch.cuda.current_stream()
    sp = s.cuda_stream
    print(f"[tune] {len(geoms)} geometries of {','.join(names)} on "
          f"{torch.cuda.get_device_properties(0).gcnArchName}", flush=True)
    t0 = time.time()
    entries, totals = [], {}

    for gi, (g, rec) in enumerate(geoms.items()):
        n, h, w, c, k, r, ss, st, pad, pad_w = g
        P, Q = (h + 2 * pad - r) // st + 1, (w + 2 * pad_w - ss) // st + 1
        sh = D.ConvShape(*g)
        x = torch.randn(n, h, w, c, device="cuda")
        wt = torch.randn(k, r, ss, c, device="cuda") * (2.0 / (r * ss * c)) ** 0.5
        y = torch.empty(n, P, Q, k, device="cuda")
        dy = torch.randn(n, P, Q, k, device="cuda") * 1e-3
        dx = torch.empty(n, h, w, c, device="cuda")
        dw = torch.empty(k, r, ss, c, device="cuda")
        line = []
        for pas in (0, 1, 2):
            if pas == 1 and rec["first"]:
                continue
            src = D.conv_plan_info(g, pas)[7]
            if src in (3, 4):   # the FC streaming kernel, the RGB layer's direct kernels
                line.append(f"{PASS_NAMES[pas]} {'FC streaming' if src == 3 else 'direct RGB-layer'} kernel")
                continue

            def run(ws, wsb, pas=pas):
                if pas == 0:
                    D.call("dc_conv2d_forward", ctypes.byref(sh), x.data_ptr(), wt.data_ptr(), None, 0,
                           y.data_ptr(), ws, wsb, sp)
                elif pas == 1:
                    D.call("dc_conv2d_backward_data", ctypes.byref(sh), dy.data_ptr(), wt.data_ptr(), 0,
                           dx.data_ptr(), ws, wsb, sp)
                else:
                    D.call("dc_conv2d_backward_filter", ctypes.byref(sh), x.data_ptr(), dy.data_ptr(),
                           dw.data_ptr(), None, ws, wsb, sp)

            def time_plan(plan, reps=None):
                D.conv_set_plan(g, pas, *plan)
                wsb = max(D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh)), 256)
                if wsb > (4 << 30):
                    return None
                buf = torch.empty(wsb + 256, dtype=torch.uint8, device="cuda")
                ws = (buf.data_ptr() + 255) // 256 * 256
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                run(ws, wsb)
                if reps is None:   # size the repetitions to about 2 ms of work
                    e0.record(s)
                    run(ws, wsb)
                    e1.record(s)
                    e1.synchronize()
                    reps = max(3, min(50, int(2.0 / max(e0.elapsed_time(e1), 1e-3))))
                e0.record(s)
                for _ in range(reps):
                    run(ws, wsb)
                e1.record(s)
                e1.synchronize()
                return e0.elapsed_time(e1) / reps, reps

            D.conv_set_plan(g, pas, -1)
            model = tuple(D.conv_plan_info(g, pas)[:3])
            first_pass = {}
            for plan in D.conv_plan_candidates(g, pas):
                t = time_plan(plan)
                if t is not None:
                    first_pass[plan] = t
            if model not in first_pass:   # only when its workspace would exceed the cap
                D.conv_set_plan(g, pas, 0)
                continue
            short = sorted(first_pass, key=lambda p: first_pass[p][0])[:3]
            if model not in short:
                short.append(model)
            med = {}
            samples = {p: [] for p in short}
            for _ in range(a.rounds):
                for p in short:
                    samples[p].append(time_plan(p, first_pass[p][1])[0])
            for p in short:
                med[p] = statistics.median(samples[p])
            D.conv_set_plan(g, pas, 0)
            best = min(med, key=med.get)
            t_model = med[model]
            use = best if (best != model and t_model > (1.0 + a.margin) * med[best]) else model
            if use != model:
                entries.append((pas, g, use, t_model, med[use]))
            for name, cnt in rec["users"].items():
                tm, tu = totals.get(name, (0.0, 0.0))
                totals[name] = (tm + cnt * t_model, tu + cnt * med.get(use, t_model))
            line.append(f"{PASS_NAMES[pas]} {model}->{use} {t_model:.3f}/{med.get(use, t_model):.3f} ms")
        del x, wt, y, dy, dx, dw
        print(f"[tune {gi + 1}/{len(geoms)} {time.time() - t0:.0f}s] {g}: " + "; ".join(line), flush=True)

    torch.cuda.synchronize()
    with open(a.out, "w") as f:
        f.write("// Measured plans: {pass, n, h, w, c, k, r, s, stride, pad, pad_w, tile M, tile N, split-K}.\n")
        f.write(f"// Written by: python -m paper_2101_07968_amd.tune {' '.join(argv or sys.argv[1:])}\n")
        f.write(f"// on {torch.cuda.get_device_properties(0).gcnArchName.split(':')[0]}; margin {a.margin}, "
                f"{a.rounds} rounds.  "
                "Comments: cost model's plan time -> this plan's time.\n")
        for pas, g, use, tm, tu in sorted(entries):
            f.write("{%d, %s, %d, %d, %d}, // %s %.4f -> %.4f ms\n"
                    % (pas, ", ".join(map(str, g)), use[0], use[1], use[2], PASS_NAMES[pas], tm, tu))
    for name, (tm, tu) in sorted(totals.items()):
        print(f"[tune] {name}: conv passes {tm:.3f} ms with the cost model, {tu:.3f} ms with the table "
              f"({100 * (1 - tu / tm):.1f}% less)", flush=True)
    print(f"[tune] {len(entries)} entries -> {a.out}", flush=True)


if __name__ == "__main__":
    main()
