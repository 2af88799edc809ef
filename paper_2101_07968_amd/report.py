"""Per-workload report: DynaComm's plan against the sequential and layer-by-layer
schedules at each workload's emulated link, measured next to the cost model f_m.

  python -m paper_2101_07968_amd.report [--only tiny,vgg16] [--vgg-sweep] [--out file.md]

For each (workload, link): profile once (Sec. IV-A), plan (Eq. 8/9), then time
dc_step with the DP decision, the sequential decision and - when it finishes in
a few seconds - the layer-by-layer decision.  Prints one markdown row per run
and a JSON line per run on stderr as it goes.
"""
from __future__ import annotations

import argparse
import json
import sys
import time

import numpy as np


def run_case(D, PN, synth, torch, name, rate_bps, paced, steps, lbl_limit_s=6.0):
    wl = PN.WORKLOADS[name]
    ops, hwc, classes = PN.build(name)
    specs = PN.param_specs(ops, hwc)
    x, y, params = synth.cnn_inputs(wl["seed"], wl["batch"], hwc, classes, specs)
    model = D.Model(ops, wl["batch"], hwc, classes)
    model.ps_write(params)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    lnk = D.link(rate_bps if paced else 1e9, 0, paced=paced)
    prof = model.profile(xd, yd, lnk, reps=3)
    t0 = time.perf_counter()
    dp = D.dc_plan(prof)
    t_plan = (time.perf_counter() - t0) * 1e6
    plans = {"dp": dp, "sequential": D.dc_plan_sequential(prof), "lbl": D.dc_plan_lbl(prof)}
    res = {"workload": name, "batch": wl["batch"], "L": model.L,
           "link": f"{rate_bps * 8 / 1e9:g} Gb/s" if paced else "unpaced",
           "p": dp.decisions()[0], "g": dp.decisions()[1], "t_plan_us": round(t_plan, 1),
           "fc_ms": round(float(prof.fc.sum()) / 1e6, 3), "bc_ms": round(float(prof.bc.sum()) / 1e6, 3),
           "pt_ms": round(float(prof.pt.sum()) / 1e6, 3), "dt_us": round(prof.dt / 1e3, 1)}
    for key, pl in plans.items():
        t_model_s = (pl.t_fwd_ns + pl.t_bwd_ns) / 1e9
        if key == "lbl" and t_model_s > lbl_limit_s:
            res[key] = {"t_model_ms": round(t_model_s * 1e3, 3), "skipped": True}
            continue
        model.ps_write(params)
        n = max(1, min(steps, int(20.0 / max(t_model_s, 1e-3))))
        if t_model_s < 2.0:
            model.step(xd, yd, pl, lnk)  # warm-up
        its, walls = [], []
        for _ in range(n):
            w0 = time.perf_counter()
            st = model.step(xd, yd, pl, lnk)
            walls.append(time.perf_counter() - w0)
            its.append(st["t_iter_ns"])
            print(f"  {name} {res['link']} {key}: t_iter {st['t_iter_ns'] / 1e6:.2f} ms", file=sys.stderr,
                  flush=True)
        t_iter = float(np.mean(its)) / 1e6
        res[key] = {"images_per_s": round(wl["batch"] / np.mean(walls), 3), "t_iter_ms": round(t_iter, 3),
                    "t_model_ms": round(t_model_s * 1e3, 3),
                    "model_err": round(abs(t_iter - t_model_s * 1e3) / (t_model_s * 1e3), 4),
                    "n_pull": st["n_pull"], "n_push": st["n_push"], "steps": n}
    model.close()
    del xd, yd
    torch.cuda.empty_cache()
    seq = res["sequential"]["t_iter_ms"]
    res["reduced_vs_sequential"] = round(1 - res["dp"]["t_iter_ms"] / seq, 4)
    return res


def row(r):
    def cell(k):
        v = r.get(k, {})
        if v.get("skipped"):
            return f"model {v['t_model_ms']:.1f}"
        return f"{v['t_iter_ms']:.1f} / {v['t_model_ms']:.1f}"
    return (f"| {r['workload']} | {r['batch']} | {r['link']} | {cell('dp')} | {cell('sequential')} | {cell('lbl')} | "
            f"{r['dp']['images_per_s']:.2f} | {100 * r['reduced_vs_sequential']:.1f}% | {r['dp']['model_err'] * 100:.2f}% | "
            f"{r['dp']['n_pull']}/{r['dp']['n_push']} | {r['fc_ms']:.1f}+{r['bc_ms']:.1f} | {r['dt_us']:.0f} |")


HEADER = ("| workload | batch | link | DP t_iter / f_m (ms) | sequential (ms) | LBL (ms) | DP img/s | "
          "time saved vs sequential | DP model error | pull/push segments | fc+bc (ms) | dt (us) |\n"
          "|---|---|---|---|---|---|---|---|---|---|---|---|")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--only", default="tiny,alexnet,resnet18,vgg16,resnet50")
    ap.add_argument("--vgg-sweep", action="store_true", help="VGG-16 at 0.1, 1, 10, 100 Gb/s and unpaced")
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--out", default="")
    a = ap.parse_args()
    import torch

    import synth
    from . import _lib as D
    from . import nets as PN
    cases = [(n, PN.WORKLOADS[n]["link"], True) for n in a.only.split(",") if n]
    if a.vgg_sweep:
        cases = [c for c in cases if c[0] != "vgg16"]
        cases += [("vgg16", g * 1e9 / 8, True) for g in (0.1, 1, 10, 100)] + [("vgg16", 0, False)]
    rows = []
    for name, rate, paced in cases:
        r = run_case(D, PN, synth, torch, name, rate, paced, a.steps)
        print(json.dumps(r), file=sys.stderr, flush=True)
        rows.append(r)
    text = HEADER + "\n" + "\n".join(row(r) for r in rows)
    print(text)
    if a.out:
        with open(a.out, "w") as f:
            f.write(text + "\n")


if __name__ == "__main__":
    main()
