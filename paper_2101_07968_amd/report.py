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


def _union(iv):
    out = []
    for a, b in sorted((int(a), int(b)) for a, b in iv if b > a):
        if out and a <= out[-1][1]:
            out[-1][1] = max(out[-1][1], b)
        else:
            out.append([a, b])
    return out


def _length(u):
    return sum(b - a for a, b in u)


def _common(u, v):
    i = j = tot = 0
    while i < len(u) and j < len(v):
        a, b = max(u[i][0], v[j][0]), min(u[i][1], v[j][1])
        tot += max(0, b - a)
        if u[i][1] < v[j][1]:
            i += 1
        else:
            j += 1
    return tot


def breakdown(tl):
    """The split of Sec. V-B for each pass, from one step's timeline (ns rows of
    pull start/end, forward start/end, backward start/end, push start/end per
    layer): computation alone, computation and communication together, and
    communication alone, in ms."""
    out = {}
    for key, comm, comp in (("fwd", tl[:, 0:2], tl[:, 2:4]), ("bwd", tl[:, 6:8], tl[:, 4:6])):
        cu, pu = _union(comm), _union(comp)
        both = _common(cu, pu)
        out[key] = [round((_length(pu) - both) / 1e6, 3), round(both / 1e6, 3), round((_length(cu) - both) / 1e6, 3)]
    return out


def link_rates(tl, layer_bytes, dt_ns):
    """Achieved pull and push rates (bytes/s) of one step: each segment's bytes over its
    duration less the per-transfer overhead dt, summed over the segments (a segment
    appears on the timeline row of every layer it carries)."""
    out = []
    for c0 in (0, 6):
        segs = {}
        for l in range(tl.shape[0]):
            key = (int(tl[l, c0]), int(tl[l, c0 + 1]))
            segs[key] = segs.get(key, 0) + layer_bytes[l]
        t = sum(max(e - s - dt_ns, 1) for s, e in segs)
        out.append(sum(segs.values()) / t * 1e9)
    return out


def run_case(D, PN, synth, torch, name, rate_bps, paced, steps, lbl_limit_s=6.0, dt_emul_ns=0):
    wl = PN.WORKLOADS[name]
    ops, hwc, classes = PN.build(name)
    specs = PN.param_specs(ops, hwc)
    x, y, params = synth.cnn_inputs(wl["seed"], wl["batch"], hwc, classes, specs)
    model = D.Model(ops, wl["batch"], hwc, classes)
    model.set_option(D.DC_OPT_LR, wl["lr"])
    model.set_option(D.DC_OPT_TIMELINE, 1)
    model.ps_write(params)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    lnk = D.link(rate_bps if paced else 1e9, dt_emul_ns, paced=paced)
    prof = model.profile(xd, yd, lnk, reps=3)
    nbytes = sum(model.layer_bytes())
    t0 = time.perf_counter()
    dp = D.dc_plan(prof)
    t_plan = (time.perf_counter() - t0) * 1e6
    plans = {"dp": dp, "sequential": D.dc_plan_sequential(prof), "lbl": D.dc_plan_lbl(prof),
             "ibatch": D.dc_plan_ibatch(prof)}
    res = {"workload": name, "batch": wl["batch"], "L": model.L,
           "link": (f"{rate_bps * 8 / 1e9:g} Gb/s" if paced else "unpaced") +
                   (f", dt {dt_emul_ns / 1e6:g} ms" if dt_emul_ns else ""),
           "link_fit_gbps": round(nbytes / max(float(prof.pt.sum()), 1.0) * 8, 3),
           "p": dp.decisions()[0], "g": dp.decisions()[1], "t_plan_us": round(t_plan, 1),
           "fc_ms": round(float(prof.fc.sum()) / 1e6, 3), "bc_ms": round(float(prof.bc.sum()) / 1e6, 3),
           "pt_ms": round(float(prof.pt.sum()) / 1e6, 3), "dt_us": round(prof.dt / 1e3, 1)}
    for key, pl in plans.items():
        t_model_s = (pl.t_fwd_ns + pl.t_bwd_ns) / 1e9
        if key in ("lbl", "ibatch") and t_model_s > lbl_limit_s:
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
                    "n_pull": st["n_pull"], "n_push": st["n_push"], "steps": n,
                    "split": breakdown(model.timeline())}
        if key == "dp":
            pr, gr = link_rates(model.timeline(), model.layer_bytes(), prof.dt)
            res["link_achieved_gbps"] = [round(pr * 8 / 1e9, 3), round(gr * 8 / 1e9, 3)]
    model.close()
    del xd, yd
    torch.cuda.empty_cache()
    seq = res["sequential"]["t_iter_ms"]
    res["reduced_vs_sequential"] = round(1 - res["dp"]["t_iter_ms"] / seq, 4)
    return res


def adapt(D, PN, synth, torch, name, rates_gbps, steps):
    """Dynamic adaptation: the link changes mid-run; compare keeping the old
    profile and plan with re-profiling and re-planning (Sec. IV-C cadence).
    Runs through dc_step_dynamic (planning in the idle windows)."""
    wl = PN.WORKLOADS[name]
    ops, hwc, classes = PN.build(name)
    x, y, params = synth.cnn_inputs(wl["seed"], wl["batch"], hwc, classes, PN.param_specs(ops, hwc))
    model = D.Model(ops, wl["batch"], hwc, classes)
    model.set_option(D.DC_OPT_LR, wl["lr"])
    model.ps_write(params)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    out = []
    prof = None
    for phase, g in enumerate(rates_gbps):
        lnk = D.link(g * 1e9 / 8, 0, paced=True)
        for fresh in ((False, True) if phase else (True,)):
            if fresh:
                t0 = time.perf_counter()
                prof = model.profile(xd, yd, lnk, reps=2)
                t_prof = time.perf_counter() - t0
            plan = D.dc_plan(prof)
            its = []
            for _ in range(steps):
                st = model.step_dynamic(xd, yd, prof, plan, lnk)
                its.append(st["t_iter_ns"])
            # what the plan in use costs on the link actually present
            truth = model.profile(xd, yd, lnk, reps=1) if not fresh else prof
            ev = D.dc_plan_eval(truth, *plan.decisions())
            best = D.dc_plan(truth)
            out.append({"link_gbps": g, "profile": "re-profiled" if fresh else "stale", "p": plan.decisions()[0],
                        "g": plan.decisions()[1], "t_iter_ms": round(float(np.mean(its)) / 1e6, 2),
                        "f_m_ms": round((ev.t_fwd_ns + ev.t_bwd_ns) / 1e6, 2),
                        "best_f_m_ms": round((best.t_fwd_ns + best.t_bwd_ns) / 1e6, 2),
                        "plan_hidden": st["plan_hidden"], "t_plan_us": round((st["t_plan_fwd_ns"] +
                                                                            st["t_plan_bwd_ns"]) / 1e3, 1),
                        "t_profile_s": round(t_prof, 3) if fresh else None})
            print(json.dumps(out[-1]), file=sys.stderr, flush=True)
    model.close()
    lines = ["| link (Gb/s) | profile | pull / push segments | measured t_iter (ms) | f_m of plan in use (ms) | "
             "f_m of the best plan (ms) | planning (us, hidden) |", "|---|---|---|---|---|---|---|"]
    for o in out:
        lines.append(f"| {o['link_gbps']:g} | {o['profile']} | {sum(o['p']) + 1} / {sum(o['g']) + 1} | "
                     f"{o['t_iter_ms']:.2f} | {o['f_m_ms']:.2f} | {o['best_f_m_ms']:.2f} | "
                     f"{o['t_plan_us']:.0f} ({'yes' if o['plan_hidden'] == 3 else 'no'}) |")
    return "\n".join(lines)


def planner_scaling(D, PN, synth, Ls, reps=20):
    """Host time of the DP (Eq. 8 + 9) and of iBatch (Algorithms 1 + 2) against L on
    generated profiles (the study of Fig. 12 / Table I), median of `reps` calls,
    minus the median time of a one-layer call (the ctypes round trip).  The L of
    the paper's four evaluation networks are always included and labelled."""
    def med(f, prof):
        ts = []
        for _ in range(reps):
            t0 = time.perf_counter_ns()
            f(prof)
            ts.append(time.perf_counter_ns() - t0)
        return float(np.median(ts))
    one = D.Profile(*synth.random_profile(0, 1)[:4], 0)
    base = min(med(D.dc_plan, one), med(D.dc_plan_ibatch, one))
    lines = ["| L | DP forward + backward (us) | iBatch forward + backward (us) |", "|---|---|---|"]
    named = {}
    for name in ("vgg19", "googlenet", "inception_v4", "resnet152"):
        ops, _, _ = PN.build(name)
        named.setdefault(max(o[1] for o in ops), []).append(name)
    for L in sorted(set(Ls) | set(named)):
        pt, fc, bc, gt, dt = synth.random_profile(1000 + L, L, hi=10 ** 7, dt_hi=10 ** 6)
        prof = D.Profile(pt, fc, bc, gt, dt)
        a = max(0.0, med(D.dc_plan, prof) - base) / 1e3
        b = max(0.0, med(D.dc_plan_ibatch, prof) - base) / 1e3
        label = f"{L} ({', '.join(named[L])})" if L in named else f"{L}"
        lines.append(f"| {label} | {a:.1f} | {b:.1f} |")
        print(lines[-1], file=sys.stderr, flush=True)
    return "\n".join(lines)


def non_gemm(D, PN, torch, name, batch=None, reps=3):
    """Bandwidth of the HBM-bound kernels (ReLU, max-pool, BN, add, GAP, concat and
    their backward passes) at every shape the workload uses, through the C ABI,
    against MI355X's 8 TB/s.  Bytes per call are what each kernel must move
    (BN: 12 B per element forward with the one-pass statistics, 16 off the
    float4 path, and 20 backward); tensors whose whole footprint fits in the
    256 MB Infinity Cache are counted apart."""
    import ctypes
    wl = PN.WORKLOADS[name]
    n = batch or wl["batch"]
    ops, hwc, _ = PN.build(name)
    shp = PN.shapes(ops, hwc)
    s = torch.cuda.current_stream()
    sp = s.cuda_stream
    stats = {}

    def timed(kind, nbytes, fn):
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(reps):
            fn()
        e1.record(s)
        e1.synchronize()
        ms = e0.elapsed_time(e1) / reps
        key = (kind, nbytes > 256e6)
        t = stats.setdefault(key, [0, 0.0, 0.0])
        t[0] += 1
        t[1] += nbytes
        t[2] += ms

    for (kind, _l, src, other, out_ch, r, ss, stride, pad, bias, in2, in3, _pw), (ho, wo, co) in zip(ops, shp[1:]):
        h, w, c = shp[src]
        ne_in, ne_out = n * h * w * c, n * ho * wo * co
        if kind == D.DC_OP_RELU:
            x = torch.randn(ne_in, device="cuda")
            y, dx = torch.empty_like(x), torch.empty_like(x)
            timed("relu fwd", 8 * ne_in, lambda: D.call("dc_relu_forward", x.data_ptr(), y.data_ptr(), ne_in, sp))
            timed("relu bwd", 12 * ne_in, lambda: D.call("dc_relu_backward", x.data_ptr(), y.data_ptr(), 0,
                                                         dx.data_ptr(), ne_in, sp))
            del x, y, dx
        elif kind == D.DC_OP_MAXPOOL:
            ps = D.PoolShape(n, h, w, c, r, ss, stride, pad)
            x = torch.randn(ne_in, device="cuda")
            y = torch.empty(ne_out, device="cuda")
            arg = torch.empty(ne_out, dtype=torch.uint8, device="cuda")
            dx = torch.empty_like(x)
            timed("maxpool fwd", 4 * ne_in + 5 * ne_out,
                  lambda: D.call("dc_maxpool_forward", ctypes.byref(ps), x.data_ptr(), y.data_ptr(), arg.data_ptr(), sp))
            timed("maxpool bwd", 5 * ne_out + 4 * ne_in,
                  lambda: D.call("dc_maxpool_backward", ctypes.byref(ps), y.data_ptr(), arg.data_ptr(), 0,
                                 dx.data_ptr(), sp))
            del x, y, arg, dx
        elif kind == D.DC_OP_BN:
            rows = n * h * w
            x = torch.randn(ne_in, device="cuda")
            y, dx = torch.empty_like(x), torch.empty_like(x)
            g, b = torch.ones(c, device="cuda"), torch.zeros(c, device="cuda")
            mean, inv, dg, db = (torch.empty(c, device="cuda") for _ in range(4))
            wsb = D.lib().dc_batchnorm_workspace_bytes(rows, c)
            ws = torch.empty(wsb + 256, dtype=torch.uint8, device="cuda")
            wsp = (ws.data_ptr() + 255) // 256 * 256
            timed("bn fwd", (12 if c % 4 == 0 else 16) * ne_in,
                  lambda: D.call("dc_batchnorm_forward", rows, c, x.data_ptr(), g.data_ptr(), b.data_ptr(),
                                 ctypes.c_float(1e-5), y.data_ptr(), mean.data_ptr(), inv.data_ptr(), wsp, wsb, sp))
            timed("bn bwd", 20 * ne_in, lambda: D.call("dc_batchnorm_backward", rows, c, y.data_ptr(), x.data_ptr(),
                                                       g.data_ptr(), mean.data_ptr(), inv.data_ptr(), 0,
                                                       dx.data_ptr(), dg.data_ptr(), db.data_ptr(), wsp, wsb, sp))
            del x, y, dx, ws
        elif kind == D.DC_OP_ADD:
            a, b2 = torch.randn(ne_in, device="cuda"), torch.randn(ne_in, device="cuda")
            y = torch.empty_like(a)
            timed("add fwd", 12 * ne_in, lambda: D.call("dc_add_forward", a.data_ptr(), b2.data_ptr(), 0,
                                                        y.data_ptr(), ne_in, sp))
            timed("add bwd (copy)", 8 * ne_in, lambda: D.call("dc_copy_grad", a.data_ptr(), 0, y.data_ptr(), ne_in, sp))
            del a, b2, y
        elif kind == D.DC_OP_GAP:
            x = torch.randn(ne_in, device="cuda")
            y = torch.empty(n * c, device="cuda")
            dx = torch.empty_like(x)
            timed("gap fwd", 4 * ne_in + 4 * n * c,
                  lambda: D.call("dc_gap_forward", n, h * w, c, x.data_ptr(), y.data_ptr(), sp))
            timed("gap bwd", 4 * ne_in + 4 * n * c,
                  lambda: D.call("dc_gap_backward", n, h * w, c, y.data_ptr(), 0, dx.data_ptr(), sp))
            del x, y, dx
        elif kind == D.DC_OP_CONCAT:
            rows = n * h * w
            y = torch.empty(rows * co, device="cuda")
            off = 0
            for t in (src, other, in2, in3):
                if t < 0:
                    continue
                ci = shp[t][2]
                x = torch.randn(rows * ci, device="cuda")
                timed("concat fwd", 8 * rows * ci, lambda: D.call("dc_concat_forward", rows, ci, co, off,
                                                                   x.data_ptr(), y.data_ptr(), sp))
                timed("concat bwd", 8 * rows * ci, lambda: D.call("dc_concat_backward", rows, ci, co, off,
                                                                   y.data_ptr(), 0, x.data_ptr(), sp))
                off += ci
                del x
            del y
    torch.cuda.synchronize()
    lines = [f"Non-GEMM kernels, {name} batch {n} (HBM peak 8000 GB/s):", "",
             "| kernel | footprint | calls | GB moved | ms | GB/s | % of 8 TB/s |", "|---|---|---|---|---|---|---|"]
    for (kind, big), (cnt, nb, ms) in sorted(stats.items()):
        gbs = nb / ms / 1e6
        lines.append(f"| {kind} | {'> 256 MB' if big else '<= 256 MB (cache)'} | {cnt} | {nb / 1e9:.2f} | "
                     f"{ms:.3f} | {gbs:.0f} | {100 * gbs / 8000:.1f}% |")
    return "\n".join(lines)


def row(r):
    def cell(k):
        v = r.get(k, {})
        if v.get("skipped"):
            return f"model {v['t_model_ms']:.1f}"
        return f"{v['t_iter_ms']:.1f} / {v['t_model_ms']:.1f}"
    return (f"| {r['workload']} | {r['batch']} | {r['link']} | {cell('dp')} | {cell('sequential')} | {cell('lbl')} | "
            f"{cell('ibatch')} | "
            f"{r['dp']['images_per_s']:.2f} | {100 * r['reduced_vs_sequential']:.1f}% | {r['dp']['model_err'] * 100:.2f}% | "
            f"{r['dp']['n_pull']}/{r['dp']['n_push']} | {r['fc_ms']:.1f}+{r['bc_ms']:.1f} | {r['dt_us']:.0f} |")


def split_rows(r):
    rows = []
    for key in ("dp", "sequential", "lbl", "ibatch"):
        v = r.get(key, {})
        if "split" not in v:
            continue
        f, b = v["split"]["fwd"], v["split"]["bwd"]
        rows.append(f"| {r['workload']} | {r['link']} | {key} | {f[0]:.1f} / {f[1]:.1f} / {f[2]:.1f} | "
                    f"{b[0]:.1f} / {b[1]:.1f} / {b[2]:.1f} | {v['t_iter_ms']:.1f} |")
    return rows


SPLIT_HEADER = ("| workload | link | plan | forward: compute only / overlapped / link only (ms) | "
                "backward: compute only / overlapped / link only (ms) | t_iter (ms) |\n|---|---|---|---|---|---|")

HEADER = ("| workload | batch | link | DP t_iter / f_m (ms) | sequential (ms) | LBL (ms) | iBatch (ms) | DP img/s | "
          "time saved vs sequential | DP model error | pull/push segments | fc+bc (ms) | dt (us) |\n"
          "|---|---|---|---|---|---|---|---|---|---|---|---|---|")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--only", default="tiny,alexnet,resnet18,vgg16,resnet50")
    ap.add_argument("--vgg-sweep", action="store_true", help="VGG-16 at 0.1, 1, 10, 100 Gb/s and unpaced")
    ap.add_argument("--rate-sweep", default="", help="workload:g1,g2,... at those link rates (Gb/s), e.g. "
                                                      "resnet152:1,5,10,25")
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--adapt", default="", help="workload for the link-change scenario, e.g. resnet50")
    ap.add_argument("--adapt-rates", default="100,10,100", help="Gb/s of the successive phases")
    ap.add_argument("--planner-scaling", action="store_true", help="DP vs iBatch planning time against L")
    ap.add_argument("--batch-sweep", default="", help="workload:b1,b2,... at its own link, e.g. resnet50:16,32,64")
    ap.add_argument("--non-gemm", default="", help="comma list of workloads: bandwidth of the HBM-bound kernels")
    ap.add_argument("--dt-sweep", action="store_true",
                    help="VGG-16 at 100 Gb/s and unpaced with an emulated per-transfer overhead of 1 and 10 ms")
    ap.add_argument("--unpaced", action="store_true", help="run the --only workloads on unpaced copies")
    ap.add_argument("--out", default="")
    a = ap.parse_args()
    import torch

    import synth
    from . import _lib as D
    from . import nets as PN
    cases = [(n, PN.WORKLOADS[n]["link"], not a.unpaced, 0) for n in a.only.split(",") if n]
    if a.vgg_sweep:
        cases = [c for c in cases if c[0] != "vgg16"]
        cases += [("vgg16", g * 1e9 / 8, True, 0) for g in (0.1, 1, 10, 100)] + [("vgg16", 0, False, 0)]
    if a.rate_sweep:
        name, gs = a.rate_sweep.split(":")
        cases += [(name, float(g) * 1e9 / 8, True, 0) for g in gs.split(",")]
    if a.dt_sweep:
        cases = [("vgg16", rate, paced, int(dt * 1e6)) for rate, paced in ((100e9 / 8, True), (0, False))
                 for dt in (0, 1, 10)]
    if a.adapt or a.planner_scaling or a.non_gemm:
        cases = []
    rows = []
    for name, rate, paced, dt in cases:
        r = run_case(D, PN, synth, torch, name, rate, paced, a.steps, dt_emul_ns=dt)
        print(json.dumps(r), file=sys.stderr, flush=True)
        rows.append(r)
    if a.batch_sweep:
        name, bs = a.batch_sweep.split(":")
        base = dict(PN.WORKLOADS[name])
        for b in bs.split(","):
            PN.WORKLOADS[name] = dict(base, batch=int(b))
            r = run_case(D, PN, synth, torch, name, base["link"], True, a.steps)
            print(json.dumps(r), file=sys.stderr, flush=True)
            rows.append(r)
        PN.WORKLOADS[name] = base
    text = ""
    if rows:
        text = HEADER + "\n" + "\n".join(row(r) for r in rows) + "\n\n" + SPLIT_HEADER + "\n" + \
            "\n".join(x for r in rows for x in split_rows(r)) + "\n\nlink rate (Gb/s), fitted by dc_profile / " + \
            "achieved by the DP step's pulls / pushes: " + \
            ", ".join(f"{r['workload']} {r['link']}: {r['link_fit_gbps']:g} / {r['link_achieved_gbps'][0]:g} / "
                      f"{r['link_achieved_gbps'][1]:g}" for r in rows)
    if a.non_gemm:
        # a 256 MiB copy of known size first: the scale for HBM byte counters
        src = torch.ones(64 << 20, device="cuda")
        dst = torch.empty_like(src)
        D.call("dc_copy_grad", src.data_ptr(), 0, dst.data_ptr(), src.numel(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        del src, dst
        text = "\n\n".join(non_gemm(D, PN, torch, w) for w in a.non_gemm.split(","))
    if a.planner_scaling:
        text = planner_scaling(D, PN, synth, [4, 8, 16, 18, 50, 100, 160, 200, 300])
    if a.adapt:
        text = adapt(D, PN, synth, torch, a.adapt, [float(g) for g in a.adapt_rates.split(",")], a.steps)
    print(text)
    if a.out:
        with open(a.out, "w") as f:
            f.write(text + "\n")


if __name__ == "__main__":
    main()
