"""Benchmark: images/s of DynaComm's segment-overlapped parameter-server iteration.

One step = one SGD iteration through dc_step: plan (Eq. 8/9 on the current
profile), paced pulls gating the forward layers, loss, backward, paced pushes
and the server's SGD update, on synthetic data already resident in HBM.  The
profile (Sec. IV-A) is taken once before timing, as the paper does once per
epoch.  Default workload: VGG-16, batch 32, 224x224x3, emulated 100 Gb/s link.

Prints one JSON line (rank 0, N = 1):
  value        images/s with the DynaComm plan (whole job = the one GPU)
  extra        the same for the sequential (no-overlap) and layer-by-layer plans,
               measured iteration times next to the time model f_m
  roofline     conv / FC implicit-GEMM passes against the fp32 MFMA peak, timed
               inside the timed DP steps with HIP events on the compute stream
               (DC_OPT_GEMM_TIMING); the same passes launched alone are reported
               beside them
  cpu_baseline the oracle (float64 loops) for one whole iteration of the same
               workload and batch on the host cores (about a minute for VGG-16)
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP32_MFMA_PEAK_TFLOPS = 157.3


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="vgg16", choices=["tiny", "alexnet", "resnet18", "vgg16", "resnet50", "googlenet", "vgg19",
                                                          "resnet152", "inception_v4"])
    ap.add_argument("--batch", type=int, default=0, help="0 = the workload's own batch")
    ap.add_argument("--link-gbps", default="100", help="emulated link in Gb/s, or 'pcie' for unpaced copies")
    ap.add_argument("--dt-emul-ms", type=float, default=0.0)
    ap.add_argument("--compare", default="sequential,lbl,ibatch", help="other plans to time ('' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-roofline", action="store_true")
    ap.add_argument("--oracle-configs", action="store_true",
                    help="time the oracle on every benchmark configuration and the planner oracle, then exit")
    ap.add_argument("--kernels-only", action="store_true",
                    help="run each conv / FC pass of the workload once plus a 256 MiB calibration copy "
                         "(for rocprofv3 --pmc), then exit")
    return ap.parse_args()


def calibration_copy(D, nbytes=256 << 20):
    """dc_copy_grad over nbytes: reads and writes exactly nbytes each (counter scale)."""
    import torch
    n = nbytes // 4
    a = torch.ones(n, device="cuda")
    b = torch.empty(n, device="cuda")
    torch.cuda.synchronize()
    D.call("dc_copy_grad", a.data_ptr(), 0, b.data_ptr(), n, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()


def traffic_from_profiles(name, batch):
    """HBM bytes per igemm launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel and plan-table sources; else None."""
    from paper_2101_07968_amd.profsum import gemm_sources_sha256
    path = os.path.join(ROOT, "profiles", f"igemm_{name}_b{batch}_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.strip().split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("gemm_sources_sha256") != gemm_sources_sha256():
        return None
    return float(kv["hbm_bytes_per_launch"]), float(kv["algorithmic_bytes_per_launch"])


def measure_convs(D, PN, ops, hwc, batch, reps=3):
    import torch
    geoms = PN.conv_geoms(ops, hwc, batch)
    s = torch.cuda.current_stream()
    sp = s.cuda_stream
    flops = 0.0
    ms_total = 0.0
    per = []
    for _i, g, first in geoms:
        n, h, w, c, k, r, ss, st, pad, pad_w = g
        P, Q = (h + 2 * pad - r) // st + 1, (w + 2 * pad_w - ss) // st + 1
        sh = D.ConvShape(*g)
        wsb = max(D.lib().dc_conv2d_workspace_bytes(ctypes.byref(sh)), 256)
        ws = torch.empty(wsb + 256, dtype=torch.uint8, device="cuda")
        wsp = (ws.data_ptr() + 255) // 256 * 256
        x = torch.randn(n, h, w, c, device="cuda")
        wt = torch.randn(k, r, ss, c, device="cuda") * (2.0 / (r * ss * c)) ** 0.5
        b = torch.zeros(k, device="cuda")
        y = torch.empty(n, P, Q, k, device="cuda")
        dy = torch.randn(n, P, Q, k, device="cuda") * 1e-3
        dx = torch.empty(n, h, w, c, device="cuda")
        dw = torch.empty(k, r, ss, c, device="cuda")
        mac = n * P * Q * k * r * ss * c
        passes = [("fwd", lambda: D.call("dc_conv2d_forward", ctypes.byref(sh), x.data_ptr(), wt.data_ptr(),
                                         b.data_ptr(), 0, y.data_ptr(), wsp, wsb, sp)),
                  ("wgrad", lambda: D.call("dc_conv2d_backward_filter", ctypes.byref(sh), x.data_ptr(),
                                           dy.data_ptr(), dw.data_ptr(), None, wsp, wsb, sp))]
        if not first:
            passes.append(("dgrad", lambda: D.call("dc_conv2d_backward_data", ctypes.byref(sh), dy.data_ptr(),
                                                   wt.data_ptr(), 0, dx.data_ptr(), wsp, wsb, sp)))
        for name, fn in passes:
            fn()  # warm
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            for _ in range(reps):
                fn()
            e1.record(s)
            e1.synchronize()
            ms = e0.elapsed_time(e1) / reps
            ms_total += ms
            flops += 2.0 * mac
            per.append({"shape": list(g), "pass": name, "ms": round(ms, 4),
                        "tflops": round(2.0 * mac / ms / 1e9, 2)})
        del x, wt, b, y, dy, dx, dw, ws
    torch.cuda.synchronize()
    return flops, ms_total, per


def cpu_model():
    """The host CPU's model string and the OpenMP threads the oracle runs with."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or os.cpu_count()
    return model, threads


def oracle_iteration(name, batch, seed):
    """One full oracle iteration (float64 loops: forward, backward, server SGD) on the
    workload's own seeded inputs; returns its wall time in seconds."""
    import synth
    from oracle import cnn as OC
    from oracle import nets as ON
    spec = ON.get(name)
    net = OC.Net(spec, batch)
    x, y, p = synth.cnn_inputs(seed, batch, spec["hwc"], spec["classes"], net.param_specs)
    t0 = time.perf_counter()
    net.step(x, y, p)
    return time.perf_counter() - t0


def cpu_baseline(name, batch, seed):
    """The oracle, untuned, for one whole iteration of the benchmarked workload and batch."""
    dt = oracle_iteration(name, batch, seed)
    model, threads = cpu_model()
    return {"value": round(batch / dt, 4), "unit": "images/s", "cores": threads, "kind": "oracle",
            "cpu": model, "seconds": round(dt, 2),
            "sample": f"one whole {name} iteration at batch {batch} (the benchmark's own seeded inputs): "
                      f"forward, backward and SGD in float64 loops with OpenMP on {threads} threads, {dt:.1f} s"}


def oracle_configs():
    """Oracle images/s for every benchmark configuration at its own batch and seed, and
    the planner oracle (Eq. 8 / 9 in Python) next to dc_plan at L = 50.  Host only."""
    from oracle import plan as OP
    from paper_2101_07968_amd import _lib as D
    from paper_2101_07968_amd import nets as PN
    import synth
    model, threads = cpu_model()
    rows = []
    for name in ("tiny", "alexnet", "resnet18", "vgg16", "resnet50"):
        wl = PN.WORKLOADS[name]
        dt = oracle_iteration(name, wl["batch"], wl["seed"])
        rows.append({"workload": name, "batch": wl["batch"], "seconds": round(dt, 3),
                     "images_per_s": round(wl["batch"] / dt, 4)})
        log(f"[oracle] {name} batch {wl['batch']}: {dt:.2f} s, {wl['batch'] / dt:.3f} images/s")
    plans = []
    for L in (50, 76, 152):
        pt, fc, bc, gt, dt = synth.random_profile(777 + L, L, hi=10 ** 7, dt_hi=10 ** 6)
        t0 = time.perf_counter()
        OP.forward_dp(pt, fc, dt)
        OP.backward_dp(bc, gt, dt)
        t_py = time.perf_counter() - t0
        prof = D.Profile(pt, fc, bc, gt, dt)
        D.dc_plan(prof)
        t0 = time.perf_counter()
        reps = 20
        for _ in range(reps):
            D.dc_plan(prof)
        t_c = (time.perf_counter() - t0) / reps
        plans.append({"L": L, "oracle_ms": round(t_py * 1e3, 2), "dc_plan_ms": round(t_c * 1e3, 4)})
        log(f"[oracle] planner L={L}: oracle (Python) {t_py * 1e3:.1f} ms, dc_plan {t_c * 1e3:.3f} ms")
    print(json.dumps({"cpu": model, "threads": threads, "oracle_iterations": rows, "planner": plans}), flush=True)


def _finite(v):
    """JSON has no NaN / Infinity: report non-finite numbers as null."""
    import math
    if isinstance(v, float) and not math.isfinite(v):
        return None
    if isinstance(v, dict):
        return {k: _finite(x) for k, x in v.items()}
    if isinstance(v, (list, tuple)):
        return [_finite(x) for x in v]
    return v


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (the library has no multi-GPU path); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)
    if args.oracle_configs:
        oracle_configs()
        return
    import numpy as np
    import torch

    import synth
    from paper_2101_07968_amd import _lib as D
    from paper_2101_07968_amd import nets as PN

    name = args.workload
    wl = PN.WORKLOADS[name]
    batch = args.batch or wl["batch"]
    ops, hwc, classes = PN.build(name)
    if args.kernels_only:
        torch.cuda.set_device(0)
        calibration_copy(D)
        measure_convs(D, PN, ops, hwc, batch, reps=1)
        log("[bench] kernels-only pass done")
        return
    specs = PN.param_specs(ops, hwc)
    x, y, params = synth.cnn_inputs(wl["seed"], batch, hwc, classes, specs)
    torch.cuda.set_device(0)
    model = D.Model(ops, batch, hwc, classes)
    model.set_option(D.DC_OPT_LR, wl["lr"])
    model.ps_write(params)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    paced = args.link_gbps != "pcie"
    rate = float(args.link_gbps) * 1e9 / 8 if paced else 1e9
    lnk = D.link(rate, int(args.dt_emul_ms * 1e6), paced=paced)
    log(f"[bench] {name} batch {batch}, link {args.link_gbps} {'Gb/s paced' if paced else '(unpaced)'}")

    t0 = time.perf_counter()
    prof = model.profile(xd, yd, lnk, reps=3)
    t_profile = time.perf_counter() - t0
    t0 = time.perf_counter()
    plan = D.dc_plan(prof)
    t_plan_us = (time.perf_counter() - t0) * 1e6
    log(f"[bench] profiled in {t_profile:.2f} s; plan p={plan.decisions()[0]} g={plan.decisions()[1]}")

    gemm = {"n": 0, "ns": 0, "flop": 0.0}
    # A one-element dc_relu_forward launch before and after the timed DP steps
    # marks them in a kernel trace (VGG-16's steps fold every ReLU, so they never
    # launch it); profsum's stats take the GEMM passes between the two marks.
    mark_buf = torch.zeros(2, device="cuda")

    def trace_mark():
        D.call("dc_relu_forward", mark_buf.data_ptr(), mark_buf.data_ptr() + 4, 1,
               torch.cuda.current_stream().cuda_stream)

    def run(kind, steps, warmup):
        # every plan starts from the same initial parameters (outside the timed region)
        model.ps_write(params)
        for _ in range(warmup):
            pl = D.dc_plan(prof) if kind == "dp" else fixed[kind]
            model.step(xd, yd, pl, lnk)
        # the DP steps time their own conv / FC GEMM passes with events on the compute stream
        model.set_option(D.DC_OPT_GEMM_TIMING, 1 if kind == "dp" else 0)
        if kind == "dp":
            trace_mark()
        torch.cuda.synchronize()
        iters, losses = [], []
        t0 = time.perf_counter()
        for i in range(steps):
            pl = D.dc_plan(prof) if kind == "dp" else fixed[kind]
            st = model.step(xd, yd, pl, lnk)
            iters.append(st["t_iter_ns"])
            losses.append(st["loss"])
            if kind == "dp":
                gemm["n"] += st["n_gemm"]
                gemm["ns"] += st["t_gemm_ns"]
                gemm["flop"] += st["gemm_flop"]
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        if kind == "dp":
            trace_mark()
        model.set_option(D.DC_OPT_GEMM_TIMING, 0)
        pl = D.dc_plan(prof) if kind == "dp" else fixed[kind]
        res = {"images_per_s": batch * steps / wall, "ms_per_step": wall / steps * 1e3,
               "t_iter_ms": float(np.mean(iters)) / 1e6, "t_model_ms": (pl.t_fwd_ns + pl.t_bwd_ns) / 1e6,
               "n_pull": st["n_pull"], "n_push": st["n_push"], "loss_first": losses[0], "loss_last": losses[-1]}
        res["model_err"] = abs(res["t_iter_ms"] - res["t_model_ms"]) / res["t_model_ms"]
        log(f"[bench] {kind}: {res['images_per_s']:.2f} img/s, {res['ms_per_step']:.2f} ms/step, "
            f"t_iter {res['t_iter_ms']:.2f} ms vs model {res['t_model_ms']:.2f} ms")
        return res

    fixed = {"sequential": D.dc_plan_sequential(prof), "lbl": D.dc_plan_lbl(prof), "ibatch": D.dc_plan_ibatch(prof)}
    main_res = run("dp", args.steps, args.warmup)
    others = {}
    for kind in [k for k in args.compare.split(",") if k]:
        others[kind] = run(kind, max(2, args.steps // 2), 1)

    roof = None
    if not args.no_roofline and gemm["n"]:
        # the timed DP steps' own GEMM passes: algorithmic FLOPs per pass / mean pass duration
        achieved = gemm["flop"] / (gemm["ns"] * 1e-9) / 1e12
        per_step = gemm["n"] / args.steps
        roof = {"bound": "mfma",
                "kernel": "igemm_kernel: the conv / FC GEMM passes (forward, dgrad, wgrad; fp32 MFMA), each with "
                          "its split-K reduction, as dispatched inside the timed steps",
                "achieved": round(achieved, 2), "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / FP32_MFMA_PEAK_TFLOPS, 4), "traffic": None,
                "launches_per_step": per_step, "gflop_per_launch": round(gemm["flop"] / gemm["n"] / 1e9, 3),
                "ms_per_launch": round(gemm["ns"] / gemm["n"] / 1e6, 4),
                "gemm_ms_per_step": round(gemm["ns"] / args.steps / 1e6, 3),
                "gflop_per_step": round(gemm["flop"] / args.steps / 1e9, 1)}
        tr = traffic_from_profiles(name, batch)
        if tr is not None:
            roof["traffic"] = round(tr[0])
            roof["traffic_algorithmic"] = round(tr[1])
        log(f"[bench] conv GEMMs in the steps: {achieved:.1f} TFLOP/s, {per_step:.0f} passes and "
            f"{gemm['ns'] / args.steps / 1e6:.2f} ms per step")
        # the same passes launched alone on random tensors, for comparison
        flops, ms, per = measure_convs(D, PN, ops, hwc, batch)
        iso = flops / (ms * 1e-3) / 1e12
        roof["isolated"] = {"achieved": round(iso, 2), "frac": round(iso / FP32_MFMA_PEAK_TFLOPS, 4),
                            "gemm_ms_per_step": round(ms, 3)}
        log(f"[bench] conv GEMMs alone: {iso:.1f} TFLOP/s over {flops / 1e9:.0f} GFLOP in {ms:.2f} ms")
        for d in sorted(per, key=lambda d: -d["ms"]):
            log(f"[bench]   {d['pass']:5s} {str(d['shape']):42s} {d['ms']:8.3f} ms {d['tflops']:7.2f} TFLOP/s")

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on the host ...")
        cpu = cpu_baseline(name, batch, wl["seed"])

    out = {
        "metric": "images/s per SGD iteration with segment-overlapped pull/push; conv MFMA %",
        "value": round(main_res["images_per_s"], 3),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_res["ms_per_step"], 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded N(0,1) images, uniform labels, He-normal weights)",
        "config": {"workload": name, "global_batch": batch, "image": list(hwc), "classes": classes,
                   "link": f"{args.link_gbps} Gb/s paced" if paced else "unpaced host interface",
                   "dt_emul_ms": args.dt_emul_ms, "lr": wl["lr"], "plan": "dynacomm-dp",
                   "parallelism": "single GPU"},
        "plan": {"p": plan.decisions()[0], "g": plan.decisions()[1], "t_plan_us": round(t_plan_us, 1),
                 "t_profile_s": round(t_profile, 3)},
        "dynacomm": {k: round(v, 4) if isinstance(v, float) else v for k, v in main_res.items()},
        "compare": {k: {kk: round(vv, 4) if isinstance(vv, float) else vv for kk, vv in v.items()}
                    for k, v in others.items()},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(_finite(out)), flush=True)
    model.close()


if __name__ == "__main__":
    main()
