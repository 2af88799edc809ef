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
  roofline     conv / FC implicit-GEMM kernels against the fp32 MFMA peak,
               timed live with HIP events on their launch stream
  cpu_baseline the oracle (float64 loops) on a bounded sample, host cores
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


def cpu_baseline(name, batch_total):
    """The oracle, untuned, on one image of the workload: forward, backward and SGD."""
    import numpy as np

    import synth
    from oracle import cnn as OC
    from oracle import nets as ON
    spec = ON.get(name)
    n = 1
    net = OC.Net(spec, n)
    x, y, p = synth.cnn_inputs(0, n, spec["hwc"], spec["classes"], net.param_specs)
    t0 = time.perf_counter()
    net.step(x, y, p)
    dt = time.perf_counter() - t0
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or os.cpu_count()
    return {"value": round(n / dt, 4), "unit": "images/s", "cores": threads, "kind": "oracle",
            "sample": f"{n} of the {batch_total} images of one {name} iteration (forward, backward, SGD), "
                      f"{dt:.1f} s, float64 loops with OpenMP"}


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

    def run(kind, steps, warmup):
        # every plan starts from the same initial parameters (outside the timed region)
        model.ps_write(params)
        for _ in range(warmup):
            pl = D.dc_plan(prof) if kind == "dp" else fixed[kind]
            model.step(xd, yd, pl, lnk)
        torch.cuda.synchronize()
        iters, losses = [], []
        t0 = time.perf_counter()
        for i in range(steps):
            pl = D.dc_plan(prof) if kind == "dp" else fixed[kind]
            st = model.step(xd, yd, pl, lnk)
            iters.append(st["t_iter_ns"])
            losses.append(st["loss"])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
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
    if not args.no_roofline:
        flops, ms, per = measure_convs(D, PN, ops, hwc, batch)
        achieved = flops / (ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "kernel": "igemm_kernel (conv/FC forward, dgrad, wgrad; fp32 MFMA)",
                "achieved": round(achieved, 2), "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / FP32_MFMA_PEAK_TFLOPS, 4), "traffic": None,
                "gflop_per_step": round(flops / 1e9, 1), "conv_ms_per_step": round(ms, 3)}
        tr = traffic_from_profiles(name, batch)
        if tr is not None:
            roof["traffic"] = round(tr[0])
            roof["traffic_algorithmic"] = round(tr[1])
        log(f"[bench] conv GEMMs: {achieved:.1f} TFLOP/s over {flops / 1e9:.0f} GFLOP in {ms:.2f} ms")
        for d in sorted(per, key=lambda d: -d["ms"]):
            log(f"[bench]   {d['pass']:5s} {str(d['shape']):42s} {d['ms']:8.3f} ms {d['tflops']:7.2f} TFLOP/s")

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on the host ...")
        cpu = cpu_baseline(name, batch)

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
