"""Summarise rocprofv3 CSV output into the short text reports kept under profiles/.

  python -m paper_2101_07968_amd.profsum stats <kernel_trace.csv> <kernel_stats.csv> --steps 10 --flops 2964.7 \
      --cmd "<command>" > profiles/igemm_<workload>_kernel_stats.md
  python -m paper_2101_07968_amd.profsum traffic <fetch counter_collection.csv> <write counter_collection.csv> \
      --workload vgg16 --batch 32 --cmd "<commands>" > profiles/igemm_<workload>_b<batch>_traffic.txt

stats: per-kernel totals from --stats, and the conv/FC GEMM passes of bench.py's
timed DP steps (the dispatches between the two relu_fwd_kernel marks it launches
around them), per step and per pass, for comparison with the bench's roofline.

traffic: FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the igemm dispatches of a
`bench.py --kernels-only` run, scaled by what the same counters read for the
256 MiB calibration copy, against the algorithmic bytes of those launches.

mfma: SQ_INSTS_VALU_MFMA_MOPS_F32 (units of 512 flops), SQ_VALU_MFMA_BUSY_CYCLES
and GRBM_GUI_ACTIVE of the same igemm dispatches, with their durations from a
kernel-trace run: MFMA flops issued against algorithmic flops, and the fraction
of SIMD cycles the matrix cores were busy.

hbm: FETCH_SIZE / WRITE_SIZE of every dispatch of a run that includes a
calibration copy (the non-GEMM report does), over durations from a
kernel-trace run of the same command, per bandwidth-bound kernel.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))


GEMM_SOURCES = ("igemm.hip", "fc.hip", "conv3.hip", "plan_table.cpp", "plan_table.inc")


def gemm_sources_sha256():
    """One hash over the conv GEMM kernels and their launch-plan table: a counter
    summary is only valid for the sources it was taken on."""
    h = hashlib.sha256()
    for name in GEMM_SOURCES:
        h.update(open(os.path.join(HERE, "csrc", name), "rb").read())
    return h.hexdigest()


def short(name):
    name = name.replace("dc::(anonymous namespace)::", "")
    name = re.sub(r"\(.*$", "", name) if not is_gemm(name) else name.split("(")[0]
    return name.replace("void ", "")[:80]


def is_gemm(name):
    """A dispatch of a conv/FC pass: the GEMM, its split-K reduction or its channel padding, the FC
    forward and data-gradient kernels, or the RGB layer's direct kernels."""
    return any(k in name for k in ("igemm_kernel", "splitk_reduce_kernel", "pad_channels_kernel",
                                   "fc_dgrad_kernel", "fc_dgrad_reduce_kernel", "fc_fwd_kernel", "fc_fwd_reduce_kernel",
                                   "conv3_"))


def is_pass(name):
    """The one dispatch of each conv/FC pass that does its multiply-adds."""
    return ("igemm_kernel" in name or any(k in name and "reduce" not in name for k in ("fc_dgrad_kernel", "fc_fwd_kernel"))
            or "conv3_fwd_kernel" in name or "conv3_wgrad_kernel" in name)


def cmd_stats(a):
    rows = list(csv.DictReader(open(a.stats)))
    out = ["# rocprofv3 kernel statistics", "", f"Command: `{a.cmd}`", "",
           "| kernel | calls | total ms | avg us | % |", "|---|---|---|---|---|"]
    for r in rows[:a.top]:
        out.append(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
                   f"{float(r['AverageNs']) / 1e3:.1f} | {float(r['Percentage']):.2f} |")
    gemm_total = sum(float(r["TotalDurationNs"]) for r in rows if is_gemm(r["Name"]))
    gemm_calls = sum(int(r["Calls"]) for r in rows if is_gemm(r["Name"]))
    out += ["", f"All conv-pass dispatches (implicit GEMM, split-K reduce, channel padding): {gemm_calls} calls, "
            f"{gemm_total / 1e6:.2f} ms."]
    trace = list(csv.DictReader(open(a.trace)))
    trace.sort(key=lambda r: int(r["Start_Timestamp"]))
    marks = [i for i, r in enumerate(trace) if "relu_fwd_kernel" in r["Kernel_Name"]]
    if len(marks) < 2:
        raise SystemExit("no pair of relu_fwd_kernel marks around the timed steps in the trace")
    win = [r for r in trace[marks[0] + 1:marks[1]] if is_gemm(r["Kernel_Name"])]
    dur = sum(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in win)
    passes = sum(1 for r in win if is_pass(r["Kernel_Name"]))
    gemm_only = sum(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in win if "igemm_kernel" in r["Kernel_Name"])
    n_igemm = sum(1 for r in win if "igemm_kernel" in r["Kernel_Name"])
    per_step = dur / a.steps / 1e6
    out += ["", "Timed steps (the dispatches between the two relu_fwd_kernel marks bench.py places around them):",
            f"{passes} conv/FC passes ({passes // a.steps} per step), {len(win)} dispatches (implicit GEMM, "
            f"split-K reduce, channel padding, FC and RGB-layer kernels), {dur / 1e6:.2f} ms in all, "
            f"{per_step:.3f} ms per step.",
            f"Mean duration per pass: {dur / max(passes, 1) / 1e3:.1f} us; igemm_kernel alone: "
            f"{n_igemm} dispatches, mean {gemm_only / max(n_igemm, 1) / 1e3:.1f} us."]
    if a.flops:
        out.append(f"Algorithmic GEMM work per step {a.flops:.1f} GFLOP -> "
                   f"{a.flops / per_step:.1f} TFLOP/s from these durations "
                   f"({100 * a.flops / per_step / 157.3:.1f}% of the 157.3 TFLOP/s fp32 matrix peak).")
    print("\n".join(out))


def read_counter(path, counter):
    rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    return rows


def conv_bytes(geoms):
    """Algorithmic bytes of each conv pass launch: every operand read once, the result written once."""
    out = []
    for _i, g, first in geoms:
        n, h, w, c, k, r, s, st, pad, pad_w = g
        P, Q = (h + 2 * pad - r) // st + 1, (w + 2 * pad_w - s) // st + 1
        x, y, wt = n * h * w * c * 4, n * P * Q * k * 4, k * r * s * c * 4
        out.append(("fwd", x + wt + y))
        out.append(("wgrad", x + y + wt))
        if not first:
            out.append(("dgrad", y + wt + x))
    return out


def cmd_traffic(a):
    from . import nets as PN
    fetch = read_counter(a.fetch, "FETCH_SIZE")
    write = read_counter(a.write, "WRITE_SIZE")
    cal_f = [float(r["Counter_Value"]) for r in fetch if "copy_grad_kernel" in r["Kernel_Name"]]
    cal_w = [float(r["Counter_Value"]) for r in write if "copy_grad_kernel" in r["Kernel_Name"]]
    known_kib = a.cal_bytes / 1024.0
    sf, sw = known_kib / cal_f[0], known_kib / cal_w[0]
    gf = [float(r["Counter_Value"]) for r in fetch if is_pass(r["Kernel_Name"])]
    gw = [float(r["Counter_Value"]) for r in write if is_pass(r["Kernel_Name"])]
    n = len(gf)
    hbm = (sum(gf) * sf + sum(gw) * sw) * 1024.0 / n
    ops, hwc, _ = PN.build(a.workload)
    passes = conv_bytes(PN.conv_geoms(ops, hwc, a.batch))
    algo = sum(b for _, b in passes) / len(passes)
    sha = gemm_sources_sha256()
    print(f"# HBM traffic of the implicit-GEMM kernel, {a.workload} batch {a.batch}")
    print(f"# commands: {a.cmd}")
    print(f"# calibration: {a.cal_bytes} B copy read as FETCH_SIZE {cal_f[0]:.1f} KiB, WRITE_SIZE {cal_w[0]:.1f} KiB")
    print(f"# pass dispatches (igemm_kernel, fc_fwd_kernel / fc_dgrad_kernel for the FC passes they take, "
          f"conv3_fwd_kernel / conv3_wgrad_kernel for the RGB layer): {n} "
          f"({len(passes)} conv/FC passes, each launched twice)")
    print(f"# raw FETCH_SIZE {sum(gf):.0f} KiB, WRITE_SIZE {sum(gw):.0f} KiB over those dispatches")
    print(f"fetch_scale={sf:.4f}")
    print(f"write_scale={sw:.4f}")
    print(f"hbm_bytes_per_launch={hbm:.0f}")
    print(f"algorithmic_bytes_per_launch={algo:.0f}")
    print(f"hbm_over_algorithmic={hbm / algo:.3f}")
    print(f"gemm_sources_sha256={sha}")


def _trace_durations(path, keep):
    """Durations (ns) of the dispatches whose kernel name passes keep(), in dispatch order."""
    rows = [r for r in csv.DictReader(open(path)) if keep(r["Kernel_Name"])]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    return [(r["Kernel_Name"], int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) for r in rows]


def _counters(path, names):
    """{dispatch id: (kernel name, {counter: value})} for the named counters."""
    out = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] not in names:
            continue
        d = out.setdefault(int(r["Dispatch_Id"]), (r["Kernel_Name"], {}))
        d[1][r["Counter_Name"]] = d[1].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return dict(sorted(out.items()))


def cmd_mfma(a):
    """MFMA work and busy fraction of the pass dispatches (implicit GEMM, FC and RGB-layer kernels, all on
    fp32 MFMA) of a `bench.py --kernels-only` run."""
    from . import nets as PN
    cnt = _counters(a.counters, {"SQ_INSTS_VALU_MFMA_MOPS_F32", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE"})
    gem = [(k, v) for k, v in cnt.values() if is_pass(k)]
    dur = [d for _, d in _trace_durations(a.trace, is_pass)]
    if len(dur) != len(gem):
        raise SystemExit(f"{len(gem)} counted pass dispatches but {len(dur)} in the trace")
    mops = sum(v.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0) for _, v in gem)
    busy = sum(v.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) for _, v in gem)
    active = sum(v.get("GRBM_GUI_ACTIVE", 0) for _, v in gem)
    ops, hwc, _ = PN.build(a.workload)
    algo = 0.0
    for _i, g, first in PN.conv_geoms(ops, hwc, a.batch):
        n, h, w, c, k, r, s_, st, pad, pad_w = g
        P, Q = (h + 2 * pad - r) // st + 1, (w + 2 * pad_w - s_) // st + 1
        algo += 2.0 * n * P * Q * k * r * s_ * c * (2 if first else 3)
    launches = len(gem) / (len(PN.conv_geoms(ops, hwc, a.batch)) * 3 - sum(1 for *_, f in
                                                                          PN.conv_geoms(ops, hwc, a.batch) if f))
    flops = mops * 512.0
    simds = a.cus * 4
    print(f"# fp32 MFMA counters of the conv/FC pass kernels, {a.workload} batch {a.batch}")
    print(f"# commands: {a.cmd}")
    print(f"# pass dispatches: {len(gem)} ({launches:g} launches of each conv/FC pass)")
    print(f"mfma_flops_per_iteration={flops / launches:.4e}")
    print(f"algorithmic_flops_per_iteration={algo:.4e}")
    print(f"mfma_over_algorithmic={flops / launches / algo:.3f}")
    print(f"kernel_time_per_iteration_ms={sum(dur) / launches / 1e6:.3f}")
    print(f"mfma_tflops_issued={flops / sum(dur) / 1e3:.1f}")
    print(f"algorithmic_tflops={algo * launches / sum(dur) / 1e3:.1f}")
    # GRBM_GUI_ACTIVE arrives summed over the XCDs; per XCD it counts the
    # cycles the GPU was busy, which all of its SIMDs share
    print(f"gpu_active_cycles_per_xcd={active / a.xcds:.4e} (over {sum(dur) / 1e6:.2f} ms: "
          f"{active / a.xcds / sum(dur):.2f} GHz)")
    print(f"mfma_busy_percent={100.0 * busy / (active / a.xcds * simds):.1f}")
    print(f"gemm_sources_sha256={gemm_sources_sha256()}")


def cmd_stalls(a):
    """Where the wave cycles of the implicit-GEMM dispatches go, from two counter passes of a
    `bench.py --kernels-only` run: fractions of SQ_WAVE_CYCLES per pass kind, LDS counters, MFMA busy."""
    pa = _counters(a.a, {"SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_WAIT_INST_LDS", "SQ_ACTIVE_INST_LDS",
                         "SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_VMEM", "SQ_ACTIVE_INST_MISC"})
    pb = _counters(a.b, {"SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_DATA_FIFO_FULL", "SQ_VALU_MFMA_BUSY_CYCLES",
                         "GRBM_GUI_ACTIVE"})

    def total(cnt, pred):
        s = {}
        for k, v in cnt.values():
            if pred(k):
                for n, x in v.items():
                    s[n] = s.get(n, 0.0) + x
        return s

    print("# wave-cycle attribution of the implicit-GEMM kernel, vgg16 batch 32")
    print(f"# commands: {a.cmd}")
    print("# fractions of SQ_WAVE_CYCLES: wait_any = s_waitcnt / barrier waits, wait_inst_any = waiting to issue "
          "(the SIMD's MFMA pipe or a dependency), active_* = issuing that instruction type")
    for label, pas in (("all", None), ("forward", "<0,"), ("data gradient", "<1,"), ("filter gradient", "<2,")):
        def pred(n, pas=pas):
            return "igemm_kernel" in n and (pas is None or pas in n.replace(" ", ""))
        x, y = total(pa, pred), total(pb, pred)
        wc = x.get("SQ_WAVE_CYCLES", 0.0) or 1.0
        simd_cycles = y.get("GRBM_GUI_ACTIVE", 0.0) / a.xcds * a.cus * 4
        print(f"{label}: wait_any={x.get('SQ_WAIT_ANY', 0) / wc:.3f} wait_inst_any={x.get('SQ_WAIT_INST_ANY', 0) / wc:.3f} "
              f"wait_inst_lds={x.get('SQ_WAIT_INST_LDS', 0) / wc:.3f} active_lds={x.get('SQ_ACTIVE_INST_LDS', 0) / wc:.3f} "
              f"active_valu={x.get('SQ_ACTIVE_INST_VALU', 0) / wc:.3f} active_vmem={x.get('SQ_ACTIVE_INST_VMEM', 0) / wc:.3f} "
              f"active_misc={x.get('SQ_ACTIVE_INST_MISC', 0) / wc:.3f} "
              f"lds_bank_conflicts_per_lds_inst={y.get('SQ_LDS_BANK_CONFLICT', 0) / max(y.get('SQ_INSTS_LDS', 0), 1):.3f} "
              f"lds_data_fifo_full_per_lds_inst={y.get('SQ_LDS_DATA_FIFO_FULL', 0) / max(y.get('SQ_INSTS_LDS', 0), 1):.3f} "
              f"mfma_busy={y.get('SQ_VALU_MFMA_BUSY_CYCLES', 0) / max(simd_cycles, 1):.3f}")
    print(f"gemm_sources_sha256={gemm_sources_sha256()}")


def cmd_table(a):
    """Calls and per-dispatch durations of the kernels whose names contain one of the patterns."""
    rows = [r for r in csv.DictReader(open(a.stats)) if any(p in r["Name"] for p in a.patterns.split(","))]
    print(f"# rocprofv3 kernel statistics: {a.title}")
    print(f"\nCommand: `{a.cmd}`\n")
    print("| kernel | calls | total ms | avg us | min us | max us |")
    print("|---|---|---|---|---|---|")
    for r in rows:
        print(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
              f"{float(r['AverageNs']) / 1e3:.1f} | {float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} |")


def cmd_hbm(a):
    """HBM GB/s of the bandwidth-bound kernels: calibrated FETCH_SIZE + WRITE_SIZE per dispatch over the
    dispatch's duration from a kernel-trace run of the same command."""
    fetch = _counters(a.fetch, {"FETCH_SIZE"})
    write = _counters(a.write, {"WRITE_SIZE"})
    cal = [v["FETCH_SIZE"] for k, v in fetch.values() if "copy_grad_kernel" in k]
    calw = [v["WRITE_SIZE"] for k, v in write.values() if "copy_grad_kernel" in k]
    known_kib = a.cal_bytes / 1024.0
    sf, sw = known_kib / max(cal), known_kib / max(calw)
    names = [k for k, _ in fetch.values()]
    dur = _trace_durations(a.trace, lambda n: True)
    if [short(k) for k, _ in dur] != [short(k) for k in names] or len(write) != len(fetch):
        raise SystemExit("the counter and trace runs dispatched different kernel sequences")
    agg = {}
    for (k, fv), (_, wv), (_, d) in zip(fetch.values(), write.values(), dur):
        key = short(k)
        if not any(t in key for t in ("relu", "maxpool", "bn_", "colred", "add_kernel", "copy_grad", "gap_",
                                      "concat")):
            continue
        t = agg.setdefault(key, [0, 0.0, 0])
        t[0] += fv["FETCH_SIZE"] * sf * 1024 + wv["WRITE_SIZE"] * sw * 1024
        t[1] += d
        t[2] += 1
    print(f"# HBM traffic of the bandwidth-bound kernels ({a.what_ran})")
    print(f"# commands: {a.cmd}")
    print(f"# calibration: {a.cal_bytes} B copy read as FETCH_SIZE {max(cal):.1f} KiB, WRITE_SIZE {max(calw):.1f} KiB")
    print("")
    print("| kernel | dispatches | HBM bytes (counters) | time (ms) | GB/s | % of 8 TB/s |")
    print("|---|---|---|---|---|---|")
    for key, (b, d, n) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        print(f"| `{key}` | {n} | {b / 1e9:.3f} GB | {d / 1e6:.3f} | {b / d:.0f} | {100 * b / d / 8000:.1f}% |")


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="what", required=True)
    s = sub.add_parser("stats")
    s.add_argument("trace")
    s.add_argument("stats")
    s.add_argument("--steps", type=int, default=10, help="timed DP steps between the two marks")
    s.add_argument("--flops", type=float, default=0.0, help="GFLOP of one iteration's GEMM passes")
    s.add_argument("--top", type=int, default=25)
    s.add_argument("--cmd", default="")
    t = sub.add_parser("traffic")
    t.add_argument("fetch")
    t.add_argument("write")
    t.add_argument("--workload", default="vgg16")
    t.add_argument("--batch", type=int, default=32)
    t.add_argument("--cal-bytes", type=int, default=256 << 20)
    t.add_argument("--cmd", default="")
    m = sub.add_parser("mfma")
    m.add_argument("counters")
    m.add_argument("trace")
    m.add_argument("--workload", default="vgg16")
    m.add_argument("--batch", type=int, default=32)
    m.add_argument("--cus", type=int, default=256)
    m.add_argument("--xcds", type=int, default=8)
    m.add_argument("--cmd", default="")
    tb = sub.add_parser("table")
    tb.add_argument("stats")
    tb.add_argument("--patterns", required=True, help="comma-separated substrings of kernel names")
    tb.add_argument("--title", default="")
    tb.add_argument("--cmd", default="")
    w = sub.add_parser("stalls")
    w.add_argument("a")
    w.add_argument("b")
    w.add_argument("--cus", type=int, default=256)
    w.add_argument("--xcds", type=int, default=8)
    w.add_argument("--cmd", default="")
    h = sub.add_parser("hbm")
    h.add_argument("fetch")
    h.add_argument("write")
    h.add_argument("trace")
    h.add_argument("--cal-bytes", type=int, default=256 << 20)
    h.add_argument("--what-ran", default="")
    h.add_argument("--cmd", default="")
    a = ap.parse_args()
    {"stats": cmd_stats, "traffic": cmd_traffic, "mfma": cmd_mfma, "hbm": cmd_hbm, "stalls": cmd_stalls, "table": cmd_table}[a.what](a)


if __name__ == "__main__":
    main()
