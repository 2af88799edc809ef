"""Host-side logic of the benchmark and of the profile summaries (no GPU).

* bench.py refuses more than one GPU before it touches the device;
* the committed implicit-GEMM counter summaries were taken on the current GEMM
  sources, so the bench's `traffic` field is live, and their algorithmic bytes
  are the sum over VGG-16's passes of every operand read once and the result
  written once, recomputed here from the layer shapes;
* profsum's traffic arithmetic on synthetic counter files: the calibration copy
  scales FETCH_SIZE and WRITE_SIZE, and the bytes are averaged per launch.
"""
import csv
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2101_07968_amd import nets as PN  # noqa: E402
from paper_2101_07968_amd import profsum  # noqa: E402

GEMM_PROFILES = ["igemm_vgg16_b32_traffic.txt", "igemm_vgg16_b32_mfma.txt", "igemm_vgg16_b32_stalls.txt"]


def _kv(path):
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith("#") and ":" not in line.split("=", 1)[0]:
            k, v = line.strip().split("=", 1)
            kv[k.strip()] = v.strip()
    return kv


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stdout + r.stderr


@pytest.mark.parametrize("name", GEMM_PROFILES)
def test_committed_gemm_profiles_are_current(name):
    text = open(os.path.join(ROOT, "profiles", name)).read()
    sha = [ln.split("=", 1)[1].strip() for ln in text.splitlines() if ln.startswith("gemm_sources_sha256=")]
    assert sha == [profsum.gemm_sources_sha256()], name


def test_traffic_figures_and_algorithmic_bytes():
    import bench
    kv = _kv(os.path.join(ROOT, "profiles", "igemm_vgg16_b32_traffic.txt"))
    hbm, algo = bench.traffic_from_profiles("vgg16", 32)
    assert hbm == float(kv["hbm_bytes_per_launch"]) and algo == float(kv["algorithmic_bytes_per_launch"])
    assert abs(hbm / algo - float(kv["hbm_over_algorithmic"])) < 1e-3
    # every operand read once and the result written once, per pass launch
    ops, hwc, _ = PN.build("vgg16")
    total, launches = 0, 0
    for _i, (n, h, w, c, k, r, s, st, pad, pad_w), first in PN.conv_geoms(ops, hwc, 32):
        p, q = (h + 2 * pad - r) // st + 1, (w + 2 * pad_w - s) // st + 1
        x, y, wt = n * h * w * c, n * p * q * k, k * r * s * c
        passes = 2 if first else 3    # the first layer has no data gradient
        total += passes * 4 * (x + y + wt)
        launches += passes
    assert launches == 47
    assert abs(algo - total / launches) < 1.0


def _counter_csv(path, counter, rows):
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        wr.writeheader()
        for i, (kernel, value) in enumerate(rows):
            wr.writerow({"Dispatch_Id": i, "Kernel_Name": kernel, "Counter_Name": counter, "Counter_Value": value})


def test_profsum_traffic_scaling(tmp_path):
    # the 256 MiB calibration copy reads as half its bytes in FETCH_SIZE and all of them in WRITE_SIZE
    cal = ("void dc::copy_grad_kernel(float const*, int, float*, long, long)", None)
    passes = [f"void dc::igemm_kernel<{i % 3}, 128, 128, 16, true, true, true>(dc::Args)" for i in range(94)]
    fetch = [(cal[0], 131072.0)] + [(k, 1000.0 + i) for i, k in enumerate(passes)] + [("void dc::relu_fwd_kernel()", 7e6)]
    write = [(cal[0], 262144.0)] + [(k, 500.0) for k in passes] + [("void dc::relu_fwd_kernel()", 7e6)]
    _counter_csv(tmp_path / "f.csv", "FETCH_SIZE", fetch)
    _counter_csv(tmp_path / "w.csv", "WRITE_SIZE", write)
    r = subprocess.run([sys.executable, "-m", "paper_2101_07968_amd.profsum", "traffic", str(tmp_path / "f.csv"),
                        str(tmp_path / "w.csv"), "--workload", "vgg16", "--batch", "32"], capture_output=True,
                       text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 0, r.stderr
    kv = {}
    for line in r.stdout.splitlines():
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k] = v
    assert float(kv["fetch_scale"]) == pytest.approx(2.0) and float(kv["write_scale"]) == pytest.approx(1.0)
    fetch_kib = sum(1000.0 + i for i in range(94))
    want = (fetch_kib * 2.0 + 94 * 500.0) * 1024.0 / 94
    assert abs(float(kv["hbm_bytes_per_launch"]) - want) <= 1.0
    assert kv["gemm_sources_sha256"] == profsum.gemm_sources_sha256()
