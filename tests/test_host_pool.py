"""Host code under stress and under the sanitizers (no GPU).

* The parameter server's thread pool under many short back-to-back jobs: a
  worker that woke after its job had finished once took an index of the next
  job through the finished job's null pointer; the stress driver gives late
  wake-ups many chances and checks that every index runs exactly once.  Run
  plain, under ThreadSanitizer, and under AddressSanitizer + UBSan.
* The planner (both DPs, iBatch, f_m) on random profiles up to L = 300 and
  near-overflow magnitudes under AddressSanitizer + UBSan.
* The multiply-high division the kernels index with, against plain division.
"""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2101_07968_amd", "csrc")


SANITIZERS = {"plain": [], "thread": ["-fsanitize=thread"],
              "address+undefined": ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined"]}


@pytest.mark.parametrize("san", list(SANITIZERS))
def test_host_pool_stress(tmp_path, san):
    exe = str(tmp_path / "host_pool_stress")
    r = subprocess.run(["g++", "-O1" if san != "plain" else "-O2", "-g", "-std=c++17", "-pthread", "-I", CSRC]
                       + SANITIZERS[san] + [os.path.join(ROOT, "tests", "host_pool_stress.cpp"),
                                            os.path.join(CSRC, "host_pool.cpp"), "-o", exe],
                       capture_output=True, text=True)
    if r.returncode != 0:
        pytest.fail(r.stderr)
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1", ASAN_OPTIONS="halt_on_error=1")
    out = subprocess.run([exe, "20000" if san != "plain" else "100000"], capture_output=True, text=True,
                         timeout=300, env=env)
    assert out.returncode == 0, (out.returncode, out.stdout, out.stderr[-3000:])
    assert out.stdout.startswith("ok"), out.stdout


def test_planner_under_sanitizers(tmp_path):
    exe = str(tmp_path / "planner_sanitize")
    r = subprocess.run(["g++", "-O1", "-g", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
                        "-I", os.path.join(ROOT, "include"), "-I", CSRC,
                        "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                        os.path.join(ROOT, "tests", "planner_sanitize.cpp"), os.path.join(CSRC, "planner.cpp"),
                        "-o", exe], capture_output=True, text=True)
    if r.returncode != 0:
        pytest.fail(r.stderr)
    out = subprocess.run([exe, "3000"], capture_output=True, text=True, timeout=300,
                         env=dict(os.environ, ASAN_OPTIONS="halt_on_error=1"))
    assert out.returncode == 0, (out.returncode, out.stdout, out.stderr[-3000:])
    assert out.stdout.startswith("ok"), out.stdout


def test_multiply_high_division(tmp_path):
    """dc::FDiv, the division by an invariant integer behind the kernels' index
    arithmetic, equals n / d for n < 2^31 (under UBSan)."""
    exe = str(tmp_path / "fdiv_check")
    r = subprocess.run(["g++", "-O1", "-g", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
                        "-I", os.path.join(ROOT, "include"), "-I", CSRC,
                        "-fsanitize=undefined", "-fno-sanitize-recover=undefined",
                        os.path.join(ROOT, "tests", "fdiv_check.cpp"), "-o", exe], capture_output=True, text=True)
    if r.returncode != 0:
        pytest.fail(r.stderr)
    out = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, (out.returncode, out.stdout, out.stderr[-3000:])
    assert out.stdout.startswith("ok"), out.stdout
