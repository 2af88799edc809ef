"""The parameter server's host thread pool under many short back-to-back jobs (no GPU).

A worker that woke after its job had finished once took an index of the next
job through the finished job's null pointer; the stress driver gives late
wake-ups many chances and checks that every index runs exactly once.
"""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2101_07968_amd", "csrc")


def test_host_pool_stress(tmp_path):
    exe = str(tmp_path / "host_pool_stress")
    r = subprocess.run(["g++", "-O2", "-std=c++17", "-pthread", "-I", CSRC,
                        os.path.join(ROOT, "tests", "host_pool_stress.cpp"), os.path.join(CSRC, "host_pool.cpp"),
                        "-o", exe], capture_output=True, text=True)
    if r.returncode != 0:
        pytest.fail(r.stderr)
    out = subprocess.run([exe, "100000"], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, (out.returncode, out.stdout, out.stderr)
    assert out.stdout.startswith("ok"), out.stdout
