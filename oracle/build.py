"""Build the oracle's C loops into ``oracle/liboracle_cnn.so`` with gcc and OpenMP.

Building the checker is not using it: ``__graft_entry__.build()`` calls this so
that the tests find the library, nothing else links against it.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))


def build(verbose=False):
    src = os.path.join(HERE, "cnn.c")
    out = os.path.join(HERE, "liboracle_cnn.so")
    tmp = out + ".tmp"
    cmd = ["gcc", "-O2", "-march=x86-64-v2", "-fno-fast-math", "-fopenmp", "-shared", "-fPIC",
           "-o", tmp, src]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
