"""Helpers shared by the GPU tests: device buffers, scratch, error metrics."""
import numpy as np


def torch():
    import torch as t
    return t


def dev(a):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(a)).cuda()


def zeros(shape, dtype="float32"):
    t = torch()
    return t.zeros(shape, dtype=getattr(t, dtype), device="cuda")


def scratch(nbytes):
    """A 256-byte aligned device scratch buffer: returns (tensor, address, size)."""
    t = torch()
    nbytes = max(int(nbytes), 256)
    buf = t.empty(nbytes + 256, dtype=t.uint8, device="cuda")
    base = buf.data_ptr()
    return buf, (base + 255) // 256 * 256, nbytes


def host(t):
    torch().cuda.synchronize()
    return t.detach().cpu().numpy()


def rel_err(x, ref):
    """max |x - ref| / max |ref| (per tensor), with 0/0 = 0."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.abs(ref).max() if ref.size else 0.0
    num = np.abs(x - ref).max() if ref.size else 0.0
    if den == 0:
        return 0.0 if num == 0 else np.inf
    return num / den


def stream():
    return torch().cuda.current_stream().cuda_stream


# Lines the GPU tests want in the session's output whether they pass or not
# (tests/conftest.py prints them in the terminal summary).
SUMMARY = []


def report(line):
    print(line, flush=True)
    SUMMARY.append(line)
