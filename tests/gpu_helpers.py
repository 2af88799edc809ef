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


def update_err(p_new, p_old, want):
    """How far the applied update p_new - p_old is from want, relative to max |want|.

    p_new is the server's float32 weight after the step, which holds w - lr g rounded
    to float32: half an ulp of each new weight is storage rounding that no accuracy of
    g removes (for a BN gamma near 1 updated by ~1e-5 it is ~5e-3 of the update), so
    each element's distance is taken less that half ulp."""
    p_new = np.asarray(p_new, dtype=np.float32)
    upd = p_new.astype(np.float64) - np.asarray(p_old, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    if not want.size:
        return 0.0
    excess = np.maximum(np.abs(upd - want) - np.spacing(np.abs(p_new)).astype(np.float64) / 2, 0.0)
    den = np.abs(want).max()
    if den == 0:
        return 0.0 if excess.max() == 0 else np.inf
    return excess.max() / den


def stream():
    return torch().cuda.current_stream().cuda_stream


# Lines the GPU tests want in the session's output whether they pass or not
# (tests/conftest.py prints them in the terminal summary).
SUMMARY = []


def report(line):
    print(line, flush=True)
    SUMMARY.append(line)
