"""ctypes binding of libdc (include/dc.h, include/dc_kernels.h).

Argument marshalling only: every function here converts Python / torch
arguments into the C structs and raw pointers of the C ABI and calls the
function of the same name.  No computation happens in Python.  If libdc.so
is missing the import of any entry point raises immediately; there is no
fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdc.so")

DC_OK, DC_EINVAL, DC_EHIP, DC_ENOMEM, DC_ESTATE, DC_ETIMEOUT = range(6)
DC_OP_CONV, DC_OP_FC, DC_OP_BN, DC_OP_RELU, DC_OP_MAXPOOL, DC_OP_GAP, DC_OP_ADD, DC_OP_CONCAT, DC_OP_AVGPOOL = range(1, 10)
DC_OPT_LR, DC_OPT_TIMELINE, DC_OPT_TIMEOUT_S, DC_OPT_SGD_THREADS, DC_OPT_GRAPHS, DC_OPT_GEMM_TIMING = range(1, 7)
DC_READ_ACT, DC_READ_ARGMAX = 0, 1

c_i32, c_i64, c_f32, c_f64, c_sz, c_vp = (ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double,
                                          ctypes.c_size_t, ctypes.c_void_p)


class DcError(RuntimeError):
    def __init__(self, status, func, msg):
        super().__init__(f"{func} failed: {msg} (status {status})")
        self.status = status


class OpDesc(ctypes.Structure):
    """dc_op_desc; pad_w defaults to pad (square padding) when not given."""
    _fields_ = [("kind", c_i32), ("layer", c_i32), ("in0", c_i32), ("in1", c_i32), ("out_ch", c_i32),
                ("r", c_i32), ("s", c_i32), ("stride", c_i32), ("pad", c_i32), ("bias", c_i32),
                ("in2", c_i32), ("in3", c_i32), ("pad_w", c_i32)]

    def __init__(self, *args, **kw):
        super().__init__(*args, **kw)
        if len(args) < 13 and "pad_w" not in kw:
            self.pad_w = self.pad


class ConvShape(ctypes.Structure):
    """dc_conv_shape; pad_w defaults to pad (square padding) when not given."""
    _fields_ = [(n, c_i32) for n in ("n", "h", "w", "c", "k", "r", "s", "stride", "pad", "pad_w")]

    def __init__(self, *args, **kw):
        super().__init__(*args, **kw)
        if len(args) < 10 and "pad_w" not in kw:
            self.pad_w = self.pad


class PoolShape(ctypes.Structure):
    _fields_ = [(n, c_i32) for n in ("n", "h", "w", "c", "r", "s", "stride", "pad")]


class Link(ctypes.Structure):
    _fields_ = [("bytes_per_s", c_f64), ("dt_emul_ns", c_i64), ("paced", c_i32)]


class Batch(ctypes.Structure):
    _fields_ = [("x_dev", c_vp), ("y_dev", c_vp), ("n", c_i32)]


class GradContrib(ctypes.Structure):
    _fields_ = [(n, c_i32) for n in ("tensor", "origin_op", "exec_op", "accumulate", "fused")]


class ProfileT(ctypes.Structure):
    _fields_ = [("L", c_i32), ("pt_ns", ctypes.POINTER(c_i64)), ("fc_ns", ctypes.POINTER(c_i64)),
                ("bc_ns", ctypes.POINTER(c_i64)), ("gt_ns", ctypes.POINTER(c_i64)), ("dt_ns", c_i64)]


class PlanT(ctypes.Structure):
    _fields_ = [("L", c_i32), ("p", ctypes.POINTER(ctypes.c_uint8)), ("g", ctypes.POINTER(ctypes.c_uint8)),
                ("t_fwd_ns", c_i64), ("t_bwd_ns", c_i64)]


class StepStats(ctypes.Structure):
    _fields_ = [("loss", c_f32), ("n_pull", c_i32), ("n_push", c_i32), ("t_iter_ns", c_i64), ("t_fwd_ns", c_i64),
                ("t_bwd_ns", c_i64), ("t_compute_ns", c_i64), ("t_link_ns", c_i64), ("t_sgd_tail_ns", c_i64),
                ("t_host_ns", c_i64), ("t_plan_bwd_ns", c_i64), ("t_plan_fwd_ns", c_i64), ("plan_hidden", c_i32),
                ("n_gemm", c_i32), ("t_gemm_ns", c_i64), ("gemm_flop", c_f64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


_P = ctypes.POINTER
_SIGS = {
    "dc_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "dc_last_error": (ctypes.c_char_p, []),
    "dc_last_hip_error": (ctypes.c_int, []),
    "dc_model_create": (ctypes.c_int, [_P(OpDesc), ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_int, _P(c_vp)]),
    "dc_model_destroy": (None, [c_vp]),
    "dc_backward_schedule": (ctypes.c_int, [_P(OpDesc), ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                            ctypes.c_int, ctypes.c_int, _P(GradContrib), ctypes.c_int, _P(c_i32)]),
    "dc_model_num_layers": (ctypes.c_int, [c_vp]),
    "dc_model_num_params": (c_sz, [c_vp]),
    "dc_workspace_bytes": (c_sz, [c_vp]),
    "dc_model_bind_workspace": (ctypes.c_int, [c_vp, c_vp, c_sz]),
    "dc_layer_range": (ctypes.c_int, [c_vp, ctypes.c_int, _P(c_sz), _P(c_sz)]),
    "dc_model_set_option": (ctypes.c_int, [c_vp, ctypes.c_int, c_f64]),
    "dc_ps_write": (ctypes.c_int, [c_vp, c_vp, c_sz]),
    "dc_ps_read": (ctypes.c_int, [c_vp, c_vp, c_vp, c_sz]),
    "dc_model_read_tensor": (ctypes.c_int, [c_vp, ctypes.c_int, ctypes.c_int, c_vp, c_sz]),
    "dc_profile": (ctypes.c_int, [c_vp, _P(Batch), _P(Link), ctypes.c_int, c_vp, _P(ProfileT)]),
    "dc_plan": (ctypes.c_int, [_P(ProfileT), _P(PlanT)]),
    "dc_plan_sequential": (ctypes.c_int, [_P(ProfileT), _P(PlanT)]),
    "dc_plan_lbl": (ctypes.c_int, [_P(ProfileT), _P(PlanT)]),
    "dc_plan_eval": (ctypes.c_int, [_P(ProfileT), _P(PlanT)]),
    "dc_plan_ibatch": (ctypes.c_int, [_P(ProfileT), _P(PlanT)]),
    "dc_step": (ctypes.c_int, [c_vp, _P(Batch), _P(PlanT), _P(Link), c_vp, _P(StepStats)]),
    "dc_step_dynamic": (ctypes.c_int, [c_vp, _P(Batch), _P(ProfileT), _P(Link), c_vp, _P(PlanT), _P(StepStats)]),
    "dc_timeline": (ctypes.c_int, [c_vp, _P(c_i64), ctypes.c_int]),
    "dc_conv2d_workspace_bytes": (c_sz, [_P(ConvShape)]),
    "dc_conv2d_plan_info": (ctypes.c_int, [_P(ConvShape), ctypes.c_int, _P(c_i32)]),
    "dc_conv2d_plan_candidates": (ctypes.c_int, [_P(ConvShape), ctypes.c_int, _P(c_i32), ctypes.c_int, _P(c_i32)]),
    "dc_conv2d_set_plan": (ctypes.c_int, [_P(ConvShape), ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "dc_conv2d_forward": (ctypes.c_int, [_P(ConvShape), c_vp, c_vp, c_vp, ctypes.c_int, c_vp, c_vp, c_sz, c_vp]),
    "dc_conv2d_backward_data": (ctypes.c_int, [_P(ConvShape), c_vp, c_vp, ctypes.c_int, c_vp, c_vp, c_sz, c_vp]),
    "dc_conv2d_forward_noalloc": (ctypes.c_int, [_P(ConvShape), c_vp, c_vp, c_vp, ctypes.c_int, c_vp, c_vp]),
    "dc_conv2d_backward_data_relu": (ctypes.c_int, [_P(ConvShape), c_vp, c_vp, c_vp, ctypes.c_int, c_vp, c_vp,
                                                    c_sz, c_vp]),
    "dc_conv2d_backward_filter": (ctypes.c_int, [_P(ConvShape), c_vp, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]),
    "dc_relu_forward": (ctypes.c_int, [c_vp, c_vp, c_i64, c_vp]),
    "dc_relu_backward": (ctypes.c_int, [c_vp, c_vp, ctypes.c_int, c_vp, c_i64, c_vp]),
    "dc_maxpool_forward": (ctypes.c_int, [_P(PoolShape), c_vp, c_vp, c_vp, c_vp]),
    "dc_maxpool_backward": (ctypes.c_int, [_P(PoolShape), c_vp, c_vp, ctypes.c_int, c_vp, c_vp]),
    "dc_maxpool_backward_relu": (ctypes.c_int, [_P(PoolShape), c_vp, c_vp, c_vp, ctypes.c_int, c_vp, c_vp]),
    "dc_avgpool_forward": (ctypes.c_int, [_P(PoolShape), c_vp, c_vp, c_vp]),
    "dc_avgpool_backward": (ctypes.c_int, [_P(PoolShape), c_vp, ctypes.c_int, c_vp, c_vp]),
    "dc_gap_forward": (ctypes.c_int, [c_i32, c_i32, c_i32, c_vp, c_vp, c_vp]),
    "dc_gap_backward": (ctypes.c_int, [c_i32, c_i32, c_i32, c_vp, ctypes.c_int, c_vp, c_vp]),
    "dc_add_forward": (ctypes.c_int, [c_vp, c_vp, ctypes.c_int, c_vp, c_i64, c_vp]),
    "dc_copy_grad": (ctypes.c_int, [c_vp, ctypes.c_int, c_vp, c_i64, c_vp]),
    "dc_add_relu_backward": (ctypes.c_int, [c_vp, c_vp, ctypes.c_int, c_vp, ctypes.c_int, c_vp, c_i64, c_vp]),
    "dc_concat_forward": (ctypes.c_int, [c_i64, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp]),
    "dc_concat_backward": (ctypes.c_int, [c_i64, c_i32, c_i32, c_i32, c_vp, ctypes.c_int, c_vp, c_vp]),
    "dc_concat_backward_relu": (ctypes.c_int, [c_i64, c_i32, c_i32, c_i32, c_vp, c_vp, ctypes.c_int, c_vp, c_vp]),
    "dc_batchnorm_workspace_bytes": (c_sz, [c_i64, c_i32]),
    "dc_batchnorm_forward": (ctypes.c_int, [c_i64, c_i32, c_vp, c_vp, c_vp, c_f32, c_vp, c_vp, c_vp, c_vp, c_sz,
                                            c_vp]),
    "dc_batchnorm_backward": (ctypes.c_int, [c_i64, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, ctypes.c_int, c_vp, c_vp,
                                             c_vp, c_vp, c_sz, c_vp]),
    "dc_batchnorm_backward_relu": (ctypes.c_int, [c_i64, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, ctypes.c_int,
                                                  c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]),
    "dc_softmax_xent_workspace_bytes": (c_sz, [c_i32]),
    "dc_softmax_xent": (ctypes.c_int, [c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]),
}

_lib = None


def lib():
    """The loaded libdc.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        # torch ships its own HIP runtime with the same soname; loading torch
        # first makes libdc bind to that copy, so the process has one runtime
        # and torch's device pointers and streams are valid here.
        import torch  # noqa: F401
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libdc.so is not built ({LIB_PATH}); run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(status, func):
    if status != DC_OK:
        msg = lib().dc_last_error().decode(errors="replace")
        raise DcError(status, func, msg or lib().dc_strerror(status).decode())


def ptr(t):
    """Raw address of a torch tensor / numpy array / int / None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def stream_ptr(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def call(name, *args):
    check(getattr(lib(), name)(*args), name)


# ---------------------------------------------------------------- planner

class Profile:
    """Cost vectors pt, fc, bc, gt (int64 ns) and dt, laid out for dc_profile_t."""

    def __init__(self, pt, fc, bc, gt, dt):
        self.pt, self.fc, self.bc, self.gt = (np.ascontiguousarray(v, dtype=np.int64) for v in (pt, fc, bc, gt))
        self.dt = int(dt)
        self.L = len(self.pt)

    @classmethod
    def empty(cls, L):
        z = np.zeros(L, dtype=np.int64)
        return cls(z, z.copy(), z.copy(), z.copy(), 0)

    def c(self):
        P = ctypes.POINTER(c_i64)
        return ProfileT(self.L, self.pt.ctypes.data_as(P), self.fc.ctypes.data_as(P), self.bc.ctypes.data_as(P),
                        self.gt.ctypes.data_as(P), self.dt)

    def as_dict(self):
        return {"pt": self.pt.tolist(), "fc": self.fc.tolist(), "bc": self.bc.tolist(), "gt": self.gt.tolist(),
                "dt": self.dt}


class Plan:
    """Decision vectors p and g (uint8, length L-1) with the model times of dc_plan_t."""

    def __init__(self, L, p=None, g=None):
        self.L = L
        n = max(L - 1, 1)
        self.p = np.zeros(n, dtype=np.uint8) if p is None else np.ascontiguousarray(p, dtype=np.uint8)
        self.g = np.zeros(n, dtype=np.uint8) if g is None else np.ascontiguousarray(g, dtype=np.uint8)
        self.t_fwd_ns = 0
        self.t_bwd_ns = 0
        self._c = None

    def c(self):
        U = ctypes.POINTER(ctypes.c_uint8)
        self._c = PlanT(self.L, self.p.ctypes.data_as(U), self.g.ctypes.data_as(U), self.t_fwd_ns, self.t_bwd_ns)
        return self._c

    def _sync(self):
        self.t_fwd_ns, self.t_bwd_ns = self._c.t_fwd_ns, self._c.t_bwd_ns
        return self

    def decisions(self):
        return self.p[:self.L - 1].tolist(), self.g[:self.L - 1].tolist()


def _run_plan(name, prof, plan):
    pc = prof.c()
    c = plan.c()
    call(name, ctypes.byref(pc), ctypes.byref(c))
    return plan._sync()


def dc_plan(prof):
    return _run_plan("dc_plan", prof, Plan(prof.L))


def dc_plan_sequential(prof):
    return _run_plan("dc_plan_sequential", prof, Plan(prof.L))


def dc_plan_lbl(prof):
    return _run_plan("dc_plan_lbl", prof, Plan(prof.L))


def dc_plan_ibatch(prof):
    return _run_plan("dc_plan_ibatch", prof, Plan(prof.L))


def dc_plan_eval(prof, p, g):
    return _run_plan("dc_plan_eval", prof, Plan(prof.L, p, g))


# ---------------------------------------------------------------- model

def conv_plan_info(shape, pas):
    """(tile M, tile N, splits, GEMM M, GEMM N, GEMM K, phases, source) of one conv pass;
    source 0 = cost model, 1 = table of measured plans, 2 = pinned, 3 = the weight-streaming
    FC data-gradient kernel (tiles 0, splits = its reduction splits), 4 = the direct kernels of
    the RGB input layer (tiles 0, split 1)."""
    out = (c_i32 * 8)()
    sh = ConvShape(*shape)
    call("dc_conv2d_plan_info", ctypes.byref(sh), pas, out)
    return tuple(out)


def conv_plan_candidates(shape, pas):
    """Every (tile M, tile N, splits) the pass can be launched with for this shape."""
    sh = ConvShape(*shape)
    n = c_i32()
    call("dc_conv2d_plan_candidates", ctypes.byref(sh), pas, None, 0, ctypes.byref(n))
    out = (c_i32 * (3 * n.value))()
    call("dc_conv2d_plan_candidates", ctypes.byref(sh), pas, out, n.value, ctypes.byref(n))
    return [tuple(out[3 * i:3 * i + 3]) for i in range(n.value)]


def conv_set_plan(shape, pas, mt, nt=0, splits=0):
    """Pin a pass's plan for this process (mt = 0 unpins, mt = -1 pins the cost model's choice)."""
    sh = ConvShape(*shape)
    call("dc_conv2d_set_plan", ctypes.byref(sh), pas, mt, nt, splits)


def backward_schedule(ops, batch, hwc, classes):
    """dc_backward_schedule: the backward pass's gradient contributions in launch order, as
    dicts with keys tensor, origin_op, exec_op, accumulate, fused."""
    arr = (OpDesc * len(ops))(*[OpDesc(*o) for o in ops])
    n = c_i32()
    st = lib().dc_backward_schedule(arr, len(ops), batch, hwc[0], hwc[1], hwc[2], classes, None, 0, ctypes.byref(n))
    if st != DC_OK and n.value == 0:
        check(st, "dc_backward_schedule")
    out = (GradContrib * max(n.value, 1))()
    call("dc_backward_schedule", arr, len(ops), batch, hwc[0], hwc[1], hwc[2], classes, out, n.value,
         ctypes.byref(n))
    return [{k: getattr(out[i], k) for k, _ in GradContrib._fields_} for i in range(n.value)]


def link(bytes_per_s=1e9, dt_emul_ns=0, paced=True):
    return Link(float(bytes_per_s), int(dt_emul_ns), 1 if paced else 0)


class Model:
    """A dc_model handle bound to a torch-allocated device workspace."""

    def __init__(self, ops, batch, hwc, classes, device=None):
        import torch
        arr = (OpDesc * len(ops))(*[OpDesc(*o) for o in ops])
        h = c_vp()
        call("dc_model_create", arr, len(ops), batch, hwc[0], hwc[1], hwc[2], classes, ctypes.byref(h))
        self.h = h
        self.batch, self.hwc, self.classes = batch, tuple(hwc), classes
        self.L = lib().dc_model_num_layers(h)
        self.n_params = lib().dc_model_num_params(h)
        nbytes = lib().dc_workspace_bytes(h)
        self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=device or "cuda")
        base = self.workspace.data_ptr()
        aligned = (base + 255) // 256 * 256
        call("dc_model_bind_workspace", h, aligned, nbytes)

    def close(self):
        if self.h:
            lib().dc_model_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def layer_range(self, l):
        off, cnt = c_sz(), c_sz()
        call("dc_layer_range", self.h, l, ctypes.byref(off), ctypes.byref(cnt))
        return off.value, cnt.value

    def layer_bytes(self):
        return [4 * self.layer_range(l)[1] for l in range(1, self.L + 1)]

    def set_option(self, opt, value):
        call("dc_model_set_option", self.h, opt, float(value))

    def ps_write(self, params):
        a = np.ascontiguousarray(params, dtype=np.float32)
        call("dc_ps_write", self.h, a.ctypes.data, a.size)

    def ps_read(self):
        p = np.empty(self.n_params, dtype=np.float32)
        g = np.empty(self.n_params, dtype=np.float32)
        call("dc_ps_read", self.h, p.ctypes.data, g.ctypes.data, self.n_params)
        return p, g

    def read_tensor(self, tensor, shape, what=0):
        """dc_model_read_tensor: tensor `tensor` of the last step (NHWC `shape`) as a float32 array
        (what = DC_READ_ACT) or the max-pool window taps as a uint8 array (DC_READ_ARGMAX)."""
        out = np.empty(shape, dtype=np.float32 if what == DC_READ_ACT else np.uint8)
        call("dc_model_read_tensor", self.h, tensor, what, out.ctypes.data, out.nbytes)
        return out

    def _batch(self, x, y):
        """dc_batch of a float32 NHWC input and int32 labels, both contiguous device tensors."""
        import torch
        h, w, c = self.hwc
        for t, dt, n, name in ((x, torch.float32, self.batch * h * w * c, "x"), (y, torch.int32, self.batch, "y")):
            if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == dt and t.is_contiguous()
                    and t.numel() == n):
                raise DcError(DC_EINVAL, "dc_batch", f"{name} must be a contiguous {dt} device tensor of {n} "
                              f"elements (batch {self.batch}, input {h}x{w}x{c})")
        return Batch(ptr(x), ptr(y), int(x.shape[0]))

    def profile(self, x, y, lnk, reps=3, stream=None):
        prof = Profile.empty(self.L)
        pc = prof.c()
        b = self._batch(x, y)
        call("dc_profile", self.h, ctypes.byref(b), ctypes.byref(lnk), reps, stream_ptr(stream), ctypes.byref(pc))
        prof.dt = pc.dt_ns
        return prof

    def step(self, x, y, plan, lnk, stream=None):
        st = StepStats()
        b = self._batch(x, y)
        c = plan.c()
        call("dc_step", self.h, ctypes.byref(b), ctypes.byref(c), ctypes.byref(lnk), stream_ptr(stream),
             ctypes.byref(st))
        return st.as_dict()

    def step_dynamic(self, x, y, prof, plan, lnk, stream=None):
        """dc_step_dynamic: uses plan.p, fills plan.g (used) and plan.p (next call)."""
        st = StepStats()
        b = self._batch(x, y)
        pc = prof.c()
        c = plan.c()
        call("dc_step_dynamic", self.h, ctypes.byref(b), ctypes.byref(pc), ctypes.byref(lnk), stream_ptr(stream),
             ctypes.byref(c), ctypes.byref(st))
        plan._sync()
        return st.as_dict()

    def timeline(self):
        out = np.zeros(8 * self.L, dtype=np.int64)
        call("dc_timeline", self.h, out.ctypes.data_as(ctypes.POINTER(c_i64)), out.size)
        return out.reshape(self.L, 8)
