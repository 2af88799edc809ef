// C ABI: error reporting, the planner entry points and the operator entry
// points of dc_kernels.h.
#include "dc_internal.h"

#include <algorithm>
#include <climits>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <vector>

namespace dc {
namespace {
thread_local char g_err[512] = "";
thread_local int g_hip_err = 0;
} // namespace

int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

int hip_fail(hipError_t e, const char *what) {
    g_hip_err = (int)e;
    snprintf(g_err, sizeof(g_err), "%s failed: %s (%d)", what, hipGetErrorString(e), (int)e);
    return DC_EHIP;
}

void clear_error() {
    g_err[0] = 0;
    g_hip_err = 0;
}

} // namespace dc

using namespace dc;

extern "C" const char *dc_strerror(int status) {
    switch (status) {
    case DC_OK: return "ok";
    case DC_EINVAL: return "invalid argument";
    case DC_EHIP: return "HIP runtime error";
    case DC_ENOMEM: return "out of memory";
    case DC_ESTATE: return "call out of order";
    case DC_ETIMEOUT: return "watchdog timeout";
    default: return "unknown status";
    }
}

extern "C" const char *dc_last_error(void) { return g_err; }
extern "C" int dc_last_hip_error(void) { return g_hip_err; }

// ---------------------------------------------------------------- planner

static int check_profile(const dc_profile_t *prof, const dc_plan_t *out) {
    if (!prof || !out)
        return fail(DC_EINVAL, "profile or plan is NULL");
    if (prof->L < 1)
        return fail(DC_EINVAL, "L must be >= 1");
    if (!prof->pt_ns || !prof->fc_ns || !prof->bc_ns || !prof->gt_ns)
        return fail(DC_EINVAL, "profile arrays are NULL");
    if (out->L != prof->L)
        return fail(DC_EINVAL, "plan L=%d differs from profile L=%d", out->L, prof->L);
    if (prof->L > 1 && (!out->p || !out->g))
        return fail(DC_EINVAL, "plan arrays are NULL");
    if (prof->dt_ns < 0)
        return fail(DC_EINVAL, "dt must be >= 0");
    for (int l = 0; l < prof->L; ++l)
        if (prof->pt_ns[l] < 0 || prof->fc_ns[l] < 0 || prof->bc_ns[l] < 0 || prof->gt_ns[l] < 0)
            return fail(DC_EINVAL, "costs must be >= 0");
    return DC_OK;
}

extern "C" int dc_plan(const dc_profile_t *prof, dc_plan_t *out) {
    clear_error();
    DC_TRY(check_profile(prof, out));
    DC_TRY(plan_forward(prof->pt_ns, prof->fc_ns, prof->dt_ns, prof->L, out->p, &out->t_fwd_ns));
    DC_TRY(plan_backward(prof->bc_ns, prof->gt_ns, prof->dt_ns, prof->L, out->g, &out->t_bwd_ns));
    return DC_OK;
}

extern "C" int dc_plan_eval(const dc_profile_t *prof, dc_plan_t *plan) {
    clear_error();
    DC_TRY(check_profile(prof, plan));
    // the dynamic program's overflow bound covers every decision; reuse it
    std::vector<uint8_t> tmp(prof->L > 1 ? prof->L - 1 : 1);
    int64_t t;
    DC_TRY(plan_forward(prof->pt_ns, prof->fc_ns, prof->dt_ns, prof->L, tmp.data(), &t));
    DC_TRY(plan_backward(prof->bc_ns, prof->gt_ns, prof->dt_ns, prof->L, tmp.data(), &t));
    plan->t_fwd_ns = fm_forward(prof->pt_ns, prof->fc_ns, prof->dt_ns, prof->L, plan->p);
    plan->t_bwd_ns = fm_backward(prof->bc_ns, prof->gt_ns, prof->dt_ns, prof->L, plan->g);
    return DC_OK;
}

extern "C" int dc_plan_ibatch(const dc_profile_t *prof, dc_plan_t *out) {
    clear_error();
    DC_TRY(check_profile(prof, out));
    DC_TRY(plan_ibatch_forward(prof->pt_ns, prof->fc_ns, prof->dt_ns, prof->L, out->p));
    DC_TRY(plan_ibatch_backward(prof->bc_ns, prof->gt_ns, prof->dt_ns, prof->L, out->g, &out->t_bwd_ns));
    out->t_fwd_ns = fm_forward(prof->pt_ns, prof->fc_ns, prof->dt_ns, prof->L, out->p);
    return DC_OK;
}

static int fixed_plan(const dc_profile_t *prof, dc_plan_t *out, uint8_t v) {
    clear_error();
    DC_TRY(check_profile(prof, out));
    for (int l = 0; l < prof->L - 1; ++l)
        out->p[l] = out->g[l] = v;
    return dc_plan_eval(prof, out);
}

extern "C" int dc_plan_sequential(const dc_profile_t *prof, dc_plan_t *out) { return fixed_plan(prof, out, 0); }
extern "C" int dc_plan_lbl(const dc_profile_t *prof, dc_plan_t *out) { return fixed_plan(prof, out, 1); }

// ---------------------------------------------------------------- operators

static int conv_setup(const dc_conv_shape *sh, ConvGeom *g) {
    if (!sh)
        return fail(DC_EINVAL, "shape is NULL");
    if (!conv_geom_from_shape(*sh, g))
        return fail(DC_EINVAL, "invalid convolution shape");
    return DC_OK;
}

static int need_ws(size_t need, void *ws, size_t ws_bytes) {
    if (need > 0 && (!ws || ws_bytes < need))
        return fail(DC_EINVAL, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
    if (ws && (uintptr_t)ws % 256 != 0)
        return fail(DC_EINVAL, "workspace must be 256-byte aligned");
    return DC_OK;
}

extern "C" size_t dc_conv2d_workspace_bytes(const dc_conv_shape *sh) {
    ConvGeom g;
    if (!sh || !conv_geom_from_shape(*sh, &g))
        return 0;
    size_t w = 0;
    for (int p = 0; p < 3; ++p)
        w = std::max(w, plan_gemm(g, p).ws_bytes);
    return std::max(w, colsum_ws_bytes((int64_t)g.N * g.P * g.Q, g.K));
}

extern "C" int dc_conv2d_plan_info(const dc_conv_shape *sh, int pass, int32_t *out) {
    clear_error();
    ConvGeom g;
    DC_TRY(conv_setup(sh, &g));
    if (pass < 0 || pass > 2 || !out)
        return fail(DC_EINVAL, "pass must be 0, 1 or 2 and out non-NULL");
    GemmPlan pl = plan_gemm(g, pass);
    const bool own = pl.fc || pl.direct; // kernels outside the implicit GEMM
    const int32_t v[8] = {own ? 0 : pl.mt, own ? 0 : pl.nt, pl.fc ? pl.fc_splits : (pl.direct ? 1 : pl.splits),
                          pl.M, pl.Ng, pl.Kg, pl.phases, pl.source};
    for (int i = 0; i < 8; ++i)
        out[i] = v[i];
    return DC_OK;
}

extern "C" int dc_conv2d_plan_candidates(const dc_conv_shape *sh, int pass, int32_t *out, int cap, int32_t *count) {
    clear_error();
    ConvGeom g;
    DC_TRY(conv_setup(sh, &g));
    if (pass < 0 || pass > 2 || !count || cap < 0 || (cap > 0 && !out))
        return fail(DC_EINVAL, "pass must be 0, 1 or 2, count non-NULL and out non-NULL when cap > 0");
    *count = plan_candidates(g, pass, out, cap);
    return DC_OK;
}

extern "C" int dc_conv2d_set_plan(const dc_conv_shape *sh, int pass, int mt, int nt, int splits) {
    clear_error();
    ConvGeom g;
    DC_TRY(conv_setup(sh, &g));
    if (pass < 0 || pass > 2)
        return fail(DC_EINVAL, "pass must be 0, 1 or 2");
    if (mt == 0 || mt == -1) {
        pin_plan(g, pass, mt, 0, 0);
        return DC_OK;
    }
    const int n = plan_candidates(g, pass, nullptr, 0);
    std::vector<int32_t> c(3 * (size_t)n);
    plan_candidates(g, pass, c.data(), n);
    for (int i = 0; i < n; ++i)
        if (c[3 * i] == mt && c[3 * i + 1] == nt && c[3 * i + 2] == splits) {
            pin_plan(g, pass, mt, nt, splits);
            return DC_OK;
        }
    return fail(DC_EINVAL, "plan (%d, %d, split %d) is not a candidate for this shape and pass", mt, nt, splits);
}

extern "C" int dc_conv2d_forward(const dc_conv_shape *sh, const float *x, const float *w, const float *bias, int relu,
                                 float *y, void *ws, size_t ws_bytes, void *stream) {
    clear_error();
    ConvGeom g;
    DC_TRY(conv_setup(sh, &g));
    if (g.N == 0)
        return DC_OK;
    if (!x || !w || !y)
        return fail(DC_EINVAL, "NULL tensor");
    GemmPlan pl = plan_gemm(g, PASS_FWD);
    DC_TRY(need_ws(pl.ws_bytes, ws, ws_bytes));
    return conv_forward(g, pl, x, w, bias, relu, y, ws, static_cast<hipStream_t>(stream));
}

// ---------------------------------------------------------------- forward conv without allocation
//
// dc_conv2d_forward_noalloc keeps the pass's scratch (split-K partial sums,
// channel-padded operand copies) in this file-scope device array instead of
// a caller workspace.  Each device holds its own copy for the life of the
// process.  In host code `noalloc_scratch` only names the array: its device
// address comes from hipGetSymbolAddress, taken once per device (with that
// device current) at the first call there, and only that address is handed
// to kernels.
namespace {
constexpr size_t NOALLOC_SCRATCH_BYTES = size_t(64) << 20;
constexpr int NOALLOC_MAX_DEVICES = 64;
static __device__ __align__(256) unsigned char noalloc_scratch[NOALLOC_SCRATCH_BYTES];
std::mutex g_noalloc_mu;
void *g_noalloc_ptr[NOALLOC_MAX_DEVICES] = {};

int noalloc_scratch_ptr(void **out) {
    int dev = -1;
    DC_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= NOALLOC_MAX_DEVICES)
        return fail(DC_EINVAL, "device %d is beyond the %d devices the static scratch serves", dev,
                    NOALLOC_MAX_DEVICES);
    std::lock_guard<std::mutex> lock(g_noalloc_mu);
    if (!g_noalloc_ptr[dev]) {
        void *p = nullptr;
        DC_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(noalloc_scratch)));
        if (!p)
            return fail(DC_EHIP, "hipGetSymbolAddress gave no address for the static scratch");
        g_noalloc_ptr[dev] = p;
    }
    *out = g_noalloc_ptr[dev];
    return DC_OK;
}
} // namespace

extern "C" int dc_conv2d_forward_noalloc(const dc_conv_shape *sh, const float *x, const float *w, const float *bias,
                                         int relu, float *y, void *stream) {
    clear_error();
    ConvGeom g;
    DC_TRY(conv_setup(sh, &g));
    if (g.N == 0)
        return DC_OK;
    if (!x || !w || !y)
        return fail(DC_EINVAL, "NULL tensor");
    GemmPlan pl = plan_gemm(g, PASS_FWD);
    if (pl.ws_bytes > NOALLOC_SCRATCH_BYTES)
        return fail(DC_EINVAL, "this shape's forward pass needs %zu bytes of scratch; the static scratch holds %zu",
                    pl.ws_bytes, NOALLOC_SCRATCH_BYTES);
    void *ws = nullptr;
    if (pl.ws_bytes > 0)
        DC_TRY(noalloc_scratch_ptr(&ws));
    return conv_forward(g, pl, x, w, bias, relu, y, ws, static_cast<hipStream_t>(stream));
}

extern "C" int dc_conv2d_backward_data(const dc_conv_shape *sh, const float *dy, const float *w, int accumulate,
                                       float *dx, void *ws, size_t ws_bytes, void *stream) {
    clear_error();
    ConvGeom g;
    DC_TRY(conv_setup(sh, &g));
    if (g.N == 0)
        return DC_OK;
    if (!dy || !w || !dx)
        return fail(DC_EINVAL, "NULL tensor");
    GemmPlan pl = plan_gemm(g, PASS_DGRAD);
    DC_TRY(need_ws(pl.ws_bytes, ws, ws_bytes));
    return conv_dgrad(g, pl, dy, w, accumulate, dx, ws, static_cast<hipStream_t>(stream));
}

extern "C" int dc_conv2d_backward_data_relu(const dc_conv_shape *sh, const float *dy, const float *w,
                                            const float *relu_y, int accumulate, float *dx, void *ws, size_t ws_bytes,
                                            void *stream) {
    clear_error();
    ConvGeom g;
    DC_TRY(conv_setup(sh, &g));
    if (g.N == 0)
        return DC_OK;
    if (!dy || !w || !relu_y || !dx)
        return fail(DC_EINVAL, "NULL tensor");
    GemmPlan pl = plan_gemm(g, PASS_DGRAD);
    DC_TRY(need_ws(pl.ws_bytes, ws, ws_bytes));
    return conv_dgrad(g, pl, dy, w, accumulate, dx, ws, static_cast<hipStream_t>(stream), relu_y);
}

extern "C" int dc_conv2d_backward_filter(const dc_conv_shape *sh, const float *x, const float *dy, float *dw,
                                         float *dbias, void *ws, size_t ws_bytes, void *stream) {
    clear_error();
    ConvGeom g;
    DC_TRY(conv_setup(sh, &g));
    if (!x || !dy || !dw)
        return fail(DC_EINVAL, "NULL tensor");
    hipStream_t s = static_cast<hipStream_t>(stream);
    GemmPlan pl = plan_gemm(g, PASS_WGRAD);
    size_t cs = dbias ? colsum_ws_bytes((int64_t)g.N * g.P * g.Q, g.K) : 0;
    DC_TRY(need_ws(std::max(pl.ws_bytes, cs), ws, ws_bytes));
    if (g.N == 0) {
        DC_HIP(hipMemsetAsync(dw, 0, sizeof(float) * (size_t)g.K * g.R * g.S * g.C, s));
        if (dbias)
            DC_HIP(hipMemsetAsync(dbias, 0, sizeof(float) * g.K, s));
        return DC_OK;
    }
    bool bias_done = false;
    DC_TRY(conv_wgrad(g, pl, x, dy, dw, ws, s, dbias, &bias_done));
    if (dbias && !bias_done)
        DC_TRY(colsum((int64_t)g.N * g.P * g.Q, g.K, dy, dbias, ws, s));
    return DC_OK;
}

extern "C" int dc_relu_forward(const float *x, float *y, int64_t n, void *stream) {
    clear_error();
    if (n < 0 || (n > 0 && (!x || !y)))
        return fail(DC_EINVAL, "bad relu arguments");
    return relu_forward(x, y, n, static_cast<hipStream_t>(stream));
}

extern "C" int dc_relu_backward(const float *dy, const float *y, int accumulate, float *dx, int64_t n, void *stream) {
    clear_error();
    if (n < 0 || (n > 0 && (!dy || !y || !dx)))
        return fail(DC_EINVAL, "bad relu arguments");
    return relu_backward(dy, y, accumulate, dx, n, static_cast<hipStream_t>(stream));
}

static int pool_check(const dc_pool_shape *sh) {
    // r and s are bounded before their product; padded extents in 64 bits
    if (!sh || sh->n < 0 || sh->h < 1 || sh->w < 1 || sh->c < 1 || sh->r < 1 || sh->s < 1 || sh->r > 256 ||
        sh->s > 256 || sh->stride < 1 || sh->pad < 0 || sh->pad >= sh->r || sh->pad >= sh->s ||
        sh->r * sh->s > 256 || (int64_t)sh->h + 2 * sh->pad < sh->r || (int64_t)sh->w + 2 * sh->pad < sh->s ||
        (int64_t)sh->h + 2 * sh->pad >= INT_MAX || (int64_t)sh->w + 2 * sh->pad >= INT_MAX)
        return fail(DC_EINVAL, "invalid pooling shape");
    return DC_OK;
}

extern "C" int dc_maxpool_forward(const dc_pool_shape *sh, const float *x, float *y, uint8_t *arg, void *stream) {
    clear_error();
    DC_TRY(pool_check(sh));
    if (sh->n > 0 && (!x || !y || !arg))
        return fail(DC_EINVAL, "NULL tensor");
    return maxpool_forward(*sh, x, y, arg, static_cast<hipStream_t>(stream));
}

extern "C" int dc_maxpool_backward(const dc_pool_shape *sh, const float *dy, const uint8_t *arg, int accumulate,
                                   float *dx, void *stream) {
    clear_error();
    DC_TRY(pool_check(sh));
    if (sh->n > 0 && (!dy || !arg || !dx))
        return fail(DC_EINVAL, "NULL tensor");
    return maxpool_backward(*sh, dy, arg, accumulate, dx, static_cast<hipStream_t>(stream));
}

extern "C" int dc_maxpool_backward_relu(const dc_pool_shape *sh, const float *dy, const uint8_t *arg,
                                        const float *y, int accumulate, float *dx, void *stream) {
    clear_error();
    DC_TRY(pool_check(sh));
    if (sh->n > 0 && (!dy || !arg || !y || !dx))
        return fail(DC_EINVAL, "NULL tensor");
    return maxpool_backward(*sh, dy, arg, accumulate, dx, static_cast<hipStream_t>(stream), y);
}

extern "C" int dc_avgpool_forward(const dc_pool_shape *sh, const float *x, float *y, void *stream) {
    clear_error();
    DC_TRY(pool_check(sh));
    if (sh->n > 0 && (!x || !y))
        return fail(DC_EINVAL, "NULL tensor");
    return avgpool_forward(*sh, x, y, static_cast<hipStream_t>(stream));
}

extern "C" int dc_avgpool_backward(const dc_pool_shape *sh, const float *dy, int accumulate, float *dx,
                                   void *stream) {
    clear_error();
    DC_TRY(pool_check(sh));
    if (sh->n > 0 && (!dy || !dx))
        return fail(DC_EINVAL, "NULL tensor");
    return avgpool_backward(*sh, dy, accumulate, dx, static_cast<hipStream_t>(stream));
}

extern "C" int dc_gap_forward(int32_t n, int32_t hw, int32_t c, const float *x, float *y, void *stream) {
    clear_error();
    if (n < 0 || hw < 1 || c < 1 || (n > 0 && (!x || !y)))
        return fail(DC_EINVAL, "bad pooling arguments");
    return gap_forward(n, hw, c, x, y, static_cast<hipStream_t>(stream));
}

extern "C" int dc_gap_backward(int32_t n, int32_t hw, int32_t c, const float *dy, int accumulate, float *dx,
                               void *stream) {
    clear_error();
    if (n < 0 || hw < 1 || c < 1 || (n > 0 && (!dy || !dx)))
        return fail(DC_EINVAL, "bad pooling arguments");
    return gap_backward(n, hw, c, dy, accumulate, dx, static_cast<hipStream_t>(stream));
}

extern "C" int dc_add_forward(const float *a, const float *b, int relu, float *y, int64_t n, void *stream) {
    clear_error();
    if (n < 0 || (n > 0 && (!a || !b || !y)))
        return fail(DC_EINVAL, "bad add arguments");
    return add_forward(a, b, relu, y, n, static_cast<hipStream_t>(stream));
}

extern "C" int dc_copy_grad(const float *dy, int accumulate, float *dx, int64_t n, void *stream) {
    clear_error();
    if (n < 0 || (n > 0 && (!dy || !dx)))
        return fail(DC_EINVAL, "bad copy arguments");
    return copy_grad(dy, accumulate, dx, n, static_cast<hipStream_t>(stream));
}

extern "C" int dc_add_relu_backward(const float *dy, const float *y, int acc0, float *dx0, int acc1, float *dx1,
                                    int64_t n, void *stream) {
    clear_error();
    if (n < 0 || (n > 0 && (!dy || !y || (!dx0 && !dx1))))
        return fail(DC_EINVAL, "bad add arguments");
    return add_relu_backward(dy, y, acc0, dx0, acc1, dx1, n, static_cast<hipStream_t>(stream));
}

extern "C" int dc_concat_forward(int64_t rows, int32_t c_in, int32_t c_out, int32_t off, const float *x, float *y,
                                 void *stream) {
    clear_error();
    if (rows < 0 || c_in < 1 || off < 0 || (int64_t)off + c_in > c_out || (rows > 0 && (!x || !y)))
        return fail(DC_EINVAL, "bad concat arguments");
    return concat_forward(rows, c_in, c_out, off, x, y, static_cast<hipStream_t>(stream));
}

extern "C" int dc_concat_backward(int64_t rows, int32_t c_in, int32_t c_out, int32_t off, const float *dy,
                                  int accumulate, float *dx, void *stream) {
    clear_error();
    if (rows < 0 || c_in < 1 || off < 0 || (int64_t)off + c_in > c_out || (rows > 0 && (!dy || !dx)))
        return fail(DC_EINVAL, "bad concat arguments");
    return concat_backward(rows, c_in, c_out, off, dy, accumulate, dx, static_cast<hipStream_t>(stream));
}

extern "C" int dc_concat_backward_relu(int64_t rows, int32_t c_in, int32_t c_out, int32_t off, const float *dy,
                                       const float *relu_y, int accumulate, float *dx, void *stream) {
    clear_error();
    if (rows < 0 || c_in < 1 || off < 0 || (int64_t)off + c_in > c_out || (rows > 0 && (!dy || !relu_y || !dx)))
        return fail(DC_EINVAL, "bad concat arguments");
    return concat_backward(rows, c_in, c_out, off, dy, accumulate, dx, static_cast<hipStream_t>(stream), relu_y);
}

extern "C" size_t dc_batchnorm_workspace_bytes(int64_t rows, int32_t c) {
    return rows > 0 && c > 0 ? bn_ws_bytes(rows, c) : 0;
}

extern "C" int dc_batchnorm_forward(int64_t rows, int32_t c, const float *x, const float *gamma, const float *beta,
                                    float eps, float *y, float *mean, float *invstd, void *ws, size_t ws_bytes,
                                    void *stream) {
    clear_error();
    if (rows < 0 || c < 1 || !(eps >= 0))
        return fail(DC_EINVAL, "bad batchnorm arguments");
    if (rows == 0)
        return DC_OK;
    if (!x || !gamma || !beta || !y || !mean || !invstd)
        return fail(DC_EINVAL, "NULL tensor");
    DC_TRY(need_ws(bn_ws_bytes(rows, c), ws, ws_bytes));
    return bn_forward(rows, c, x, gamma, beta, eps, 0, y, mean, invstd, ws, static_cast<hipStream_t>(stream));
}

extern "C" int dc_batchnorm_backward(int64_t rows, int32_t c, const float *dy, const float *x, const float *gamma,
                                     const float *mean, const float *invstd, int accumulate, float *dx, float *dgamma,
                                     float *dbeta, void *ws, size_t ws_bytes, void *stream) {
    clear_error();
    if (rows < 0 || c < 1)
        return fail(DC_EINVAL, "bad batchnorm arguments");
    if (rows == 0)
        return DC_OK;
    if (!dy || !x || !gamma || !mean || !invstd || !dgamma || !dbeta)
        return fail(DC_EINVAL, "NULL tensor");
    DC_TRY(need_ws(bn_ws_bytes(rows, c), ws, ws_bytes));
    return bn_backward(rows, c, dy, x, gamma, mean, invstd, accumulate, dx, dgamma, dbeta, ws,
                       static_cast<hipStream_t>(stream));
}

extern "C" int dc_batchnorm_backward_relu(int64_t rows, int32_t c, const float *dy, const float *relu_y,
                                          const float *x, const float *gamma, const float *mean, const float *invstd,
                                          int accumulate, float *dx, float *dgamma, float *dbeta, void *ws,
                                          size_t ws_bytes, void *stream) {
    clear_error();
    if (rows < 0 || c < 1)
        return fail(DC_EINVAL, "bad batchnorm arguments");
    if (rows == 0)
        return DC_OK;
    if (!dy || !relu_y || !x || !gamma || !mean || !invstd || !dgamma || !dbeta)
        return fail(DC_EINVAL, "NULL tensor");
    DC_TRY(need_ws(bn_ws_bytes(rows, c), ws, ws_bytes));
    return bn_backward(rows, c, dy, x, gamma, mean, invstd, accumulate, dx, dgamma, dbeta, ws,
                       static_cast<hipStream_t>(stream), relu_y);
}

extern "C" size_t dc_softmax_xent_workspace_bytes(int32_t n) { return xent_ws_bytes(n); }

extern "C" int dc_softmax_xent(int32_t n, int32_t classes, const float *logits, const int32_t *labels, float *loss,
                               float *dlogits, void *ws, size_t ws_bytes, void *stream) {
    clear_error();
    if (n < 0 || classes < 1)
        return fail(DC_EINVAL, "bad loss arguments");
    if (n == 0)
        return DC_OK;
    if (!logits || !labels || !loss || !dlogits)
        return fail(DC_EINVAL, "NULL tensor");
    DC_TRY(need_ws(xent_ws_bytes(n), ws, ws_bytes));
    return softmax_xent(n, classes, logits, labels, loss, dlogits, ws, static_cast<hipStream_t>(stream));
}
