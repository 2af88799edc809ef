// Internal declarations shared by the libdc sources (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "dc.h"
#include "dc_kernels.h"

namespace dc {

// ---------------------------------------------------------------- errors
int fail(int code, const char *fmt, ...);
int hip_fail(hipError_t e, const char *what);
void clear_error();

#define DC_HIP(call)                                  \
    do {                                              \
        hipError_t e_ = (call);                       \
        if (e_ != hipSuccess)                         \
            return ::dc::hip_fail(e_, #call);         \
    } while (0)

#define DC_TRY(call)                                  \
    do {                                              \
        int s_ = (call);                              \
        if (s_ != DC_OK)                              \
            return s_;                                \
    } while (0)

// ---------------------------------------------------------------- conv / GEMM
enum Pass { PASS_FWD = 0, PASS_DGRAD = 1, PASS_WGRAD = 2 };

// Division by a runtime constant d via multiply-high (valid for n < 2^31):
// the round-up method for unsigned division by an invariant integer.
struct FDiv {
    uint32_t d, m, s;
    __host__ __device__ __forceinline__ uint32_t div(uint32_t n) const {
        const uint32_t hi = (uint32_t)(((uint64_t)n * m) >> 32); // the high word of n * m
        return (uint32_t)(((uint64_t)hi + n) >> s);
    }
};

inline __host__ __device__ FDiv make_fdiv(uint32_t d) {
    FDiv f;
    f.d = d;
    if (d <= 1) {
        f.m = 0;
        f.s = 0;
        return f;
    }
    uint32_t l = 32 - __builtin_clz(d - 1);
    uint64_t one = 1;
    f.m = (uint32_t)(((one << 32) * ((one << l) - d)) / d + 1);
    f.s = l;
    return f;
}

struct ConvGeom {
    int N, H, W, C, K, R, S, st, pad, pad_w, P, Q; // pad: rows; pad_w: columns
};

// Launch configuration of one implicit-GEMM pass, chosen on the host.
struct GemmPlan {
    int pass;
    int M, Ng, Kg;        // GEMM sizes (DGRAD: maxima over the stride phases)
    int phases;           // DGRAD: stride^2, otherwise 1
    int mt, nt;           // workgroup tile
    int kt;               // K depth of one LDS stage (16 or 32)
    int tiles_m, tiles_n; // tiles per phase
    int splits;           // split-K factor (1 = no split)
    int kt_per_split;     // K stages (of depth kt) per split
    bool av, bv;          // float4 operand loads possible
    bool tu;              // lean address mode: FWD C % 16 == 0; DGRAD K % 16 == 0, C % 4 == 0; WGRAD K, C % 4 == 0, Q >= 16
    int cpad;             // FWD / WGRAD with C % 4 != 0: padded channel count, else 0
    size_t pad_x_off;     // workspace offsets of the padded x and of the padded w (FWD) or dw (WGRAD)
    size_t pad_w_off;
    size_t ws_bytes;      // split-K partial sums, then the padded copies
    int source;           // PLAN_MODEL, PLAN_TABLE, PLAN_PINNED or PLAN_FC
    // PLAN_FC: the pass (an FC data gradient) runs on the weight-streaming
    // kernel (fc.hip) with fc_splits reduction splits of fc_chunk rows each;
    // the implicit-GEMM fields above still hold the plan used when an operand
    // is not 16-byte aligned, and ws_bytes covers both.
    bool fc;
    int fc_splits, fc_chunk;
    // PLAN_DIRECT: a forward or filter-gradient pass of the RGB input layer
    // runs on the direct kernels (conv3.hip); the fields above still hold the
    // implicit-GEMM plan used when an operand is not 16-byte aligned.
    bool direct;
};

enum PlanSource { PLAN_MODEL = 0, PLAN_TABLE = 1, PLAN_PINNED = 2, PLAN_FC = 3, PLAN_DIRECT = 4 };

bool conv_geom_from_shape(const dc_conv_shape &sh, ConvGeom *g);
GemmPlan plan_gemm(const ConvGeom &g, int pass);
// Every (tile M, tile N, split-K factor) the planner can launch for this pass;
// writes up to cap triples and returns how many there are.
int plan_candidates(const ConvGeom &g, int pass, int32_t *out, int cap);

// Plans chosen by measurement, looked up before the cost model: first a plan
// pinned for this process (pin_plan), then the table built into the library.
// Returns PLAN_PINNED or PLAN_TABLE with (mt, nt, splits) in out, PLAN_MODEL
// when neither holds the shape, or -1 when the shape is pinned to the cost
// model itself.
int lookup_plan(const ConvGeom &g, int pass, int out[3]);
// mt > 0 pins (mt, nt, splits); mt == 0 removes the pin; mt == -1 pins the
// cost model's choice (the built-in table is then skipped for this shape).
void pin_plan(const ConvGeom &g, int pass, int mt, int nt, int splits);

// The data gradient of a large FC layer with at most 32 rows (fc.hip):
// whether the weight-streaming kernel takes the pass, its split of the
// reduction and scratch, and the pass (relu_mask as for conv_dgrad).
// Direct kernels for the RGB input layer (C = 3, a 3 x 3 filter; conv3.hip):
// forward pass and filter gradient, the latter with the bias gradient.
bool conv3_direct(const ConvGeom &g, int pass);
size_t conv3_ws_bytes(const ConvGeom &g, int pass);
int conv3_forward(const ConvGeom &g, const float *x, const float *w, const float *bias, int relu, float *y,
                  hipStream_t s);
int conv3_wgrad(const ConvGeom &g, const float *x, const float *dy, float *dw, float *dbias, void *ws,
                hipStream_t s);
bool fc_streaming(const ConvGeom &g, int pass);
void fc_plan(const ConvGeom &g, int pass, int splits_out[1], int *chunk, size_t *ws_bytes);
int fc_forward(const ConvGeom &g, int splits, int chunk, const float *x, const float *w, const float *bias, int relu,
               float *y, void *ws, hipStream_t s);
int fc_dgrad(const ConvGeom &g, int splits, int chunk, const float *dy, const float *w, int accumulate, float *dx,
             void *ws, hipStream_t s, const float *relu_mask);

int conv_forward(const ConvGeom &g, const GemmPlan &pl, const float *x, const float *w,
                 const float *bias, int relu, float *y, void *ws, hipStream_t s);
// relu_mask, if given, is the output of a ReLU whose input gradient dx is:
// dx (+)= (relu_mask > 0 ? dgrad : 0), laid out like dx.
int conv_dgrad(const ConvGeom &g, const GemmPlan &pl, const float *dy, const float *w,
               int accumulate, float *dx, void *ws, hipStream_t s, const float *relu_mask = nullptr);
// Filter gradient.  When the pass's kernel also forms the bias gradient (the
// direct RGB-layer kernel, given bias_done), it writes dbias (if not NULL)
// and sets *bias_done; otherwise the caller computes the bias gradient.
int conv_wgrad(const ConvGeom &g, const GemmPlan &pl, const float *x, const float *dy, float *dw,
               void *ws, hipStream_t s, float *dbias = nullptr, bool *bias_done = nullptr);

// ---------------------------------------------------------------- elementwise and reductions
size_t colsum_ws_bytes(int64_t rows, int c);
int colsum(int64_t rows, int c, const float *x, float *out, void *ws, hipStream_t s);
size_t bn_ws_bytes(int64_t rows, int c);
int bn_forward(int64_t rows, int c, const float *x, const float *gamma, const float *beta,
               float eps, int relu, float *y, float *mean, float *invstd, void *ws, hipStream_t s);
// relu_y, if given, is the output of a ReLU applied to this BN's output: dy is
// then the ReLU's output gradient and passes through the ReLU's backward
// (kept where relu_y > 0) on the way in, so no separate ReLU pass is needed.
int bn_backward(int64_t rows, int c, const float *dy, const float *x, const float *gamma,
                const float *mean, const float *invstd, int accumulate, float *dx, float *dgamma,
                float *dbeta, void *ws, hipStream_t s, const float *relu_y = nullptr);
int relu_forward(const float *x, float *y, int64_t n, hipStream_t s);
int relu_backward(const float *dy, const float *y, int accumulate, float *dx, int64_t n,
                  hipStream_t s);
int add_forward(const float *a, const float *b, int relu, float *y, int64_t n, hipStream_t s);
int copy_grad(const float *dy, int accumulate, float *dx, int64_t n, hipStream_t s);
// Backward of relu(a + b): dx0 (+)= dx1 (+)= (y > 0 ? dy : 0); a null dx is skipped.
int add_relu_backward(const float *dy, const float *y, int acc0, float *dx0, int acc1, float *dx1, int64_t n,
                      hipStream_t s);
int concat_forward(int64_t rows, int c_in, int c_out, int off, const float *x, float *y, hipStream_t s);
// relu_y, if given (laid out like dx), masks dy: dx is then the gradient of
// the input of a ReLU whose output was this concatenation's input.
int concat_backward(int64_t rows, int c_in, int c_out, int off, const float *dy, int accumulate, float *dx,
                    hipStream_t s, const float *relu_y = nullptr);
int avgpool_forward(const dc_pool_shape &sh, const float *x, float *y, hipStream_t s);
int avgpool_backward(const dc_pool_shape &sh, const float *dy, int accumulate, float *dx, hipStream_t s);
int maxpool_forward(const dc_pool_shape &sh, const float *x, float *y, uint8_t *arg,
                    hipStream_t s);
// relu_y, if given, is the pool's output: dx is then the gradient of the
// input of a ReLU whose output the pool read, masked by that ReLU.
int maxpool_backward(const dc_pool_shape &sh, const float *dy, const uint8_t *arg, int accumulate,
                     float *dx, hipStream_t s, const float *relu_y = nullptr);
int gap_forward(int n, int hw, int c, const float *x, float *y, hipStream_t s);
int gap_backward(int n, int hw, int c, const float *dy, int accumulate, float *dx, hipStream_t s);
size_t xent_ws_bytes(int n);
int softmax_xent(int n, int classes, const float *logits, const int32_t *labels, float *loss,
                 float *dlogits, void *ws, hipStream_t s);

// ---------------------------------------------------------------- link pacing
// Write the device wall clock into *slot.
int pace_mark(uint64_t *slot, hipStream_t s);
// Spin until the wall clock reaches *slot + ticks (never longer than cap_ticks).
int pace_until(const uint64_t *slot, uint64_t ticks, uint64_t cap_ticks, hipStream_t s);
// Wall-clock ticks per second of the current device.
int wall_clock_hz(double *hz);

// ---------------------------------------------------------------- planner (host)
int plan_forward(const int64_t *pt, const int64_t *fc, int64_t dt, int L, uint8_t *p,
                 int64_t *t_fwd);
int plan_backward(const int64_t *bc, const int64_t *gt, int64_t dt, int L, uint8_t *g,
                  int64_t *t_bwd);
int plan_ibatch_forward(const int64_t *pt, const int64_t *fc, int64_t dt, int L, uint8_t *p);
int plan_ibatch_backward(const int64_t *bc, const int64_t *gt, int64_t dt, int L, uint8_t *g, int64_t *t_bwd);
int64_t fm_forward(const int64_t *pt, const int64_t *fc, int64_t dt, int L, const uint8_t *p);
int64_t fm_backward(const int64_t *bc, const int64_t *gt, int64_t dt, int L, const uint8_t *g);

} // namespace dc
