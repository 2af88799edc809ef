// Bandwidth-bound kernels of the forward and backward mini-procedures:
// ReLU, residual add, max-pooling, global average pooling, BatchNorm,
// per-channel sums (bias gradients) and the softmax cross-entropy loss.
//
// Activations are NHWC, so a channel is the fastest index: threads of a wave
// walk consecutive channels and every global access is coalesced.  Per-channel
// reductions over n*h*w rows are two-stage and deterministic: workgroups of a
// fixed row partition write partial sums to fixed slots, a second kernel adds
// them in a fixed tree order in double precision.  Nothing uses atomics, so
// results are bit-identical from run to run.
#include "dc_internal.h"

#include <algorithm>
#include <climits>
#include <cstdint>
#include <numeric>
#include <type_traits>

namespace dc {
namespace {

constexpr int EW_THREADS = 256;

inline int ew_blocks(int64_t n, int per_thread = 1) {
    int64_t b = (n / per_thread + EW_THREADS - 1) / EW_THREADS;
    return (int)std::max<int64_t>(1, std::min<int64_t>(b, 1 << 20));
}

// ---------------------------------------------------------------- elementwise

__global__ void relu_fwd_kernel(const float *__restrict__ x, float *__restrict__ y, int64_t n, int64_t n4) {
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    float4 *y4 = reinterpret_cast<float4 *>(y);
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x) {
        float4 v = x4[i];
        v.x = fmaxf(v.x, 0.f); v.y = fmaxf(v.y, 0.f); v.z = fmaxf(v.z, 0.f); v.w = fmaxf(v.w, 0.f);
        y4[i] = v;
    }
    for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        y[i] = fmaxf(x[i], 0.f);
}

__device__ __forceinline__ float relu_grad(float dy, float y) { return y > 0.f ? dy : 0.f; }

__global__ void relu_bwd_kernel(const float *__restrict__ dy, const float *__restrict__ y, int acc,
                                float *__restrict__ dx, int64_t n, int64_t n4) {
    const float4 *d4 = reinterpret_cast<const float4 *>(dy);
    const float4 *y4 = reinterpret_cast<const float4 *>(y);
    float4 *o4 = reinterpret_cast<float4 *>(dx);
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x) {
        float4 d = d4[i], v = y4[i], o;
        o.x = relu_grad(d.x, v.x); o.y = relu_grad(d.y, v.y); o.z = relu_grad(d.z, v.z); o.w = relu_grad(d.w, v.w);
        if (acc) {
            float4 p = o4[i];
            o.x += p.x; o.y += p.y; o.z += p.z; o.w += p.w;
        }
        o4[i] = o;
    }
    for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        float o = relu_grad(dy[i], y[i]);
        dx[i] = acc ? dx[i] + o : o;
    }
}

// Backward of relu(a + b) into both inputs at once: dx0 (+)= m and dx1 (+)=
// m with m = (y > 0 ? dy : 0), y the ReLU's output.  One read of dy and y
// replaces a ReLU pass and two copies.  dx0 and dx1 may be the same tensor (a
// thread updates both in order) or null (no gradient wanted).
__global__ void add_relu_bwd_kernel(const float *__restrict__ dy, const float *__restrict__ y, int acc0, float *dx0,
                                    int acc1, float *dx1, int64_t n, int64_t n4) {
    const float4 *d4 = reinterpret_cast<const float4 *>(dy);
    const float4 *y4 = reinterpret_cast<const float4 *>(y);
    float4 *a4 = reinterpret_cast<float4 *>(dx0);
    float4 *b4 = reinterpret_cast<float4 *>(dx1);
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x) {
        const float4 d = d4[i], v = y4[i];
        float4 g;
        g.x = relu_grad(d.x, v.x); g.y = relu_grad(d.y, v.y); g.z = relu_grad(d.z, v.z); g.w = relu_grad(d.w, v.w);
        if (a4) {
            float4 o = g;
            if (acc0) {
                const float4 p = a4[i];
                o.x += p.x; o.y += p.y; o.z += p.z; o.w += p.w;
            }
            a4[i] = o;
        }
        if (b4) {
            float4 o = g;
            if (acc1) {
                const float4 p = b4[i];
                o.x += p.x; o.y += p.y; o.z += p.z; o.w += p.w;
            }
            b4[i] = o;
        }
    }
    for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const float g = relu_grad(dy[i], y[i]);
        if (dx0)
            dx0[i] = acc0 ? g + dx0[i] : g;
        if (dx1)
            dx1[i] = acc1 ? g + dx1[i] : g;
    }
}

__global__ void add_fwd_kernel(const float *__restrict__ a, const float *__restrict__ b, int relu,
                               float *__restrict__ y, int64_t n, int64_t n4) {
    const float4 *a4 = reinterpret_cast<const float4 *>(a);
    const float4 *b4 = reinterpret_cast<const float4 *>(b);
    float4 *y4 = reinterpret_cast<float4 *>(y);
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x) {
        float4 u = a4[i], v = b4[i], o;
        o.x = u.x + v.x; o.y = u.y + v.y; o.z = u.z + v.z; o.w = u.w + v.w;
        if (relu) {
            o.x = fmaxf(o.x, 0.f); o.y = fmaxf(o.y, 0.f); o.z = fmaxf(o.z, 0.f); o.w = fmaxf(o.w, 0.f);
        }
        y4[i] = o;
    }
    for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        float o = a[i] + b[i];
        y[i] = relu ? fmaxf(o, 0.f) : o;
    }
}

__global__ void copy_grad_kernel(const float *__restrict__ dy, int acc, float *__restrict__ dx, int64_t n, int64_t n4) {
    const float4 *d4 = reinterpret_cast<const float4 *>(dy);
    float4 *o4 = reinterpret_cast<float4 *>(dx);
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x) {
        float4 o = d4[i];
        if (acc) {
            float4 p = o4[i];
            o.x += p.x; o.y += p.y; o.z += p.z; o.w += p.w;
        }
        o4[i] = o;
    }
    for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        dx[i] = acc ? dx[i] + dy[i] : dy[i];
}

// Channel slice copies: a thread per float4 (or float) of the slice, rows
// outermost, so consecutive threads touch consecutive channels of one row.
// With I32 (fewer than 2^31 slice elements) the row is found by a multiply-high
// division by cv (fcv); else by a 64-bit division.
template <int V, bool I32>
__global__ void concat_kernel(int64_t rows, int c_in, int c_out, int off, FDiv fcv, const float *__restrict__ x,
                              float *__restrict__ y) {
    const int cv = c_in / V;
    const int64_t total = rows * cv;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t m = I32 ? (int64_t)fcv.div((uint32_t)e) : e / cv;
        int c = (int)(e - m * cv) * V;
        if (V == 4)
            *reinterpret_cast<float4 *>(y + m * c_out + off + c) = *reinterpret_cast<const float4 *>(x + m * c_in + c);
        else
            y[m * c_out + off + c] = x[m * c_in + c];
    }
}

// relu_y (may be null, laid out like dx): dx is the gradient of the input of
// a ReLU whose output was this concatenation's input; dy is kept where
// relu_y > 0.
template <int V, bool I32>
__global__ void concat_bwd_kernel(int64_t rows, int c_in, int c_out, int off, FDiv fcv, const float *__restrict__ dy,
                                  int acc, float *__restrict__ dx, const float *__restrict__ relu_y) {
    const int cv = c_in / V;
    const int64_t total = rows * cv;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t m = I32 ? (int64_t)fcv.div((uint32_t)e) : e / cv;
        int c = (int)(e - m * cv) * V;
        if (V == 4) {
            float4 g = *reinterpret_cast<const float4 *>(dy + m * c_out + off + c);
            if (relu_y) {
                const float4 v = *reinterpret_cast<const float4 *>(relu_y + m * c_in + c);
                g.x = relu_grad(g.x, v.x); g.y = relu_grad(g.y, v.y); g.z = relu_grad(g.z, v.z); g.w = relu_grad(g.w, v.w);
            }
            float4 *o = reinterpret_cast<float4 *>(dx + m * c_in + c);
            if (acc) {
                float4 p = *o;
                g.x += p.x; g.y += p.y; g.z += p.z; g.w += p.w;
            }
            *o = g;
        } else {
            float g = dy[m * c_out + off + c];
            if (relu_y)
                g = relu_grad(g, relu_y[m * c_in + c]);
            dx[m * c_in + c] = acc ? dx[m * c_in + c] + g : g;
        }
    }
}

// ---------------------------------------------------------------- pooling

__global__ void maxpool_fwd_kernel(dc_pool_shape sh, int P, int Q, const float *__restrict__ x,
                                   float *__restrict__ y, uint8_t *__restrict__ arg) {
    const int64_t total = (int64_t)sh.n * P * Q * sh.c;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        int c = (int)(e % sh.c);
        int64_t pix = e / sh.c;
        int q = (int)(pix % Q);
        int64_t t = pix / Q;
        int p = (int)(t % P);
        int n = (int)(t / P);
        int best = -1;
        float bv = 0.f;
        for (int r = 0; r < sh.r; ++r) {
            int h = p * sh.stride + r - sh.pad;
            if ((unsigned)h >= (unsigned)sh.h)
                continue;
            for (int s = 0; s < sh.s; ++s) {
                int w = q * sh.stride + s - sh.pad;
                if ((unsigned)w >= (unsigned)sh.w)
                    continue;
                float v = x[(((int64_t)n * sh.h + h) * sh.w + w) * sh.c + c];
                if (best < 0 || v > bv) {
                    best = r * sh.s + s;
                    bv = v;
                }
            }
        }
        y[e] = bv;
        arg[e] = (uint8_t)(best < 0 ? 0 : best);
    }
}

// MASK: dx is the gradient of a ReLU's input whose output the pool read; a
// window adds its dy only where its maximum (the pool's output y) is > 0,
// which is the ReLU's mask at the window's argmax.
template <bool MASK>
__global__ void maxpool_bwd_kernel(dc_pool_shape sh, int P, int Q, const float *__restrict__ dy,
                                   const uint8_t *__restrict__ arg, int acc, float *__restrict__ dx,
                                   const float *__restrict__ y) {
    const int64_t total = (int64_t)sh.n * sh.h * sh.w * sh.c;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        int c = (int)(e % sh.c);
        int64_t pix = e / sh.c;
        int w = (int)(pix % sh.w);
        int64_t t = pix / sh.w;
        int h = (int)(t % sh.h);
        int n = (int)(t / sh.h);
        // output windows that contain (h, w): p*stride - pad <= h <= p*stride - pad + r - 1
        int hp = h + sh.pad, wp = w + sh.pad;
        int p_lo = hp - sh.r + 1 > 0 ? (hp - sh.r + 1 + sh.stride - 1) / sh.stride : 0;
        int p_hi = min(P - 1, hp / sh.stride);
        int q_lo = wp - sh.s + 1 > 0 ? (wp - sh.s + 1 + sh.stride - 1) / sh.stride : 0;
        int q_hi = min(Q - 1, wp / sh.stride);
        float g = 0.f;
        for (int p = p_lo; p <= p_hi; ++p)
            for (int q = q_lo; q <= q_hi; ++q) {
                int64_t o = (((int64_t)n * P + p) * Q + q) * sh.c + c;
                int a = (hp - p * sh.stride) * sh.s + (wp - q * sh.stride);
                if (arg[o] == a && (!MASK || y[o] > 0.f))
                    g += dy[o];
            }
        dx[e] = acc ? dx[e] + g : g;
    }
}

// Float4 variants for c % 4 == 0: a thread owns one channel quad of one
// output (forward) or input (backward) pixel, so the index arithmetic is
// paid once per four channels and in 32 bits (the host checks the sizes).
// The grid-stride step stays in 32 bits too: total4 < 2^29 and the grid has at
// most 2^28 threads, so e + stride never passes INT_MAX.
// Per channel they make exactly the decisions and sums of the scalar kernels.
// Element e of the float4 output is decoded with multiply-high divisions by
// the invariant c4, Q and P (fc4, fQ, fP), not integer divisions.
__global__ void maxpool_fwd4_kernel(dc_pool_shape sh, int P, int Q, int c4, int total4, FDiv fc4, FDiv fQ, FDiv fP,
                                    const float4 *__restrict__ x, float4 *__restrict__ y,
                                    uchar4 *__restrict__ arg) {
    for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < total4; e += gridDim.x * blockDim.x) {
        const int pix = (int)fc4.div((uint32_t)e);
        const int q4 = e - pix * c4;
        const int t = (int)fQ.div((uint32_t)pix);
        const int q = pix - t * Q;
        const int n = (int)fP.div((uint32_t)t);
        const int p = t - n * P;
        float bv[4] = {0.f, 0.f, 0.f, 0.f};
        int best[4] = {-1, -1, -1, -1};
        for (int r = 0; r < sh.r; ++r) {
            const int h = p * sh.stride + r - sh.pad;
            if ((unsigned)h >= (unsigned)sh.h)
                continue;
            for (int s = 0; s < sh.s; ++s) {
                const int w = q * sh.stride + s - sh.pad;
                if ((unsigned)w >= (unsigned)sh.w)
                    continue;
                const float4 v = x[((n * sh.h + h) * sh.w + w) * c4 + q4];
                const float vv[4] = {v.x, v.y, v.z, v.w};
                const int k = r * sh.s + s;
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (best[j] < 0 || vv[j] > bv[j]) {
                        best[j] = k;
                        bv[j] = vv[j];
                    }
            }
        }
        y[e] = make_float4(bv[0], bv[1], bv[2], bv[3]);
        arg[e] = make_uchar4((unsigned char)max(best[0], 0), (unsigned char)max(best[1], 0),
                             (unsigned char)max(best[2], 0), (unsigned char)max(best[3], 0));
    }
}

template <bool MASK>
// Element e of the float4 input gradient is decoded, and its window range
// found, with multiply-high divisions by the invariant c4, W, H and stride.
__global__ void maxpool_bwd4_kernel(dc_pool_shape sh, int P, int Q, int c4, int total4, FDiv fc4, FDiv fW, FDiv fH,
                                    FDiv fst, const float4 *__restrict__ dy, const uchar4 *__restrict__ arg, int acc,
                                    float4 *__restrict__ dx, const float4 *__restrict__ y) {
    for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < total4; e += gridDim.x * blockDim.x) {
        const int pix = (int)fc4.div((uint32_t)e);
        const int q4 = e - pix * c4;
        const int t = (int)fW.div((uint32_t)pix);
        const int w = pix - t * sh.w;
        const int n = (int)fH.div((uint32_t)t);
        const int h = t - n * sh.h;
        const int hp = h + sh.pad, wp = w + sh.pad;
        // windows p with p * stride <= hp < p * stride + r (all operands >= 0)
        const int p_lo = hp - sh.r + 1 > 0 ? (int)fst.div((uint32_t)(hp - sh.r + sh.stride)) : 0;
        const int p_hi = min(P - 1, (int)fst.div((uint32_t)hp));
        const int q_lo = wp - sh.s + 1 > 0 ? (int)fst.div((uint32_t)(wp - sh.s + sh.stride)) : 0;
        const int q_hi = min(Q - 1, (int)fst.div((uint32_t)wp));
        float4 g = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int p = p_lo; p <= p_hi; ++p)
            for (int q = q_lo; q <= q_hi; ++q) {
                const int o = ((n * P + p) * Q + q) * c4 + q4;
                const int a = (hp - p * sh.stride) * sh.s + (wp - q * sh.stride);
                const uchar4 ar = arg[o];
                const float4 d = dy[o];
                const float4 ym = MASK ? y[o] : make_float4(1.f, 1.f, 1.f, 1.f);
                if (ar.x == a && ym.x > 0.f)
                    g.x += d.x;
                if (ar.y == a && ym.y > 0.f)
                    g.y += d.y;
                if (ar.z == a && ym.z > 0.f)
                    g.z += d.z;
                if (ar.w == a && ym.w > 0.f)
                    g.w += d.w;
            }
        if (acc) {
            const float4 o = dx[e];
            g.x = o.x + g.x; g.y = o.y + g.y; g.z = o.z + g.z; g.w = o.w + g.w;
        }
        dx[e] = g;
    }
}

// Backward of windows that tile the input exactly (stride = r = s, no padding,
// P r = H, Q s = W): every input element lies in one window, so a thread owns
// one output channel quad and writes its window's r x s input quads, dy where
// the tap is the argmax (and, with MASK, the maximum is positive), zero
// elsewhere.  The index arithmetic is paid once per output quad; each element
// gets exactly the gather kernel's value (0 + dy, or the accumulated sum).
template <bool MASK>
__global__ void maxpool_bwd4_tiled_kernel(dc_pool_shape sh, int P, int Q, int c4, int total4, FDiv fc4, FDiv fQ,
                                          FDiv fP, const float4 *__restrict__ dy, const uchar4 *__restrict__ arg,
                                          int acc, float4 *__restrict__ dx, const float4 *__restrict__ y) {
    for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < total4; e += gridDim.x * blockDim.x) {
        const int pix = (int)fc4.div((uint32_t)e);
        const int q4 = e - pix * c4;
        const int t = (int)fQ.div((uint32_t)pix);
        const int q = pix - t * Q;
        const int n = (int)fP.div((uint32_t)t);
        const int p = t - n * P;
        const uchar4 ar = arg[e];
        const float4 d = dy[e];
        const float4 ym = MASK ? y[e] : make_float4(1.f, 1.f, 1.f, 1.f);
        for (int i = 0; i < sh.r; ++i) {
            const int row = (n * sh.h + p * sh.r + i) * sh.w + q * sh.s;
            for (int j = 0; j < sh.s; ++j) {
                const int a = i * sh.s + j;
                float4 g = make_float4(0.f, 0.f, 0.f, 0.f);
                if (ar.x == a && ym.x > 0.f)
                    g.x += d.x;
                if (ar.y == a && ym.y > 0.f)
                    g.y += d.y;
                if (ar.z == a && ym.z > 0.f)
                    g.z += d.z;
                if (ar.w == a && ym.w > 0.f)
                    g.w += d.w;
                const int o = (row + j) * c4 + q4;
                if (acc) {
                    const float4 v = dx[o];
                    g.x = v.x + g.x; g.y = v.y + g.y; g.z = v.z + g.z; g.w = v.w + g.w;
                }
                dx[o] = g;
            }
        }
    }
}

// Average pooling over the window positions that lie inside the input (the
// padded ones are not counted).  V channels per thread (4 when c % 4 == 0 and
// the tensors are 16-byte aligned); the host keeps every element count below
// 2^31, so an element and its offsets fit in 32 bits, but the grid-stride step
// is taken in 64 bits: near 2^31 elements e + stride would pass INT_MAX.
// Backward gathers, for each input element, dy / count of every
// window that contains it, in window order: deterministic, no atomics.
__device__ __forceinline__ int pool_count(const dc_pool_shape &sh, int p, int q) {
    const int h0 = p * sh.stride - sh.pad, w0 = q * sh.stride - sh.pad;
    const int nh = min(h0 + sh.r, sh.h) - max(h0, 0), nw = min(w0 + sh.s, sh.w) - max(w0, 0);
    return max(nh, 0) * max(nw, 0);
}

template <int V>
__global__ void avgpool_fwd_kernel(dc_pool_shape sh, int P, int Q, int cv, int total, FDiv fcv, FDiv fQ, FDiv fP,
                                   const float *__restrict__ x, float *__restrict__ y) {
    using T = typename std::conditional<V == 4, float4, float>::type;
    const T *xv = reinterpret_cast<const T *>(x);
    T *yv = reinterpret_cast<T *>(y);
    for (int64_t e64 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e64 < total;
         e64 += (int64_t)gridDim.x * blockDim.x) {
        const int e = (int)e64;
        const int pix = (int)fcv.div((uint32_t)e), qc = e - pix * cv;
        const int t = (int)fQ.div((uint32_t)pix), q = pix - t * Q;
        const int n = (int)fP.div((uint32_t)t), p = t - n * P;
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        for (int r = 0; r < sh.r; ++r) {
            const int h = p * sh.stride + r - sh.pad;
            if ((unsigned)h >= (unsigned)sh.h)
                continue;
            for (int s = 0; s < sh.s; ++s) {
                const int w = q * sh.stride + s - sh.pad;
                if ((unsigned)w >= (unsigned)sh.w)
                    continue;
                const T v = xv[((n * sh.h + h) * sh.w + w) * cv + qc];
                if constexpr (V == 4) {
                    acc[0] += v.x; acc[1] += v.y; acc[2] += v.z; acc[3] += v.w;
                } else {
                    acc[0] += v;
                }
            }
        }
        const float inv = 1.0f / (float)max(pool_count(sh, p, q), 1);
        if constexpr (V == 4)
            yv[e] = make_float4(acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
        else
            yv[e] = acc[0] * inv;
    }
}

template <int V>
__global__ void avgpool_bwd_kernel(dc_pool_shape sh, int P, int Q, int cv, int total, FDiv fcv, FDiv fW, FDiv fH,
                                   FDiv fst, const float *__restrict__ dy, int acc_in, float *__restrict__ dx) {
    using T = typename std::conditional<V == 4, float4, float>::type;
    const T *dv = reinterpret_cast<const T *>(dy);
    T *xv = reinterpret_cast<T *>(dx);
    for (int64_t e64 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e64 < total;
         e64 += (int64_t)gridDim.x * blockDim.x) {
        const int e = (int)e64;
        const int pix = (int)fcv.div((uint32_t)e), qc = e - pix * cv;
        const int t = (int)fW.div((uint32_t)pix), w = pix - t * sh.w;
        const int n = (int)fH.div((uint32_t)t), h = t - n * sh.h;
        const int hp = h + sh.pad, wp = w + sh.pad;
        const int p_lo = hp - sh.r + 1 > 0 ? (int)fst.div((uint32_t)(hp - sh.r + sh.stride)) : 0;
        const int p_hi = min(P - 1, (int)fst.div((uint32_t)hp));
        const int q_lo = wp - sh.s + 1 > 0 ? (int)fst.div((uint32_t)(wp - sh.s + sh.stride)) : 0;
        const int q_hi = min(Q - 1, (int)fst.div((uint32_t)wp));
        float g[4] = {0.f, 0.f, 0.f, 0.f};
        for (int p = p_lo; p <= p_hi; ++p)
            for (int q = q_lo; q <= q_hi; ++q) {
                const float inv = 1.0f / (float)max(pool_count(sh, p, q), 1);
                const T d = dv[((n * P + p) * Q + q) * cv + qc];
                if constexpr (V == 4) {
                    g[0] += d.x * inv; g[1] += d.y * inv; g[2] += d.z * inv; g[3] += d.w * inv;
                } else {
                    g[0] += d * inv;
                }
            }
        if constexpr (V == 4) {
            float4 o = make_float4(g[0], g[1], g[2], g[3]);
            if (acc_in) {
                const float4 prev = xv[e];
                o.x += prev.x; o.y += prev.y; o.z += prev.z; o.w += prev.w;
            }
            xv[e] = o;
        } else {
            xv[e] = acc_in ? xv[e] + g[0] : g[0];
        }
    }
}

__global__ void gap_fwd_kernel(int n, int hw, int c, const float *__restrict__ x, float *__restrict__ y) {
    int64_t total = (int64_t)n * c;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        int ch = (int)(e % c);
        int64_t b = e / c;
        const float *src = x + b * hw * c + ch;
        float s = 0.f;
        for (int i = 0; i < hw; ++i)
            s += src[(int64_t)i * c];
        y[e] = s / (float)hw;
    }
}

// With I32 (fewer than 2^31 elements) the channel and image of element e come
// from multiply-high divisions by c and hw (fc, fhw); else 64-bit divisions.
template <bool I32>
__global__ void gap_bwd_kernel(int n, int hw, int c, FDiv fc, FDiv fhw, const float *__restrict__ dy, int acc,
                               float *__restrict__ dx) {
    int64_t total = (int64_t)n * hw * c;
    float inv = 1.0f / (float)hw;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        int ch;
        int64_t b;
        if (I32) {
            const uint32_t q = fc.div((uint32_t)e); // pixel index b * hw + i
            ch = (int)((uint32_t)e - q * (uint32_t)c);
            b = fhw.div(q);
        } else {
            ch = (int)(e % c);
            b = e / ((int64_t)hw * c);
        }
        float g = dy[b * c + ch] * inv;
        dx[e] = acc ? dx[e] + g : g;
    }
}

// ---------------------------------------------------------------- per-channel reductions
//
// Stage 1: workgroup (chunk, group) sums rows [chunk*rows_per_chunk, ...) of
// channels [group*CG, group*CG + CG) of a [rows][c] matrix.  256 threads =
// CG channels x (256 / CG) row lanes; lanes are combined in a fixed order.
// Mode 0: sum x.  Mode 1: sum (x - mean)^2.  Mode 2: sum dy and sum dy*xhat
// with xhat = (x - mean) * invstd (two outputs).
constexpr int CG = 64;
constexpr int RL = EW_THREADS / CG;

template <int MODE>
__global__ __launch_bounds__(EW_THREADS) void colred_partial_kernel(
    int64_t rows, int c, int64_t rows_per_chunk, const float *__restrict__ x, const float *__restrict__ dy,
    const float *__restrict__ mean, const float *__restrict__ invstd, float *__restrict__ part0,
    float *__restrict__ part1, const float *__restrict__ relu_y) {
    __shared__ float s0[RL][CG];
    __shared__ float s1[RL][CG];
    const int lane_c = threadIdx.x % CG, rl = threadIdx.x / CG;
    const int ch = blockIdx.y * CG + lane_c;
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_chunk;
    const int64_t r1 = min(rows, r0 + rows_per_chunk);
    float a0 = 0.f, a1 = 0.f;
    if (ch < c) {
        float mu = (MODE != 0) ? mean[ch] : 0.f;
        float is = (MODE == 2) ? invstd[ch] : 0.f;
        for (int64_t r = r0 + rl; r < r1; r += RL) {
            int64_t o = r * c + ch;
            if (MODE == 0) {
                a0 += x[o];
            } else if (MODE == 1) {
                float d = x[o] - mu;
                a0 += d * d;
            } else {
                float g = relu_y ? relu_grad(dy[o], relu_y[o]) : dy[o];
                a0 += g;
                a1 += g * ((x[o] - mu) * is);
            }
        }
    }
    s0[rl][lane_c] = a0;
    s1[rl][lane_c] = a1;
    __syncthreads();
    if (rl == 0 && ch < c) {
        float t0 = 0.f, t1 = 0.f;
        for (int i = 0; i < RL; ++i) {
            t0 += s0[i][lane_c];
            t1 += s1[i][lane_c];
        }
        part0[(int64_t)blockIdx.x * c + ch] = t0;
        if (MODE == 2)
            part1[(int64_t)blockIdx.x * c + ch] = t1;
    }
}

// Stage 2: one workgroup per channel adds the chunk partials with a fixed
// tree in double precision.  Output kind: 0 -> out0 = sum; 1 -> out0 = sum/rows
// (mean); 2 -> out0 = 1/sqrt(sum/rows + eps) (invstd); 3 -> out0 = sum0, out1 = sum1.
// 4 -> from the shifted sums of mode 1: out0 = K + S1/rows (mean),
// out1 = 1/sqrt(S2/rows - (S1/rows)^2 + eps) (invstd), K = shift[ch].
template <int KIND>
__global__ __launch_bounds__(EW_THREADS) void colred_final_kernel(int nchunks, int c, int64_t rows, float eps,
                                                                  const float *__restrict__ part0,
                                                                  const float *__restrict__ part1,
                                                                  float *__restrict__ out0, float *__restrict__ out1,
                                                                  const float *__restrict__ shift) {
    __shared__ double s0[EW_THREADS];
    __shared__ double s1[EW_THREADS];
    const int ch = blockIdx.x;
    double a0 = 0.0, a1 = 0.0;
    for (int i = threadIdx.x; i < nchunks; i += EW_THREADS) {
        a0 += (double)part0[(int64_t)i * c + ch];
        if (KIND >= 3)
            a1 += (double)part1[(int64_t)i * c + ch];
    }
    s0[threadIdx.x] = a0;
    s1[threadIdx.x] = a1;
    __syncthreads();
    for (int w = EW_THREADS / 2; w > 0; w >>= 1) {
        if (threadIdx.x < w) {
            s0[threadIdx.x] += s0[threadIdx.x + w];
            s1[threadIdx.x] += s1[threadIdx.x + w];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        double v = s0[0];
        if (KIND == 0) {
            out0[ch] = (float)v;
        } else if (KIND == 1) {
            out0[ch] = (float)(v / (double)rows);
        } else if (KIND == 2) {
            out0[ch] = (float)(1.0 / sqrt(v / (double)rows + (double)eps));
        } else if (KIND == 3) {
            out0[ch] = (float)v;
            out1[ch] = (float)s1[0];
        } else {
            const double m1 = v / (double)rows;
            const double var = std::max(0.0, s1[0] / (double)rows - m1 * m1);
            out0[ch] = (float)((double)shift[ch] + m1);
            out1[ch] = (float)(1.0 / sqrt(var + (double)eps));
        }
    }
}

__global__ void bn_apply_kernel(int64_t rows, int c, const float *__restrict__ x, const float *__restrict__ gamma,
                                const float *__restrict__ beta, const float *__restrict__ mean,
                                const float *__restrict__ invstd, int relu, float *__restrict__ y) {
    const int64_t total = rows * c;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        int ch = (int)(e % c);
        float v = gamma[ch] * ((x[e] - mean[ch]) * invstd[ch]) + beta[ch];
        y[e] = relu ? fmaxf(v, 0.f) : v;
    }
}

__global__ void bn_bwd_apply_kernel(int64_t rows, int c, const float *__restrict__ dy, const float *__restrict__ x,
                                    const float *__restrict__ gamma, const float *__restrict__ mean,
                                    const float *__restrict__ invstd, const float *__restrict__ dgamma,
                                    const float *__restrict__ dbeta, int acc, float *__restrict__ dx,
                                    const float *__restrict__ relu_y) {
    const int64_t total = rows * c;
    const float inv_rows = 1.0f / (float)rows;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        int ch = (int)(e % c);
        float is = invstd[ch];
        float xhat = (x[e] - mean[ch]) * is;
        const float d = relu_y ? relu_grad(dy[e], relu_y[e]) : dy[e];
        float g = gamma[ch] * is * (d - dbeta[ch] * inv_rows - xhat * dgamma[ch] * inv_rows);
        dx[e] = acc ? dx[e] + g : g;
    }
}

// Float4 path of the per-channel reductions, for c % 4 == 0 and 16-byte
// aligned tensors.  A workgroup's 256 threads are G channel quads x RL row
// lanes (G = min(c/4, 64), RL = 256 / G rounded down; leftover threads stay
// idle); it owns rows [chunk*rpc, ...) of channels [blk*4G, ...).  A thread
// sums rows rl, rl + RL, ... into two independent float4 accumulators, the
// row lanes are added in lane order through LDS, and the partials go to fixed
// slots.  Mode 0: sum x.  Mode 1: sum (x - K) and sum (x - K)^2 with K the
// channel's value in row 0, a shift that keeps the one-pass variance free of
// cancellation.  Mode 2: sum dy and sum dy * (x - mean) * invstd.
// The float4 of dy at element o, passed through ReLU's backward (kept where
// the ReLU's output relu_y is positive) when relu_y is given.
__device__ __forceinline__ float4 dy4_at(const float *dy, const float *relu_y, int64_t o) {
    float4 d = *reinterpret_cast<const float4 *>(dy + o);
    if (relu_y) {
        const float4 y = *reinterpret_cast<const float4 *>(relu_y + o);
        d = make_float4(relu_grad(d.x, y.x), relu_grad(d.y, y.y), relu_grad(d.z, y.z), relu_grad(d.w, y.w));
    }
    return d;
}

template <int MODE>
__device__ __forceinline__ void col4_acc(float4 &a0, float4 &a1, const float4 v, const float4 d, const float4 mu,
                                         const float4 is) {
    if (MODE == 0) {
        a0.x += v.x; a0.y += v.y; a0.z += v.z; a0.w += v.w;
    } else if (MODE == 1) {
        const float x0 = v.x - mu.x, x1 = v.y - mu.y, x2 = v.z - mu.z, x3 = v.w - mu.w;
        a0.x += x0; a0.y += x1; a0.z += x2; a0.w += x3;
        a1.x += x0 * x0; a1.y += x1 * x1; a1.z += x2 * x2; a1.w += x3 * x3;
    } else {
        a0.x += d.x; a0.y += d.y; a0.z += d.z; a0.w += d.w;
        a1.x += d.x * ((v.x - mu.x) * is.x);
        a1.y += d.y * ((v.y - mu.y) * is.y);
        a1.z += d.z * ((v.z - mu.z) * is.z);
        a1.w += d.w * ((v.w - mu.w) * is.w);
    }
}

__device__ __forceinline__ float4 add4(float4 a, float4 b) {
    return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

template <int MODE>
__global__ __launch_bounds__(EW_THREADS) void colred4_partial_kernel(
    int64_t rows, int c, int64_t rpc, int g, int rl_n, const float *__restrict__ x, const float *__restrict__ dy,
    const float *__restrict__ mean, const float *__restrict__ invstd, float *__restrict__ part0,
    float *__restrict__ part1, const float *__restrict__ relu_y) {
    __shared__ float4 s0[EW_THREADS];
    __shared__ float4 s1[EW_THREADS];
    const int t = threadIdx.x;
    const int q = t % g, rl = t / g;
    const int ch = (blockIdx.y * g + q) * 4;
    const int64_t r0 = (int64_t)blockIdx.x * rpc;
    const int64_t r1 = min(rows, r0 + rpc);
    const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
    float4 a0 = z4, a1 = z4, b0 = z4, b1 = z4;
    if (rl < rl_n && ch < c) {
        float4 mu = z4, is = z4;
        if (MODE == 1)
            mu = *reinterpret_cast<const float4 *>(x + ch);
        if (MODE == 2) {
            mu = *reinterpret_cast<const float4 *>(mean + ch);
            is = *reinterpret_cast<const float4 *>(invstd + ch);
        }
        const float *src = MODE == 2 ? dy : x;
        int64_t r = r0 + rl;
        for (; r + rl_n < r1; r += 2 * (int64_t)rl_n) {
            const int64_t o0 = r * c + ch, o1 = (r + rl_n) * c + ch;
            const float4 v0 = *reinterpret_cast<const float4 *>(x + o0);
            const float4 v1 = *reinterpret_cast<const float4 *>(x + o1);
            const float4 d0 = MODE == 2 ? dy4_at(src, relu_y, o0) : z4;
            const float4 d1 = MODE == 2 ? dy4_at(src, relu_y, o1) : z4;
            col4_acc<MODE>(a0, a1, v0, d0, mu, is);
            col4_acc<MODE>(b0, b1, v1, d1, mu, is);
        }
        if (r < r1) {
            const int64_t o0 = r * c + ch;
            const float4 v0 = *reinterpret_cast<const float4 *>(x + o0);
            const float4 d0 = MODE == 2 ? dy4_at(src, relu_y, o0) : z4;
            col4_acc<MODE>(a0, a1, v0, d0, mu, is);
        }
    }
    s0[t] = add4(a0, b0);
    s1[t] = add4(a1, b1);
    __syncthreads();
    if (rl == 0 && ch < c) {
        float4 t0 = s0[t], t1 = s1[t];
        for (int i = 1; i < rl_n; ++i) {
            t0 = add4(t0, s0[i * g + q]);
            t1 = add4(t1, s1[i * g + q]);
        }
        *reinterpret_cast<float4 *>(part0 + (int64_t)blockIdx.x * c + ch) = t0;
        if (MODE != 0)
            *reinterpret_cast<float4 *>(part1 + (int64_t)blockIdx.x * c + ch) = t1;
    }
}

// y = gamma * (x - mean) * invstd + beta over n4 float4 groups of [rows][c],
// c % 4 == 0.  The grid's thread count is a multiple of c/4 (bn4_blocks), so
// a thread keeps one channel quad, and its parameters, for the whole loop.
__global__ void bn_apply4_kernel(int64_t n4, int c4, const float4 *__restrict__ x, const float4 *__restrict__ gamma,
                                 const float4 *__restrict__ beta, const float4 *__restrict__ mean,
                                 const float4 *__restrict__ invstd, int relu, float4 *__restrict__ y) {
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int q = (int)(t0 % c4);
    const float4 g = gamma[q], b = beta[q], m = mean[q], is = invstd[q];
    for (int64_t i = t0; i < n4; i += stride) {
        const float4 v = x[i];
        float4 o;
        o.x = g.x * ((v.x - m.x) * is.x) + b.x;
        o.y = g.y * ((v.y - m.y) * is.y) + b.y;
        o.z = g.z * ((v.z - m.z) * is.z) + b.z;
        o.w = g.w * ((v.w - m.w) * is.w) + b.w;
        if (relu) {
            o.x = fmaxf(o.x, 0.f); o.y = fmaxf(o.y, 0.f); o.z = fmaxf(o.z, 0.f); o.w = fmaxf(o.w, 0.f);
        }
        y[i] = o;
    }
}

__device__ __forceinline__ float bn_dx(float dy, float x, float g, float m, float is, float dg, float db,
                                       float inv_rows) {
    const float xhat = (x - m) * is;
    return g * is * (dy - db * inv_rows - xhat * dg * inv_rows);
}

__global__ void bn_bwd_apply4_kernel(int64_t n4, int c4, int64_t rows, const float4 *__restrict__ dy,
                                     const float4 *__restrict__ x, const float4 *__restrict__ gamma,
                                     const float4 *__restrict__ mean, const float4 *__restrict__ invstd,
                                     const float4 *__restrict__ dgamma, const float4 *__restrict__ dbeta, int acc,
                                     float4 *__restrict__ dx, const float4 *__restrict__ relu_y) {
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int q = (int)(t0 % c4);
    const float inv_rows = 1.0f / (float)rows;
    const float4 g = gamma[q], m = mean[q], is = invstd[q], dg = dgamma[q], db = dbeta[q];
    for (int64_t i = t0; i < n4; i += stride) {
        float4 d = dy[i];
        const float4 v = x[i];
        if (relu_y) {
            const float4 y = relu_y[i];
            d = make_float4(relu_grad(d.x, y.x), relu_grad(d.y, y.y), relu_grad(d.z, y.z), relu_grad(d.w, y.w));
        }
        float4 o;
        o.x = bn_dx(d.x, v.x, g.x, m.x, is.x, dg.x, db.x, inv_rows);
        o.y = bn_dx(d.y, v.y, g.y, m.y, is.y, dg.y, db.y, inv_rows);
        o.z = bn_dx(d.z, v.z, g.z, m.z, is.z, dg.z, db.z, inv_rows);
        o.w = bn_dx(d.w, v.w, g.w, m.w, is.w, dg.w, db.w, inv_rows);
        if (acc) {
            const float4 p = dx[i];
            o.x = p.x + o.x; o.y = p.y + o.y; o.z = p.z + o.z; o.w = p.w + o.w;
        }
        dx[i] = o;
    }
}

struct ColPlan {
    int nchunks;
    int64_t rows_per_chunk;
};

ColPlan col_plan(int64_t rows, int c) {
    int groups = (c + CG - 1) / CG;
    // about 1024 workgroups in all, at most 256 chunks (one per stage-2 thread
    // slot), at least RL*8 rows each
    int64_t want = std::max<int64_t>(1, std::min<int64_t>(256, 1024 / std::max(groups, 1)));
    int64_t rpc = std::max<int64_t>((rows + want - 1) / want, RL * 8);
    ColPlan p;
    p.rows_per_chunk = rpc;
    p.nchunks = (int)((rows + rpc - 1) / rpc);
    return p;
}

struct Col4Plan {
    int g, rl_n, blocks, nchunks;
    int64_t rpc;
};

Col4Plan col4_plan(int64_t rows, int c) {
    Col4Plan p;
    p.g = std::min(c / 4, 64);
    p.rl_n = EW_THREADS / p.g;
    p.blocks = (c / 4 + p.g - 1) / p.g;
    // about 2048 workgroups in all, at least 8 rows per row lane
    int64_t want = std::max<int64_t>(1, 2048 / p.blocks);
    p.rpc = std::max<int64_t>((rows + want - 1) / want, (int64_t)p.rl_n * 8);
    p.nchunks = (int)((rows + p.rpc - 1) / p.rpc);
    return p;
}

inline bool col4_ok(int c, const void *a, const void *b = nullptr) {
    return c % 4 == 0 && ((uintptr_t)a & 15) == 0 && ((uintptr_t)b & 15) == 0;
}

// Blocks for a float4 loop over [rows][c] whose threads each keep one channel
// quad: the thread count is rounded up to a multiple of c/4.
int bn4_blocks(int64_t n4, int c4) {
    int64_t b = std::max<int64_t>(1, std::min<int64_t>((n4 + EW_THREADS - 1) / EW_THREADS, 1 << 16));
    int64_t m = c4 / std::gcd(c4, EW_THREADS);
    return (int)((b + m - 1) / m * m);
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

// Number of float4 groups the vector path may take: n/4 when every pointer is
// 16-byte aligned, else 0 (everything goes through the scalar tail loop).
inline bool al16(const void *p) { return ((uintptr_t)p & 15) == 0; }
inline int64_t vec4(int64_t n, const void *a, const void *b) { return al16(a) && al16(b) ? n >> 2 : 0; }
inline int64_t vec4(int64_t n, const void *a, const void *b, const void *c) { return al16(c) ? vec4(n, a, b) : 0; }

// ---------------------------------------------------------------- softmax cross-entropy

// One workgroup per sample: loss_i = logsumexp(z_i) - z_i[y_i],
// dz_i = (softmax(z_i) - onehot(y_i)) / n.
__global__ __launch_bounds__(EW_THREADS) void xent_row_kernel(int n, int classes, const float *__restrict__ z,
                                                              const int32_t *__restrict__ y, float *__restrict__ loss_i,
                                                              float *__restrict__ dz) {
    __shared__ float red[EW_THREADS];
    const int i = blockIdx.x;
    const float *zi = z + (int64_t)i * classes;
    float m = -INFINITY;
    for (int k = threadIdx.x; k < classes; k += EW_THREADS)
        m = fmaxf(m, zi[k]);
    red[threadIdx.x] = m;
    __syncthreads();
    for (int w = EW_THREADS / 2; w > 0; w >>= 1) {
        if (threadIdx.x < w)
            red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + w]);
        __syncthreads();
    }
    m = red[0];
    __syncthreads();
    float s = 0.f;
    for (int k = threadIdx.x; k < classes; k += EW_THREADS)
        s += expf(zi[k] - m);
    red[threadIdx.x] = s;
    __syncthreads();
    for (int w = EW_THREADS / 2; w > 0; w >>= 1) {
        if (threadIdx.x < w)
            red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    s = red[0];
    const int label = y[i];
    const float inv_n = 1.0f / (float)n;
    const float inv_s = 1.0f / s;
    for (int k = threadIdx.x; k < classes; k += EW_THREADS) {
        float p = expf(zi[k] - m) * inv_s;
        dz[(int64_t)i * classes + k] = (p - (k == label ? 1.f : 0.f)) * inv_n;
    }
    if (threadIdx.x == 0) {
        float zl = (label >= 0 && label < classes) ? zi[label] : 0.f;
        loss_i[i] = m + logf(s) - zl;
    }
}

__global__ void xent_mean_kernel(int n, const float *__restrict__ loss_i, float *__restrict__ loss) {
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        double s = 0.0;
        for (int i = 0; i < n; ++i)
            s += (double)loss_i[i];
        loss[0] = (float)(s / (double)n);
    }
}

// ---------------------------------------------------------------- link pacing

__global__ void pace_mark_kernel(uint64_t *slot) {
    if (threadIdx.x == 0)
        *slot = wall_clock64();
}

// Spins until the wall clock passes *slot + ticks.  It always ends: the wall
// clock only moves forward and the wait never exceeds cap_ticks.
__global__ void pace_until_kernel(const uint64_t *slot, uint64_t ticks, uint64_t cap_ticks) {
    if (threadIdx.x != 0)
        return;
    const uint64_t start = wall_clock64();
    const uint64_t deadline = *slot + ticks;
    for (;;) {
        uint64_t now = wall_clock64();
        if (now >= deadline || now - start >= cap_ticks)
            break;
        __builtin_amdgcn_s_sleep(2);
    }
}

} // namespace

// ---------------------------------------------------------------- launchers

int relu_forward(const float *x, float *y, int64_t n, hipStream_t s) {
    if (n <= 0)
        return DC_OK;
    hipLaunchKernelGGL(relu_fwd_kernel, dim3(ew_blocks(n, 4)), dim3(EW_THREADS), 0, s, x, y, n, vec4(n, x, y));
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int relu_backward(const float *dy, const float *y, int accumulate, float *dx, int64_t n, hipStream_t s) {
    if (n <= 0)
        return DC_OK;
    hipLaunchKernelGGL(relu_bwd_kernel, dim3(ew_blocks(n, 4)), dim3(EW_THREADS), 0, s, dy, y, accumulate, dx, n,
                       vec4(n, dy, y, dx));
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int add_forward(const float *a, const float *b, int relu, float *y, int64_t n, hipStream_t s) {
    if (n <= 0)
        return DC_OK;
    hipLaunchKernelGGL(add_fwd_kernel, dim3(ew_blocks(n, 4)), dim3(EW_THREADS), 0, s, a, b, relu, y, n, vec4(n, a, b, y));
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int add_relu_backward(const float *dy, const float *y, int acc0, float *dx0, int acc1, float *dx1, int64_t n,
                      hipStream_t s) {
    if (n <= 0)
        return DC_OK;
    const int64_t n4 = al16(dx0) && al16(dx1) ? vec4(n, dy, y) : 0;
    hipLaunchKernelGGL(add_relu_bwd_kernel, dim3(ew_blocks(n, 4)), dim3(EW_THREADS), 0, s, dy, y, acc0, dx0, acc1, dx1,
                       n, n4);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int copy_grad(const float *dy, int accumulate, float *dx, int64_t n, hipStream_t s) {
    if (n <= 0)
        return DC_OK;
    hipLaunchKernelGGL(copy_grad_kernel, dim3(ew_blocks(n, 4)), dim3(EW_THREADS), 0, s, dy, accumulate, dx, n,
                       vec4(n, dy, dx));
    DC_HIP(hipGetLastError());
    return DC_OK;
}

static bool concat_vec(int c_in, int c_out, int off, const void *a, const void *b) {
    return c_in % 4 == 0 && c_out % 4 == 0 && off % 4 == 0 && al16(a) && al16(b);
}

int concat_forward(int64_t rows, int c_in, int c_out, int off, const float *x, float *y, hipStream_t s) {
    if (rows <= 0 || c_in <= 0)
        return DC_OK;
    const bool i32 = rows * c_in < INT_MAX;
    if (concat_vec(c_in, c_out, off, x, y)) {
        const FDiv f = make_fdiv(c_in / 4);
        if (i32)
            hipLaunchKernelGGL((concat_kernel<4, true>), dim3(ew_blocks(rows * c_in, 4)), dim3(EW_THREADS), 0, s, rows,
                               c_in, c_out, off, f, x, y);
        else
            hipLaunchKernelGGL((concat_kernel<4, false>), dim3(ew_blocks(rows * c_in, 4)), dim3(EW_THREADS), 0, s, rows,
                               c_in, c_out, off, f, x, y);
    } else {
        const FDiv f = make_fdiv(c_in);
        if (i32)
            hipLaunchKernelGGL((concat_kernel<1, true>), dim3(ew_blocks(rows * c_in)), dim3(EW_THREADS), 0, s, rows,
                               c_in, c_out, off, f, x, y);
        else
            hipLaunchKernelGGL((concat_kernel<1, false>), dim3(ew_blocks(rows * c_in)), dim3(EW_THREADS), 0, s, rows,
                               c_in, c_out, off, f, x, y);
    }
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int concat_backward(int64_t rows, int c_in, int c_out, int off, const float *dy, int accumulate, float *dx,
                    hipStream_t s, const float *relu_y) {
    if (rows <= 0 || c_in <= 0)
        return DC_OK;
    const bool i32 = rows * c_in < INT_MAX;
    if (concat_vec(c_in, c_out, off, dy, dx) && al16(relu_y)) {
        const FDiv f = make_fdiv(c_in / 4);
        if (i32)
            hipLaunchKernelGGL((concat_bwd_kernel<4, true>), dim3(ew_blocks(rows * c_in, 4)), dim3(EW_THREADS), 0, s,
                               rows, c_in, c_out, off, f, dy, accumulate, dx, relu_y);
        else
            hipLaunchKernelGGL((concat_bwd_kernel<4, false>), dim3(ew_blocks(rows * c_in, 4)), dim3(EW_THREADS), 0, s,
                               rows, c_in, c_out, off, f, dy, accumulate, dx, relu_y);
    } else {
        const FDiv f = make_fdiv(c_in);
        if (i32)
            hipLaunchKernelGGL((concat_bwd_kernel<1, true>), dim3(ew_blocks(rows * c_in)), dim3(EW_THREADS), 0, s,
                               rows, c_in, c_out, off, f, dy, accumulate, dx, relu_y);
        else
            hipLaunchKernelGGL((concat_bwd_kernel<1, false>), dim3(ew_blocks(rows * c_in)), dim3(EW_THREADS), 0, s,
                               rows, c_in, c_out, off, f, dy, accumulate, dx, relu_y);
    }
    DC_HIP(hipGetLastError());
    return DC_OK;
}

// The float4 pooling kernels index in 32 bits: every input and output
// element count must stay below 2^31, and c % 4 == 0 with aligned pointers.
static bool pool4_ok(const dc_pool_shape &sh, int P, int Q, const void *a, const void *b, const void *arg) {
    return sh.c % 4 == 0 && ((uintptr_t)a & 15) == 0 && ((uintptr_t)b & 15) == 0 && ((uintptr_t)arg & 3) == 0 &&
           (int64_t)sh.n * sh.h * sh.w * sh.c < INT_MAX && (int64_t)sh.n * P * Q * sh.c < INT_MAX;
}

int maxpool_forward(const dc_pool_shape &sh, const float *x, float *y, uint8_t *arg, hipStream_t s) {
    int P = (sh.h + 2 * sh.pad - sh.r) / sh.stride + 1;
    int Q = (sh.w + 2 * sh.pad - sh.s) / sh.stride + 1;
    int64_t total = (int64_t)sh.n * P * Q * sh.c;
    if (total <= 0)
        return DC_OK;
    if (pool4_ok(sh, P, Q, x, y, arg)) {
        const int total4 = (int)(total / 4);
        hipLaunchKernelGGL(maxpool_fwd4_kernel, dim3(ew_blocks(total4)), dim3(EW_THREADS), 0, s, sh, P, Q, sh.c / 4,
                           total4, make_fdiv(sh.c / 4), make_fdiv(Q), make_fdiv(P), reinterpret_cast<const float4 *>(x),
                           reinterpret_cast<float4 *>(y), reinterpret_cast<uchar4 *>(arg));
    } else {
        hipLaunchKernelGGL(maxpool_fwd_kernel, dim3(ew_blocks(total)), dim3(EW_THREADS), 0, s, sh, P, Q, x, y, arg);
    }
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int maxpool_backward(const dc_pool_shape &sh, const float *dy, const uint8_t *arg, int accumulate, float *dx,
                     hipStream_t s, const float *relu_y) {
    int P = (sh.h + 2 * sh.pad - sh.r) / sh.stride + 1;
    int Q = (sh.w + 2 * sh.pad - sh.s) / sh.stride + 1;
    int64_t total = (int64_t)sh.n * sh.h * sh.w * sh.c;
    if (total <= 0)
        return DC_OK;
    if (pool4_ok(sh, P, Q, dy, dx, arg) && ((uintptr_t)relu_y & 15) == 0) {
        const int total4 = (int)(total / 4);
        const auto *dy4 = reinterpret_cast<const float4 *>(dy);
        const auto *arg4 = reinterpret_cast<const uchar4 *>(arg);
        const auto *y4 = reinterpret_cast<const float4 *>(relu_y);
        auto *dx4 = reinterpret_cast<float4 *>(dx);
        if (sh.pad == 0 && sh.stride == sh.r && sh.stride == sh.s && P * sh.r == sh.h && Q * sh.s == sh.w) {
            // windows tile the input: one thread per output quad writes its window
            const int out4 = (int)((int64_t)sh.n * P * Q * sh.c / 4);
            const FDiv fc4 = make_fdiv(sh.c / 4), fQ = make_fdiv(Q), fP = make_fdiv(P);
            if (relu_y)
                hipLaunchKernelGGL(maxpool_bwd4_tiled_kernel<true>, dim3(ew_blocks(out4)), dim3(EW_THREADS), 0, s, sh,
                                   P, Q, sh.c / 4, out4, fc4, fQ, fP, dy4, arg4, accumulate, dx4, y4);
            else
                hipLaunchKernelGGL(maxpool_bwd4_tiled_kernel<false>, dim3(ew_blocks(out4)), dim3(EW_THREADS), 0, s,
                                   sh, P, Q, sh.c / 4, out4, fc4, fQ, fP, dy4, arg4, accumulate, dx4, y4);
            DC_HIP(hipGetLastError());
            return DC_OK;
        }
        const FDiv fc4 = make_fdiv(sh.c / 4), fW = make_fdiv(sh.w), fH = make_fdiv(sh.h), fst = make_fdiv(sh.stride);
        if (relu_y)
            hipLaunchKernelGGL(maxpool_bwd4_kernel<true>, dim3(ew_blocks(total4)), dim3(EW_THREADS), 0, s, sh, P, Q,
                               sh.c / 4, total4, fc4, fW, fH, fst, dy4, arg4, accumulate, dx4, y4);
        else
            hipLaunchKernelGGL(maxpool_bwd4_kernel<false>, dim3(ew_blocks(total4)), dim3(EW_THREADS), 0, s, sh, P, Q,
                               sh.c / 4, total4, fc4, fW, fH, fst, dy4, arg4, accumulate, dx4, y4);
    } else if (relu_y) {
        hipLaunchKernelGGL(maxpool_bwd_kernel<true>, dim3(ew_blocks(total)), dim3(EW_THREADS), 0, s, sh, P, Q, dy, arg,
                           accumulate, dx, relu_y);
    } else {
        hipLaunchKernelGGL(maxpool_bwd_kernel<false>, dim3(ew_blocks(total)), dim3(EW_THREADS), 0, s, sh, P, Q, dy,
                           arg, accumulate, dx, relu_y);
    }
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int avgpool_forward(const dc_pool_shape &sh, const float *x, float *y, hipStream_t s) {
    const int P = (sh.h + 2 * sh.pad - sh.r) / sh.stride + 1;
    const int Q = (sh.w + 2 * sh.pad - sh.s) / sh.stride + 1;
    const int64_t total = (int64_t)sh.n * P * Q * sh.c;
    if (total <= 0)
        return DC_OK;
    if ((int64_t)sh.n * sh.h * sh.w * sh.c >= INT_MAX || total >= INT_MAX)
        return fail(DC_EINVAL, "average pooling of %lld elements exceeds the 2^31 limit", (long long)total);
    if (sh.c % 4 == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)y & 15) == 0)
        hipLaunchKernelGGL(avgpool_fwd_kernel<4>, dim3(ew_blocks(total / 4)), dim3(EW_THREADS), 0, s, sh, P, Q,
                           sh.c / 4, (int)(total / 4), make_fdiv(sh.c / 4), make_fdiv(Q), make_fdiv(P), x, y);
    else
        hipLaunchKernelGGL(avgpool_fwd_kernel<1>, dim3(ew_blocks(total)), dim3(EW_THREADS), 0, s, sh, P, Q, sh.c,
                           (int)total, make_fdiv(sh.c), make_fdiv(Q), make_fdiv(P), x, y);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int avgpool_backward(const dc_pool_shape &sh, const float *dy, int accumulate, float *dx, hipStream_t s) {
    const int P = (sh.h + 2 * sh.pad - sh.r) / sh.stride + 1;
    const int Q = (sh.w + 2 * sh.pad - sh.s) / sh.stride + 1;
    const int64_t total = (int64_t)sh.n * sh.h * sh.w * sh.c;
    if (total <= 0)
        return DC_OK;
    if (total >= INT_MAX || (int64_t)sh.n * P * Q * sh.c >= INT_MAX)
        return fail(DC_EINVAL, "average pooling of %lld elements exceeds the 2^31 limit", (long long)total);
    if (sh.c % 4 == 0 && ((uintptr_t)dy & 15) == 0 && ((uintptr_t)dx & 15) == 0)
        hipLaunchKernelGGL(avgpool_bwd_kernel<4>, dim3(ew_blocks(total / 4)), dim3(EW_THREADS), 0, s, sh, P, Q,
                           sh.c / 4, (int)(total / 4), make_fdiv(sh.c / 4), make_fdiv(sh.w), make_fdiv(sh.h),
                           make_fdiv(sh.stride), dy, accumulate, dx);
    else
        hipLaunchKernelGGL(avgpool_bwd_kernel<1>, dim3(ew_blocks(total)), dim3(EW_THREADS), 0, s, sh, P, Q, sh.c,
                           (int)total, make_fdiv(sh.c), make_fdiv(sh.w), make_fdiv(sh.h), make_fdiv(sh.stride), dy,
                           accumulate, dx);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int gap_forward(int n, int hw, int c, const float *x, float *y, hipStream_t s) {
    int64_t total = (int64_t)n * c;
    if (total <= 0)
        return DC_OK;
    hipLaunchKernelGGL(gap_fwd_kernel, dim3(ew_blocks(total)), dim3(EW_THREADS), 0, s, n, hw, c, x, y);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int gap_backward(int n, int hw, int c, const float *dy, int accumulate, float *dx, hipStream_t s) {
    int64_t total = (int64_t)n * hw * c;
    if (total <= 0)
        return DC_OK;
    if (total < INT_MAX)
        hipLaunchKernelGGL(gap_bwd_kernel<true>, dim3(ew_blocks(total)), dim3(EW_THREADS), 0, s, n, hw, c, make_fdiv(c),
                           make_fdiv(hw), dy, accumulate, dx);
    else
        hipLaunchKernelGGL(gap_bwd_kernel<false>, dim3(ew_blocks(total)), dim3(EW_THREADS), 0, s, n, hw, c,
                           make_fdiv(c), make_fdiv(hw), dy, accumulate, dx);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

static int col_slots(int64_t rows, int c) { return std::max(col_plan(rows, c).nchunks, c % 4 == 0 ? col4_plan(rows, c).nchunks : 0); }

size_t colsum_ws_bytes(int64_t rows, int c) { return align256((size_t)col_slots(rows, c) * c * sizeof(float)); }

int colsum(int64_t rows, int c, const float *x, float *out, void *ws, hipStream_t s) {
    if (c <= 0)
        return DC_OK;
    if (rows <= 0) {
        DC_HIP(hipMemsetAsync(out, 0, sizeof(float) * c, s));
        return DC_OK;
    }
    float *part = static_cast<float *>(ws);
    int nchunks;
    if (col4_ok(c, x, part)) {
        Col4Plan p = col4_plan(rows, c);
        hipLaunchKernelGGL(colred4_partial_kernel<0>, dim3(p.nchunks, p.blocks), dim3(EW_THREADS), 0, s, rows, c,
                           p.rpc, p.g, p.rl_n, x, (const float *)nullptr, (const float *)nullptr,
                           (const float *)nullptr, part, (float *)nullptr, (const float *)nullptr);
        nchunks = p.nchunks;
    } else {
        ColPlan p = col_plan(rows, c);
        dim3 g1(p.nchunks, (c + CG - 1) / CG);
        hipLaunchKernelGGL(colred_partial_kernel<0>, g1, dim3(EW_THREADS), 0, s, rows, c, p.rows_per_chunk, x,
                           (const float *)nullptr, (const float *)nullptr, (const float *)nullptr, part,
                           (float *)nullptr, (const float *)nullptr);
        nchunks = p.nchunks;
    }
    DC_HIP(hipGetLastError());
    hipLaunchKernelGGL(colred_final_kernel<0>, dim3(c), dim3(EW_THREADS), 0, s, nchunks, c, rows, 0.f, part,
                       (const float *)nullptr, out, (float *)nullptr, (const float *)nullptr);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

size_t bn_ws_bytes(int64_t rows, int c) { return 2 * align256((size_t)col_slots(rows, c) * c * sizeof(float)); }

int bn_forward(int64_t rows, int c, const float *x, const float *gamma, const float *beta, float eps, int relu,
               float *y, float *mean, float *invstd, void *ws, hipStream_t s) {
    if (rows <= 0 || c <= 0)
        return DC_OK;
    float *part = static_cast<float *>(ws);
    float *part1 = reinterpret_cast<float *>(static_cast<char *>(ws) +
                                             align256((size_t)col_slots(rows, c) * c * sizeof(float)));
    if (col4_ok(c, x, y) && col4_ok(c, gamma, beta) && col4_ok(c, mean, invstd) && col4_ok(c, part, part1)) {
        // one statistics pass (shifted sums), then the normalisation: 12 bytes per element
        Col4Plan p = col4_plan(rows, c);
        hipLaunchKernelGGL(colred4_partial_kernel<1>, dim3(p.nchunks, p.blocks), dim3(EW_THREADS), 0, s, rows, c,
                           p.rpc, p.g, p.rl_n, x, (const float *)nullptr, (const float *)nullptr,
                           (const float *)nullptr, part, part1, (const float *)nullptr);
        DC_HIP(hipGetLastError());
        hipLaunchKernelGGL(colred_final_kernel<4>, dim3(c), dim3(EW_THREADS), 0, s, p.nchunks, c, rows, eps, part,
                           (const float *)part1, mean, invstd, x);
        DC_HIP(hipGetLastError());
        const int64_t n4 = rows * c / 4;
        hipLaunchKernelGGL(bn_apply4_kernel, dim3(bn4_blocks(n4, c / 4)), dim3(EW_THREADS), 0, s, n4, c / 4,
                           reinterpret_cast<const float4 *>(x), reinterpret_cast<const float4 *>(gamma),
                           reinterpret_cast<const float4 *>(beta), reinterpret_cast<const float4 *>(mean),
                           reinterpret_cast<const float4 *>(invstd), relu, reinterpret_cast<float4 *>(y));
        DC_HIP(hipGetLastError());
        return DC_OK;
    }
    ColPlan p = col_plan(rows, c);
    dim3 g1(p.nchunks, (c + CG - 1) / CG);
    hipLaunchKernelGGL(colred_partial_kernel<0>, g1, dim3(EW_THREADS), 0, s, rows, c, p.rows_per_chunk, x,
                       (const float *)nullptr, (const float *)nullptr, (const float *)nullptr, part, (float *)nullptr,
                       (const float *)nullptr);
    DC_HIP(hipGetLastError());
    hipLaunchKernelGGL(colred_final_kernel<1>, dim3(c), dim3(EW_THREADS), 0, s, p.nchunks, c, rows, eps, part,
                       (const float *)nullptr, mean, (float *)nullptr, (const float *)nullptr);
    DC_HIP(hipGetLastError());
    hipLaunchKernelGGL(colred_partial_kernel<1>, g1, dim3(EW_THREADS), 0, s, rows, c, p.rows_per_chunk, x,
                       (const float *)nullptr, (const float *)mean, (const float *)nullptr, part, (float *)nullptr,
                       (const float *)nullptr);
    DC_HIP(hipGetLastError());
    hipLaunchKernelGGL(colred_final_kernel<2>, dim3(c), dim3(EW_THREADS), 0, s, p.nchunks, c, rows, eps, part,
                       (const float *)nullptr, invstd, (float *)nullptr, (const float *)nullptr);
    DC_HIP(hipGetLastError());
    int64_t total = rows * c;
    hipLaunchKernelGGL(bn_apply_kernel, dim3(ew_blocks(total)), dim3(EW_THREADS), 0, s, rows, c, x, gamma, beta, mean,
                       invstd, relu, y);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int bn_backward(int64_t rows, int c, const float *dy, const float *x, const float *gamma, const float *mean,
                const float *invstd, int accumulate, float *dx, float *dgamma, float *dbeta, void *ws, hipStream_t s,
                const float *relu_y) {
    if (rows <= 0 || c <= 0)
        return DC_OK;
    float *part0 = static_cast<float *>(ws);
    float *part1 = reinterpret_cast<float *>(static_cast<char *>(ws) +
                                             align256((size_t)col_slots(rows, c) * c * sizeof(float)));
    const bool v4 = col4_ok(c, dy, x) && col4_ok(c, gamma, mean) && col4_ok(c, invstd, dgamma) &&
                    col4_ok(c, dbeta, part0) && col4_ok(c, part1) && (!dx || col4_ok(c, dx)) &&
                    (!relu_y || col4_ok(c, relu_y));
    int nchunks;
    if (v4) {
        Col4Plan p = col4_plan(rows, c);
        hipLaunchKernelGGL(colred4_partial_kernel<2>, dim3(p.nchunks, p.blocks), dim3(EW_THREADS), 0, s, rows, c,
                           p.rpc, p.g, p.rl_n, x, dy, mean, invstd, part0, part1, relu_y);
        nchunks = p.nchunks;
    } else {
        ColPlan p = col_plan(rows, c);
        dim3 g1(p.nchunks, (c + CG - 1) / CG);
        hipLaunchKernelGGL(colred_partial_kernel<2>, g1, dim3(EW_THREADS), 0, s, rows, c, p.rows_per_chunk, x, dy,
                           mean, invstd, part0, part1, relu_y);
        nchunks = p.nchunks;
    }
    DC_HIP(hipGetLastError());
    hipLaunchKernelGGL(colred_final_kernel<3>, dim3(c), dim3(EW_THREADS), 0, s, nchunks, c, rows, 0.f, part0,
                       (const float *)part1, dbeta, dgamma, (const float *)nullptr);
    DC_HIP(hipGetLastError());
    if (dx) {
        if (v4) {
            const int64_t n4 = rows * c / 4;
            hipLaunchKernelGGL(bn_bwd_apply4_kernel, dim3(bn4_blocks(n4, c / 4)), dim3(EW_THREADS), 0, s, n4, c / 4,
                               rows, reinterpret_cast<const float4 *>(dy), reinterpret_cast<const float4 *>(x),
                               reinterpret_cast<const float4 *>(gamma), reinterpret_cast<const float4 *>(mean),
                               reinterpret_cast<const float4 *>(invstd), reinterpret_cast<const float4 *>(dgamma),
                               reinterpret_cast<const float4 *>(dbeta), accumulate, reinterpret_cast<float4 *>(dx),
                               reinterpret_cast<const float4 *>(relu_y));
        } else {
            int64_t total = rows * c;
            hipLaunchKernelGGL(bn_bwd_apply_kernel, dim3(ew_blocks(total)), dim3(EW_THREADS), 0, s, rows, c, dy, x,
                               gamma, mean, invstd, dgamma, dbeta, accumulate, dx, relu_y);
        }
        DC_HIP(hipGetLastError());
    }
    return DC_OK;
}

size_t xent_ws_bytes(int n) { return align256((size_t)std::max(n, 1) * sizeof(float)); }

int softmax_xent(int n, int classes, const float *logits, const int32_t *labels, float *loss, float *dlogits,
                 void *ws, hipStream_t s) {
    if (n <= 0 || classes <= 0)
        return DC_OK;
    float *loss_i = static_cast<float *>(ws);
    hipLaunchKernelGGL(xent_row_kernel, dim3(n), dim3(EW_THREADS), 0, s, n, classes, logits, labels, loss_i, dlogits);
    DC_HIP(hipGetLastError());
    hipLaunchKernelGGL(xent_mean_kernel, dim3(1), dim3(64), 0, s, n, (const float *)loss_i, loss);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int pace_mark(uint64_t *slot, hipStream_t s) {
    hipLaunchKernelGGL(pace_mark_kernel, dim3(1), dim3(64), 0, s, slot);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int pace_until(const uint64_t *slot, uint64_t ticks, uint64_t cap_ticks, hipStream_t s) {
    hipLaunchKernelGGL(pace_until_kernel, dim3(1), dim3(64), 0, s, slot, ticks, cap_ticks);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int wall_clock_hz(double *hz) {
    int dev = 0;
    DC_HIP(hipGetDevice(&dev));
    int khz = 0;
    DC_HIP(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev));
    if (khz <= 0)
        return fail(DC_EHIP, "device reports no wall-clock rate");
    *hz = (double)khz * 1000.0;
    return DC_OK;
}

} // namespace dc
