// Direct convolution for the RGB input layer: three input channels and a
// 3 x 3 filter, forward pass and filter gradient on gfx950 fp32 matrix cores
// without LDS staging.
//
// With C = 3 the forward and filter-gradient GEMMs of Sec. III-A have a
// reduction depth of only R*S*C = 27.  The implicit GEMM must pad the
// channels to 4 (a third more work, plus padded copies of the input), and
// its tiles spend most of their time in prologue and epilogue.  Here each
// wave builds its MFMA operands straight from global memory:
//
// * v_mfma_f32_32x32x2f32 takes, per lane l, one element of a 32 x 2 block of
//   A (row l % 32, k = l / 32) and of a 2 x 32 block of B (k = l / 32,
//   column l % 32); element v of the 32 x 32 result in lane l is row
//   8 (v / 4) + 4 (l / 32) + v % 4, column l % 32.
// * Forward, Y[pixel][k] = sum_t X[pixel][t] W[k][t]: a wave takes 32 output
//   pixels, lane l the pixel l % 32, whose 27 inputs are nine 12-byte raw
//   buffer loads (out-of-image offsets read as zero: the padding).  The taps
//   are consumed two per MFMA (the 28th is zero); the weights sit in
//   registers, 14 per lane and 32-channel block.  The next tile's loads are
//   issued before the current tile's MFMAs.
// * Filter gradient, dW[k][t] = sum_pixel dY[pixel][k] X[pixel][t] and
//   db[k] = sum_pixel dY[pixel][k]: the reduction runs over pixels, two per
//   MFMA; lane l reads dY of its channel l % 32 and X of its tap l % 32, and
//   tap 27 reads 1 for a live pixel, so the bias gradient comes out of the
//   same products.  The four waves of a workgroup are added in wave order
//   through LDS, each workgroup writes its partial sums to a fixed slot, and
//   a second kernel adds the slots in order: results are deterministic.
#include "dc_internal.h"

#include <algorithm>

namespace dc {
namespace {

typedef float f3v __attribute__((ext_vector_type(3)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int NT = 256;                 // 4 waves
constexpr int TAPS = 27;                // 3 x 3 x 3
constexpr int PER_K = TAPS + 1;         // partial sums per channel: 27 weight taps, then the bias
constexpr unsigned OOB = 0x80000000u;   // a byte offset that reads as zero
constexpr int WGRAD_WGS = 1024;         // filter-gradient workgroups (partial slots)
constexpr int FWD_WGS = 2048;

struct Geo {
    int N, H, W, K, st, pad, pad_w, P, Q;
    int64_t npq; // output pixels N * P * Q
    int64_t per; // filter gradient: output pixels per workgroup, a multiple of 128
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const float *p, int64_t elems) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p), (short)0, (int)(4 * elems), 0x00020000);
}

// Position of one output pixel.
struct Pix {
    int n, p, q;
};

// (pixel indices fit in 32 bits: conv3_direct bounds N P Q K below 2^29)
__device__ __forceinline__ Pix pix_at(const Geo &g, int64_t i) {
    Pix x;
    const int pq = g.P * g.Q, ii = (int)i;
    x.n = ii / pq;
    const int r = ii - x.n * pq;
    x.p = r / g.Q;
    x.q = r - x.p * g.Q;
    return x;
}

// Two pixels on, without a loop or branch (Q >= 2, so the column wraps at
// most once).
__device__ __forceinline__ void pix_step2(const Geo &g, Pix &x) {
    x.q += 2;
    const bool wq = x.q >= g.Q;
    x.q = wq ? x.q - g.Q : x.q;
    x.p += wq ? 1 : 0;
    const bool wp = x.p == g.P;
    x.p = wp ? 0 : x.p;
    x.n += wp ? 1 : 0;
}

// The nine 3-channel input pixels under output pixel i (zeros outside the
// image, and everywhere when !live).
// Offsets are formed with selects (bitwise conditions, no short-circuit), so
// no branch separates a load from the next and the loads stay in flight.
__device__ __forceinline__ void gather(const Geo &g, __amdgpu_buffer_rsrc_t rx, int64_t i, bool live, f3v xs[9]) {
    const Pix x = pix_at(g, live ? i : 0);
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int s = 0; s < 3; ++s) {
            const int ih = x.p * g.st - g.pad + r, iw = x.q * g.st - g.pad_w + s;
            const bool ok = live & (ih >= 0) & (ih < g.H) & (iw >= 0) & (iw < g.W);
            const int e = (x.n * g.H + ih) * g.W + iw;
            const unsigned off = ok ? (unsigned)(12 * e) : OOB;
            xs[r * 3 + s] = __builtin_bit_cast(f3v, __builtin_amdgcn_raw_buffer_load_b96(rx, off, 0, 0));
        }
}

// Tap t (< 28) of a gathered pixel; tap 27 is the zero padding of the depth.
__device__ __forceinline__ float tap_of(const f3v xs[9], int t) { return t < TAPS ? xs[t / 3][t % 3] : 0.f; }

// Forward: NB blocks of 32 output channels (K = 32 NB).  Each wave walks
// 32-pixel tiles with a stride of all waves of the grid.
template <int NB>
__global__ __launch_bounds__(NT) void conv3_fwd_kernel(Geo g, const float *__restrict__ x,
                                                       const float *__restrict__ w,
                                                       const float *__restrict__ bias, int relu,
                                                       float *__restrict__ y) {
    const int lane = threadIdx.x & 63, h = lane >> 5, col = lane & 31;
    const int64_t tiles = (g.npq + 31) / 32, stride = (int64_t)gridDim.x * (NT / 64);
    int64_t tile = (int64_t)blockIdx.x * (NT / 64) + (threadIdx.x >> 6);
    if (tile >= tiles)
        return; // the whole wave; this kernel has no barrier
    // B operand: W[k = 32 blk + col][t = 2 i + h]
    float wb[NB][14], bv[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
#pragma unroll
        for (int i = 0; i < 14; ++i)
            wb[b][i] = 2 * i + h < TAPS ? w[(32 * b + col) * TAPS + 2 * i + h] : 0.f;
        bv[b] = bias ? bias[32 * b + col] : 0.f;
    }
    const __amdgpu_buffer_rsrc_t rx = rsrc(x, (int64_t)g.N * g.H * g.W * 3);
    f3v xs[9];
    gather(g, rx, tile * 32 + col, tile * 32 + col < g.npq, xs);
    while (tile < tiles) {
        const int64_t next = tile + stride;
        f3v xn[9];
        gather(g, rx, next * 32 + col, next * 32 + col < g.npq, xn);
        f32x16 acc[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                acc[b][v] = bv[b];
#pragma unroll
        for (int i = 0; i < 14; ++i) {
            // A operand: X[pixel = col][t = 2 i + h]
            const float a = h ? tap_of(xs, 2 * i + 1) : tap_of(xs, 2 * i);
#pragma unroll
            for (int b = 0; b < NB; ++b)
                acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, wb[b][i], acc[b], 0, 0, 0);
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int64_t pix = tile * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
            if (pix < g.npq) {
                float *dst = y + pix * g.K + col;
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    dst[32 * b] = relu ? fmaxf(acc[b][v], 0.f) : acc[b][v];
            }
        }
        tile = next;
#pragma unroll
        for (int t = 0; t < 9; ++t)
            xs[t] = xn[t];
    }
}

// Filter gradient, K = 32 NB: workgroup b takes pixels [b per, (b + 1) per),
// wave w the 32-pixel chunks w, w + 4, ... of that range.
template <int NB>
__global__ __launch_bounds__(NT) void conv3_wgrad_kernel(Geo g, const float *__restrict__ x,
                                                         const float *__restrict__ dy, float *__restrict__ part) {
    __shared__ float red[NB * 16 * 64];
    const int lane = threadIdx.x & 63, h = lane >> 5, col = lane & 31, wave = threadIdx.x >> 6;
    const __amdgpu_buffer_rsrc_t rx = rsrc(x, (int64_t)g.N * g.H * g.W * 3), rd = rsrc(dy, g.npq * g.K);
    // this lane's tap: (r, s, c) of t = col < 27; t = 27 reads 1 for a live pixel
    const int t = col, tr = t / 9, ts = (t / 3) % 3, tc = t % 3;
    // pixel indices fit in 32 bits (conv3_direct)
    const int lo = (int)min((int64_t)blockIdx.x * g.per, g.npq), hi = (int)min(g.npq, (int64_t)lo + g.per);
    f32x16 acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b)
        acc[b] = f32x16{};
    // operands of one 32-pixel chunk: pixel c0 + 2 i + h for i < 16
    struct Ops {
        float a[NB][16], bx[16];
    };
    auto load = [&](Ops &o, int c0) {
        const int i0 = c0 + h;
        Pix px = pix_at(g, i0 < hi ? i0 : lo);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int pix = c0 + 2 * i + h;
            const bool live = pix < hi;
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const unsigned off = live ? (unsigned)(4 * (pix * g.K + 32 * b + col)) : OOB;
                o.a[b][i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rd, off, 0, 0));
            }
            const int ih = px.p * g.st - g.pad + tr, iw = px.q * g.st - g.pad_w + ts;
            const bool ok = live & (t < TAPS) & (ih >= 0) & (ih < g.H) & (iw >= 0) & (iw < g.W);
            const int e = ((px.n * g.H + ih) * g.W + iw) * 3 + tc;
            const unsigned off = ok ? (unsigned)(4 * e) : OOB;
            // tap 27 reads zero and adds 1 for a live pixel: the bias gradient
            o.bx[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rx, off, 0, 0)) +
                      ((t == TAPS) & live ? 1.f : 0.f);
            pix_step2(g, px);
        }
    };
    int c0 = lo + 32 * wave;
    if (c0 < hi) {
        Ops cur, nxt;
        load(cur, c0);
        while (c0 < hi) {
            const int c1 = c0 + 32 * (NT / 64);
            load(nxt, c1); // past hi every load reads zero
#pragma unroll
            for (int i = 0; i < 16; ++i)
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(cur.a[b][i], cur.bx[i], acc[b], 0, 0, 0);
            c0 = c1;
            cur = nxt;
        }
    }
    // the waves in wave order
    for (int wv = 0; wv < NT / 64; ++wv) {
        if (wave == wv)
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    float &r = red[(b * 16 + v) * 64 + lane];
                    r = wv == 0 ? acc[b][v] : r + acc[b][v];
                }
        __syncthreads();
    }
    // slot layout [k][28]: k = 32 b + row (v, lane / 32), tap = lane % 32 < 28
    float *dst = part + (int64_t)blockIdx.x * g.K * PER_K;
    for (int e = threadIdx.x; e < NB * 16 * 64; e += NT) {
        const int l = e & 63, v = (e >> 6) & 15, b = e >> 10;
        const int tap = l & 31;
        if (tap < PER_K)
            dst[(32 * b + 8 * (v >> 2) + 4 * (l >> 5) + (v & 3)) * PER_K + tap] = red[e];
    }
}

// dw[k][t] = sum over slots in order of part[slot][k][t]; db[k] likewise from
// t = 27.  16 lanes per output, each adding every 16th slot, then the lanes
// in lane order.
__global__ __launch_bounds__(NT) void conv3_wgrad_reduce_kernel(const float *__restrict__ part, int slots, int K,
                                                                float *__restrict__ dw, float *__restrict__ db) {
    const int lane = threadIdx.x & 15;
    const int e = blockIdx.x * (NT / 16) + (threadIdx.x >> 4);
    const int n = K * PER_K;
    float s = 0.f;
    if (e < n)
        for (int i = lane; i < slots; i += 16)
            s += part[(int64_t)i * n + e];
    float v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i)
        v[i] = __shfl(s, (int)((threadIdx.x & 63) & ~15u) + i, 64);
    if (lane != 0 || e >= n)
        return;
    float t = v[0];
#pragma unroll
    for (int i = 1; i < 16; ++i)
        t += v[i];
    const int k = e / PER_K, tap = e - k * PER_K;
    if (tap < TAPS)
        dw[k * TAPS + tap] = t;
    else if (db)
        db[k] = t;
}

Geo geo_of(const ConvGeom &g, int wgs) {
    Geo o;
    o.N = g.N; o.H = g.H; o.W = g.W; o.K = g.K; o.st = g.st; o.pad = g.pad; o.pad_w = g.pad_w; o.P = g.P; o.Q = g.Q;
    o.npq = (int64_t)g.N * g.P * g.Q;
    o.per = ((o.npq + wgs - 1) / wgs + 127) / 128 * 128;
    return o;
}

int64_t tiles_of(const ConvGeom &g) { return ((int64_t)g.N * g.P * g.Q + 31) / 32; }

int fwd_wgs(const ConvGeom &g) { return (int)std::min<int64_t>(FWD_WGS, (tiles_of(g) + 3) / 4); }

// at least 4 chunks of 32 pixels per workgroup
int wgrad_wgs(const ConvGeom &g) { return (int)std::max<int64_t>(1, std::min<int64_t>(WGRAD_WGS, tiles_of(g) / 16)); }

template <typename F>
void by_blocks(int K, F &&f) {
    switch (K / 32) {
    case 1: f(std::integral_constant<int, 1>{}); break;
    case 2: f(std::integral_constant<int, 2>{}); break;
    case 3: f(std::integral_constant<int, 3>{}); break;
    default: f(std::integral_constant<int, 4>{}); break;
    }
}

} // namespace

bool conv3_direct(const ConvGeom &g, int pass) {
    if (pass != PASS_FWD && pass != PASS_WGRAD)
        return false;
    if (g.C != 3 || g.R != 3 || g.S != 3 || g.K % 32 != 0 || g.K < 32 || g.K > 128 || g.P < 1 || g.Q < 2)
        return false;
    // byte offsets into x and dy are 32-bit, offsets from 2^31 up reading as zero
    const int64_t lim = (int64_t)1 << 31;
    return 12 * (int64_t)g.N * g.H * g.W < lim && 4 * (int64_t)g.N * g.P * g.Q * g.K < lim;
}

size_t conv3_ws_bytes(const ConvGeom &g, int pass) {
    return pass == PASS_WGRAD ? (size_t)wgrad_wgs(g) * g.K * PER_K * sizeof(float) : 0;
}

int conv3_forward(const ConvGeom &g, const float *x, const float *w, const float *bias, int relu, float *y,
                  hipStream_t s) {
    const int wgs = fwd_wgs(g);
    const Geo geo = geo_of(g, wgs);
    by_blocks(g.K, [&](auto nb) {
        hipLaunchKernelGGL((conv3_fwd_kernel<decltype(nb)::value>), dim3(wgs), dim3(NT), 0, s, geo, x, w, bias, relu,
                           y);
    });
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int conv3_wgrad(const ConvGeom &g, const float *x, const float *dy, float *dw, float *dbias, void *ws,
                hipStream_t s) {
    if (!ws)
        return fail(DC_EINVAL, "the RGB-layer filter gradient needs a workspace");
    const int wgs = wgrad_wgs(g);
    const Geo geo = geo_of(g, wgs);
    float *part = static_cast<float *>(ws);
    by_blocks(g.K, [&](auto nb) {
        hipLaunchKernelGGL((conv3_wgrad_kernel<decltype(nb)::value>), dim3(wgs), dim3(NT), 0, s, geo, x, dy, part);
    });
    DC_HIP(hipGetLastError());
    const int n = g.K * PER_K;
    hipLaunchKernelGGL(conv3_wgrad_reduce_kernel, dim3((n + NT / 16 - 1) / (NT / 16)), dim3(NT), 0, s,
                       (const float *)part, wgs, g.K, dw, dbias);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

} // namespace dc
