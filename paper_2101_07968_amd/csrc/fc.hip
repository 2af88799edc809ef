// The data gradient of a large FC layer with few rows: a weight-streaming
// GEMM on gfx950 fp32 matrix cores.
//
// For an FC layer with weights W [O][I] and M <= 32 rows (the batch), the
// backward compute mini-procedure's data gradient (Sec. III-A)
//
//   dX[m][i] = sum_o dY[m][o] W[o][i]
//
// moves the O x I weights once and little else: 2 M flops per 4 weight
// bytes, near the balance point of HBM and the fp32 matrix cores.  This
// kernel streams W straight from HBM into registers, in rows of 512
// contiguous bytes per half-wave, with no LDS staging of the operands:
//
// * v_mfma_f32_32x32x2f32 takes, per lane l, one element of a 32 x 2 block
//   of A (row l % 32, k = l / 32) and of a 2 x 32 block of B (k = l / 32,
//   column l % 32).
// * Lane (j = l % 32, h = l / 32) holds dY[m = j][o + 4h .. +3] and
//   W[o + 4h + u][i + 4j .. +3] for u = 0..3.  Product (u, e) takes element u
//   of the dY quad and element e of the u-th W quad, so it adds row pair
//   (o + u, o + 4 + u) into the column set {i + 4j + e}: four accumulators
//   cover 128 contiguous columns, written back as float4.
// * Three register buffers form a ring, so the loads of the next two steps
//   are in flight while a step multiplies; operands are read with raw buffer
//   loads whose out-of-range offsets read as zero, which masks the ragged
//   edges without a branch around a load.
//
// * The four waves of a workgroup share one 128-column strip and take
//   interleaved groups of 8 rows, so a workgroup reads 32 consecutive rows of
//   the strip per round (measured on 25088 -> 4096 at 32 rows: 97 us, against
//   104 us with the waves on neighbouring strips); the waves' sums are then
//   added in wave order through LDS.
//
// The reduction over o is split over workgroups: fixed-slot partial sums,
// then a fixed-order reduction that applies a folded ReLU's mask and the
// accumulate flag, so results are deterministic.
//
// The forward pass of such a layer has its own kernel here too:
// Y[m][o] = sum_i X[m][i] W[o][i] reduces along the weight rows, so lanes
// cannot read W straight into MFMA operands with coalesced loads.  A
// workgroup stages a 128-row x 32-column block of W (rows of 128 contiguous
// bytes per 8 lanes) and the 32 x 32 block of X in LDS, double buffered, and
// each wave multiplies 32 rows of X by 32 rows of W.  The implicit GEMM's
// smallest tile has 64 rows, so at M <= 32 half of its matrix work multiplied
// zero rows.  Split over i into fixed slots, then a fixed-order reduction
// adds the bias and applies the ReLU.  The filter gradient stays on the
// implicit GEMM: a register-operand kernel writing 32 x 128 blocks of dW ran
// VGG-16's 25088 -> 4096 layer in 131 us against its 102.
#include "dc_internal.h"

#include <algorithm>
#include <climits>

namespace dc {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int WAVES = 4;              // waves per workgroup
constexpr int TARGET_WGS = 1152;      // data gradient: about 4.5 workgroups of 4 waves per CU
constexpr unsigned OOB = 0x80000000u; // a byte offset that reads as zero
constexpr int64_t FWD_MIN = 16000000; // weights from which the forward kernel runs

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const float *p, int64_t elems) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p), (short)0, (int)(4 * elems), 0x00020000);
}

__device__ __forceinline__ float4 ld4_sel(__amdgpu_buffer_rsrc_t r, int64_t elem, bool ok) {
    return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, ok ? (unsigned)(4 * elem) : OOB, 0, 0));
}

__device__ __forceinline__ float ld_sel(__amdgpu_buffer_rsrc_t r, int64_t elem, bool ok) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, ok ? (unsigned)(4 * elem) : OOB, 0, 0));
}

__device__ __forceinline__ float el(const float4 &v, int e) {
    return e == 0 ? v.x : (e == 1 ? v.y : (e == 2 ? v.z : v.w));
}

// One workgroup: columns i0 .. i0+127 for rows 0 .. M-1 (M <= 32), over the o
// range of split `sp` (ochunk rows, a multiple of 96).  The o range is taken
// in rounds of 32 rows, wave w reading rows 8w .. 8w+7 of each round, so the
// four waves stream one 512-byte strip of 32 consecutive weight rows; their
// sums are added in wave order through LDS.  partial[sp][m][i].
__global__ __launch_bounds__(64 * WAVES) void fc_dgrad_kernel(const float *__restrict__ dY,
                                                              const float *__restrict__ W,
                                                              float *__restrict__ partial, int M, int I, int O,
                                                              int tiles_i, int ochunk) {
    __shared__ float red[64 * 64];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, j = lane & 31, h = lane >> 5;
    const int tile = blockIdx.x % tiles_i, sp = blockIdx.x / tiles_i;
    const int i = tile * 128 + 4 * j;
    const bool iok = i < I;
    const int ob = sp * ochunk, oe = min(O, ob + ochunk);
    f32x16 acc[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
        acc[e] = f32x16{};
    const __amdgpu_buffer_rsrc_t rw = rsrc(W, (int64_t)O * I), ra = rsrc(dY, (int64_t)M * O);
    const bool aok = j < M;
    const int64_t arow = (int64_t)j * O;
    // dY rows are read as float4 only when O % 4 == 0; else element by element
    const bool a4 = O % 4 == 0;
    struct Buf {
        float4 w[4], a;
    };
    auto load = [&](Buf &b, int o0) {
        const int oa = o0 + 8 * wave + 4 * h;
#pragma unroll
        for (int u = 0; u < 4; ++u)
            b.w[u] = ld4_sel(rw, (int64_t)(oa + u) * I + i, iok && oa + u < oe);
        if (a4) {
            b.a = ld4_sel(ra, arow + oa, aok && oa < oe);
        } else {
            float t[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                t[u] = ld_sel(ra, arow + oa + u, aok && oa + u < oe);
            b.a = make_float4(t[0], t[1], t[2], t[3]);
        }
    };
    auto step = [&](const Buf &b) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                acc[e] = __builtin_amdgcn_mfma_f32_32x32x2f32(el(b.a, u), el(b.w[u], e), acc[e], 0, 0, 0);
    };
    // rounds past oe load zeros and add nothing
    Buf b0, b1, b2;
    load(b0, ob);
    load(b1, ob + 32);
    for (int o0 = ob; o0 < oe; o0 += 96) {
        load(b2, o0 + 64);
        step(b0);
        load(b0, o0 + 96);
        step(b1);
        load(b1, o0 + 128);
        step(b2);
    }
    // the waves in order: red = ((w0 + w1) + w2) + w3, element by element
    for (int wv = 0; wv < WAVES; ++wv) {
        if (wave == wv)
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    float &r = red[(e * 16 + v) * 64 + lane];
                    r = wv == 0 ? acc[e][v] : r + acc[e][v];
                }
        __syncthreads();
    }
    if (!iok)
        return;
    // element v of lane l is row 8*(v/4) + 4*(l/32) + v%4 of a 32 x 32 block;
    // wave w writes the rows of v = 4w .. 4w+3
    float *dst = partial + (size_t)sp * M * I;
#pragma unroll
    for (int vv = 0; vv < 4; ++vv) {
        const int v = 4 * wave + vv;
        const int m = 8 * (v >> 2) + 4 * h + (v & 3);
        if (m < M)
            *reinterpret_cast<float4 *>(dst + (size_t)m * I + i) =
                make_float4(red[(0 * 16 + v) * 64 + lane], red[(1 * 16 + v) * 64 + lane],
                            red[(2 * 16 + v) * 64 + lane], red[(3 * 16 + v) * 64 + lane]);
    }
}

// dX[m][i] (+)= (mask?) sum over splits in order of partial[s][m][i]; a
// float4 of columns per thread (I % 4 == 0).
__global__ __launch_bounds__(256) void fc_dgrad_reduce_kernel(const float4 *__restrict__ partial, int splits,
                                                              int64_t n4, const float4 *__restrict__ relu_mask,
                                                              int accumulate, float4 *__restrict__ dX) {
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n4;
         idx += (int64_t)gridDim.x * blockDim.x) {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int s = 0; s < splits; ++s) {
            const float4 p = partial[(size_t)s * n4 + idx];
            v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
        }
        if (relu_mask) {
            const float4 r = relu_mask[idx];
            if (!(r.x > 0.f)) v.x = 0.f;
            if (!(r.y > 0.f)) v.y = 0.f;
            if (!(r.z > 0.f)) v.z = 0.f;
            if (!(r.w > 0.f)) v.w = 0.f;
        }
        if (accumulate) {
            const float4 d = dX[idx];
            v.x += d.x; v.y += d.y; v.z += d.z; v.w += d.w;
        }
        dX[idx] = v;
    }
}

constexpr int FKT = 32;            // forward: i per LDS stage
constexpr int FOT = 128;           // forward: o per workgroup
constexpr int FLD = FKT + 4;       // forward: LDS row stride in floats (conflict-free b128 reads)

// Forward partial sums: workgroup (tile, sp) takes o in [128 tile, +128) and
// i in [sp chunk, +chunk) (chunk a multiple of FKT); partial[sp][m][o].
__global__ __launch_bounds__(256) void fc_fwd_kernel(const float *__restrict__ X, const float *__restrict__ W,
                                                     float *__restrict__ partial, int M, int I, int O, int tiles_o,
                                                     int chunk) {
    __shared__ float sw[2][FOT * FLD];
    __shared__ float sx[2][32 * FLD];
    const int t = threadIdx.x, wave = t >> 6, lane = t & 63, h = lane >> 5, col = lane & 31;
    const int tile = blockIdx.x % tiles_o, sp = blockIdx.x / tiles_o;
    const int o0 = tile * FOT, ib = sp * chunk, ie = min(I, ib + chunk);
    const __amdgpu_buffer_rsrc_t rw = rsrc(W, (int64_t)O * I), rx = rsrc(X, (int64_t)M * I);
    // stage loads: W rows t / 8 + 32 q, X row t / 8; 4 columns at 4 (t % 8)
    const int lr = t >> 3, lc = 4 * (t & 7);
    float4 gw[4], gx;
    auto gload = [&](int i0) {
        const int i = i0 + lc;
        const bool iok = i < ie;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int row = o0 + lr + 32 * q;
            gw[q] = ld4_sel(rw, (int64_t)row * I + i, iok & (row < O));
        }
        gx = ld4_sel(rx, (int64_t)lr * I + i, iok & (lr < M));
    };
    auto sstore = [&](int b) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            *reinterpret_cast<float4 *>(&sw[b][(lr + 32 * q) * FLD + lc]) = gw[q];
        *reinterpret_cast<float4 *>(&sx[b][lr * FLD + lc]) = gx;
    };
    f32x16 acc = f32x16{};
    const int nst = ie > ib ? (ie - ib + FKT - 1) / FKT : 0;
    gload(ib);
    sstore(0);
    __syncthreads();
    for (int s = 0; s < nst; ++s) {
        const int b = s & 1;
        gload(ib + (s + 1) * FKT); // past ie every load reads zero
        const float *wrow = &sw[b][(32 * wave + col) * FLD + 4 * h];
        const float *xrow = &sx[b][col * FLD + 4 * h];
#pragma unroll
        for (int g = 0; g < FKT / 8; ++g) {
            // lane half h holds i = 8 g + 4 h + u: A = X[m = col][i], B = W[o = col][i]
            const float4 wv = *reinterpret_cast<const float4 *>(wrow + 8 * g);
            const float4 xv = *reinterpret_cast<const float4 *>(xrow + 8 * g);
#pragma unroll
            for (int u = 0; u < 4; ++u)
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(el(xv, u), el(wv, u), acc, 0, 0, 0);
        }
        sstore(b ^ 1);
        __syncthreads();
    }
    // element v of lane l: m = 8 (v / 4) + 4 h + v % 4, o = o0 + 32 wave + col
    const int o = o0 + 32 * wave + col;
    float *dst = partial + (size_t)sp * M * O;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const int m = 8 * (v >> 2) + 4 * h + (v & 3);
        if (m < M && o < O)
            dst[(size_t)m * O + o] = acc[v];
    }
}

// Y[m][o] = (ReLU) bias[o] + sum over splits in order of partial[s][m][o];
// a float4 of o per thread (O % 4 == 0).
__global__ __launch_bounds__(256) void fc_fwd_reduce_kernel(const float4 *__restrict__ partial, int splits,
                                                            int64_t n4, int o4, const float4 *__restrict__ bias,
                                                            int relu, float4 *__restrict__ Y) {
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n4;
         idx += (int64_t)gridDim.x * blockDim.x) {
        float4 v = bias ? bias[idx % o4] : make_float4(0.f, 0.f, 0.f, 0.f);
        for (int s = 0; s < splits; ++s) {
            const float4 p = partial[(size_t)s * n4 + idx];
            v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
        }
        if (relu) {
            v.x = fmaxf(v.x, 0.f); v.y = fmaxf(v.y, 0.f); v.z = fmaxf(v.z, 0.f); v.w = fmaxf(v.w, 0.f);
        }
        Y[idx] = v;
    }
}

} // namespace

bool fc_streaming(const ConvGeom &g, int pass) {
    const bool fc = g.H == 1 && g.W == 1 && g.R == 1 && g.S == 1 && g.st == 1 && g.pad == 0 && g.pad_w == 0;
    if (!fc || g.N < 1 || g.N > 32 || g.C % 4 != 0)
        return false;
    // every operand is read through 32-bit byte offsets, offsets from 2^31 up
    // reading as zero: each below 2^31 bytes (with the data gradient ring's 32
    // rows past the end), as are the partial sums
    const int64_t lim = (int64_t)1 << 31;
    if (4 * ((int64_t)g.K + 32) * g.C >= lim || 4 * (int64_t)g.N * std::max(g.C, g.K) * 64 >= lim)
        return false;
    const int64_t weights = (int64_t)g.K * g.C;
    // Measured on MI355X against the implicit GEMM's plans (VGG-16's and
    // AlexNet's FC layers at 32 rows): the streaming data gradient wins from
    // about 4 M weights (25088 -> 4096: 97 against 133 us); the forward from
    // about 16 M (25088 -> 4096: 97 against 119 us, 9216 -> 4096: 39 against
    // 51, 4096 -> 4096: 25 against 28.5) and loses below (4096 -> 1000: 28
    // against 14).
    if (pass == PASS_DGRAD)
        return weights >= 4000000;
    if (pass == PASS_FWD)
        return g.K % 4 == 0 && weights >= FWD_MIN;
    return false;
}

// Data gradient: splits of the reduction over o, about TARGET_WGS workgroups
// in chunks of 96 rows (the ring's three rounds of 32), while the partial sums
// (splits x M x I) stay within a quarter of the weight bytes.  Forward: about 768
// workgroups (three per CU), splits of the reduction over i in whole LDS
// stages.
void fc_plan(const ConvGeom &g, int pass, int splits_out[1], int *chunk, size_t *ws_bytes) {
    const int64_t M = g.N, I = g.C, O = g.K;
    if (pass == PASS_FWD) {
        const int64_t tiles = (O + FOT - 1) / FOT, stages = (I + FKT - 1) / FKT;
        const int64_t s = std::min<int64_t>(stages, std::max<int64_t>(1, (768 + tiles - 1) / tiles));
        const int64_t per = (stages + s - 1) / s;
        *chunk = (int)(per * FKT);
        splits_out[0] = (int)((stages + per - 1) / per);
        *ws_bytes = (size_t)splits_out[0] * M * O * sizeof(float);
        return;
    }
    const int64_t tiles = (I + 127) / 128;
    const int64_t steps = (O + 95) / 96;
    int64_t s = std::max<int64_t>(1, (TARGET_WGS + tiles - 1) / tiles);
    s = std::min<int64_t>(s, std::max<int64_t>(1, O / (4 * M)));
    s = std::min<int64_t>(s, steps);
    const int64_t per = (steps + s - 1) / s;
    *chunk = (int)(per * 96);
    splits_out[0] = (int)((steps + per - 1) / per);
    *ws_bytes = (size_t)splits_out[0] * M * I * sizeof(float);
}

int fc_forward(const ConvGeom &g, int splits, int chunk, const float *x, const float *w, const float *bias, int relu,
               float *y, void *ws, hipStream_t s) {
    const int M = g.N, I = g.C, O = g.K;
    if (!ws)
        return fail(DC_EINVAL, "FC forward needs a workspace");
    float *partial = static_cast<float *>(ws);
    const int tiles = (O + FOT - 1) / FOT;
    hipLaunchKernelGGL(fc_fwd_kernel, dim3(tiles * splits), dim3(256), 0, s, x, w, partial, M, I, O, tiles, chunk);
    DC_HIP(hipGetLastError());
    const int64_t n4 = (int64_t)M * O / 4;
    hipLaunchKernelGGL(fc_fwd_reduce_kernel, dim3((int)std::min<int64_t>((n4 + 255) / 256, 4096)), dim3(256), 0, s,
                       reinterpret_cast<const float4 *>(partial), splits, n4, O / 4,
                       reinterpret_cast<const float4 *>(bias), relu, reinterpret_cast<float4 *>(y));
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int fc_dgrad(const ConvGeom &g, int splits, int chunk, const float *dy, const float *w, int accumulate, float *dx,
             void *ws, hipStream_t s, const float *relu_mask) {
    const int M = g.N, I = g.C, O = g.K;
    if (!ws)
        return fail(DC_EINVAL, "FC dgrad needs a workspace");
    float *partial = static_cast<float *>(ws);
    const int tiles = (I + 127) / 128;
    hipLaunchKernelGGL(fc_dgrad_kernel, dim3(tiles * splits), dim3(64 * WAVES), 0, s, dy, w, partial, M, I, O, tiles,
                       chunk);
    DC_HIP(hipGetLastError());
    const int64_t n4 = (int64_t)M * I / 4;
    hipLaunchKernelGGL(fc_dgrad_reduce_kernel, dim3((int)std::min<int64_t>((n4 + 255) / 256, 4096)), dim3(256), 0,
                       s, reinterpret_cast<const float4 *>(partial), splits, n4,
                       reinterpret_cast<const float4 *>(relu_mask), accumulate, reinterpret_cast<float4 *>(dx));
    DC_HIP(hipGetLastError());
    return DC_OK;
}

} // namespace dc
