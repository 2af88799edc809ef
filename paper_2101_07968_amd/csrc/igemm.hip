// Convolution and FC layers as implicit GEMM on gfx950 fp32 matrix cores.
//
// The forward and backward compute mini-procedures of a conv or FC layer
// (Sec. III-A) are three GEMMs over the NHWC activations and KRSC filters:
//
//   forward  Y[m][k]  = sum_kk X~[m][kk] W[k][kk]     m = (n,p,q), kk = (r,s,c)
//   dgrad    dX[m][c] = sum_kk dY~[m][kk] W~[kk][c]   m = (n,h,w) in one stride phase,
//                                                      kk = (tap r, tap s, k)
//   wgrad    dW[k][kk] = sum_m dY[m][k] X~[m][kk]     m = (n,p,q), kk = (r,s,c)
//
// where ~ marks an operand gathered on the fly (no im2col buffer).  For a
// strided convolution, output rows h with the same residue modulo the stride
// see the same filter taps, so dgrad runs one GEMM per residue pair ("phase")
// holding only the taps that hit; no structurally zero products are formed.
//
// One kernel template serves all three passes.  A workgroup of 256 threads
// (4 waves of 64) owns an MT x NT output tile; each wave owns a quarter and
// issues v_mfma_f32_32x32x2f32.  Operand tiles of depth KT are staged through
// LDS in the layout of their contiguous global dimension (float4 loads,
// ds_write_b128), double buffered with one barrier per K step; the next
// step's global loads are in flight while the current step multiplies.
// Split-K writes fixed-position partial sums that a second kernel adds in a
// fixed order, so every result is deterministic.  Workgroup ids are remapped
// so that consecutive tiles land on the same XCD and share its L2.
#include "dc_internal.h"

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>
#include <type_traits>

namespace dc {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int NTHR = 256;
constexpr int PADK = 4;  // padding of k-contiguous LDS rows (floats)
constexpr int PADR = 4;  // padding of row-contiguous LDS rows (floats)

struct Args {
    int N, H, W, C, K, R, S, st, pad, pad_w, P, Q;
    int M, Ng, Kg;          // FWD / WGRAD sizes; DGRAD: maxima over phases
    int tiles_m, tiles_n, tiles;
    int splits, kt_per_split, phases;
    const float *A;         // FWD: x   DGRAD: dy   WGRAD: dy
    const float *B;         // FWD: w   DGRAD: w    WGRAD: x
    float *out;             // FWD: y   DGRAD: dx   WGRAD: dw
    const float *bias;      // FWD only, may be null
    float *partial;         // split-K scratch
    int relu, accumulate;
    FDiv fC, fS, fK, fQ, fPQ;
    unsigned a_bytes, b_bytes; // sizes of A and B (lean mode: each below 2^31)
    const float *relu_mask;    // DGRAD, may be null: zero dx where this tensor (laid out like dx) is not > 0
};

// Per-phase geometry of dgrad (stride residues rh, rw).
struct Phase {
    int Hh, Wh;     // output rows / cols of this residue
    int Rt, St;     // filter taps that reach them
    int r0, s0;     // first tap
    int dh, dw;     // p = i + dh - tr, q = j + dw - ts
    int M, Kg;
    FDiv fW, fHW;   // stride > 1: division by Wh and by Hh * Wh
};

__device__ __forceinline__ Phase make_phase(const Args &a, int z) {
    Phase ph;
    int rh = z / a.st, rw = z % a.st;
    ph.Hh = a.H > rh ? (a.H - rh + a.st - 1) / a.st : 0;
    ph.Wh = a.W > rw ? (a.W - rw + a.st - 1) / a.st : 0;
    ph.r0 = (rh + a.pad) % a.st;
    ph.s0 = (rw + a.pad_w) % a.st;
    ph.Rt = ph.r0 < a.R ? (a.R - ph.r0 + a.st - 1) / a.st : 0;
    ph.St = ph.s0 < a.S ? (a.S - ph.s0 + a.st - 1) / a.st : 0;
    ph.dh = (rh + a.pad - ph.r0) / a.st;
    ph.dw = (rw + a.pad_w - ph.s0) / a.st;
    ph.M = a.N * ph.Hh * ph.Wh;
    ph.Kg = ph.Rt * ph.St * a.K;
    if (a.st > 1) { // out_row decodes rows of this phase
        ph.fW = make_fdiv((uint32_t)ph.Wh);
        ph.fHW = make_fdiv((uint32_t)(ph.Hh * ph.Wh));
    }
    return ph;
}

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }

// Fragment idx (of NTHR * F) of a k-contiguous tile [row][KT + PADK] -> (row,
// k quad).  A wave's 64 fragments cover 64 / (KT/4) rows; within each run of
// 16 lanes the row changes fastest and the quad is fixed, so the 16 float4
// LDS writes of a run land on disjoint banks (rows are KT + 4 floats apart);
// the global addresses a wave loads are the same set as with the quad
// fastest, so coalescing is unchanged.
template <int KT>
__device__ __forceinline__ void kc_map_t(int idx, int *row, int *kc) {
    constexpr int Q4 = KT / 4;               // quads per row
    constexpr int RW = 64 / Q4;              // rows per wave
    const int lane = idx & 63;
    *row = (idx >> 6) * RW + lane % RW;
    *kc = lane / RW;
}

// Raw buffer loads for the lean address mode: a 32-bit byte offset into a
// tensor described by base and size; an offset at or past the size reads as
// zeros, which is how the kernel fetches padding and tails without branches.
constexpr unsigned OOB = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tensor_rsrc(const float *p, unsigned bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ float4 bld4(__amdgpu_buffer_rsrc_t r, unsigned elem_off, bool ok) {
    return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, ok ? elem_off * 4u : OOB, 0, 0));
}

// Address of output row m of a pass in its destination tensor (row-major
// [rows][Ng] for FWD / WGRAD, the NHWC pixel of the phase for DGRAD).
__device__ __forceinline__ size_t out_row(const Args &a, int pass, const Phase &ph, int z, int m) {
    // a stride-1 data gradient has one phase holding every pixel in NHWC order,
    // so its rows are the pixels themselves (no division per row)
    if (pass != PASS_DGRAD || a.st == 1)
        return (size_t)m * a.Ng;
    const int n = (int)ph.fHW.div((uint32_t)m);
    const int rem = m - n * (ph.Hh * ph.Wh);
    const int i = (int)ph.fW.div((uint32_t)rem);
    const int j = rem - i * ph.Wh;
    int h = z / a.st + a.st * i;
    int w = z % a.st + a.st * j;
    return (((size_t)n * a.H + h) * a.W + w) * a.C;
}

__device__ __forceinline__ float epilogue(const Args &a, int pass, float v, int n, const float *dst) {
    if (pass == PASS_FWD) {
        if (a.bias)
            v += a.bias[n];
        if (a.relu)
            v = fmaxf(v, 0.0f);
    } else if (pass == PASS_DGRAD) {
        // a folded ReLU's backward: its output gradient v, kept where its output is positive
        if (a.relu_mask && !(a.relu_mask[dst - a.out] > 0.0f))
            v = 0.0f;
        if (a.accumulate)
            v += *dst;
    }
    return v;
}

// TU, the lean address mode (the host checks that every tensor has fewer
// than 2^31 elements, so element offsets are 32-bit):
//  * forward with C % KT == 0, dgrad with K % KT == 0 and C % 4 == 0: every K
//    stage lies inside one filter tap, so the tap and first channel of a
//    stage are workgroup-uniform scalars and every stage is full; a
//    fragment's offset is its row's base offset plus a per-stage delta.  The
//    stages run through every tap of one block of KT channels before the next
//    block: the taps' overlapping input windows are then re-read while they
//    are still in L2 (with channels innermost, the resident workgroups sweep
//    all channels between two taps, more than an XCD's L2 holds, and the
//    forward / dgrad passes fetched 4x more from memory);
//  * wgrad with K % 4 == 0, C % 4 == 0 and Q >= KT: every B fragment's pixel
//    advances by KT per stage (at most one row wrap), so its (q, p), input
//    origin and offset are carried from stage to stage with uniform
//    increments instead of being decoded.
template <int PASS, int MT, int NT, int KT, bool AV, bool BV, bool TU>
__global__ __launch_bounds__(NTHR, TU ? 4 : 1) void igemm_kernel(Args a) {
    static_assert(!TU || (AV && BV), "the lean address mode needs float4 operands");
    constexpr bool A_KC = (PASS != PASS_WGRAD); // A tile stored [row][k]
    constexpr bool B_KC = (PASS == PASS_FWD);   // B tile stored [col][k]
    constexpr int A_LD = A_KC ? (KT + PADK) : (MT + PADR);
    constexpr int B_LD = B_KC ? (KT + PADK) : (NT + PADR);
    constexpr int A_SZ = A_KC ? MT * A_LD : KT * A_LD;
    constexpr int B_SZ = B_KC ? NT * B_LD : KT * B_LD;
    constexpr int FA = MT * KT / 4 / NTHR; // float4 fragments per thread
    constexpr int FB = NT * KT / 4 / NTHR;
    static_assert(FA >= 1 && FB >= 1, "tile too small");
    // The 4 waves form a WM x WN grid over the tile (4 x 1 for tall tiles,
    // 1 x 4 for wide ones, 2 x 2 otherwise); each owns BM x BN 32x32 blocks.
    constexpr int WM = MT >= 4 * NT ? 4 : (NT >= 4 * MT ? 1 : 2);
    constexpr int WN = 4 / WM;
    constexpr int BM = MT / (32 * WM), BN = NT / (32 * WN);
    static_assert(BM >= 1 && BN >= 1 && BM * 32 * WM == MT && BN * 32 * WN == NT, "tile shape");

    __shared__ __attribute__((aligned(16))) float lds[2 * (A_SZ + B_SZ)];

    const int t = threadIdx.x;
    // XCD-aware order: workgroups are dealt to the 8 XCDs round-robin by
    // linear id.  Each stride phase owns a range of ids padded to a multiple
    // of 8 (phase-major dispatch); inside it, id -> (id % 8) * (range / 8) +
    // id / 8 gives each XCD one contiguous run of (split, tile): neighbouring
    // tiles of the same split, which share operand rows in that XCD's L2, and
    // the splits of a GEMM with few tiles spread over every XCD.
    const int per_phase = a.tiles * a.splits;
    const int range = (per_phase + 7) & ~7;
    const int z = blockIdx.x / range;
    int bid = blockIdx.x - z * range;
    bid = (bid & 7) * (range >> 3) + (bid >> 3);
    if (bid >= per_phase)
        return;
    const int split = bid / a.tiles;
    const int tile = bid - split * a.tiles;
    const int tm = tile / a.tiles_n;
    const int tn = tile - tm * a.tiles_n;

    Phase ph{};
    int M = a.M, Kg = a.Kg;
    if (PASS == PASS_DGRAD) {
        ph = make_phase(a, z);
        M = ph.M;
        Kg = ph.Kg;
        if (tm * MT >= M)
            return;
    }
    const int ktiles = (Kg + KT - 1) / KT;
    const int kt0 = split * a.kt_per_split;
    const int kt1 = min(kt0 + a.kt_per_split, ktiles);
    const int nkt = max(kt1 - kt0, 0);

    // ------------------------------------------------ per-thread load state
    auto kc_map = [](int idx, int *row, int *kc) { kc_map_t<KT>(idx, row, kc); };
    // A fragments: k-contiguous -> kc_map (row, k quad);
    // row-contiguous -> (krow = idx / (MT/4), mc = idx % (MT/4)).
    int a_row[FA];
    int a_kc = 0;
    bool a_ok[FA];
    // FWD: pixel base and (h, w) origin per row; DGRAD: (n, i+dh, j+dw) per row.
    int a_n[FA], a_h[FA], a_w[FA];
#pragma unroll
    for (int f = 0; f < FA; ++f) {
        int idx = t + NTHR * f;
        if (A_KC) {
            kc_map(idx, &a_row[f], &a_kc);
            int m = tm * MT + a_row[f];
            a_ok[f] = m < M;
            int mm = a_ok[f] ? m : 0;
            if (PASS == PASS_FWD) {
                int n = a.fPQ.div(mm);
                int rem = mm - n * a.P * a.Q;
                int p = a.fQ.div(rem);
                int q = rem - p * a.Q;
                a_n[f] = n;
                a_h[f] = p * a.st - a.pad;
                a_w[f] = q * a.st - a.pad_w;
            } else {
                int hw = ph.Hh * ph.Wh;
                int n = hw ? mm / hw : 0;
                int rem = mm - n * hw;
                int i = ph.Wh ? rem / ph.Wh : 0;
                int j = rem - i * ph.Wh;
                a_n[f] = n;
                a_h[f] = i + ph.dh;
                a_w[f] = j + ph.dw;
            }
        } else {
            a_row[f] = idx / (MT / 4); // k row (pixel) within the stage
            a_kc = idx % (MT / 4);     // output-channel quad
            a_ok[f] = true;
            a_n[f] = a_h[f] = a_w[f] = 0;
        }
    }
    // TU: element offset of each A fragment's (possibly padded-out) window
    // origin, and of each B fragment's first k.
    int a_base[FA], b_base[FB];
    if (TU && PASS == PASS_FWD) {
#pragma unroll
        for (int f = 0; f < FA; ++f)
            a_base[f] = ((a_n[f] * a.H + a_h[f]) * a.W + a_w[f]) * a.C + 4 * a_kc;
    }
    if (TU && PASS == PASS_DGRAD) {
#pragma unroll
        for (int f = 0; f < FA; ++f)
            a_base[f] = ((a_n[f] * a.P + a_h[f]) * a.Q + a_w[f]) * a.K + 4 * a_kc;
    }
    // B fragments: k-contiguous -> kc_map (row, k quad); n-contiguous ->
    // (krow = idx / (NT/4), nc = idx % (NT/4)).
    int b_row[FB];
    int b_kc = 0;
    // WGRAD: filter tap (r, s) and channel c of the thread's column quad (or
    // of each of its 4 columns in the scalar path).
    int b_r[4], b_s[4], b_c[4];
    bool b_cok[4];
#pragma unroll
    for (int f = 0; f < FB; ++f) {
        int idx = t + NTHR * f;
        if (B_KC) {
            kc_map(idx, &b_row[f], &b_kc);
        } else {
            b_row[f] = idx / (NT / 4);
            b_kc = idx % (NT / 4);
        }
    }
    if (TU && PASS == PASS_FWD) {
#pragma unroll
        for (int f = 0; f < FB; ++f)
            b_base[f] = (tn * NT + b_row[f]) * a.Kg + 4 * b_kc;
    }
    if (TU && PASS == PASS_DGRAD) {
#pragma unroll
        for (int f = 0; f < FB; ++f)
            b_base[f] = b_row[f] * (a.R * a.S * a.C) + tn * NT + 4 * b_kc;
    }
    if (PASS == PASS_WGRAD) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            int kk = tn * NT + 4 * b_kc + e;
            b_cok[e] = kk < a.Ng;
            int k2 = b_cok[e] ? kk : 0;
            int rs = a.fC.div(k2);
            b_c[e] = k2 - rs * a.C;
            b_r[e] = a.fS.div(rs);
            b_s[e] = rs - b_r[e] * a.S;
        }
    }

    // WGRAD TU: A fragment offsets (stage 0) and each B fragment's pixel
    // state (q, p, window origin hh/ww, element offset) for its next stage.
    int wa_off[FA];
    int bq[FB], bp[FB], bhh[FB], bww[FB], boff[FB];
    if (PASS == PASS_WGRAD && TU) {
#pragma unroll
        for (int f = 0; f < FA; ++f)
            wa_off[f] = a_row[f] * a.K + tm * MT + 4 * a_kc;
    }
    auto wpix_init = [&](int kt) {
#pragma unroll
        for (int f = 0; f < FB; ++f) {
            const int mp = min(kt * KT + b_row[f], max(a.Kg - 1, 0));
            const int n = a.fPQ.div(mp);
            const int rem = mp - n * a.P * a.Q;
            const int pp = a.fQ.div(rem);
            bq[f] = rem - pp * a.Q;
            bp[f] = pp;
            bhh[f] = pp * a.st - a.pad + b_r[0];
            bww[f] = bq[f] * a.st - a.pad_w + b_s[0];
            boff[f] = ((n * a.H + bhh[f]) * a.W + bww[f]) * a.C + b_c[0];
        }
    };
    auto wpix_next = [&]() {
        const int row_step = (a.st * a.W - a.Q * a.st) * a.C, img_step = (a.H - a.P * a.st) * a.W * a.C;
#pragma unroll
        for (int f = 0; f < FB; ++f) {
            bq[f] += KT;
            bww[f] += KT * a.st;
            boff[f] += KT * a.st * a.C;
            if (bq[f] >= a.Q) { // Q >= KT: at most one row wrap per stage
                bq[f] -= a.Q;
                bww[f] -= a.Q * a.st;
                ++bp[f];
                bhh[f] += a.st;
                boff[f] += row_step;
                if (bp[f] >= a.P) {
                    bp[f] -= a.P;
                    bhh[f] -= a.P * a.st;
                    boff[f] += img_step;
                }
            }
        }
    };

    float4 ra[FA], rb[FB];
    const __amdgpu_buffer_rsrc_t rs_a = tensor_rsrc(a.A, a.a_bytes), rs_b = tensor_rsrc(a.B, a.b_bytes);

    // TU stage cursor, uniform over the workgroup: first channel c0 of the
    // next stage to load and its tap, (r, s) for the forward pass or (tr, ts)
    // for dgrad.  Stage kt covers channel block kt / T and tap kt % T (T taps,
    // row-major).  Set once by division, then advanced one stage at a time.
    constexpr bool FW = PASS == PASS_FWD;
    int cur_c0 = 0, cur_t1 = 0, cur_t2 = 0;
    auto cursor_init = [&](int kt) {
        const int t1n = FW ? a.R : ph.Rt, t2n = FW ? a.S : ph.St;
        const int cb = kt / (t1n * t2n), tap = kt - cb * (t1n * t2n);
        cur_c0 = cb * KT;
        cur_t1 = tap / t2n;
        cur_t2 = tap - cur_t1 * t2n;
    };
    auto cursor_next = [&]() {
        if (++cur_t2 == (FW ? a.S : ph.St)) {
            cur_t2 = 0;
            if (++cur_t1 == (FW ? a.R : ph.Rt)) {
                cur_t1 = 0;
                cur_c0 += KT;
            }
        }
    };

    // ------------------------------------------------ global -> registers
    auto load_a = [&](int kt) {
        const int kbase = kt * KT;
        if (PASS == PASS_FWD && TU) {
            const int r = cur_t1, s = cur_t2;
            const int delta = (r * a.W + s) * a.C + cur_c0;
#pragma unroll
            for (int f = 0; f < FA; ++f) {
                const int h = a_h[f] + r, w = a_w[f] + s;
                const bool ok = a_ok[f] && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
                ra[f] = bld4(rs_a, (unsigned)(a_base[f] + delta), ok);
            }
        } else if (PASS == PASS_FWD) {
            if (AV) {
                int kk = kbase + 4 * a_kc;
                bool kok = kk < Kg;
                int k2 = kok ? kk : 0;
                int rs = a.fC.div(k2);
                int c = k2 - rs * a.C;
                int r = a.fS.div(rs);
                int s = rs - r * a.S;
#pragma unroll
                for (int f = 0; f < FA; ++f) {
                    int h = a_h[f] + r, w = a_w[f] + s;
                    bool ok = kok && a_ok[f] && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
                    ra[f] = ok ? ld4(a.A + (((size_t)a_n[f] * a.H + h) * a.W + w) * a.C + c)
                               : make_float4(0.f, 0.f, 0.f, 0.f);
                }
            } else {
                float v[4][FA];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    int kk = kbase + 4 * a_kc + e;
                    bool kok = kk < Kg;
                    int k2 = kok ? kk : 0;
                    int rs = a.fC.div(k2);
                    int c = k2 - rs * a.C;
                    int r = a.fS.div(rs);
                    int s = rs - r * a.S;
#pragma unroll
                    for (int f = 0; f < FA; ++f) {
                        int h = a_h[f] + r, w = a_w[f] + s;
                        bool ok = kok && a_ok[f] && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
                        v[e][f] = ok ? a.A[(((size_t)a_n[f] * a.H + h) * a.W + w) * a.C + c] : 0.f;
                    }
                }
#pragma unroll
                for (int f = 0; f < FA; ++f)
                    ra[f] = make_float4(v[0][f], v[1][f], v[2][f], v[3][f]);
            }
        } else if (PASS == PASS_DGRAD && TU) {
            const int tr = cur_t1, ts = cur_t2;
            const int delta = cur_c0 - (tr * a.Q + ts) * a.K;
#pragma unroll
            for (int f = 0; f < FA; ++f) {
                const int p = a_h[f] - tr, q = a_w[f] - ts;
                const bool ok = a_ok[f] && (unsigned)p < (unsigned)a.P && (unsigned)q < (unsigned)a.Q;
                ra[f] = bld4(rs_a, (unsigned)(a_base[f] + delta), ok);
            }
        } else if (PASS == PASS_DGRAD) {
            // kk = (tr, ts, k) with k fastest
            float v[4][FA];
            const int nel = AV ? 1 : 4;
#pragma unroll
            for (int e = 0; e < nel; ++e) {
                int kk = kbase + 4 * a_kc + e;
                bool kok = kk < Kg;
                int k2 = kok ? kk : 0;
                int tt = a.fK.div(k2);
                int k = k2 - tt * a.K;
                int tr = ph.St ? tt / ph.St : 0;
                int ts = tt - tr * ph.St;
#pragma unroll
                for (int f = 0; f < FA; ++f) {
                    int p = a_h[f] - tr, q = a_w[f] - ts;
                    bool ok = kok && a_ok[f] && (unsigned)p < (unsigned)a.P && (unsigned)q < (unsigned)a.Q;
                    const float *src = a.A + (((size_t)a_n[f] * a.P + p) * a.Q + q) * a.K + k;
                    if (AV) {
                        ra[f] = ok ? ld4(src) : make_float4(0.f, 0.f, 0.f, 0.f);
                    } else {
                        v[e][f] = ok ? *src : 0.f;
                    }
                }
            }
            if (!AV) {
#pragma unroll
                for (int f = 0; f < FA; ++f)
                    ra[f] = make_float4(v[0][f], v[1][f], v[2][f], v[3][f]);
            }
        } else if (PASS == PASS_WGRAD && TU) {
            const bool kok = tm * MT + 4 * a_kc < a.M;
#pragma unroll
            for (int f = 0; f < FA; ++f) {
                const bool ok = kok && kbase + a_row[f] < Kg;
                ra[f] = bld4(rs_a, (unsigned)(wa_off[f] + kbase * a.K), ok);
            }
        } else { // WGRAD: A = dY^T, rows are output channels (contiguous), k = pixel
#pragma unroll
            for (int f = 0; f < FA; ++f) {
                int mp = kbase + a_row[f];
                int ko = tm * MT + 4 * a_kc;
                const float *src = a.A + (size_t)mp * a.K + ko;
                bool pok = mp < Kg;
                if (AV) {
                    ra[f] = (pok && ko < a.M) ? ld4(src) : make_float4(0.f, 0.f, 0.f, 0.f);
                } else {
                    float v0 = (pok && ko + 0 < a.M) ? src[0] : 0.f;
                    float v1 = (pok && ko + 1 < a.M) ? src[1] : 0.f;
                    float v2 = (pok && ko + 2 < a.M) ? src[2] : 0.f;
                    float v3 = (pok && ko + 3 < a.M) ? src[3] : 0.f;
                    ra[f] = make_float4(v0, v1, v2, v3);
                }
            }
        }
    };

    auto load_b = [&](int kt) {
        const int kbase = kt * KT;
        if (PASS == PASS_FWD && TU) {
#pragma unroll
            for (int f = 0; f < FB; ++f) {
                const bool jok = tn * NT + b_row[f] < a.Ng;
                rb[f] = bld4(rs_b, (unsigned)(b_base[f] + (cur_t1 * a.S + cur_t2) * a.C + cur_c0), jok);
            }
        } else if (PASS == PASS_FWD) { // B = W[k][kk], k-contiguous
#pragma unroll
            for (int f = 0; f < FB; ++f) {
                int j = tn * NT + b_row[f];
                int kk = kbase + 4 * b_kc;
                const float *src = a.B + (size_t)j * a.Kg + kk;
                bool jok = j < a.Ng;
                if (BV) {
                    rb[f] = (jok && kk < Kg) ? ld4(src) : make_float4(0.f, 0.f, 0.f, 0.f);
                } else {
                    float v0 = (jok && kk + 0 < Kg) ? src[0] : 0.f;
                    float v1 = (jok && kk + 1 < Kg) ? src[1] : 0.f;
                    float v2 = (jok && kk + 2 < Kg) ? src[2] : 0.f;
                    float v3 = (jok && kk + 3 < Kg) ? src[3] : 0.f;
                    rb[f] = make_float4(v0, v1, v2, v3);
                }
            }
        } else if (PASS == PASS_DGRAD && TU) {
            const int r = ph.r0 + a.st * cur_t1, s = ph.s0 + a.st * cur_t2;
            const int delta = cur_c0 * (a.R * a.S * a.C) + (r * a.S + s) * a.C;
            const bool cok = tn * NT + 4 * b_kc < a.C;
#pragma unroll
            for (int f = 0; f < FB; ++f)
                rb[f] = bld4(rs_b, (unsigned)(b_base[f] + delta), cok);
        } else if (PASS == PASS_DGRAD) { // B[kk][c] = W[k][r][s][c], c contiguous
#pragma unroll
            for (int f = 0; f < FB; ++f) {
                int kk = kbase + b_row[f];
                bool kok = kk < Kg;
                int k2 = kok ? kk : 0;
                int tt = a.fK.div(k2);
                int k = k2 - tt * a.K;
                int tr = ph.St ? tt / ph.St : 0;
                int ts = tt - tr * ph.St;
                int r = ph.r0 + a.st * tr, s = ph.s0 + a.st * ts;
                int c = tn * NT + 4 * b_kc;
                const float *src = a.B + (((size_t)k * a.R + r) * a.S + s) * a.C + c;
                if (BV) {
                    rb[f] = (kok && c < a.C) ? ld4(src) : make_float4(0.f, 0.f, 0.f, 0.f);
                } else {
                    float v0 = (kok && c + 0 < a.C) ? src[0] : 0.f;
                    float v1 = (kok && c + 1 < a.C) ? src[1] : 0.f;
                    float v2 = (kok && c + 2 < a.C) ? src[2] : 0.f;
                    float v3 = (kok && c + 3 < a.C) ? src[3] : 0.f;
                    rb[f] = make_float4(v0, v1, v2, v3);
                }
            }
        } else if (PASS == PASS_WGRAD && TU) {
#pragma unroll
            for (int f = 0; f < FB; ++f) {
                const bool ok = b_cok[0] && kbase + b_row[f] < Kg && (unsigned)bhh[f] < (unsigned)a.H &&
                                (unsigned)bww[f] < (unsigned)a.W;
                rb[f] = bld4(rs_b, (unsigned)boff[f], ok);
            }
        } else { // WGRAD: B[pixel][kk] = X~, c contiguous within a tap
#pragma unroll
            for (int f = 0; f < FB; ++f) {
                int mp = kbase + b_row[f];
                bool pok = mp < Kg;
                int m2 = pok ? mp : 0;
                int n = a.fPQ.div(m2);
                int rem = m2 - n * a.P * a.Q;
                int p = a.fQ.div(rem);
                int q = rem - p * a.Q;
                int hb = p * a.st - a.pad, wb = q * a.st - a.pad_w;
                if (BV) {
                    int h = hb + b_r[0], w = wb + b_s[0];
                    bool ok = pok && b_cok[0] && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
                    rb[f] = ok ? ld4(a.B + (((size_t)n * a.H + h) * a.W + w) * a.C + b_c[0])
                               : make_float4(0.f, 0.f, 0.f, 0.f);
                } else {
                    float v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        int h = hb + b_r[e], w = wb + b_s[e];
                        bool ok = pok && b_cok[e] && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
                        v[e] = ok ? a.B[(((size_t)n * a.H + h) * a.W + w) * a.C + b_c[e]] : 0.f;
                    }
                    rb[f] = make_float4(v[0], v[1], v[2], v[3]);
                }
            }
        }
    };

    // ------------------------------------------------ registers -> LDS
    auto store = [&](int buf) {
        float *As = lds + buf * (A_SZ + B_SZ);
        float *Bs = As + A_SZ;
#pragma unroll
        for (int f = 0; f < FA; ++f)
            st4(As + a_row[f] * A_LD + 4 * a_kc, ra[f]);
#pragma unroll
        for (int f = 0; f < FB; ++f)
            st4(Bs + b_row[f] * B_LD + 4 * b_kc, rb[f]);
    };

    // ------------------------------------------------ MFMA on one stage
    const int wave = t >> 6, lane = t & 63;
    const int lr = lane & 31, lh = lane >> 5;
    const int wm = (wave % WM) * (MT / WM), wn = (wave / WM) * (NT / WN);
    f32x16 acc[BM][BN];
#pragma unroll
    for (int i = 0; i < BM; ++i)
#pragma unroll
        for (int j = 0; j < BN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                acc[i][j][v] = 0.f;

    constexpr int STORE_ST = KT / 2 - 2;
    // Within a stage, lane half lh multiplies k = lh*KT/2 + step: any fixed
    // bijection of k is a valid order for the sum, and this one lets a lane
    // read its KT/2 values of a k-contiguous row with two ds_read_b128.
    auto compute = [&](int buf, bool more) {
        const float *As = lds + buf * (A_SZ + B_SZ);
        const float *Bs = As + A_SZ;
        float av[BM][KT / 2], bv[BN][KT / 2];
#pragma unroll
        for (int i = 0; i < BM; ++i) {
            int row = wm + 32 * i + lr;
            if (A_KC) {
#pragma unroll
                for (int q4 = 0; q4 < KT / 8; ++q4) {
                    float4 x = ld4(As + row * A_LD + lh * (KT / 2) + 4 * q4);
                    av[i][4 * q4 + 0] = x.x;
                    av[i][4 * q4 + 1] = x.y;
                    av[i][4 * q4 + 2] = x.z;
                    av[i][4 * q4 + 3] = x.w;
                }
            } else {
#pragma unroll
                for (int st = 0; st < KT / 2; ++st)
                    av[i][st] = As[(lh * (KT / 2) + st) * A_LD + row];
            }
        }
#pragma unroll
        for (int j = 0; j < BN; ++j) {
            int col = wn + 32 * j + lr;
            if (B_KC) {
#pragma unroll
                for (int q4 = 0; q4 < KT / 8; ++q4) {
                    float4 x = ld4(Bs + col * B_LD + lh * (KT / 2) + 4 * q4);
                    bv[j][4 * q4 + 0] = x.x;
                    bv[j][4 * q4 + 1] = x.y;
                    bv[j][4 * q4 + 2] = x.z;
                    bv[j][4 * q4 + 3] = x.w;
                }
            } else {
#pragma unroll
                for (int st = 0; st < KT / 2; ++st)
                    bv[j][st] = Bs[(lh * (KT / 2) + st) * B_LD + col];
            }
        }
#pragma unroll
        for (int st = 0; st < KT / 2; ++st) {
            // The lean kernels write the next stage's tile (buf ^ 1, last read
            // before the previous barrier) between their MFMAs, three quarters
            // through the stage, so a wave reaches the barrier straight from its
            // last MFMAs (measured: 1% on VGG-16's and ResNet-50's GEMMs; half-
            // way or with the loads issued right after, no better).
            if (TU && st == STORE_ST && more) {
                __builtin_amdgcn_sched_barrier(0);
                store(buf ^ 1);
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int i = 0; i < BM; ++i)
#pragma unroll
                for (int j = 0; j < BN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i][st], bv[j][st], acc[i][j], 0, 0, 0);
        }
    };

    // ------------------------------------------------ pipeline
    int buf = 0;
    if (nkt > 0) {
        if (TU && PASS != PASS_WGRAD)
            cursor_init(kt0);
        if (TU && PASS == PASS_WGRAD)
            wpix_init(kt0);
        load_a(kt0);
        load_b(kt0);
        if (TU && PASS != PASS_WGRAD)
            cursor_next();
        if (TU && PASS == PASS_WGRAD)
            wpix_next();
        store(0);
    }
    __syncthreads();
    for (int it = 0; it < nkt; ++it) {
        const bool more = it + 1 < nkt;
        if (more) {
            load_a(kt0 + it + 1);
            load_b(kt0 + it + 1);
            if (TU && PASS != PASS_WGRAD)
                cursor_next();
            if (TU && PASS == PASS_WGRAD)
                wpix_next();
        }
        // Four workgroups share each SIMD's matrix core.  Raising this wave's
        // issue priority while it runs its MFMAs keeps the core fed by one
        // wave at a time instead of interleaving it with the other waves'
        // load and barrier phases (measured: forward and data-gradient passes
        // gain 1-5%; filter-gradient passes, whose operand loads are
        // costlier, lose up to 2%, so they keep the default priority).
        constexpr bool PRIO = TU && PASS != PASS_WGRAD;
        if (PRIO)
            __builtin_amdgcn_s_setprio(1);
        compute(buf, more);
        if (PRIO)
            __builtin_amdgcn_s_setprio(0);
        if (more && !TU)
            store(buf ^ 1);
        __syncthreads();
        buf ^= 1;
    }

    // ------------------------------------------------ epilogue
    // 32x32 accumulator layout: element v of lane l is row
    // 8*(v/4) + 4*(l/32) + v%4 and column l%32 of the block.
    const int Ng = a.Ng;
#pragma unroll
    for (int i = 0; i < BM; ++i) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            int m = tm * MT + wm + 32 * i + 8 * (v >> 2) + 4 * lh + (v & 3);
            if (m >= M)
                continue;
            if (a.splits > 1) {
                float *dst = a.partial + ((size_t)(z * a.splits + split) * a.M + m) * Ng;
#pragma unroll
                for (int j = 0; j < BN; ++j) {
                    int n = tn * NT + wn + 32 * j + lr;
                    if (n < Ng)
                        dst[n] = acc[i][j][v];
                }
            } else {
                float *dst = a.out + out_row(a, PASS, ph, z, m);
#pragma unroll
                for (int j = 0; j < BN; ++j) {
                    int n = tn * NT + wn + 32 * j + lr;
                    if (n < Ng)
                        dst[n] = epilogue(a, PASS, acc[i][j][v], n, dst + n);
                }
            }
        }
    }
}

// Adds the split-K partial sums of each output, then applies the pass's
// epilogue.  A workgroup owns G = 256 / R consecutive output groups (four
// elements when VEC, else one); the R lanes of a group each sum the slots
// s = lane, lane + R, ... into four independent accumulators (many loads in
// flight), and lane 0 then adds the R lane sums in ascending lane order.  R
// depends on the plan alone, so every result is deterministic.
template <int PASS, bool VEC>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(Args a, int lg_r) {
    using V = typename std::conditional<VEC, float4, float>::type;
    constexpr int W = VEC ? 4 : 1;
    __shared__ V part[256];
    const int z = blockIdx.y;
    Phase ph{};
    int M = a.M;
    if (PASS == PASS_DGRAD) {
        ph = make_phase(a, z);
        M = ph.M;
    }
    const int R = 1 << lg_r, G = 256 >> lg_r;
    const int col = threadIdx.x & (G - 1), lane = threadIdx.x >> (8 - lg_r);
    const size_t groups = (size_t)M * a.Ng / W;
    const size_t slab = (size_t)a.M * a.Ng; // elements per split slot
    const float *base = a.partial + (size_t)z * a.splits * slab;
    auto ld = [&](const float *p) -> V {
        if constexpr (VEC)
            return *reinterpret_cast<const float4 *>(p);
        else
            return *p;
    };
    for (size_t g0 = (size_t)blockIdx.x * G; g0 < groups; g0 += (size_t)gridDim.x * G) {
        const size_t g = g0 + col;
        V s0{}, s1{}, s2{}, s3{};
        if (g < groups) {
            const float *p = base + g * W;
            int s = lane;
            for (; s + 3 * R < a.splits; s += 4 * R) {
                s0 += ld(p + (size_t)s * slab);
                s1 += ld(p + (size_t)(s + R) * slab);
                s2 += ld(p + (size_t)(s + 2 * R) * slab);
                s3 += ld(p + (size_t)(s + 3 * R) * slab);
            }
            for (; s < a.splits; s += R)
                s0 += ld(p + (size_t)s * slab);
        }
        part[threadIdx.x] = (s0 + s1) + (s2 + s3);
        __syncthreads();
        if (lane == 0 && g < groups) {
            V v = part[col];
            for (int r = 1; r < R; ++r)
                v += part[r * G + col];
            const size_t e = g * W;
            const int m = (int)(e / a.Ng);
            const int n = (int)(e - (size_t)m * a.Ng);
            float *dst = a.out + out_row(a, PASS, ph, z, m) + n;
            if constexpr (VEC) {
                dst[0] = epilogue(a, PASS, v.x, n, dst);
                dst[1] = epilogue(a, PASS, v.y, n + 1, dst + 1);
                dst[2] = epilogue(a, PASS, v.z, n + 2, dst + 2);
                dst[3] = epilogue(a, PASS, v.w, n + 3, dst + 3);
            } else {
                dst[0] = epilogue(a, PASS, v, n, dst);
            }
        }
        __syncthreads();
    }
}

// Channel padding for C % 4 != 0: with C rounded up to a multiple of 4 every
// operand of the forward and wgrad GEMMs is read as aligned float4 (one
// 16-byte load per filter tap instead of four gathered scalars).  Padded
// channels are zero, so they add nothing to any sum.
__global__ __launch_bounds__(256) void pad_channels_kernel(const float *in, float4 *out, int64_t rows, int c,
                                                           int cp4) {
    const int64_t total = rows * cp4;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = i / cp4;
        const int c0 = 4 * (int)(i - row * cp4);
        const float *src = in + row * c;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
            v[e] = c0 + e < c ? src[c0 + e] : 0.f;
        out[i] = make_float4(v[0], v[1], v[2], v[3]);
    }
}

__global__ __launch_bounds__(256) void unpad_channels_kernel(const float *in, float *out, int64_t rows, int c,
                                                             int cp) {
    const int64_t total = rows * c;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = i / c;
        out[i] = in[row * cp + (i - row * c)];
    }
}

int pad_channels(const float *in, float *out, int64_t rows, int c, int cp, hipStream_t s) {
    const int64_t total = rows * (cp / 4);
    const int blocks = (int)std::min<int64_t>((total + 255) / 256, 8192);
    hipLaunchKernelGGL(pad_channels_kernel, dim3(blocks), dim3(256), 0, s, in, reinterpret_cast<float4 *>(out),
                       rows, c, cp / 4);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

int unpad_channels(const float *in, float *out, int64_t rows, int c, int cp, hipStream_t s) {
    const int64_t total = rows * c;
    const int blocks = (int)std::min<int64_t>((total + 255) / 256, 8192);
    hipLaunchKernelGGL(unpad_channels_kernel, dim3(blocks), dim3(256), 0, s, in, out, rows, c, cp);
    DC_HIP(hipGetLastError());
    return DC_OK;
}

template <int PASS, int MT, int NT, int KT, bool AV, bool BV, bool TU = false>
void launch_t(const Args &a, int grid_x, hipStream_t s) {
    hipLaunchKernelGGL((igemm_kernel<PASS, MT, NT, KT, AV, BV, TU>), dim3(grid_x), dim3(NTHR), 0, s, a);
}

template <int PASS, int MT, int NT, int KT>
void launch_v(const Args &a, bool av, bool bv, bool tu, int grid_x, hipStream_t s) {
    if (tu) {
        launch_t<PASS, MT, NT, KT, true, true, true>(a, grid_x, s);
        return;
    }
    if (av && bv)
        launch_t<PASS, MT, NT, KT, true, true>(a, grid_x, s);
    else if (av)
        launch_t<PASS, MT, NT, KT, true, false>(a, grid_x, s);
    else if (bv)
        launch_t<PASS, MT, NT, KT, false, true>(a, grid_x, s);
    else
        launch_t<PASS, MT, NT, KT, false, false>(a, grid_x, s);
}

template <int PASS, int KT>
void launch_k(const Args &a, const GemmPlan &pl, int grid_x, hipStream_t s) {
    if (pl.mt == 128 && pl.nt == 128)
        launch_v<PASS, 128, 128, KT>(a, pl.av, pl.bv, pl.tu, grid_x, s);
    else if (pl.mt == 128 && pl.nt == 64)
        launch_v<PASS, 128, 64, KT>(a, pl.av, pl.bv, pl.tu, grid_x, s);
    else if (pl.mt == 64 && pl.nt == 128)
        launch_v<PASS, 64, 128, KT>(a, pl.av, pl.bv, pl.tu, grid_x, s);
    else
        launch_v<PASS, 64, 64, KT>(a, pl.av, pl.bv, pl.tu, grid_x, s);
}

template <int PASS>
void launch_p(const Args &a, const GemmPlan &pl, int grid_x, hipStream_t s) {
    launch_k<PASS, 16>(a, pl, grid_x, s);
}

Args make_args(const ConvGeom &g, const GemmPlan &pl) {
    Args a{};
    a.N = g.N; a.H = g.H; a.W = g.W; a.C = g.C; a.K = g.K; a.R = g.R; a.S = g.S;
    a.st = g.st; a.pad = g.pad; a.pad_w = g.pad_w; a.P = g.P; a.Q = g.Q;
    a.M = pl.M; a.Ng = pl.Ng; a.Kg = pl.Kg;
    a.tiles_m = pl.tiles_m; a.tiles_n = pl.tiles_n; a.tiles = pl.tiles_m * pl.tiles_n;
    a.splits = pl.splits; a.kt_per_split = pl.kt_per_split; a.phases = pl.phases;
    a.fC = make_fdiv(g.C); a.fS = make_fdiv(g.S); a.fK = make_fdiv(g.K);
    a.fQ = make_fdiv(g.Q); a.fPQ = make_fdiv(g.P * g.Q);
    const int64_t x_el = (int64_t)g.N * g.H * g.W * g.C, y_el = (int64_t)g.N * g.P * g.Q * g.K,
                  w_el = (int64_t)g.K * g.R * g.S * g.C;
    const int64_t a_el = pl.pass == PASS_FWD ? x_el : y_el, b_el = pl.pass == PASS_WGRAD ? x_el : w_el;
    a.a_bytes = (unsigned)std::min<int64_t>(4 * a_el, OOB);
    a.b_bytes = (unsigned)std::min<int64_t>(4 * b_el, OOB);
    return a;
}

int run(const ConvGeom &g, const GemmPlan &pl, Args a, void *ws, hipStream_t s) {
    if ((int64_t)pl.M * pl.Ng == 0)
        return DC_OK;
    if (pl.splits > 1) {
        if (!ws)
            return fail(DC_EINVAL, "conv pass %d needs %zu bytes of workspace", pl.pass, pl.ws_bytes);
        a.partial = static_cast<float *>(ws);
    }
    const int64_t range = ((int64_t)pl.tiles_m * pl.tiles_n * pl.splits + 7) / 8 * 8;
    if (range * pl.phases > INT_MAX)
        return fail(DC_EINVAL, "conv pass %d needs %lld workgroups", pl.pass, (long long)(range * pl.phases));
    const int grid_x = (int)(range * pl.phases);
    switch (pl.pass) {
    case PASS_FWD: launch_p<PASS_FWD>(a, pl, grid_x, s); break;
    case PASS_DGRAD: launch_p<PASS_DGRAD>(a, pl, grid_x, s); break;
    default: launch_p<PASS_WGRAD>(a, pl, grid_x, s); break;
    }
    DC_HIP(hipGetLastError());
    if (pl.splits > 1) {
        // Lanes per output group: about one lane per four slots, at most 16
        // (so a group row of the partial buffer is read as >= 256 bytes).
        int lg_r = 0;
        while (lg_r < 4 && (4 << (lg_r + 1)) <= pl.splits)
            ++lg_r;
        const bool vec = pl.Ng % 4 == 0 && (uintptr_t)ws % 16 == 0;
        const size_t groups = (size_t)pl.M * pl.Ng / (vec ? 4 : 1);
        const size_t per_wg = (size_t)256 >> lg_r;
        const int blocks = (int)std::min<size_t>((groups + per_wg - 1) / per_wg, 8192);
        const dim3 grid(blocks, pl.pass == PASS_DGRAD ? pl.phases : 1);
        switch (pl.pass * 2 + (vec ? 1 : 0)) {
        case PASS_FWD * 2: hipLaunchKernelGGL((splitk_reduce_kernel<PASS_FWD, false>), grid, dim3(256), 0, s, a, lg_r); break;
        case PASS_FWD * 2 + 1: hipLaunchKernelGGL((splitk_reduce_kernel<PASS_FWD, true>), grid, dim3(256), 0, s, a, lg_r); break;
        case PASS_DGRAD * 2: hipLaunchKernelGGL((splitk_reduce_kernel<PASS_DGRAD, false>), grid, dim3(256), 0, s, a, lg_r); break;
        case PASS_DGRAD * 2 + 1: hipLaunchKernelGGL((splitk_reduce_kernel<PASS_DGRAD, true>), grid, dim3(256), 0, s, a, lg_r); break;
        case PASS_WGRAD * 2: hipLaunchKernelGGL((splitk_reduce_kernel<PASS_WGRAD, false>), grid, dim3(256), 0, s, a, lg_r); break;
        default: hipLaunchKernelGGL((splitk_reduce_kernel<PASS_WGRAD, true>), grid, dim3(256), 0, s, a, lg_r); break;
        }
        DC_HIP(hipGetLastError());
    }
    return DC_OK;
}

} // namespace

bool conv_geom_from_shape(const dc_conv_shape &sh, ConvGeom *g) {
    if (sh.n < 0 || sh.h < 1 || sh.w < 1 || sh.c < 1 || sh.k < 1 || sh.r < 1 || sh.s < 1 ||
        sh.stride < 1 || sh.pad < 0 || sh.pad >= sh.r || sh.pad_w < 0 || sh.pad_w >= sh.s)
        return false;
    // padded extents in 64 bits: pad is bounded only by the filter size
    const int64_t hp = (int64_t)sh.h + 2 * (int64_t)sh.pad, wp = (int64_t)sh.w + 2 * (int64_t)sh.pad_w;
    if (hp < sh.r || wp < sh.s)
        return false;
    const int64_t P = (hp - sh.r) / sh.stride + 1, Q = (wp - sh.s) / sh.stride + 1;
    // every index the kernels form must stay below 2^31
    const int64_t big = std::max<int64_t>({(int64_t)sh.n * sh.h * sh.w * sh.c, (int64_t)sh.n * P * Q * sh.k,
                                           (int64_t)sh.k * sh.r * sh.s * sh.c, hp, wp});
    if (big >= INT_MAX)
        return false;
    g->N = sh.n; g->H = sh.h; g->W = sh.w; g->C = sh.c; g->K = sh.k;
    g->R = sh.r; g->S = sh.s; g->st = sh.stride; g->pad = sh.pad; g->pad_w = sh.pad_w;
    g->P = (int)P;
    g->Q = (int)Q;
    return true;
}

// force (mt, nt, splits), if given, restricts the choice to that plan; the
// result then has mt == 0 when the shape cannot run it.
static GemmPlan plan_core(const ConvGeom &g, int pass, const int *force) {
    GemmPlan pl{};
    pl.pass = pass;
    pl.phases = 1;
    if (pass == PASS_FWD) {
        pl.M = g.N * g.P * g.Q; pl.Ng = g.K; pl.Kg = g.R * g.S * g.C;
        pl.av = g.C % 4 == 0;
        pl.bv = (g.R * g.S * g.C) % 4 == 0;
        pl.tu = g.C % 16 == 0;
    } else if (pass == PASS_DGRAD) {
        pl.phases = g.st * g.st;
        int hh = (g.H + g.st - 1) / g.st, wh = (g.W + g.st - 1) / g.st;
        int rt = (g.R + g.st - 1) / g.st, stt = (g.S + g.st - 1) / g.st;
        pl.M = g.N * hh * wh; pl.Ng = g.C; pl.Kg = rt * stt * g.K;
        pl.av = g.K % 4 == 0;
        pl.bv = g.C % 4 == 0;
        pl.tu = g.K % 16 == 0 && g.C % 4 == 0;
    } else {
        pl.M = g.K; pl.Ng = g.R * g.S * g.C; pl.Kg = g.N * g.P * g.Q;
        pl.av = g.K % 4 == 0;
        pl.bv = g.C % 4 == 0;
        pl.tu = pl.av && pl.bv && g.Q >= 16;
    }
    // The lean mode reads each operand through a 32-bit byte offset and needs
    // offsets at or past 2^31 to read as zeros: every operand below 2 GB.
    const int64_t x_el = (int64_t)g.N * g.H * g.W * g.C, y_el = (int64_t)g.N * g.P * g.Q * g.K,
                  w_el = (int64_t)g.K * g.R * g.S * g.C;
    if (4 * std::max({x_el, y_el, w_el}) >= (int64_t)OOB)
        pl.tu = false;
    // Pick the tile and split-K factor with the least estimated time.  A CU
    // holds at most occ[c] workgroups of a tile at once (registers and LDS)
    // and, holding k of them, keeps its matrix cores busy a fraction util(k)
    // of the time (one workgroup cannot hide its own global-load latency).
    // A CU that receives n workgroups runs n / occ full rounds and then a
    // partial round of n % occ at the lower utilisation of that count (the
    // tail).  Smaller tiles move more operand bytes per flop (eff, fitted to
    // measured VGG-16 / ResNet-50 / GoogLeNet / AlexNet passes); a split pays
    // for writing and re-reading its partial sums.
    static const int cand[4][2] = {{128, 128}, {128, 64}, {64, 128}, {64, 64}};
    static const double eff[4] = {1.0, 0.9, 0.85, 0.85};
    // workgroups per CU of each tile (registers and 160 KB of LDS): the lean
    // and wgrad 128 x 128 kernels fit four, the others three
    const int occ[4] = {(pl.tu || pass == PASS_WGRAD) ? 4 : 3, 5, 5, 8};
    auto util = [](int k) { return std::min(0.95, 0.35 + 0.3 * k); };
    double best = 1e300;
    const int KT = 16;
    const int ktiles = std::max(1, (pl.Kg + KT - 1) / KT);
    for (int c = 0; c < 4; ++c) {
        int mt = cand[c][0], nt = cand[c][1];
        if (force && (mt != force[0] || nt != force[1]))
            continue;
        int tm = (pl.M + mt - 1) / mt, tn = (pl.Ng + nt - 1) / nt;
        int64_t tiles = (int64_t)tm * tn * pl.phases;
        for (int sp = 1; sp <= 1024; sp *= 2) {
            if (sp > 1 && (ktiles / sp) < 4)
                break;
            int kps = (ktiles + sp - 1) / sp;
            int spe = (ktiles + kps - 1) / kps;
            if (force) {
                if (spe != force[2])
                    continue;
                pl.mt = mt; pl.nt = nt; pl.kt = KT; pl.splits = spe; pl.kt_per_split = kps;
                pl.tiles_m = tm; pl.tiles_n = tn;
                break;
            }
            int64_t wgs = tiles * spe;
            const int64_t per_cu = (wgs + 255) / 256; // workgroups the busiest CU works through
            const int64_t full = per_cu / occ[c], rem = per_cu % occ[c];
            const double wg_cycles = 2.0 * mt * nt * KT * kps / (256.0 * eff[c]);
            double t_main = (double)full * occ[c] * wg_cycles / util(occ[c]);
            if (rem)
                t_main += (double)rem * wg_cycles / util((int)rem);
            t_main /= 2.4; // ns at 2.4 GHz
            double t_red = 0;
            if (spe > 1)
                t_red = 4000.0 + 2.0 * (double)(spe + 1) * pl.M * pl.Ng * pl.phases * 4.0 / 4000.0; // ns
            double cost = t_main + t_red;
            if (cost < best * 0.97) {
                best = cost;
                pl.mt = mt; pl.nt = nt; pl.kt = KT; pl.splits = spe; pl.kt_per_split = kps;
                pl.tiles_m = tm; pl.tiles_n = tn;
            }
        }
    }
    pl.ws_bytes = pl.splits > 1 ? (size_t)pl.splits * pl.phases * pl.M * pl.Ng * sizeof(float) : 0;
    return pl;
}

// The (tile, split) pairs the search above visits, with repeats of the same
// effective split removed.
static int candidates_core(const ConvGeom &g, int pass, int32_t *out, int cap) {
    const GemmPlan base = plan_core(g, pass, nullptr);
    static const int cand[4][2] = {{128, 128}, {128, 64}, {64, 128}, {64, 64}};
    const int ktiles = std::max(1, (base.Kg + 15) / 16);
    int n = 0;
    for (int c = 0; c < 4; ++c) {
        int last = 0;
        for (int sp = 1; sp <= 1024; sp *= 2) {
            if (sp > 1 && (ktiles / sp) < 4)
                break;
            const int kps = (ktiles + sp - 1) / sp, spe = (ktiles + kps - 1) / kps;
            if (spe == last)
                continue;
            last = spe;
            if (n < cap && out) {
                out[3 * n] = cand[c][0];
                out[3 * n + 1] = cand[c][1];
                out[3 * n + 2] = spe;
            }
            ++n;
        }
    }
    return n;
}

static size_t round256(size_t b) { return (b + 255) / 256 * 256; }

// Forward and wgrad with C % 4 != 0 run on channel-padded copies of x (and of
// w, or of dw) held in the workspace after the split-K partial sums.
static bool pads_channels(const ConvGeom &g, int pass) {
    if (pass == PASS_DGRAD || g.C % 4 == 0)
        return false;
    const int64_t cp = (g.C + 3) / 4 * 4;
    return (int64_t)g.N * g.H * g.W * cp < INT_MAX && (int64_t)g.K * g.R * g.S * cp < INT_MAX;
}

static ConvGeom padded(const ConvGeom &g) {
    ConvGeom gp = g;
    gp.C = (g.C + 3) / 4 * 4;
    return gp;
}

int plan_candidates(const ConvGeom &g, int pass, int32_t *out, int cap) {
    return candidates_core(pads_channels(g, pass) ? padded(g) : g, pass, out, cap);
}

GemmPlan plan_gemm(const ConvGeom &g, int pass) {
    const bool pads = pads_channels(g, pass);
    const ConvGeom gp = pads ? padded(g) : g;
    int force[3];
    const int src = lookup_plan(g, pass, force);
    GemmPlan pl{};
    if (src == PLAN_TABLE || src == PLAN_PINNED) {
        pl = plan_core(gp, pass, force);
        pl.source = src;
    }
    if (pl.mt == 0) { // no measured plan, or one this shape cannot run
        pl = plan_core(gp, pass, nullptr);
        pl.source = PLAN_MODEL;
    }
    if (src != PLAN_PINNED && src != -1 && fc_streaming(g, pass)) {
        size_t fws = 0;
        fc_plan(g, pass, &pl.fc_splits, &pl.fc_chunk, &fws);
        pl.fc = true;
        pl.source = PLAN_FC;
        pl.ws_bytes = std::max(pl.ws_bytes, fws);
    }
    if (src != PLAN_PINNED && src != -1 && conv3_direct(g, pass)) {
        pl.direct = true;
        pl.source = PLAN_DIRECT;
        pl.ws_bytes = std::max(pl.ws_bytes, conv3_ws_bytes(g, pass));
    }
    if (!pads)
        return pl;
    pl.cpad = gp.C;
    pl.pad_x_off = round256(pl.ws_bytes);
    pl.pad_w_off = pl.pad_x_off + round256((size_t)g.N * g.H * g.W * gp.C * sizeof(float));
    pl.ws_bytes = pl.pad_w_off + round256((size_t)g.K * g.R * g.S * gp.C * sizeof(float));
    return pl;
}

static bool al16(const void *p) { return (uintptr_t)p % 16 == 0; }

int conv_forward(const ConvGeom &g, const GemmPlan &pl, const float *x, const float *w,
                 const float *bias, int relu, float *y, void *ws, hipStream_t s) {
    if (pl.direct && al16(y))
        return conv3_forward(g, x, w, bias, relu, y, s);
    if (pl.fc && ws && al16(x) && al16(w) && al16(y) && al16(bias) && al16(ws))
        return fc_forward(g, pl.fc_splits, pl.fc_chunk, x, w, bias, relu, y, ws, s);
    if (pl.cpad) {
        if (!ws)
            return fail(DC_EINVAL, "conv forward needs %zu bytes of workspace", pl.ws_bytes);
        float *xp = reinterpret_cast<float *>(static_cast<char *>(ws) + pl.pad_x_off);
        float *wp = reinterpret_cast<float *>(static_cast<char *>(ws) + pl.pad_w_off);
        DC_TRY(pad_channels(x, xp, (int64_t)g.N * g.H * g.W, g.C, pl.cpad, s));
        DC_TRY(pad_channels(w, wp, (int64_t)g.K * g.R * g.S, g.C, pl.cpad, s));
        const ConvGeom gp = padded(g);
        Args a = make_args(gp, pl);
        a.A = xp; a.B = wp; a.out = y; a.bias = bias; a.relu = relu;
        return run(gp, pl, a, ws, s);
    }
    Args a = make_args(g, pl);
    a.A = x; a.B = w; a.out = y; a.bias = bias; a.relu = relu;
    return run(g, pl, a, ws, s);
}

int conv_dgrad(const ConvGeom &g, const GemmPlan &pl, const float *dy, const float *w,
               int accumulate, float *dx, void *ws, hipStream_t s, const float *relu_mask) {
    if (pl.fc && al16(dy) && al16(w) && al16(dx) && al16(ws) && al16(relu_mask))
        return fc_dgrad(g, pl.fc_splits, pl.fc_chunk, dy, w, accumulate, dx, ws, s, relu_mask);
    Args a = make_args(g, pl);
    a.A = dy; a.B = w; a.out = dx; a.accumulate = accumulate; a.relu_mask = relu_mask;
    return run(g, pl, a, ws, s);
}

int conv_wgrad(const ConvGeom &g, const GemmPlan &pl, const float *x, const float *dy, float *dw,
               void *ws, hipStream_t s, float *dbias, bool *bias_done) {
    if (bias_done)
        *bias_done = false;
    if (pl.direct && ws && bias_done && al16(dy)) {
        *bias_done = true;
        return conv3_wgrad(g, x, dy, dw, dbias, ws, s);
    }
    if (pl.cpad) {
        if (!ws)
            return fail(DC_EINVAL, "conv wgrad needs %zu bytes of workspace", pl.ws_bytes);
        float *xp = reinterpret_cast<float *>(static_cast<char *>(ws) + pl.pad_x_off);
        float *dwp = reinterpret_cast<float *>(static_cast<char *>(ws) + pl.pad_w_off);
        DC_TRY(pad_channels(x, xp, (int64_t)g.N * g.H * g.W, g.C, pl.cpad, s));
        const ConvGeom gp = padded(g);
        Args a = make_args(gp, pl);
        a.A = dy; a.B = xp; a.out = dwp;
        DC_TRY(run(gp, pl, a, ws, s));
        return unpad_channels(dwp, dw, (int64_t)g.K * g.R * g.S, g.C, pl.cpad, s);
    }
    Args a = make_args(g, pl);
    a.A = dy; a.B = x; a.out = dw;
    return run(g, pl, a, ws, s);
}

} // namespace dc
