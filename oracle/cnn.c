/*
 * Oracle CNN primitives (test infrastructure only).
 *
 * Plain, slow reference loops for the layers of the parameter-server CNN
 * training iteration: the operators a worker runs between pulling the
 * parameters and pushing the gradients (the forward and backward
 * mini-procedures of Sec. III-A).  Only the tests, the smoke check and the
 * CPU baseline of the benchmark load this library; the product library
 * shares no code with it.
 *
 * Every tensor is double precision.  Activations are NHWC, filters KRSC
 * (k = output channel, then filter row r, filter column s, input channel c).
 * Each output element is one sum accumulated in the order its definition
 * lists the indices; loops only run over independent outputs in a different
 * order so that the compiler can vectorise across them.  OpenMP splits the
 * work across independent outputs only.
 *
 * Argmax decisions of max-pooling are taken on the values rounded to
 * float32, the precision the GPU kernels decide in; the first maximum in
 * row-major window order wins.
 */
#include <stdlib.h>
#include <string.h>

#define IDX4(a, b, c, d, B, C, D) ((((size_t)(a) * (B) + (b)) * (C) + (c)) * (D) + (d))

/* Convolution (cross-correlation, zero padding: pad rows above and below,
 * pad_w columns left and right):
 *   y[n,p,q,k] = b[k] + sum over r, s, c of x[n, p*st+r-pad, q*st+s-pad_w, c] * w[k,r,s,c]
 * Taps that fall into the padding contribute nothing.  b may be NULL. */
void or_conv2d_forward(int N, int H, int W, int C, int K, int R, int S, int st, int pad, int pad_w,
                       int P, int Q, const double *x, const double *w, const double *b,
                       double *y)
{
    /* wt[r][s][c][k] = w[k][r][s][c]: a copy, so the innermost loop runs over
     * independent outputs k with unit stride */
    double *wt = (double *)malloc(sizeof(double) * (size_t)K * R * S * C);
    for (int k = 0; k < K; ++k)
        for (int r = 0; r < R; ++r)
            for (int s = 0; s < S; ++s)
                for (int c = 0; c < C; ++c)
                    wt[IDX4(r, s, c, k, S, C, K)] = w[IDX4(k, r, s, c, R, S, C)];
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int n = 0; n < N; ++n)
        for (int p = 0; p < P; ++p)
            for (int q = 0; q < Q; ++q) {
                double *acc = y + IDX4(n, p, q, 0, P, Q, K);
                for (int k = 0; k < K; ++k)
                    acc[k] = b ? b[k] : 0.0;
                for (int r = 0; r < R; ++r) {
                    int h = p * st + r - pad;
                    if (h < 0 || h >= H)
                        continue;
                    for (int s = 0; s < S; ++s) {
                        int ww = q * st + s - pad_w;
                        if (ww < 0 || ww >= W)
                            continue;
                        const double *xp = x + IDX4(n, h, ww, 0, H, W, C);
                        for (int c = 0; c < C; ++c) {
                            const double xv = xp[c];
                            const double *wp = wt + IDX4(r, s, c, 0, S, C, K);
                            for (int k = 0; k < K; ++k)
                                acc[k] += xv * wp[k];
                        }
                    }
                }
            }
    free(wt);
}

/* Gradient of the convolution with respect to its input:
 *   dx[n,h,w,c] = sum over r, s, k of dy[n,p,q,k] * w[k,r,s,c]
 * over the taps with h = p*st + r - pad and w = q*st + s - pad_w for an output
 * position (p, q) inside the output. */
void or_conv2d_backward_data(int N, int H, int W, int C, int K, int R, int S, int st, int pad, int pad_w,
                             int P, int Q, const double *dy, const double *w, double *dx)
{
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int n = 0; n < N; ++n)
        for (int h = 0; h < H; ++h)
            for (int ww = 0; ww < W; ++ww) {
                double *acc = dx + IDX4(n, h, ww, 0, H, W, C);
                for (int c = 0; c < C; ++c)
                    acc[c] = 0.0;
                for (int r = 0; r < R; ++r) {
                    int t = h + pad - r;
                    if (t < 0 || t % st != 0 || t / st >= P)
                        continue;
                    int p = t / st;
                    for (int s = 0; s < S; ++s) {
                        int u = ww + pad_w - s;
                        if (u < 0 || u % st != 0 || u / st >= Q)
                            continue;
                        int q = u / st;
                        const double *dyp = dy + IDX4(n, p, q, 0, P, Q, K);
                        for (int k = 0; k < K; ++k) {
                            const double g = dyp[k];
                            const double *wp = w + IDX4(k, r, s, 0, R, S, C);
                            for (int c = 0; c < C; ++c)
                                acc[c] += g * wp[c];
                        }
                    }
                }
            }
}

/* Gradient of the convolution with respect to its filter:
 *   dw[k,r,s,c] = sum over n, p, q of dy[n,p,q,k] * x[n, p*st+r-pad, q*st+s-pad_w, c] */
void or_conv2d_backward_filter(int N, int H, int W, int C, int K, int R, int S, int st, int pad, int pad_w,
                               int P, int Q, const double *x, const double *dy, double *dw)
{
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int k = 0; k < K; ++k)
        for (int r = 0; r < R; ++r)
            for (int s = 0; s < S; ++s) {
                double *acc = dw + IDX4(k, r, s, 0, R, S, C);
                for (int c = 0; c < C; ++c)
                    acc[c] = 0.0;
                for (int n = 0; n < N; ++n)
                    for (int p = 0; p < P; ++p) {
                        int h = p * st + r - pad;
                        if (h < 0 || h >= H)
                            continue;
                        for (int q = 0; q < Q; ++q) {
                            int ww = q * st + s - pad_w;
                            if (ww < 0 || ww >= W)
                                continue;
                            const double g = dy[IDX4(n, p, q, k, P, Q, K)];
                            const double *xp = x + IDX4(n, h, ww, 0, H, W, C);
                            for (int c = 0; c < C; ++c)
                                acc[c] += g * xp[c];
                        }
                    }
            }
}

/* Max-pooling over R x S windows with stride st and padding pad (padded
 * positions never win).  arg[n,p,q,c] = r*S + s of the chosen element. */
void or_maxpool_forward(int N, int H, int W, int C, int R, int S, int st, int pad, int P, int Q,
                        const double *x, double *y, int *arg)
{
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int p = 0; p < P; ++p)
            for (int q = 0; q < Q; ++q)
                for (int c = 0; c < C; ++c) {
                    int best = -1;
                    float bestv = 0.0f;
                    double besty = 0.0;
                    for (int r = 0; r < R; ++r) {
                        int h = p * st + r - pad;
                        if (h < 0 || h >= H)
                            continue;
                        for (int s = 0; s < S; ++s) {
                            int ww = q * st + s - pad;
                            if (ww < 0 || ww >= W)
                                continue;
                            double v = x[IDX4(n, h, ww, c, H, W, C)];
                            float vf = (float)v;
                            if (best < 0 || vf > bestv) {
                                best = r * S + s;
                                bestv = vf;
                                besty = v;
                            }
                        }
                    }
                    y[IDX4(n, p, q, c, P, Q, C)] = besty;
                    arg[IDX4(n, p, q, c, P, Q, C)] = best;
                }
}

/* Backward of max-pooling: each output gradient goes to the input element its
 * window chose; overlapping windows add up. */
void or_maxpool_backward(int N, int H, int W, int C, int R, int S, int st, int pad, int P, int Q,
                         const double *dy, const int *arg, double *dx)
{
#pragma omp parallel for schedule(static)
    for (int n = 0; n < N; ++n) {
        memset(dx + IDX4(n, 0, 0, 0, H, W, C), 0, sizeof(double) * (size_t)H * W * C);
        for (int p = 0; p < P; ++p)
            for (int q = 0; q < Q; ++q)
                for (int c = 0; c < C; ++c) {
                    int a = arg[IDX4(n, p, q, c, P, Q, C)];
                    int h = p * st + a / S - pad;
                    int ww = q * st + a % S - pad;
                    dx[IDX4(n, h, ww, c, H, W, C)] += dy[IDX4(n, p, q, c, P, Q, C)];
                }
    }
}

/* Sampled outputs of the three convolution sums, one at a time, for layers
 * too large to evaluate whole.  Inputs are the float32 tensors themselves
 * (every float32 is exact in double); each sample is accumulated in double in
 * the order of its definition.  idx holds 4 indices per sample:
 *   forward (n, p, q, k); data gradient (n, h, w, c); filter gradient (k, r, s, c). */
void or_conv2d_forward_samples(int N, int H, int W, int C, int K, int R, int S, int st, int pad, int pad_w,
                               int P, int Q, const float *x, const float *w, const float *b,
                               int ns, const int *idx, double *out)
{
    (void)N;
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < ns; ++i) {
        int n = idx[4 * i], p = idx[4 * i + 1], q = idx[4 * i + 2], k = idx[4 * i + 3];
        double acc = b ? (double)b[k] : 0.0;
        for (int r = 0; r < R; ++r) {
            int h = p * st + r - pad;
            if (h < 0 || h >= H)
                continue;
            for (int s = 0; s < S; ++s) {
                int ww = q * st + s - pad_w;
                if (ww < 0 || ww >= W)
                    continue;
                for (int c = 0; c < C; ++c)
                    acc += (double)x[IDX4(n, h, ww, c, H, W, C)] * (double)w[IDX4(k, r, s, c, R, S, C)];
            }
        }
        (void)P;
        (void)Q;
        out[i] = acc;
    }
}

void or_conv2d_backward_data_samples(int N, int H, int W, int C, int K, int R, int S, int st, int pad, int pad_w,
                                     int P, int Q, const float *dy, const float *w,
                                     int ns, const int *idx, double *out)
{
    (void)N;
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < ns; ++i) {
        int n = idx[4 * i], h = idx[4 * i + 1], ww = idx[4 * i + 2], c = idx[4 * i + 3];
        double acc = 0.0;
        for (int r = 0; r < R; ++r) {
            int t = h + pad - r;
            if (t < 0 || t % st != 0 || t / st >= P)
                continue;
            int p = t / st;
            for (int s = 0; s < S; ++s) {
                int u = ww + pad_w - s;
                if (u < 0 || u % st != 0 || u / st >= Q)
                    continue;
                int q = u / st;
                for (int k = 0; k < K; ++k)
                    acc += (double)dy[IDX4(n, p, q, k, P, Q, K)] * (double)w[IDX4(k, r, s, c, R, S, C)];
            }
        }
        out[i] = acc;
    }
}

void or_conv2d_backward_filter_samples(int N, int H, int W, int C, int K, int R, int S, int st, int pad, int pad_w,
                                       int P, int Q, const float *x, const float *dy,
                                       int ns, const int *idx, double *out)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < ns; ++i) {
        int k = idx[4 * i], r = idx[4 * i + 1], s = idx[4 * i + 2], c = idx[4 * i + 3];
        double acc = 0.0;
        for (int n = 0; n < N; ++n)
            for (int p = 0; p < P; ++p) {
                int h = p * st + r - pad;
                if (h < 0 || h >= H)
                    continue;
                for (int q = 0; q < Q; ++q) {
                    int ww = q * st + s - pad_w;
                    if (ww < 0 || ww >= W)
                        continue;
                    acc += (double)dy[IDX4(n, p, q, k, P, Q, K)] * (double)x[IDX4(n, h, ww, c, H, W, C)];
                }
            }
        out[i] = acc;
    }
}
