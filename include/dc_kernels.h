/*
 * libdc operator entry points: the gfx950 kernels that the executor runs for
 * each forward and backward mini-procedure (Sec. III-A), callable one at a
 * time.  Conventions (status codes, device pointers, void* streams, NHWC
 * activations, KRSC filters) are those of dc.h.  Every call only enqueues
 * work on `stream`; inputs and outputs are caller-owned device buffers.
 * Where a call takes `ws`, it is caller-owned device scratch of at least the
 * size its *_workspace_bytes() query returns (256-byte aligned); calls on one
 * stream may share it.  `accumulate` = 1 adds the result into the output
 * instead of overwriting it.  Shapes are validated on the host (DC_EINVAL);
 * empty shapes (a zero dimension) are a no-op.
 */
#ifndef DC_KERNELS_H
#define DC_KERNELS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Convolution geometry: input n x h x w x c, k filters of r x s x c, stride,
 * `pad` zero rows above and below and `pad_w` zero columns left and right
 * (pad < r, pad_w < s).  Output p x q with p = (h + 2 pad - r) / stride + 1,
 * q = (w + 2 pad_w - s) / stride + 1.  An FC layer of in -> out features is
 * the case h = w = r = s = 1, c = in, k = out, stride = 1, pad = pad_w = 0. */
typedef struct dc_conv_shape {
    int32_t n, h, w, c, k, r, s, stride, pad, pad_w;
} dc_conv_shape;

/* Scratch needed by the three conv passes of this shape (split-K partials). */
size_t dc_conv2d_workspace_bytes(const dc_conv_shape *sh);

/* y[n,p,q,k] = bias[k] + sum over r, s, c of x[n, p*stride+r-pad, q*stride+s-pad_w, c] * w[k,r,s,c],
 * then max(., 0) if relu; implicit GEMM on fp32 MFMA.  bias may be NULL. */
int dc_conv2d_forward(const dc_conv_shape *sh, const float *x, const float *w, const float *bias,
                      int relu, float *y, void *ws, size_t ws_bytes, void *stream);

/* For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): dc_conv2d_forward with no
 * workspace argument.  Its scratch (split-K partial sums, the channel-padded
 * copies of a C % 4 != 0 input) lives in a static device array of 64 MiB
 * (67,108,864 bytes) that each device holds until the process ends.  The call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine) and
 * gives the same result as dc_conv2d_forward under the same launch plan.  A
 * shape whose forward pass needs more scratch than that (at most
 * dc_conv2d_workspace_bytes) is refused with DC_EINVAL before anything is
 * launched.  Every call on one device shares its array and leaves its own
 * contents there: calls that overlap on a device (other streams, other host
 * threads) race; order them on one stream or synchronise between them.  The
 * first call on a device looks up that device's array address
 * (hipGetSymbolAddress) with the device current. */
int dc_conv2d_forward_noalloc(const dc_conv_shape *sh, const float *x, const float *w, const float *bias,
                              int relu, float *y, void *stream);

/* dx[n,h,w,c] (+)= sum over the (r, s, k) that reach (h, w) of dy[n,p,q,k] * w[k,r,s,c];
 * strided convolutions are split into stride^2 phase GEMMs with only the taps that hit. */
int dc_conv2d_backward_data(const dc_conv_shape *sh, const float *dy, const float *w,
                            int accumulate, float *dx, void *ws, size_t ws_bytes, void *stream);

/* The data gradient through a ReLU that feeds this convolution (its output
 * relu_y is the conv's input x): dx (+)= (relu_y > 0 ? the data gradient
 * above : 0), the ReLU's input gradient in one pass (chain rule of
 * Sec. III-A's backward procedure through both ops).  relu_y is laid out like
 * dx.  This is the launch a model makes when a ReLU's only reader is a conv or
 * FC. */
int dc_conv2d_backward_data_relu(const dc_conv_shape *sh, const float *dy, const float *w, const float *relu_y,
                                 int accumulate, float *dx, void *ws, size_t ws_bytes, void *stream);

/* dw[k,r,s,c] = sum over n, p, q of dy[n,p,q,k] * x[n, p*stride+r-pad, q*stride+s-pad_w, c];
 * dbias[k] = sum over n, p, q of dy[n,p,q,k] if dbias != NULL.  Deterministic
 * (fixed-order split-K). */
int dc_conv2d_backward_filter(const dc_conv_shape *sh, const float *x, const float *dy,
                              float *dw, float *dbias, void *ws, size_t ws_bytes, void *stream);

/* Launch plan the conv passes use for this shape (pass: 0 forward, 1 data
 * gradient, 2 filter gradient).  out[0..7] = workgroup tile M, tile N, split-K
 * factor, GEMM M, GEMM N, GEMM K, stride phases, and where the plan came from
 * (0 the occupancy cost model, 1 the library's table of measured plans, 2 a
 * plan pinned with dc_conv2d_set_plan, 3 the weight-streaming FC kernel, which
 * takes the data gradient of an FC shape (h = w = r = s = 1) of at most 32
 * rows, c % 4 == 0 and at least 4,000,000 weights unless a plan is pinned; its
 * tiles read as 0 and the split as its reduction splits; 4 the direct kernels
 * of the RGB input layer, which take the forward pass and filter gradient of
 * c = 3, r = s = 3, k a multiple of 32 from 32 to 128 unless a plan is
 * pinned; tiles 0, split 1).  out holds at least 8 int32.  Host only; for
 * inspection and tuning. */
int dc_conv2d_plan_info(const dc_conv_shape *sh, int pass, int32_t *out);

/* Every plan the pass can be launched with for this shape, as (tile M, tile N,
 * split-K factor) triples: writes min(cap, count) triples to out (3 int32
 * each; out may be NULL when cap is 0) and the number available to *count.
 * Host only. */
int dc_conv2d_plan_candidates(const dc_conv_shape *sh, int pass, int32_t *out, int cap, int32_t *count);

/* Pins the plan of one pass of one shape for the rest of the process: the conv
 * entry points, dc_conv2d_workspace_bytes and models created afterwards use
 * it (models already created keep their plans).  (mt, nt, splits) must be one
 * of dc_conv2d_plan_candidates' triples, else DC_EINVAL.  mt = 0 removes the
 * pin; mt = -1 pins the occupancy cost model's own choice, bypassing the table
 * of measured plans.  Every plan computes the same sums; they differ in speed
 * and in the rounding order of split-K partial sums.  Thread-safe.  Host
 * only; for tuning (timing candidates through the conv entry points). */
int dc_conv2d_set_plan(const dc_conv_shape *sh, int pass, int mt, int nt, int splits);

/* y = max(x, 0) over n floats. */
int dc_relu_forward(const float *x, float *y, int64_t n, void *stream);
/* dx (+)= dy where y > 0, else 0 (relu'(0) = 0). */
int dc_relu_backward(const float *dy, const float *y, int accumulate, float *dx, int64_t n,
                     void *stream);

/* Max-pooling geometry: input n x h x w x c, window r x s, stride, padding. */
typedef struct dc_pool_shape {
    int32_t n, h, w, c, r, s, stride, pad;
} dc_pool_shape;

/* y = window max; arg = r*s_win + s of the first maximum in row-major window order. */
int dc_maxpool_forward(const dc_pool_shape *sh, const float *x, float *y, uint8_t *arg,
                       void *stream);
/* dx (+)= the sum of dy over the windows whose argmax is this element. */
int dc_maxpool_backward(const dc_pool_shape *sh, const float *dy, const uint8_t *arg,
                        int accumulate, float *dx, void *stream);

/* The same through a ReLU that feeds the pool (x = relu(u)): du (+)= the sum
 * of dy over the windows whose argmax is this element, where that window's
 * maximum y (this pool's output) is positive.  The maximum is the ReLU's
 * output at the argmax, so this is the ReLU's mask.  The launch a model makes
 * when a ReLU's only reader is the max-pool after it. */
int dc_maxpool_backward_relu(const dc_pool_shape *sh, const float *dy, const uint8_t *arg, const float *y,
                             int accumulate, float *dx, void *stream);

/* Average pooling: y = the mean of x over the window positions that lie
 * inside the input (padded positions are not counted).  Backward: dx (+)=
 * the sum, over the windows containing each element, of dy / that window's
 * count.  Element counts must stay below 2^31 (else DC_EINVAL). */
int dc_avgpool_forward(const dc_pool_shape *sh, const float *x, float *y, void *stream);
int dc_avgpool_backward(const dc_pool_shape *sh, const float *dy, int accumulate, float *dx, void *stream);

/* Global average pooling: y[n,c] = mean over hw of x[n,hw,c]; backward spreads dy / hw. */
int dc_gap_forward(int32_t n, int32_t hw, int32_t c, const float *x, float *y, void *stream);
int dc_gap_backward(int32_t n, int32_t hw, int32_t c, const float *dy, int accumulate, float *dx,
                    void *stream);

/* y = a + b over n floats; relu = 1 gives max(a + b, 0). */
int dc_add_forward(const float *a, const float *b, int relu, float *y, int64_t n, void *stream);
/* dx (+)= dy over n floats. */
int dc_copy_grad(const float *dy, int accumulate, float *dx, int64_t n, void *stream);

/* Backward of relu(a + b) over n floats: with m = (y > 0 ? dy : 0), y the
 * ReLU's output and dy its gradient, dx0 (+)= m and dx1 (+)= m (acc0 / acc1
 * choose add or write for each); either dx may be NULL (skipped).  The launch
 * a model makes for a residual add followed by a ReLU. */
int dc_add_relu_backward(const float *dy, const float *y, int acc0, float *dx0, int acc1, float *dx1, int64_t n,
                         void *stream);

/* Channel concatenation of NHWC tensors viewed as [rows][channels]:
 * forward y[m][off + c] = x[m][c] for c < c_in, y having c_out channels;
 * backward dx[m][c] (+)= dy[m][off + c]. */
int dc_concat_forward(int64_t rows, int32_t c_in, int32_t c_out, int32_t off, const float *x, float *y,
                      void *stream);
int dc_concat_backward(int64_t rows, int32_t c_in, int32_t c_out, int32_t off, const float *dy,
                       int accumulate, float *dx, void *stream);

/* The concatenation's backward into the input of a ReLU whose output is this
 * input (relu_y, laid out like dx): dx[m][c] (+)= (relu_y[m][c] > 0 ?
 * dy[m][off + c] : 0).  The launch a model makes when a ReLU's only reader is
 * a concatenation. */
int dc_concat_backward_relu(int64_t rows, int32_t c_in, int32_t c_out, int32_t off, const float *dy,
                            const float *relu_y, int accumulate, float *dx, void *stream);

/* BatchNorm over rows = n*h*w rows of c channels (NHWC viewed as [rows][c]). */
size_t dc_batchnorm_workspace_bytes(int64_t rows, int32_t c);
/* mean, invstd (c floats each, outputs) = batch statistics with the biased
 * variance; y = gamma * (x - mean) * invstd + beta; invstd = 1/sqrt(var + eps). */
int dc_batchnorm_forward(int64_t rows, int32_t c, const float *x, const float *gamma,
                         const float *beta, float eps, float *y, float *mean, float *invstd,
                         void *ws, size_t ws_bytes, void *stream);
/* dgamma = sum dy*xhat, dbeta = sum dy,
 * dx (+)= gamma*invstd*(dy - dbeta/rows - xhat*dgamma/rows), xhat = (x-mean)*invstd. */
int dc_batchnorm_backward(int64_t rows, int32_t c, const float *dy, const float *x,
                          const float *gamma, const float *mean, const float *invstd,
                          int accumulate, float *dx, float *dgamma, float *dbeta, void *ws,
                          size_t ws_bytes, void *stream);

/* BatchNorm backward through the ReLU applied to its output: dy is the
 * ReLU's output gradient and relu_y = relu(y) the ReLU's output; the
 * backward above runs on (relu_y > 0 ? dy : 0).  The launch a model makes for
 * a BatchNorm followed by a ReLU.  dx may be NULL (no data gradient). */
int dc_batchnorm_backward_relu(int64_t rows, int32_t c, const float *dy, const float *relu_y, const float *x,
                               const float *gamma, const float *mean, const float *invstd, int accumulate,
                               float *dx, float *dgamma, float *dbeta, void *ws, size_t ws_bytes, void *stream);

/* loss[0] = mean over n of (logsumexp(z_i) - z_i[y_i]); dz = (softmax(z) - onehot(y)) / n.
 * logits n x classes.  Labels are not range-checked: a label outside
 * [0, classes) is taken as "no target" (that sample contributes
 * logsumexp(z_i) to the loss and softmax(z_i) / n to dz), and no memory
 * outside the logits is read. */
size_t dc_softmax_xent_workspace_bytes(int32_t n);
int dc_softmax_xent(int32_t n, int32_t classes, const float *logits, const int32_t *labels,
                    float *loss, float *dlogits, void *ws, size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* DC_KERNELS_H */
