/*
 * libdc - one parameter-server CNN training iteration with DynaComm's
 * segment-overlapped pulls and pushes, on one MI355X (gfx950).
 *
 * The iteration of the default parameter server has four procedures run in
 * sequence: pull the parameters, forward, backward, push the gradients
 * (Sec. III-A).  Each procedure splits into one mini-procedure per layer, and
 * DynaComm batches the per-layer transmissions into segments chosen by two
 * dynamic programs over per-layer timing profiles (Sec. IV-B, Eq. 8 and 9).
 * This library provides the profiler (dc_profile), the planner (dc_plan) and
 * the executor (dc_step) of that scheme.  The parameter server is pinned host
 * memory owned by the library; the link between it and the GPU is the host
 * interface, paced to an emulated rate when asked.
 *
 * Conventions for every call:
 *  - Return value: DC_OK (0) or one of the DC_E* codes; no call throws or
 *    aborts.  dc_strerror() names a code, dc_last_error() describes the last
 *    failure on the calling thread, dc_last_hip_error() gives the hipError_t
 *    behind the last DC_EHIP.
 *  - "device" pointers are HIP device memory of the current device; "host"
 *    pointers are ordinary host memory.  Streams are hipStream_t passed as
 *    void*; NULL is the null stream.
 *  - Activations are NHWC float32; conv filters are KRSC (output channel,
 *    filter row, filter column, input channel); FC weights are [out][in]
 *    over the NHWC-flattened input.
 *  - Costs and times are int64 nanoseconds.
 */
#ifndef DC_H
#define DC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------ status */

enum {
    DC_OK = 0,
    DC_EINVAL = 1,   /* an argument is out of range or inconsistent */
    DC_EHIP = 2,     /* a HIP runtime call failed; see dc_last_hip_error() */
    DC_ENOMEM = 3,   /* host allocation failed or the workspace is too small */
    DC_ESTATE = 4,   /* call out of order (e.g. no workspace bound yet) */
    DC_ETIMEOUT = 5  /* the watchdog of dc_step / dc_profile expired */
};

const char *dc_strerror(int status);
/* Text of the last failure on this thread ("" if none). */
const char *dc_last_error(void);
/* hipError_t value of the last DC_EHIP on this thread (0 if none). */
int dc_last_hip_error(void);

/* ------------------------------------------------------------ network */

enum {
    DC_OP_CONV = 1,    /* 2-D convolution (cross-correlation), zero padding, optional bias */
    DC_OP_FC = 2,      /* fully connected layer over the NHWC-flattened input, optional bias */
    DC_OP_BN = 3,      /* BatchNorm, training mode: batch statistics, biased variance */
    DC_OP_RELU = 4,
    DC_OP_MAXPOOL = 5, /* r x s window, stride, padding; padded positions never win */
    DC_OP_GAP = 6,     /* global average pooling to N x 1 x 1 x C */
    DC_OP_ADD = 7,     /* elementwise sum of in0 and in1 (residual connection) */
    DC_OP_CONCAT = 8,  /* channel concatenation of in0, in1 and, if not -1, in2 and in3 */
    DC_OP_AVGPOOL = 9  /* r x s window, stride, padding; the mean over the window's positions inside the input */
};

/*
 * One operation of the network, in forward order.  Tensor 0 is the input
 * batch; tensor i+1 is the output of operation i.  `layer` is the planner
 * layer (1-based): layers are contiguous and non-decreasing along the list,
 * and each layer's first operation is a CONV or FC.  Following Sec. III-A, a
 * layer is one weighted operation with the parameter-less operations that
 * follow it; branches at the same depth (a residual block's projection, the
 * parallel convs of an Inception module) may share a layer.  A layer's parameters are one contiguous byte range of the
 * parameter server: its operations in order, each weight then bias
 * (CONV/FC) or gamma then beta (BN).  The last operation must produce
 * N x 1 x 1 x classes logits; the loss is the batch mean of the softmax
 * cross-entropy, folded into the last layer.
 */
typedef struct dc_op_desc {
    int32_t kind;    /* DC_OP_* */
    int32_t layer;   /* planner layer, 1..L */
    int32_t in0;     /* input tensor id (< own id) */
    int32_t in1;     /* DC_OP_ADD / DC_OP_CONCAT: second input tensor id; otherwise -1 */
    int32_t out_ch;  /* CONV: output channels; FC: output features */
    int32_t r, s;    /* CONV / MAXPOOL / AVGPOOL window (rows, columns) */
    int32_t stride;  /* CONV / MAXPOOL / AVGPOOL */
    int32_t pad;     /* CONV / MAXPOOL / AVGPOOL: zero rows above and below */
    int32_t bias;    /* CONV / FC: 1 if the op has a bias */
    int32_t in2;     /* DC_OP_CONCAT: third input tensor id or -1; otherwise -1 */
    int32_t in3;     /* DC_OP_CONCAT: fourth input tensor id or -1; otherwise -1 */
    int32_t pad_w;   /* CONV: zero columns left and right (pad_w < s); pools: equal to pad */
} dc_op_desc;

typedef struct dc_model dc_model;

/*
 * One contribution to a tensor's gradient in the backward pass: the chain-rule
 * term of op `origin_op` for its input `tensor`, performed by the launch of op
 * `exec_op` (a ReLU's term can be carried out by the op that reads its
 * output, or by the BN / ADD that produced its input).  accumulate = 1 adds
 * it to what earlier contributions wrote, 0 writes it.  fused = 1: the term is
 * formed inside that launch and never stored.
 */
typedef struct dc_grad_contrib {
    int32_t tensor;
    int32_t origin_op;
    int32_t exec_op;
    int32_t accumulate;
    int32_t fused;
} dc_grad_contrib;

/*
 * Build a model for `batch` images of in_h x in_w x in_c and `classes`
 * classes.  Allocates the pinned parameter-server buffers (parameters and
 * gradients, zero-filled) and the library's side streams and events on the
 * current device.  *out is owned by the caller and released with
 * dc_model_destroy().  Errors: DC_EINVAL for an inconsistent description,
 * DC_ENOMEM, DC_EHIP.
 */
int dc_model_create(const dc_op_desc *ops, int n_ops, int batch, int in_h, int in_w, int in_c,
                    int classes, dc_model **out);
/* Waits for the library's own work (side streams, and what dc_step queued last
 * on the caller's stream), then frees the model.  The caller's workspace and
 * any other work on its stream stay the caller's to synchronise. */
void dc_model_destroy(dc_model *m);

/*
 * The backward pass's tensor-gradient contributions for a network, in the
 * order the launches of dc_step make them (layers L..1, each layer's ops last
 * to first).  The description is validated as by dc_model_create; no HIP call
 * is made and no device is needed.  Sec. III-A's backward procedure applies
 * the chain rule op by op in reverse; a tensor read by several ops receives
 * their terms in reverse op order, the first written and the rest added, so
 * each gradient is one fixed sum whatever the segmentation.  This call shows
 * where a folded ReLU's term is carried out.  Writes up to `cap` entries to
 * `out` (caller-owned; may be NULL when cap is 0) and the number of entries
 * into *n_out.  Errors: those of dc_model_create's validation; DC_EINVAL when
 * cap is smaller than the number of entries (*n_out is still set).
 */
int dc_backward_schedule(const dc_op_desc *ops, int n_ops, int batch, int in_h, int in_w, int in_c, int classes,
                         dc_grad_contrib *out, int cap, int *n_out);

int dc_model_num_layers(const dc_model *m);      /* L */
size_t dc_model_num_params(const dc_model *m);   /* float32 parameters in total */

/* Bytes of device workspace the model needs: parameters, gradients,
 * activations and their gradients, saved statistics and kernel scratch. */
size_t dc_workspace_bytes(const dc_model *m);

/* Hand the model a device buffer of at least dc_workspace_bytes() bytes,
 * 256-byte aligned.  The caller keeps ownership and must keep it alive while
 * the model is used.  Errors: DC_EINVAL (NULL, misaligned), DC_ENOMEM (too
 * small). */
int dc_model_bind_workspace(dc_model *m, void *dev, size_t bytes);

/* Parameter range of planner layer `layer` (1..L): first float and count. */
int dc_layer_range(const dc_model *m, int layer, size_t *off, size_t *count);

/* Options (dc_model_set_option). */
enum {
    DC_OPT_LR = 1,          /* SGD learning rate at the server (default 0.01) */
    DC_OPT_TIMELINE = 2,    /* 1: dc_step records per-layer timestamps (default 0) */
    DC_OPT_TIMEOUT_S = 3,   /* watchdog for one dc_step / dc_profile in seconds (default 600) */
    DC_OPT_SGD_THREADS = 4, /* host threads of the server update (default: hardware threads, max 16) */
    DC_OPT_GRAPHS = 5,      /* 1: each layer's forward and backward kernels run as one captured HIP graph
                               launch (default 0: launched one by one).  The graphs are captured at the first
                               dc_step / dc_profile for a workspace and batch address (a one-time cost) and
                               recaptured when either changes; results are identical either way.  A graph
                               launch costs more than it saves unless a layer is many kernels of ~1 us */
    DC_OPT_GEMM_TIMING = 6  /* 1: dc_step brackets every conv / FC GEMM pass it launches (forward, data and
                               filter gradient, each with its split-K reduction) with a pair of HIP events on
                               the compute stream and reports their summed durations and algorithmic FLOPs in
                               dc_step_stats (default 0).  Ignored while DC_OPT_GRAPHS is on */
};
int dc_model_set_option(dc_model *m, int option, double value);

/* ------------------------------------------------------------ parameter server */

/* Copy n = dc_model_num_params() host floats into the server's parameters. */
int dc_ps_write(dc_model *m, const float *host_params, size_t n);
/* Copy the server's parameters and/or last pushed gradients out (either
 * pointer may be NULL). */
int dc_ps_read(const dc_model *m, float *params_out, float *grads_out, size_t n);

/* Copy one tensor of the last dc_step / dc_profile out of the workspace, for
 * checks against an oracle (the discrete decisions of Sec. III-A's forward:
 * which ReLU inputs were positive, which window tap each max-pool took).
 * tensor 0 is the input batch, tensor i + 1 the output of op i.
 *   what = DC_READ_ACT:    the activation, n*h*w*c float32 (NHWC) -> host;
 *   what = DC_READ_ARGMAX: when op tensor-1 is a max-pool, its window tap per
 *                          output element (r * S + s), n*h*w*c uint8 -> host.
 * bytes must equal the tensor's size.  DC_EINVAL for a bad tensor or size,
 * DC_READ_ACT of tensor 0 (the caller's own buffer) or of an activation the
 * model does not keep (the output of a conv / FC / BN / add whose ReLU is
 * folded into it: only the ReLU's output is written), or DC_READ_ARGMAX on
 * anything but a max-pool output; DC_ESTATE when no workspace is bound.
 * Waits for the model's work to finish first. */
enum { DC_READ_ACT = 0, DC_READ_ARGMAX = 1 };
int dc_model_read_tensor(const dc_model *m, int tensor, int what, void *host, size_t bytes);

/* ------------------------------------------------------------ link and batch */

/*
 * The emulated link between the parameter server and the worker.  A
 * transmission mini-procedure of `bytes` occupies the link for
 * dt_emul_ns + bytes / bytes_per_s when paced, or dt_emul_ns plus the real
 * copy time when not; its data is usable when it ends.  Transmissions run
 * one at a time in each direction.
 */
typedef struct dc_link {
    double bytes_per_s;  /* emulated rate (paced = 1), > 0 */
    int64_t dt_emul_ns;  /* extra per-transmission set-up time, >= 0 */
    int32_t paced;       /* 1: pace copies to bytes_per_s; 0: host interface speed */
} dc_link;

/* One batch, resident in device memory: x is N x H x W x C float32 (NHWC),
 * y holds N int32 labels in [0, classes). */
typedef struct dc_batch {
    const float *x_dev;
    const int32_t *y_dev;
    int32_t n;           /* must equal the model's batch */
} dc_batch;

/* ------------------------------------------------------------ profiler (Sec. IV-A) */

/*
 * Per-layer cost vectors pt, fc, bc, gt and the per-transmission overhead dt
 * that the schedulers take as input (Sec. III-B, IV-A).  The caller owns
 * the four arrays of L entries.
 */
typedef struct dc_profile_t {
    int32_t L;
    int64_t *pt_ns;  /* pull time of each layer's parameters */
    int64_t *fc_ns;  /* forward compute time of each layer (the loss folds into layer L) */
    int64_t *bc_ns;  /* backward compute time of each layer */
    int64_t *gt_ns;  /* push time of each layer's gradients */
    int64_t dt_ns;   /* overhead of one transmission mini-procedure */
} dc_profile_t;

/*
 * Fill *out for this model, batch and link: fc and bc are the mean over
 * `reps` timed forward+backward passes (after one warm-up) of per-layer
 * event intervals on `stream`; dt and the host-interface rate come from a
 * least-squares fit t = a + bytes / rate over probe copies; pt = gt =
 * bytes / rate at the emulated rate when paced, the fitted one otherwise;
 * dt = a + h + dt_emul_ns, where h is the measured latency of the
 * cross-stream handoff every segment adds (compute waiting for a pull, a
 * push waiting for the backward).  Pulls all parameters to the device first.
 * Errors: DC_EINVAL (L or batch mismatch, reps < 1), DC_ESTATE, DC_EHIP.
 */
int dc_profile(dc_model *m, const dc_batch *b, const dc_link *link, int reps, void *stream,
               dc_profile_t *out);

/* ------------------------------------------------------------ planner (Sec. IV-B) */

/*
 * Pull / push decisions.  p[l-1] is p_l and g[k-1] is g_k for l, k = 1..L-1
 * (Sec. III-B): p_l = 1 starts a new pull mini-procedure at layer l+1;
 * g_k = 1 puts a push boundary between layer L-k+1 and layer L-k.  The
 * caller owns p and g (L-1 bytes each).  t_fwd_ns and t_bwd_ns are the
 * model's estimates f_m for the decision.
 */
typedef struct dc_plan_t {
    int32_t L;
    uint8_t *p;
    uint8_t *g;
    int64_t t_fwd_ns;
    int64_t t_bwd_ns;
} dc_plan_t;

/*
 * DynaComm's optimal decisions: the forward dynamic program of Eq. 8 with
 * Algorithm 3's traceback, and the backward one of Eq. 9 with Algorithm 4's,
 * in exact int64 arithmetic.  Ties keep the smallest split point and then
 * the fewest segments.  Pure host code, thread-safe, O(L^3) time and O(L^2)
 * space.  Errors: DC_EINVAL for L < 1, negative costs or int64 overflow.
 */
int dc_plan(const dc_profile_t *prof, dc_plan_t *out);
/* The default parameter server (one pull, one push) and layer-by-layer
 * (every position enabled) decisions, with f_m filled from prof. */
int dc_plan_sequential(const dc_profile_t *prof, dc_plan_t *out);
int dc_plan_lbl(const dc_profile_t *prof, dc_plan_t *out);
/* iBatch, the greedy baseline of Sec. III-C: Algorithm 1 (front-to-back
 * forward batching; its reverse twin is not given in the paper) and
 * Algorithm 2 (gradient batching over every second position, keeping the
 * candidate of least f_m), with f_m filled in.  Same errors as dc_plan. */
int dc_plan_ibatch(const dc_profile_t *prof, dc_plan_t *out);
/* Fill t_fwd_ns / t_bwd_ns of a given decision with the cost function f_m. */
int dc_plan_eval(const dc_profile_t *prof, dc_plan_t *plan);

/* ------------------------------------------------------------ executor */

typedef struct dc_step_stats {
    float loss;            /* batch mean of the softmax cross-entropy */
    int32_t n_pull;        /* pull segments */
    int32_t n_push;        /* push segments */
    int64_t t_iter_ns;     /* start of the first pull to the end of the last push */
    int64_t t_fwd_ns;      /* start of the first pull to the end of the forward pass and loss */
    int64_t t_bwd_ns;      /* end of the forward pass to the end of the last push */
    int64_t t_compute_ns;  /* forward + backward kernel time on the compute stream */
    int64_t t_link_ns;     /* sum of the pull and push segment durations */
    int64_t t_sgd_tail_ns; /* server update after the last push ended (outside t_iter) */
    int64_t t_host_ns;     /* wall time of the whole dc_step call */
    int64_t t_plan_bwd_ns; /* dc_step_dynamic: host time of the backward DP (0 otherwise) */
    int64_t t_plan_fwd_ns; /* dc_step_dynamic: host time of the next forward DP (0 otherwise) */
    int32_t plan_hidden;   /* dc_step_dynamic: bit 0 set if the backward DP ended before the forward
                              pass did, bit 1 if the next forward DP ended before the last push did */
    int32_t n_gemm;        /* DC_OPT_GEMM_TIMING: conv / FC GEMM passes timed in this step (0 otherwise) */
    int64_t t_gemm_ns;     /* DC_OPT_GEMM_TIMING: their summed durations, from events on the compute stream */
    double gemm_flop;      /* DC_OPT_GEMM_TIMING: their algorithmic FLOPs, 2 per multiply-add */
} dc_step_stats;

/*
 * One training iteration (Sec. III-A) under the given decisions:
 * pull segment j (a side stream) copies its layers' parameters from the
 * server to the device and records an event; the forward kernels of a layer
 * wait only for the segment holding that layer (Eq. 1); backward runs layers
 * L..1 (Eq. 6) and records an event when it finishes the lowest layer of a
 * push segment; push segment j (another side stream) then copies those
 * gradients to the server (Eq. 2, 7), where host threads apply SGD to the
 * range as soon as it lands.  Returns when every push and every update is
 * done.  `stream` is the compute stream.  The results do not depend on the
 * decisions.  Errors: DC_EINVAL (plan L or batch size mismatch, bad link),
 * DC_ESTATE (no workspace), DC_EHIP, DC_ETIMEOUT.  After DC_ETIMEOUT (the
 * DC_OPT_TIMEOUT_S watchdog), copies and kernels of the iteration may still
 * be running; they end on their own (every pacing wait is bounded), the
 * server update of the unfinished segments is not applied, and
 * dc_model_destroy waits for them.
 */
int dc_step(dc_model *m, const dc_batch *b, const dc_plan_t *plan, const dc_link *link,
            void *stream, dc_step_stats *out);

/*
 * One iteration in DynaComm's run-time mode with the idle-event trigger
 * (Sec. IV-C): this iteration's pulls and forward pass use plan->p; the
 * backward decision is computed by the backward DP (Eq. 9, Algorithm 4) on
 * `prof` while the pulls and the forward pass are in flight (the host has
 * already enqueued them), and the forward decision of the
 * next iteration (Eq. 8, Algorithm 3) while the last push is in flight, so
 * planning stays off the critical path.  On return plan->g holds the
 * backward decision that was used and plan->p the decision for the next
 * call (with t_fwd_ns / t_bwd_ns from f_m).  `prof` is typically refreshed by
 * dc_profile once per epoch.  Errors as dc_step, plus those of dc_plan.
 */
int dc_step_dynamic(dc_model *m, const dc_batch *b, const dc_profile_t *prof, const dc_link *link,
                    void *stream, dc_plan_t *plan, dc_step_stats *out);

/*
 * Per-layer timestamps of the last dc_step run with DC_OPT_TIMELINE on, in
 * ns from the start of the first pull: out[8*(l-1) + 0..7] = pull start,
 * pull end, forward start, forward end, backward start, backward end, push
 * start, push end of layer l (pull/push times are those of its segment).
 * `out` holds 8*L entries.  Errors: DC_ESTATE if no timeline was recorded.
 */
int dc_timeline(const dc_model *m, int64_t *out, int n);

#ifdef __cplusplus
}
#endif

#endif /* DC_H */
