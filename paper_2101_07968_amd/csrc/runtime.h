// The model object behind the dc_model handle of the C ABI.
#pragma once

#include "dc_internal.h"
#include "host_pool.h"

#include <condition_variable>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

namespace dc {

constexpr size_t NONE = (size_t)-1;

struct TensorInfo {
    int n = 0, h = 0, w = 0, c = 0;
    size_t act = NONE;   // byte offset of the activation in the workspace
    size_t grad = NONE;  // byte offset of its gradient
    int64_t size() const { return (int64_t)n * h * w * c; }
};

struct OpInfo {
    dc_op_desc d{};
    int out = 0;                     // output tensor id
    size_t w_off = NONE, b_off = NONE; // float offsets into the parameter vector (gamma/beta for BN)
    ConvGeom geom{};
    GemmPlan fwd{}, dgrad{}, wgrad{};
    dc_pool_shape pool{};
    size_t aux = NONE;               // BN: mean then invstd; MAXPOOL: argmax bytes
    int n_in = 1;                    // inputs: in0, in1, in2, in3 (ADD 2, CONCAT 2-4)
    int in[4] = {-1, -1, -1, -1};
    int ch_off[4] = {0, 0, 0, 0};    // CONCAT: channel offset of each input in the output
    bool grad_in[4] = {false, false, false, false};
    int acc_in[4] = {0, 0, 0, 0};    // backward adds into the input gradient
    // Forward ReLU folded into its producer: a CONV / FC / BN / ADD whose only
    // consumer is the next op, a ReLU of the same layer, writes max(., 0)
    // straight into the ReLU's output (relu_into = that tensor), and the ReLU
    // does nothing in the forward pass.  The producer's own output tensor is
    // then never written; nothing reads it (the ReLU's backward reads the
    // ReLU's output, the producer's backward reads its inputs).
    int relu_into = -1;
    bool fwd_folded = false;
    // Backward ReLU folding, for a BN or ADD with relu_into set: the
    // producer's backward reads the ReLU's output gradient and masks it with
    // the ReLU's output, and the ReLU's backward (bwd_folded) does nothing.
    bool bwd_folded = false;
    // Backward ReLU folding into a max-pool: a ReLU (not folded into a BN)
    // whose only consumer is the next op, a MAXPOOL of the same layer.  The
    // pool's backward writes the ReLU's input gradient directly, adding a
    // window's dy only where the window's maximum (the pool's output) is
    // positive; that maximum is the ReLU's output at the argmax, so this is
    // exactly the ReLU's mask.  relu_bwd_from is the ReLU's op index, set on
    // the MAXPOOL; the ReLU gets bwd_folded.
    int relu_bwd_from = -1;
    // The same for a ReLU whose only consumer is the next op, a CONV / FC
    // (possibly of the next layer): its data gradient is the ReLU's output
    // gradient, so the GEMM's epilogue keeps it where the ReLU's output is
    // positive and writes the ReLU's input gradient.  Set on the CONV / FC.
    int dgrad_relu_from = -1;
    // The same for a ReLU whose output is input k of a CONCAT (its only
    // consumer): the concatenation's backward masks that slice of its output
    // gradient and writes the ReLU's input gradient.
    int concat_relu_from[4] = {-1, -1, -1, -1};
};

} // namespace dc

struct dc_model {
    int batch = 0, in_h = 0, in_w = 0, in_c = 0, classes = 0, L = 0;
    int device = 0;
    std::vector<dc::OpInfo> ops;
    std::vector<dc::TensorInfo> tensors;
    size_t n_params = 0;
    std::vector<size_t> layer_off, layer_cnt;     // index 1..L
    std::vector<int> layer_first, layer_last;     // op index range of each layer

    // parameter server: pinned host memory
    float *ps_params = nullptr;
    float *ps_grads = nullptr;
    float *probe_host = nullptr;
    size_t probe_bytes = 0;

    // device workspace (caller-owned)
    char *ws = nullptr;
    size_t ws_bytes = 0;
    size_t ws_need = 0;
    size_t off_params = 0, off_grads = 0, off_scratch = 0, scratch_bytes = 0;
    size_t off_loss = 0, off_slots = 0;

    hipStream_t pull_s = nullptr, push_s = nullptr;
    std::vector<hipEvent_t> ev_pull_start, ev_pull_done, ev_bwd_done, ev_push_start, ev_push_done;
    std::vector<hipEvent_t> ev_fwd_start, ev_fwd_end, ev_bwd_end; // per layer, index 1..L (+ [0] / [L+1] sentinels)
    hipEvent_t ev_t0 = nullptr;
    // last work dc_step enqueues on the caller's stream (the loss copy into
    // probe_host); dc_model_destroy waits for it before freeing that buffer
    hipEvent_t ev_cs_done = nullptr;

    double lr = 0.01;
    int timeline = 0;
    double timeout_s = 600.0;
    int sgd_threads = 0;
    dc::HostPool *pool = nullptr;
    double wall_hz = 0;

    std::vector<int64_t> timeline_ns;
    bool timeline_valid = false;

    // Per-layer HIP graphs (DC_OPT_GRAPHS): the kernels of each layer's
    // forward and backward mini-procedures, captured once on a private
    // stream and replayed with one launch each.  They hold the workspace and
    // batch addresses they were captured with and are rebuilt when those
    // change.
    int use_graphs = 0;
    hipStream_t cap_s = nullptr;
    std::vector<hipGraphExec_t> g_fwd, g_bwd; // index 1..L
    const char *g_ws = nullptr;
    const float *g_x = nullptr;
    const int32_t *g_y = nullptr;

    // DC_OPT_GEMM_TIMING: an event before and after every GEMM pass of a step
    int gemm_timing = 0;
    std::vector<hipEvent_t> gemm_ev;  // 2 per pass, grown on demand
    std::vector<double> gemm_flop;    // algorithmic FLOPs of each timed pass
    size_t gemm_n = 0;                // passes timed in the current step

    float *dparams() const { return reinterpret_cast<float *>(ws + off_params); }
    float *dgrads() const { return reinterpret_cast<float *>(ws + off_grads); }
    float *act(int t) const { return reinterpret_cast<float *>(ws + tensors[t].act); }
    float *grad(int t) const { return reinterpret_cast<float *>(ws + tensors[t].grad); }
    void *scratch() const { return ws + off_scratch; }
    float *dloss() const { return reinterpret_cast<float *>(ws + off_loss); }
    uint64_t *slots() const { return reinterpret_cast<uint64_t *>(ws + off_slots); }
};

namespace dc {
// The tensor-gradient contributions of the backward pass in launch order
// (dc_backward_schedule).
struct BwdRecorder {
    std::vector<dc_grad_contrib> v;
};
// Enqueue the forward mini-procedures of layer l (and the loss after layer L)
// on stream s; x is the input batch, y its labels.
int run_forward_layer(dc_model *m, int l, const float *x, const int32_t *y, hipStream_t s);
// Enqueue the backward mini-procedures of layer l (x: the input batch).  With
// rec set, nothing is launched: the contributions the launches would make are
// appended to rec instead.
int run_backward_layer(dc_model *m, int l, const float *x, hipStream_t s, BwdRecorder *rec = nullptr);
// The same work through the layer's HIP graph when DC_OPT_GRAPHS is on (the
// graphs are captured at the first call for a workspace and batch).
int launch_forward_layer(dc_model *m, int l, const float *x, const int32_t *y, hipStream_t s);
int launch_backward_layer(dc_model *m, int l, const float *x, hipStream_t s);
void drop_graphs(dc_model *m);
// DC_OPT_GEMM_TIMING: record the event opening (start = true) or closing a
// GEMM pass of `flop` algorithmic FLOPs on stream s; a no-op when the option is
// off or the layer is being captured into a graph.
int gemm_mark(dc_model *m, bool start, double flop, hipStream_t s);
void free_gemm_events(dc_model *m);
} // namespace dc
