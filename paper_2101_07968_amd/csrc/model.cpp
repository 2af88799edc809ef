// Model construction, workspace layout, the parameter server's buffers and
// the per-layer forward / backward mini-procedures.
//
// A layer (Sec. III-A) is one weighted op plus the parameter-less ops after
// it; its parameters are one contiguous range of the parameter vector, so a
// pull or push segment of consecutive layers is one contiguous copy.  Every
// tensor gets its own activation and gradient buffer in the caller's device
// workspace; a tensor read by several ops receives the backward contributions
// in reverse op order, the first one writing and the rest accumulating, so
// the result never depends on timing.
#include "runtime.h"

#include <algorithm>
#include <climits>
#include <cstring>

namespace dc {

namespace {

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int check_desc(const dc_op_desc *ops, int n_ops, int batch, int in_h, int in_w, int in_c, int classes) {
    if (!ops || n_ops < 1)
        return fail(DC_EINVAL, "no operations");
    if (batch < 1 || in_h < 1 || in_w < 1 || in_c < 1 || classes < 1)
        return fail(DC_EINVAL, "batch and input sizes must be positive");
    if ((int64_t)batch * in_h * in_w * in_c >= INT_MAX)
        return fail(DC_EINVAL, "input batch of %lld elements (the limit is 2^31 - 1)",
                    (long long)batch * in_h * in_w * in_c);
    int prev_layer = 0;
    for (int i = 0; i < n_ops; ++i) {
        const dc_op_desc &d = ops[i];
        if (d.kind < DC_OP_CONV || d.kind > DC_OP_AVGPOOL)
            return fail(DC_EINVAL, "op %d: unknown kind %d", i, d.kind);
        if (d.in0 < 0 || d.in0 > i)
            return fail(DC_EINVAL, "op %d: input tensor %d is not an earlier tensor", i, d.in0);
        if ((d.kind == DC_OP_ADD || d.kind == DC_OP_CONCAT) && (d.in1 < 0 || d.in1 > i))
            return fail(DC_EINVAL, "op %d: second input tensor %d is not an earlier tensor", i, d.in1);
        if (d.kind == DC_OP_CONCAT) {
            if (d.in2 < -1 || d.in2 > i || d.in3 < -1 || d.in3 > i || (d.in2 < 0 && d.in3 >= 0))
                return fail(DC_EINVAL, "op %d: concat inputs in2 / in3 must be earlier tensors or -1", i);
        }
        // The input batch (tensor 0) has no activation or gradient buffer of
        // its own: only a CONV / FC reads it, and its backward skips dgrad.
        const bool weighted_op = d.kind == DC_OP_CONV || d.kind == DC_OP_FC;
        const bool multi = d.kind == DC_OP_ADD || d.kind == DC_OP_CONCAT;
        if ((!weighted_op && d.in0 == 0) || (multi && d.in1 == 0) ||
            (d.kind == DC_OP_CONCAT && (d.in2 == 0 || d.in3 == 0)))
            return fail(DC_EINVAL, "op %d: only a CONV or FC may read the input batch (tensor 0)", i);
        if (d.layer != prev_layer && d.layer != prev_layer + 1)
            return fail(DC_EINVAL, "op %d: layers must be contiguous and non-decreasing", i);
        bool weighted = d.kind == DC_OP_CONV || d.kind == DC_OP_FC;
        if (d.layer == prev_layer + 1 && !weighted)
            return fail(DC_EINVAL, "op %d: layer %d must start with a CONV or FC op", i, d.layer);
        prev_layer = d.layer;
    }
    if (ops[0].layer != 1)
        return fail(DC_EINVAL, "the first op must belong to layer 1");
    return DC_OK;
}

} // namespace

static int build_model(dc_model *m, const dc_op_desc *ops, int n_ops) {
    m->ops.resize(n_ops);
    m->tensors.resize(n_ops + 1);
    m->tensors[0] = TensorInfo{m->batch, m->in_h, m->in_w, m->in_c};
    size_t poff = 0;
    m->L = ops[n_ops - 1].layer;
    m->layer_off.assign(m->L + 2, 0);
    m->layer_cnt.assign(m->L + 2, 0);
    m->layer_first.assign(m->L + 2, -1);
    m->layer_last.assign(m->L + 2, -1);
    for (int i = 0; i < n_ops; ++i) {
        OpInfo &o = m->ops[i];
        o.d = ops[i];
        o.out = i + 1;
        o.in[0] = o.d.in0;
        o.n_in = 1;
        if (o.d.kind == DC_OP_ADD || o.d.kind == DC_OP_CONCAT) {
            o.in[1] = o.d.in1;
            o.n_in = 2;
        }
        if (o.d.kind == DC_OP_CONCAT) {
            if (o.d.in2 >= 0)
                o.in[o.n_in++] = o.d.in2;
            if (o.d.in3 >= 0)
                o.in[o.n_in++] = o.d.in3;
        }
        const TensorInfo in = m->tensors[o.d.in0];
        TensorInfo out = in;
        int l = o.d.layer;
        if (m->layer_first[l] < 0) {
            m->layer_first[l] = i;
            m->layer_off[l] = poff;
        }
        m->layer_last[l] = i;
        size_t start = poff;
        switch (o.d.kind) {
        case DC_OP_CONV:
        case DC_OP_FC: {
            dc_conv_shape sh;
            if (o.d.kind == DC_OP_CONV) {
                sh = dc_conv_shape{in.n, in.h, in.w, in.c, o.d.out_ch, o.d.r, o.d.s, o.d.stride, o.d.pad, o.d.pad_w};
            } else {
                sh = dc_conv_shape{in.n, 1, 1, in.h * in.w * in.c, o.d.out_ch, 1, 1, 1, 0};
            }
            if (o.d.out_ch < 1 || !conv_geom_from_shape(sh, &o.geom))
                return fail(DC_EINVAL, "op %d: invalid %s geometry", i, o.d.kind == DC_OP_CONV ? "conv" : "fc");
            o.fwd = plan_gemm(o.geom, PASS_FWD);
            o.dgrad = plan_gemm(o.geom, PASS_DGRAD);
            o.wgrad = plan_gemm(o.geom, PASS_WGRAD);
            o.w_off = poff;
            poff += (size_t)o.geom.K * o.geom.R * o.geom.S * o.geom.C;
            if (o.d.bias) {
                o.b_off = poff;
                poff += o.geom.K;
            }
            if (o.d.kind == DC_OP_CONV)
                out = TensorInfo{in.n, o.geom.P, o.geom.Q, o.geom.K};
            else
                out = TensorInfo{in.n, 1, 1, o.geom.K};
            break;
        }
        case DC_OP_BN:
            o.w_off = poff;          // gamma
            o.b_off = poff + in.c;   // beta
            poff += 2 * (size_t)in.c;
            break;
        case DC_OP_RELU:
            break;
        case DC_OP_MAXPOOL:
        case DC_OP_AVGPOOL: {
            if (o.d.r < 1 || o.d.s < 1 || o.d.r > 256 || o.d.s > 256 || o.d.stride < 1 || o.d.pad < 0 ||
                o.d.pad >= o.d.r || o.d.pad >= o.d.s || o.d.r * o.d.s > 256 || in.h + 2 * o.d.pad < o.d.r ||
                in.w + 2 * o.d.pad < o.d.s || o.d.pad_w != o.d.pad)
                return fail(DC_EINVAL, "op %d: invalid pooling geometry (pad_w must equal pad)", i);
            o.pool = dc_pool_shape{in.n, in.h, in.w, in.c, o.d.r, o.d.s, o.d.stride, o.d.pad};
            out.h = (in.h + 2 * o.d.pad - o.d.r) / o.d.stride + 1;
            out.w = (in.w + 2 * o.d.pad - o.d.s) / o.d.stride + 1;
            break;
        }
        case DC_OP_GAP:
            out.h = out.w = 1;
            break;
        case DC_OP_ADD: {
            const TensorInfo &b = m->tensors[o.d.in1];
            if (b.n != in.n || b.h != in.h || b.w != in.w || b.c != in.c)
                return fail(DC_EINVAL, "op %d: ADD inputs differ in shape", i);
            break;
        }
        case DC_OP_CONCAT: {
            int64_t c = 0;
            for (int k = 0; k < o.n_in; ++k) {
                const TensorInfo &b = m->tensors[o.in[k]];
                if (b.n != in.n || b.h != in.h || b.w != in.w)
                    return fail(DC_EINVAL, "op %d: CONCAT inputs differ in n, h or w", i);
                o.ch_off[k] = (int)c;
                c += b.c;
            }
            if (c >= INT_MAX)
                return fail(DC_EINVAL, "op %d: CONCAT output has too many channels", i);
            out.c = (int)c;
            break;
        }
        }
        // every tensor is indexed with 32-bit element offsets somewhere
        if (out.size() >= INT_MAX)
            return fail(DC_EINVAL, "op %d: output tensor of %lld elements (the limit is 2^31 - 1)", i,
                        (long long)out.size());
        m->layer_cnt[l] += poff - start;
        m->tensors[o.out] = out;
    }
    for (int l = 1; l <= m->L; ++l)
        if (m->layer_cnt[l] == 0)
            return fail(DC_EINVAL, "layer %d has no parameters", l);
    const TensorInfo &lg = m->tensors[n_ops];
    if (lg.h != 1 || lg.w != 1 || lg.c != m->classes)
        return fail(DC_EINVAL, "the last op must produce N x 1 x 1 x classes logits");
    m->n_params = poff;

    // backward: which input gradients are needed and whether they accumulate
    std::vector<char> written(n_ops + 1, 0);
    for (int i = n_ops - 1; i >= 0; --i) {
        OpInfo &o = m->ops[i];
        for (int k = 0; k < o.n_in; ++k) {
            int t = o.in[k];
            if (t <= 0)
                continue; // the input batch needs no gradient
            o.grad_in[k] = true;
            o.acc_in[k] = written[t] ? 1 : 0;
            written[t] = 1;
        }
    }
    for (int t = 1; t <= n_ops; ++t)
        if (!written[t] && t != n_ops)
            return fail(DC_EINVAL, "tensor %d is never used", t);

    // forward ReLU folding (see OpInfo::relu_into)
    std::vector<int> consumers(n_ops + 1, 0);
    for (const OpInfo &o : m->ops)
        for (int k = 0; k < o.n_in; ++k)
            if (o.in[k] >= 0)
                ++consumers[o.in[k]];
    for (int i = 0; i + 1 < n_ops; ++i) {
        OpInfo &o = m->ops[i], &nx = m->ops[i + 1];
        const int kd = o.d.kind;
        if ((kd == DC_OP_CONV || kd == DC_OP_FC || kd == DC_OP_BN || kd == DC_OP_ADD) && !o.fwd_folded &&
            nx.d.kind == DC_OP_RELU && nx.d.in0 == o.out && consumers[o.out] == 1 && nx.d.layer == o.d.layer) {
            o.relu_into = nx.out;
            nx.fwd_folded = true;
            nx.bwd_folded = kd == DC_OP_BN || kd == DC_OP_ADD;
        }
    }

    for (int i = 0; i + 1 < n_ops; ++i) {
        OpInfo &r = m->ops[i], &mp = m->ops[i + 1];
        if (r.d.kind == DC_OP_RELU && !r.bwd_folded && r.grad_in[0] && mp.d.kind == DC_OP_MAXPOOL &&
            mp.d.in0 == r.out && consumers[r.out] == 1 && mp.d.layer == r.d.layer) {
            mp.relu_bwd_from = i;
            r.bwd_folded = true;
        }
    }
    // A ReLU whose only consumer is a CONV / FC or a CONCAT: that op's backward
    // applies the mask.  The ReLU's input gradient then receives this
    // contribution at the consumer's turn instead of the ReLU's; that keeps the
    // order of contributions when the consumer is the next op, or when the
    // ReLU is the only reader of its input (one contribution in all).
    std::vector<int> consumer_of(n_ops + 1, -1);
    for (int j = 0; j < n_ops; ++j)
        for (int k = 0; k < m->ops[j].n_in; ++k)
            if (m->ops[j].in[k] >= 0)
                consumer_of[m->ops[j].in[k]] = j;
    for (int i = 0; i < n_ops; ++i) {
        OpInfo &r = m->ops[i];
        if (r.d.kind != DC_OP_RELU || r.bwd_folded || !r.grad_in[0] || consumers[r.out] != 1)
            continue;
        const int j = consumer_of[r.out];
        if (j < 0 || (j != i + 1 && consumers[r.d.in0] != 1))
            continue;
        OpInfo &c = m->ops[j];
        if ((c.d.kind == DC_OP_CONV || c.d.kind == DC_OP_FC) && c.d.in0 == r.out && c.grad_in[0]) {
            c.dgrad_relu_from = i;
            r.bwd_folded = true;
        } else if (c.d.kind == DC_OP_CONCAT) {
            // The concatenation hands its slices back in slot order, so a slot
            // that reads the ReLU's input directly would receive its term on
            // the wrong side of the ReLU's: no fold then.
            bool direct = false;
            for (int k = 0; k < c.n_in; ++k)
                direct |= c.in[k] == r.d.in0;
            if (direct)
                continue;
            for (int k = 0; k < c.n_in; ++k)
                if (c.in[k] == r.out && c.grad_in[k]) {
                    c.concat_relu_from[k] = i;
                    r.bwd_folded = true;
                }
        }
    }

    // workspace layout
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align_up(off + std::max<size_t>(bytes, 1), 256);
        return o;
    };
    m->off_params = take(m->n_params * sizeof(float));
    m->off_grads = take(m->n_params * sizeof(float));
    for (int t = 1; t <= n_ops; ++t) {
        m->tensors[t].act = take((size_t)m->tensors[t].size() * sizeof(float));
        m->tensors[t].grad = take((size_t)m->tensors[t].size() * sizeof(float));
    }
    size_t scratch = xent_ws_bytes(m->batch);
    for (int i = 0; i < n_ops; ++i) {
        OpInfo &o = m->ops[i];
        const TensorInfo &in = m->tensors[o.d.in0];
        const TensorInfo &out = m->tensors[o.out];
        if (o.d.kind == DC_OP_CONV || o.d.kind == DC_OP_FC) {
            scratch = std::max({scratch, o.fwd.ws_bytes, o.dgrad.ws_bytes, o.wgrad.ws_bytes});
            if (o.d.bias)
                scratch = std::max(scratch, colsum_ws_bytes((int64_t)out.n * out.h * out.w, out.c));
        } else if (o.d.kind == DC_OP_BN) {
            o.aux = take(2 * (size_t)in.c * sizeof(float));
            scratch = std::max(scratch, bn_ws_bytes((int64_t)in.n * in.h * in.w, in.c));
        } else if (o.d.kind == DC_OP_MAXPOOL) {
            o.aux = take((size_t)out.size());
        }
    }
    m->scratch_bytes = scratch;
    m->off_scratch = take(scratch);
    m->off_loss = take(sizeof(float));
    m->off_slots = take(sizeof(uint64_t) * 2 * (m->L + 1));
    m->ws_need = off;
    return DC_OK;
}

// ---------------------------------------------------------------- mini-procedures

// Algorithmic FLOPs of one GEMM pass (forward, data or filter gradient):
// 2 per multiply-add, N*P*Q*K*R*S*C multiply-adds.
static double gemm_flop(const ConvGeom &g) {
    return 2.0 * g.N * g.P * g.Q * (double)g.K * g.R * g.S * g.C;
}

int gemm_mark(dc_model *m, bool start, double flop, hipStream_t s) {
    if (!m->gemm_timing || m->use_graphs)
        return DC_OK;
    const size_t i = 2 * m->gemm_n + (start ? 0 : 1);
    while (m->gemm_ev.size() <= i) {
        hipEvent_t e = nullptr;
        DC_HIP(hipEventCreate(&e));
        m->gemm_ev.push_back(e);
    }
    if (start) {
        if (m->gemm_flop.size() <= m->gemm_n)
            m->gemm_flop.resize(m->gemm_n + 1);
        m->gemm_flop[m->gemm_n] = flop;
    }
    DC_HIP(hipEventRecord(m->gemm_ev[i], s));
    if (!start)
        ++m->gemm_n;
    return DC_OK;
}

void free_gemm_events(dc_model *m) {
    for (hipEvent_t e : m->gemm_ev)
        if (e)
            (void)hipEventDestroy(e);
    m->gemm_ev.clear();
    m->gemm_flop.clear();
    m->gemm_n = 0;
}

int run_forward_layer(dc_model *m, int l, const float *x, const int32_t *y, hipStream_t s) {
    const float *P = m->dparams();
    for (int i = m->layer_first[l]; i <= m->layer_last[l]; ++i) {
        OpInfo &o = m->ops[i];
        if (o.fwd_folded)
            continue; // computed by the producer (OpInfo::relu_into)
        const float *in = o.d.in0 == 0 ? x : m->act(o.d.in0);
        const int relu = o.relu_into >= 0 ? 1 : 0;
        float *out = m->act(relu ? o.relu_into : o.out);
        const TensorInfo &ti = m->tensors[o.d.in0];
        switch (o.d.kind) {
        case DC_OP_CONV:
        case DC_OP_FC:
            DC_TRY(gemm_mark(m, true, gemm_flop(o.geom), s));
            DC_TRY(conv_forward(o.geom, o.fwd, in, P + o.w_off, o.b_off != NONE ? P + o.b_off : nullptr, relu, out,
                                m->scratch(), s));
            DC_TRY(gemm_mark(m, false, 0, s));
            break;
        case DC_OP_BN: {
            float *mean = reinterpret_cast<float *>(m->ws + o.aux);
            DC_TRY(bn_forward((int64_t)ti.n * ti.h * ti.w, ti.c, in, P + o.w_off, P + o.b_off, 1e-5f, relu, out, mean,
                              mean + ti.c, m->scratch(), s));
            break;
        }
        case DC_OP_RELU:
            DC_TRY(relu_forward(in, out, ti.size(), s));
            break;
        case DC_OP_MAXPOOL:
            DC_TRY(maxpool_forward(o.pool, in, out, reinterpret_cast<uint8_t *>(m->ws + o.aux), s));
            break;
        case DC_OP_AVGPOOL:
            DC_TRY(avgpool_forward(o.pool, in, out, s));
            break;
        case DC_OP_GAP:
            DC_TRY(gap_forward(ti.n, ti.h * ti.w, ti.c, in, out, s));
            break;
        case DC_OP_ADD:
            DC_TRY(add_forward(in, m->act(o.d.in1), relu, out, ti.size(), s));
            break;
        case DC_OP_CONCAT: {
            const TensorInfo &to = m->tensors[o.out];
            for (int k = 0; k < o.n_in; ++k) {
                const TensorInfo &tk = m->tensors[o.in[k]];
                const float *src = o.in[k] == 0 ? x : m->act(o.in[k]);
                DC_TRY(concat_forward((int64_t)tk.n * tk.h * tk.w, tk.c, to.c, o.ch_off[k], src, out, s));
            }
            break;
        }
        }
    }
    if (l == m->L) {
        int last = (int)m->ops.size();
        DC_TRY(softmax_xent(m->batch, m->classes, m->act(last), y, m->dloss(), m->grad(last), m->scratch(), s));
    }
    return DC_OK;
}

int run_backward_layer(dc_model *m, int l, const float *x, hipStream_t s, BwdRecorder *rec) {
    const float *P = m->dparams();
    float *G = m->dgrads();
    for (int i = m->layer_last[l]; i >= m->layer_first[l]; --i) {
        OpInfo &o = m->ops[i];
        // With rec set, each launch below is replaced by the records of the
        // tensor-gradient contributions it makes, in the order it makes them:
        // (tensor, op whose chain-rule term it is, accumulate, fused).
        auto note = [&](int t, int origin, int acc, int fused) {
            if (rec)
                rec->v.push_back(dc_grad_contrib{t, origin, i, acc, fused});
        };
        const float *in = o.d.in0 == 0 ? x : m->act(o.d.in0);
        const float *dy = m->grad(o.out);
        float *dx = o.grad_in[0] ? m->grad(o.d.in0) : nullptr;
        const TensorInfo &ti = m->tensors[o.d.in0];
        const TensorInfo &to = m->tensors[o.out];
        switch (o.d.kind) {
        case DC_OP_CONV:
        case DC_OP_FC:
            if (!rec) {
                DC_TRY(gemm_mark(m, true, gemm_flop(o.geom), s));
                bool bias_done = false;
                DC_TRY(conv_wgrad(o.geom, o.wgrad, in, dy, G + o.w_off, m->scratch(), s,
                                  o.b_off != NONE ? G + o.b_off : nullptr, &bias_done));
                DC_TRY(gemm_mark(m, false, 0, s));
                if (o.b_off != NONE && !bias_done)
                    DC_TRY(colsum((int64_t)to.n * to.h * to.w, to.c, dy, G + o.b_off, m->scratch(), s));
            }
            if (o.dgrad_relu_from >= 0) { // through the folded ReLU into its input's gradient
                const OpInfo &r = m->ops[o.dgrad_relu_from];
                note(r.out, i, o.acc_in[0], 1);
                note(r.d.in0, o.dgrad_relu_from, r.acc_in[0], 0);
                if (!rec) {
                    DC_TRY(gemm_mark(m, true, gemm_flop(o.geom), s));
                    DC_TRY(conv_dgrad(o.geom, o.dgrad, dy, P + o.w_off, r.acc_in[0], m->grad(r.d.in0), m->scratch(),
                                      s, m->act(r.out)));
                    DC_TRY(gemm_mark(m, false, 0, s));
                }
            } else if (dx) {
                note(o.d.in0, i, o.acc_in[0], 0);
                if (!rec) {
                    DC_TRY(gemm_mark(m, true, gemm_flop(o.geom), s));
                    DC_TRY(conv_dgrad(o.geom, o.dgrad, dy, P + o.w_off, o.acc_in[0], dx, m->scratch(), s));
                    DC_TRY(gemm_mark(m, false, 0, s));
                }
            }
            break;
        case DC_OP_BN: {
            const float *mean = reinterpret_cast<const float *>(m->ws + o.aux);
            // a folded ReLU: take its output gradient and mask it on the way in
            const bool fold = o.relu_into >= 0 && m->ops[i + 1].bwd_folded;
            if (fold)
                note(o.out, i + 1, m->ops[i + 1].acc_in[0], 1);
            note(o.d.in0, i, o.acc_in[0], 0);
            if (!rec)
                DC_TRY(bn_backward((int64_t)ti.n * ti.h * ti.w, ti.c, fold ? m->grad(o.relu_into) : dy, in,
                                   P + o.w_off, mean, mean + ti.c, o.acc_in[0], dx, G + o.w_off, G + o.b_off,
                                   m->scratch(), s, fold ? m->act(o.relu_into) : nullptr));
            break;
        }
        case DC_OP_RELU:
            if (o.bwd_folded)
                break; // done by the BN / add that produced its input, or by the op that reads its output
            note(o.d.in0, i, o.acc_in[0], 0);
            if (!rec)
                DC_TRY(relu_backward(dy, m->act(o.out), o.acc_in[0], dx, ti.size(), s));
            break;
        case DC_OP_MAXPOOL:
            if (o.relu_bwd_from >= 0) { // through the folded ReLU into its input's gradient
                const OpInfo &r = m->ops[o.relu_bwd_from];
                note(r.out, i, o.acc_in[0], 1);
                note(r.d.in0, o.relu_bwd_from, r.acc_in[0], 0);
                if (!rec)
                    DC_TRY(maxpool_backward(o.pool, dy, reinterpret_cast<const uint8_t *>(m->ws + o.aux),
                                            r.acc_in[0], m->grad(r.d.in0), s, m->act(o.out)));
            } else {
                note(o.d.in0, i, o.acc_in[0], 0);
                if (!rec)
                    DC_TRY(maxpool_backward(o.pool, dy, reinterpret_cast<const uint8_t *>(m->ws + o.aux),
                                            o.acc_in[0], dx, s));
            }
            break;
        case DC_OP_AVGPOOL:
            note(o.d.in0, i, o.acc_in[0], 0);
            if (!rec)
                DC_TRY(avgpool_backward(o.pool, dy, o.acc_in[0], dx, s));
            break;
        case DC_OP_GAP:
            note(o.d.in0, i, o.acc_in[0], 0);
            if (!rec)
                DC_TRY(gap_backward(ti.n, ti.h * ti.w, ti.c, dy, o.acc_in[0], dx, s));
            break;
        case DC_OP_ADD:
            if (o.relu_into >= 0 && m->ops[i + 1].bwd_folded) { // the folded ReLU's gradient, masked, into both inputs
                note(o.out, i + 1, m->ops[i + 1].acc_in[0], 1);
                note(o.d.in0, i, o.acc_in[0], 0);
                if (o.grad_in[1])
                    note(o.d.in1, i, o.acc_in[1], 0);
                if (!rec)
                    DC_TRY(add_relu_backward(m->grad(o.relu_into), m->act(o.relu_into), o.acc_in[0], dx,
                                             o.acc_in[1], o.grad_in[1] ? m->grad(o.d.in1) : nullptr, ti.size(), s));
            } else {
                note(o.d.in0, i, o.acc_in[0], 0);
                note(o.d.in1, i, o.acc_in[1], 0);
                if (!rec) {
                    DC_TRY(copy_grad(dy, o.acc_in[0], dx, ti.size(), s));
                    DC_TRY(copy_grad(dy, o.acc_in[1], m->grad(o.d.in1), ti.size(), s));
                }
            }
            break;
        case DC_OP_CONCAT:
            for (int k = 0; k < o.n_in; ++k) {
                if (!o.grad_in[k])
                    continue;
                const TensorInfo &tk = m->tensors[o.in[k]];
                if (o.concat_relu_from[k] >= 0) { // through the folded ReLU into its input's gradient
                    const OpInfo &r = m->ops[o.concat_relu_from[k]];
                    note(r.out, i, o.acc_in[k], 1);
                    note(r.d.in0, o.concat_relu_from[k], r.acc_in[0], 0);
                    if (!rec)
                        DC_TRY(concat_backward((int64_t)tk.n * tk.h * tk.w, tk.c, to.c, o.ch_off[k], dy, r.acc_in[0],
                                               m->grad(r.d.in0), s, m->act(r.out)));
                } else {
                    note(o.in[k], i, o.acc_in[k], 0);
                    if (!rec)
                        DC_TRY(concat_backward((int64_t)tk.n * tk.h * tk.w, tk.c, to.c, o.ch_off[k], dy,
                                               o.acc_in[k], m->grad(o.in[k]), s));
                }
            }
            break;
        }
    }
    return DC_OK;
}

// ---------------------------------------------------------------- per-layer HIP graphs

void drop_graphs(dc_model *m) {
    for (auto *v : {&m->g_fwd, &m->g_bwd})
        for (auto &g : *v)
            if (g) {
                (void)hipGraphExecDestroy(g);
                g = nullptr;
            }
    m->g_ws = nullptr;
    m->g_x = nullptr;
    m->g_y = nullptr;
}

// Capture the work of one layer and direction on the private stream.  The
// capture is always ended, also when enqueueing fails, so the stream never
// stays in capture mode.
static int capture_layer(dc_model *m, int l, bool fwd, const float *x, const int32_t *y, hipGraphExec_t *out) {
    DC_HIP(hipStreamBeginCapture(m->cap_s, hipStreamCaptureModeThreadLocal));
    const int st = fwd ? run_forward_layer(m, l, x, y, m->cap_s) : run_backward_layer(m, l, x, m->cap_s);
    hipGraph_t g = nullptr;
    const hipError_t e = hipStreamEndCapture(m->cap_s, &g);
    if (st != DC_OK) {
        if (g)
            (void)hipGraphDestroy(g);
        return st;
    }
    if (e != hipSuccess)
        return hip_fail(e, "hipStreamEndCapture");
    const hipError_t ei = hipGraphInstantiate(out, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (ei != hipSuccess)
        return hip_fail(ei, "hipGraphInstantiate");
    return DC_OK;
}

static int ensure_graphs(dc_model *m, const float *x, const int32_t *y) {
    if (m->g_ws == m->ws && m->g_x == x && m->g_y == y && (int)m->g_fwd.size() == m->L + 1)
        return DC_OK;
    drop_graphs(m);
    if (!m->cap_s)
        DC_HIP(hipStreamCreateWithFlags(&m->cap_s, hipStreamNonBlocking));
    m->g_fwd.assign(m->L + 1, nullptr);
    m->g_bwd.assign(m->L + 1, nullptr);
    for (int l = 1; l <= m->L; ++l) {
        int st = capture_layer(m, l, true, x, y, &m->g_fwd[l]);
        if (st == DC_OK)
            st = capture_layer(m, l, false, x, y, &m->g_bwd[l]);
        if (st != DC_OK) {
            drop_graphs(m);
            return st;
        }
    }
    m->g_ws = m->ws;
    m->g_x = x;
    m->g_y = y;
    return DC_OK;
}

int launch_forward_layer(dc_model *m, int l, const float *x, const int32_t *y, hipStream_t s) {
    if (!m->use_graphs)
        return run_forward_layer(m, l, x, y, s);
    DC_TRY(ensure_graphs(m, x, y));
    DC_HIP(hipGraphLaunch(m->g_fwd[l], s));
    return DC_OK;
}

int launch_backward_layer(dc_model *m, int l, const float *x, hipStream_t s) {
    // the forward call for the same batch captured the graphs; without them
    // (graphs off, or a batch the forward pass has not seen) launch directly
    if (!m->use_graphs || m->g_ws != m->ws || m->g_x != x || (int)m->g_bwd.size() != m->L + 1)
        return run_backward_layer(m, l, x, s);
    DC_HIP(hipGraphLaunch(m->g_bwd[l], s));
    return DC_OK;
}

} // namespace dc

// ---------------------------------------------------------------- C ABI: model and parameter server

using namespace dc;

extern "C" int dc_model_create(const dc_op_desc *ops, int n_ops, int batch, int in_h, int in_w, int in_c,
                               int classes, dc_model **out) {
    clear_error();
    if (!out)
        return fail(DC_EINVAL, "out is NULL");
    *out = nullptr;
    DC_TRY(check_desc(ops, n_ops, batch, in_h, in_w, in_c, classes));
    dc_model *m = new (std::nothrow) dc_model();
    if (!m)
        return fail(DC_ENOMEM, "out of host memory");
    m->batch = batch;
    m->in_h = in_h;
    m->in_w = in_w;
    m->in_c = in_c;
    m->classes = classes;
    int st = build_model(m, ops, n_ops);
    if (st != DC_OK) {
        delete m;
        return st;
    }
    auto cleanup = [&](int code) {
        dc_model_destroy(m);
        return code;
    };
    hipError_t e = hipGetDevice(&m->device);
    if (e != hipSuccess)
        return cleanup(hip_fail(e, "hipGetDevice"));
    const size_t pbytes = std::max<size_t>(m->n_params * sizeof(float), 256);
    if ((e = hipHostMalloc((void **)&m->ps_params, pbytes, hipHostMallocDefault)) != hipSuccess)
        return cleanup(hip_fail(e, "hipHostMalloc(parameters)"));
    if ((e = hipHostMalloc((void **)&m->ps_grads, pbytes, hipHostMallocDefault)) != hipSuccess)
        return cleanup(hip_fail(e, "hipHostMalloc(gradients)"));
    std::memset(m->ps_params, 0, pbytes);
    std::memset(m->ps_grads, 0, pbytes);
    m->probe_bytes = 16u << 20;
    if ((e = hipHostMalloc((void **)&m->probe_host, m->probe_bytes, hipHostMallocDefault)) != hipSuccess)
        return cleanup(hip_fail(e, "hipHostMalloc(probe)"));
    if ((e = hipStreamCreateWithFlags(&m->pull_s, hipStreamNonBlocking)) != hipSuccess)
        return cleanup(hip_fail(e, "hipStreamCreate(pull)"));
    if ((e = hipStreamCreateWithFlags(&m->push_s, hipStreamNonBlocking)) != hipSuccess)
        return cleanup(hip_fail(e, "hipStreamCreate(push)"));
    auto mk = [&](std::vector<hipEvent_t> &v, int n) -> hipError_t {
        v.assign(n, nullptr);
        for (auto &ev : v) {
            hipError_t r = hipEventCreate(&ev);
            if (r != hipSuccess)
                return r;
        }
        return hipSuccess;
    };
    const int L = m->L;
    for (auto *v : {&m->ev_pull_start, &m->ev_pull_done, &m->ev_bwd_done, &m->ev_push_start, &m->ev_push_done})
        if ((e = mk(*v, L)) != hipSuccess)
            return cleanup(hip_fail(e, "hipEventCreate"));
    for (auto *v : {&m->ev_fwd_start, &m->ev_fwd_end, &m->ev_bwd_end})
        if ((e = mk(*v, L + 2)) != hipSuccess)
            return cleanup(hip_fail(e, "hipEventCreate"));
    if ((e = hipEventCreate(&m->ev_t0)) != hipSuccess)
        return cleanup(hip_fail(e, "hipEventCreate"));
    if ((e = hipEventCreate(&m->ev_cs_done)) != hipSuccess)
        return cleanup(hip_fail(e, "hipEventCreate"));
    int wall = wall_clock_hz(&m->wall_hz);
    if (wall != DC_OK)
        return cleanup(wall);
    unsigned hw = std::thread::hardware_concurrency();
    m->sgd_threads = (int)std::max(1u, std::min(hw ? hw : 1u, 16u));
    m->pool = new HostPool(m->sgd_threads);
    *out = m;
    return DC_OK;
}

extern "C" void dc_model_destroy(dc_model *m) {
    if (!m)
        return;
    if (m->pull_s)
        (void)hipStreamSynchronize(m->pull_s);
    if (m->push_s)
        (void)hipStreamSynchronize(m->push_s);
    // a step that ended on the watchdog can leave the loss copy into
    // probe_host queued on the caller's stream
    if (m->ev_cs_done)
        (void)hipEventSynchronize(m->ev_cs_done);
    for (auto *v : {&m->ev_pull_start, &m->ev_pull_done, &m->ev_bwd_done, &m->ev_push_start, &m->ev_push_done,
                    &m->ev_fwd_start, &m->ev_fwd_end, &m->ev_bwd_end})
        for (auto ev : *v)
            if (ev)
                (void)hipEventDestroy(ev);
    if (m->ev_t0)
        (void)hipEventDestroy(m->ev_t0);
    if (m->ev_cs_done)
        (void)hipEventDestroy(m->ev_cs_done);
    drop_graphs(m);
    free_gemm_events(m);
    if (m->cap_s)
        (void)hipStreamDestroy(m->cap_s);
    if (m->pull_s)
        (void)hipStreamDestroy(m->pull_s);
    if (m->push_s)
        (void)hipStreamDestroy(m->push_s);
    if (m->ps_params)
        (void)hipHostFree(m->ps_params);
    if (m->ps_grads)
        (void)hipHostFree(m->ps_grads);
    if (m->probe_host)
        (void)hipHostFree(m->probe_host);
    delete m->pool;
    delete m;
}

extern "C" int dc_backward_schedule(const dc_op_desc *ops, int n_ops, int batch, int in_h, int in_w, int in_c,
                                    int classes, dc_grad_contrib *out, int cap, int *n_out) {
    clear_error();
    if (!n_out || cap < 0 || (cap > 0 && !out))
        return fail(DC_EINVAL, "n_out is NULL, or out is NULL with cap > 0");
    *n_out = 0;
    DC_TRY(check_desc(ops, n_ops, batch, in_h, in_w, in_c, classes));
    dc_model m;
    m.batch = batch;
    m.in_h = in_h;
    m.in_w = in_w;
    m.in_c = in_c;
    m.classes = classes;
    DC_TRY(build_model(&m, ops, n_ops));
    BwdRecorder rec;
    for (int l = m.L; l >= 1; --l)
        DC_TRY(run_backward_layer(&m, l, nullptr, nullptr, &rec));
    *n_out = (int)rec.v.size();
    if ((size_t)cap < rec.v.size())
        return fail(DC_EINVAL, "the schedule has %zu entries, cap is %d", rec.v.size(), cap);
    std::copy(rec.v.begin(), rec.v.end(), out);
    return DC_OK;
}

extern "C" int dc_model_num_layers(const dc_model *m) { return m ? m->L : 0; }
extern "C" size_t dc_model_num_params(const dc_model *m) { return m ? m->n_params : 0; }
extern "C" size_t dc_workspace_bytes(const dc_model *m) { return m ? m->ws_need : 0; }

extern "C" int dc_model_bind_workspace(dc_model *m, void *dev, size_t bytes) {
    clear_error();
    if (!m || !dev)
        return fail(DC_EINVAL, "model or workspace is NULL");
    if ((uintptr_t)dev % 256 != 0)
        return fail(DC_EINVAL, "workspace must be 256-byte aligned");
    if (bytes < m->ws_need)
        return fail(DC_ENOMEM, "workspace has %zu bytes, the model needs %zu", bytes, m->ws_need);
    drop_graphs(m); // they hold the old workspace's addresses
    m->ws = static_cast<char *>(dev);
    m->ws_bytes = bytes;
    return DC_OK;
}

extern "C" int dc_layer_range(const dc_model *m, int layer, size_t *off, size_t *count) {
    clear_error();
    if (!m || layer < 1 || layer > m->L)
        return fail(DC_EINVAL, "layer %d out of range", layer);
    if (off)
        *off = m->layer_off[layer];
    if (count)
        *count = m->layer_cnt[layer];
    return DC_OK;
}

extern "C" int dc_model_set_option(dc_model *m, int option, double value) {
    clear_error();
    if (!m)
        return fail(DC_EINVAL, "model is NULL");
    switch (option) {
    case DC_OPT_LR:
        m->lr = value;
        return DC_OK;
    case DC_OPT_TIMELINE:
        m->timeline = value != 0.0;
        return DC_OK;
    case DC_OPT_TIMEOUT_S:
        if (!(value > 0))
            return fail(DC_EINVAL, "timeout must be positive");
        m->timeout_s = value;
        return DC_OK;
    case DC_OPT_GRAPHS:
        m->use_graphs = value != 0.0;
        return DC_OK;
    case DC_OPT_GEMM_TIMING:
        m->gemm_timing = value != 0.0;
        return DC_OK;
    case DC_OPT_SGD_THREADS: {
        int t = (int)value;
        if (t < 1 || t > 256)
            return fail(DC_EINVAL, "SGD threads must be in [1, 256]");
        delete m->pool;
        m->sgd_threads = t;
        m->pool = new HostPool(t);
        return DC_OK;
    }
    default:
        return fail(DC_EINVAL, "unknown option %d", option);
    }
}

extern "C" int dc_ps_write(dc_model *m, const float *host_params, size_t n) {
    clear_error();
    if (!m || !host_params || n != m->n_params)
        return fail(DC_EINVAL, "dc_ps_write needs exactly %zu floats", m ? m->n_params : (size_t)0);
    std::memcpy(m->ps_params, host_params, n * sizeof(float));
    return DC_OK;
}

extern "C" int dc_model_read_tensor(const dc_model *m, int tensor, int what, void *host, size_t bytes) {
    clear_error();
    if (!m || !host)
        return fail(DC_EINVAL, "NULL model or destination");
    if (tensor < 0 || tensor >= (int)m->tensors.size())
        return fail(DC_EINVAL, "tensor %d outside 0..%zu", tensor, m->tensors.size() - 1);
    if (!m->ws)
        return fail(DC_ESTATE, "no workspace is bound");
    const TensorInfo &ti = m->tensors[tensor];
    size_t off = NONE, need = 0;
    if (what == DC_READ_ACT) {
        if (tensor == 0)
            return fail(DC_EINVAL, "tensor 0 is the caller's input batch");
        // a producer with a folded ReLU writes only the ReLU's output
        if (m->ops[tensor - 1].relu_into >= 0 || ti.act == NONE)
            return fail(DC_EINVAL, "tensor %d is not kept (the input of a folded ReLU)", tensor);
        off = ti.act;
        need = (size_t)ti.size() * sizeof(float);
    } else if (what == DC_READ_ARGMAX) {
        if (tensor == 0 || m->ops[tensor - 1].d.kind != DC_OP_MAXPOOL)
            return fail(DC_EINVAL, "tensor %d is not a max-pool output", tensor);
        off = m->ops[tensor - 1].aux;
        need = (size_t)ti.size();
    } else {
        return fail(DC_EINVAL, "what must be DC_READ_ACT or DC_READ_ARGMAX");
    }
    if (bytes != need)
        return fail(DC_EINVAL, "tensor %d needs %zu bytes, got %zu", tensor, need, bytes);
    DC_HIP(hipDeviceSynchronize());
    DC_HIP(hipMemcpy(host, m->ws + off, bytes, hipMemcpyDeviceToHost));
    return DC_OK;
}

extern "C" int dc_ps_read(const dc_model *m, float *params_out, float *grads_out, size_t n) {
    clear_error();
    if (!m || n != m->n_params)
        return fail(DC_EINVAL, "dc_ps_read needs exactly %zu floats", m ? m->n_params : (size_t)0);
    if (params_out)
        std::memcpy(params_out, m->ps_params, n * sizeof(float));
    if (grads_out)
        std::memcpy(grads_out, m->ps_grads, n * sizeof(float));
    return DC_OK;
}
