// Segment-pipelined executor and real-time profiler.
//
// dc_step enqueues one iteration on three streams (Sec. III-A):
//   pull stream    - per pull segment: [mark, overhead spin], H2D copy of the
//                    segment's contiguous parameter range, [pacing spin],
//                    event pull_done[j];
//   compute stream - forward layers 1..L, each gated only by the pull_done
//                    event of its own segment (Eq. 1, 5), the loss, then
//                    backward layers L..1 (Eq. 3, 6), recording bwd_done[j]
//                    when the lowest layer of push segment j is finished;
//   push stream    - per push segment, top first: wait bwd_done[j] (Eq. 2),
//                    [mark, overhead spin], D2H copy of the gradient range
//                    into the server, [pacing spin], event push_done[j] (Eq. 7).
// The host thread then walks the push segments in order and applies SGD to
// each range as soon as its push_done fires.  Ordering comes from events
// only, and no kernel uses atomics, so the numbers are the same for every
// segmentation.
//
// Link emulation: a transmission of B bytes occupies its stream for
// dt_emul + B / rate (paced) measured from a wall-clock mark taken when the
// transmission starts; a spin kernel on the stream holds it until then, so
// the data becomes visible when the emulated transfer ends.
#include "runtime.h"

#include <chrono>
#include <cmath>
#include <cstring>

namespace dc {
namespace {

using Clock = std::chrono::steady_clock;

int64_t ns_since(Clock::time_point t0) {
    return std::chrono::duration_cast<std::chrono::nanoseconds>(Clock::now() - t0).count();
}

int elapsed_ns(hipEvent_t a, hipEvent_t b, int64_t *out) {
    float ms = 0.f;
    DC_HIP(hipEventElapsedTime(&ms, a, b));
    *out = (int64_t)llround((double)ms * 1e6);
    return DC_OK;
}

// Poll an event until it completes or the deadline passes.
int wait_event(hipEvent_t e, Clock::time_point deadline) {
    for (;;) {
        hipError_t r = hipEventQuery(e);
        if (r == hipSuccess)
            return DC_OK;
        if (r != hipErrorNotReady)
            return hip_fail(r, "hipEventQuery");
        if (Clock::now() > deadline)
            return fail(DC_ETIMEOUT, "watchdog expired while waiting for the GPU");
        std::this_thread::sleep_for(std::chrono::microseconds(20));
    }
}

struct Seg {
    int lo, hi;
};

std::vector<Seg> pull_segs(const dc_plan_t *plan, int L) {
    std::vector<Seg> s;
    int lo = 1;
    for (int l = 1; l < L; ++l)
        if (plan->p[l - 1]) {
            s.push_back({lo, l});
            lo = l + 1;
        }
    s.push_back({lo, L});
    return s;
}

// push order: top segment first; g_k = 1 splits between layer L-k+1 and L-k
std::vector<Seg> push_segs(const dc_plan_t *plan, int L) {
    std::vector<Seg> s;
    int hi = L;
    for (int k = 1; k < L; ++k)
        if (plan->g[k - 1]) {
            s.push_back({L - k + 1, hi});
            hi = L - k;
        }
    s.push_back({1, hi});
    return s;
}

uint64_t to_ticks(double ns, double hz) { return (uint64_t)std::ceil(ns * hz * 1e-9); }

// One transmission mini-procedure of `bytes` on stream s.
int transmit(dc_model *m, void *dst, const void *src, size_t bytes, hipMemcpyKind kind, const dc_link *link,
             uint64_t *slot, hipEvent_t ev_start, hipEvent_t ev_done, hipStream_t s) {
    if (ev_start)
        DC_HIP(hipEventRecord(ev_start, s));
    const bool mark = link->paced || link->dt_emul_ns > 0;
    const uint64_t one_s = to_ticks(1e9, m->wall_hz);
    if (mark)
        DC_TRY(pace_mark(slot, s));
    if (link->dt_emul_ns > 0) {
        uint64_t t = to_ticks((double)link->dt_emul_ns, m->wall_hz);
        DC_TRY(pace_until(slot, t, t + one_s, s));
    }
    if (bytes)
        DC_HIP(hipMemcpyAsync(dst, src, bytes, kind, s));
    if (link->paced) {
        double ns = (double)link->dt_emul_ns + (double)bytes / link->bytes_per_s * 1e9;
        uint64_t t = to_ticks(ns, m->wall_hz);
        DC_TRY(pace_until(slot, t, t + one_s, s));
    }
    if (ev_done)
        DC_HIP(hipEventRecord(ev_done, s));
    return DC_OK;
}

void sgd_range(dc_model *m, size_t off, size_t cnt) {
    float *w = m->ps_params + off;
    const float *g = m->ps_grads + off;
    const float lr = (float)m->lr;
    const size_t chunk = 1 << 18;
    int nchunks = (int)((cnt + chunk - 1) / chunk);
    m->pool->run(nchunks, [&](int i, int) {
        size_t a = (size_t)i * chunk, b = std::min(cnt, a + chunk);
        for (size_t k = a; k < b; ++k)
            w[k] = w[k] - lr * g[k];
    });
}

int check_link(const dc_link *link) {
    if (!link)
        return fail(DC_EINVAL, "link is NULL");
    if (link->dt_emul_ns < 0)
        return fail(DC_EINVAL, "dt_emul_ns must be >= 0");
    if (link->paced && !(link->bytes_per_s > 0) )
        return fail(DC_EINVAL, "a paced link needs bytes_per_s > 0");
    return DC_OK;
}

int check_batch(const dc_model *m, const dc_batch *b) {
    if (!b || !b->x_dev || !b->y_dev)
        return fail(DC_EINVAL, "batch or its buffers are NULL");
    if (b->n != m->batch)
        return fail(DC_EINVAL, "batch has %d images, the model was built for %d", b->n, m->batch);
    return DC_OK;
}

size_t seg_bytes(const dc_model *m, Seg s, size_t *off) {
    *off = m->layer_off[s.lo];
    return (m->layer_off[s.hi] + m->layer_cnt[s.hi] - m->layer_off[s.lo]) * sizeof(float);
}

} // namespace
} // namespace dc

using namespace dc;

namespace dc {
namespace {

// The body of dc_step and dc_step_dynamic.  With `prof` non-null the backward
// decision is planned after the forward work is enqueued (while the pulls and
// the forward pass are in flight) and the next forward decision before the
// last push is awaited, both written into `plan`.
int step_impl(dc_model *m, const dc_batch *b, dc_plan_t *plan, const dc_profile_t *prof, const dc_link *link,
              void *stream, dc_step_stats *out) {
    const auto t_host0 = Clock::now();
    if (!m)
        return fail(DC_EINVAL, "model is NULL");
    if (!m->ws)
        return fail(DC_ESTATE, "no workspace bound");
    DC_TRY(check_batch(m, b));
    DC_TRY(check_link(link));
    if (!plan || plan->L != m->L || (m->L > 1 && (!plan->p || !plan->g)))
        return fail(DC_EINVAL, "plan is for L=%d, the model has L=%d", plan ? plan->L : -1, m->L);
    if (prof && (prof->L != m->L || !prof->pt_ns || !prof->fc_ns || !prof->bc_ns || !prof->gt_ns))
        return fail(DC_EINVAL, "profile does not match the model");
    const int L = m->L;
    hipStream_t cs = static_cast<hipStream_t>(stream);
    const auto pulls = pull_segs(plan, L);
    const Clock::time_point deadline = t_host0 + std::chrono::microseconds((int64_t)(m->timeout_s * 1e6));
    m->timeline_valid = false;
    m->gemm_n = 0;
    int64_t t_plan_bwd = 0, t_plan_fwd = 0;
    int32_t hidden = 0;

    // pull stream
    DC_HIP(hipEventRecord(m->ev_t0, m->pull_s));
    for (size_t j = 0; j < pulls.size(); ++j) {
        size_t off;
        size_t bytes = seg_bytes(m, pulls[j], &off);
        DC_TRY(transmit(m, m->dparams() + off, m->ps_params + off, bytes, hipMemcpyHostToDevice, link,
                        m->slots() + j, m->ev_pull_start[j], m->ev_pull_done[j], m->pull_s));
    }
    // compute stream: forward, gated per pull segment
    size_t j = 0;
    for (int l = 1; l <= L; ++l) {
        if (j < pulls.size() && pulls[j].lo == l) {
            DC_HIP(hipStreamWaitEvent(cs, m->ev_pull_done[j], 0));
            ++j;
        }
        if (m->timeline)
            DC_HIP(hipEventRecord(m->ev_fwd_start[l], cs));
        DC_TRY(launch_forward_layer(m, l, b->x_dev, b->y_dev, cs));
        if (m->timeline || l == L)
            DC_HIP(hipEventRecord(m->ev_fwd_end[l], cs));
    }
    if (prof) {
        // idle-event trigger: the backward plan while the first pull is in flight
        const auto t0 = Clock::now();
        DC_TRY(plan_backward(prof->bc_ns, prof->gt_ns, prof->dt_ns, L, plan->g, &plan->t_bwd_ns));
        t_plan_bwd = ns_since(t0);
        // the backward kernels are needed once the forward pass (already
        // enqueued) ends; planning before that costs the GPU nothing
        if (hipEventQuery(m->ev_fwd_end[L]) == hipErrorNotReady)
            hidden |= 1;
    }
    const auto pushes = push_segs(plan, L);
    // backward, closing push segments as their lowest layer finishes
    size_t k = 0;
    for (int l = L; l >= 1; --l) {
        DC_TRY(launch_backward_layer(m, l, b->x_dev, cs));
        if (m->timeline)
            DC_HIP(hipEventRecord(m->ev_bwd_end[l], cs));
        if (k < pushes.size() && pushes[k].lo == l) {
            DC_HIP(hipEventRecord(m->ev_bwd_done[k], cs));
            ++k;
        }
    }
    float *loss_host = m->probe_host; // first float of the pinned probe buffer
    DC_HIP(hipMemcpyAsync(loss_host, m->dloss(), sizeof(float), hipMemcpyDeviceToHost, cs));
    DC_HIP(hipEventRecord(m->ev_cs_done, cs));
    // push stream
    for (size_t i = 0; i < pushes.size(); ++i) {
        size_t off;
        size_t bytes = seg_bytes(m, pushes[i], &off);
        DC_HIP(hipStreamWaitEvent(m->push_s, m->ev_bwd_done[i], 0));
        DC_TRY(transmit(m, m->ps_grads + off, m->dgrads() + off, bytes, hipMemcpyDeviceToHost, link,
                        m->slots() + L + 1 + i, m->ev_push_start[i], m->ev_push_done[i], m->push_s));
    }
    // parameter server: update each range as soon as it has landed
    Clock::time_point t_last_push{};
    for (size_t i = 0; i < pushes.size(); ++i) {
        if (prof && i + 1 == pushes.size()) {
            // idle-event trigger: the next forward plan during the last push
            const auto t0 = Clock::now();
            int64_t t_fwd;
            DC_TRY(plan_forward(prof->pt_ns, prof->fc_ns, prof->dt_ns, L, plan->p, &t_fwd));
            plan->t_fwd_ns = t_fwd;
            t_plan_fwd = ns_since(t0);
            if (hipEventQuery(m->ev_push_done[i]) == hipErrorNotReady)
                hidden |= 2;
        }
        DC_TRY(wait_event(m->ev_push_done[i], deadline));
        if (i + 1 == pushes.size())
            t_last_push = Clock::now();
        size_t off;
        size_t bytes = seg_bytes(m, pushes[i], &off);
        sgd_range(m, off, bytes / sizeof(float));
    }
    const int64_t sgd_tail = ns_since(t_last_push);
    DC_HIP(hipStreamSynchronize(cs));

    if (out) {
        std::memset(out, 0, sizeof(*out));
        out->loss = loss_host[0];
        out->n_pull = (int32_t)pulls.size();
        out->n_push = (int32_t)pushes.size();
        DC_TRY(elapsed_ns(m->ev_t0, m->ev_push_done[pushes.size() - 1], &out->t_iter_ns));
        DC_TRY(elapsed_ns(m->ev_t0, m->ev_fwd_end[L], &out->t_fwd_ns));
        out->t_bwd_ns = out->t_iter_ns - out->t_fwd_ns;
        int64_t link_ns = 0, d;
        for (size_t i = 0; i < pulls.size(); ++i) {
            DC_TRY(elapsed_ns(m->ev_pull_start[i], m->ev_pull_done[i], &d));
            link_ns += d;
        }
        for (size_t i = 0; i < pushes.size(); ++i) {
            DC_TRY(elapsed_ns(m->ev_push_start[i], m->ev_push_done[i], &d));
            link_ns += d;
        }
        out->t_link_ns = link_ns;
        out->t_compute_ns = -1;
        out->t_sgd_tail_ns = sgd_tail;
        out->t_plan_bwd_ns = t_plan_bwd;
        out->t_plan_fwd_ns = t_plan_fwd;
        out->plan_hidden = hidden;
        for (size_t i = 0; i < m->gemm_n; ++i) {
            DC_TRY(elapsed_ns(m->gemm_ev[2 * i], m->gemm_ev[2 * i + 1], &d));
            out->t_gemm_ns += d;
            out->gemm_flop += m->gemm_flop[i];
        }
        out->n_gemm = (int32_t)m->gemm_n;
    }
    if (m->timeline) {
        m->timeline_ns.assign(8 * (size_t)L, 0);
        int64_t comp = 0;
        for (size_t s = 0; s < pulls.size(); ++s) {
            int64_t a, e;
            DC_TRY(elapsed_ns(m->ev_t0, m->ev_pull_start[s], &a));
            DC_TRY(elapsed_ns(m->ev_t0, m->ev_pull_done[s], &e));
            for (int l = pulls[s].lo; l <= pulls[s].hi; ++l) {
                m->timeline_ns[8 * (l - 1) + 0] = a;
                m->timeline_ns[8 * (l - 1) + 1] = e;
            }
        }
        for (size_t s = 0; s < pushes.size(); ++s) {
            int64_t a, e;
            DC_TRY(elapsed_ns(m->ev_t0, m->ev_push_start[s], &a));
            DC_TRY(elapsed_ns(m->ev_t0, m->ev_push_done[s], &e));
            for (int l = pushes[s].lo; l <= pushes[s].hi; ++l) {
                m->timeline_ns[8 * (l - 1) + 6] = a;
                m->timeline_ns[8 * (l - 1) + 7] = e;
            }
        }
        for (int l = 1; l <= L; ++l) {
            int64_t fs, fe, bs, be;
            DC_TRY(elapsed_ns(m->ev_t0, m->ev_fwd_start[l], &fs));
            DC_TRY(elapsed_ns(m->ev_t0, m->ev_fwd_end[l], &fe));
            DC_TRY(elapsed_ns(m->ev_t0, l == L ? m->ev_fwd_end[L] : m->ev_bwd_end[l + 1], &bs));
            DC_TRY(elapsed_ns(m->ev_t0, m->ev_bwd_end[l], &be));
            int64_t *row = &m->timeline_ns[8 * (l - 1)];
            row[2] = fs;
            row[3] = fe;
            row[4] = bs;
            row[5] = be;
            comp += (fe - fs) + (be - bs);
        }
        m->timeline_valid = true;
        if (out)
            out->t_compute_ns = comp;
    }
    if (prof) // f_m of the decisions now held in plan (p for the next call, g just used)
        plan->t_bwd_ns = fm_backward(prof->bc_ns, prof->gt_ns, prof->dt_ns, L, plan->g);
    if (out)
        out->t_host_ns = ns_since(t_host0);
    return DC_OK;
}

} // namespace
} // namespace dc

extern "C" int dc_step(dc_model *m, const dc_batch *b, const dc_plan_t *plan, const dc_link *link, void *stream,
                       dc_step_stats *out) {
    clear_error();
    return step_impl(m, b, const_cast<dc_plan_t *>(plan), nullptr, link, stream, out);
}

extern "C" int dc_step_dynamic(dc_model *m, const dc_batch *b, const dc_profile_t *prof, const dc_link *link,
                               void *stream, dc_plan_t *plan, dc_step_stats *out) {
    clear_error();
    if (!prof)
        return fail(DC_EINVAL, "profile is NULL");
    return step_impl(m, b, plan, prof, link, stream, out);
}

extern "C" int dc_timeline(const dc_model *m, int64_t *out, int n) {
    clear_error();
    if (!m || !out)
        return fail(DC_EINVAL, "model or out is NULL");
    if (!m->timeline_valid)
        return fail(DC_ESTATE, "no timeline recorded (enable DC_OPT_TIMELINE and run dc_step)");
    if (n < 8 * m->L)
        return fail(DC_EINVAL, "timeline needs %d entries", 8 * m->L);
    std::memcpy(out, m->timeline_ns.data(), sizeof(int64_t) * 8 * m->L);
    return DC_OK;
}

namespace {

// Least-squares fit of t = a + b * x.
void fit_line(const std::vector<double> &x, const std::vector<double> &t, double *a, double *b) {
    double n = (double)x.size(), sx = 0, st = 0, sxx = 0, sxt = 0;
    for (size_t i = 0; i < x.size(); ++i) {
        sx += x[i];
        st += t[i];
        sxx += x[i] * x[i];
        sxt += x[i] * t[i];
    }
    double den = n * sxx - sx * sx;
    *b = den != 0 ? (n * sxt - sx * st) / den : 0.0;
    *a = (st - *b * sx) / n;
}

// Time `reps` transmissions of each size in one direction through the same
// path a segment takes.  Returns (bytes, ns) samples.
int probe_link(dc_model *m, const dc_link *link, bool h2d, const std::vector<size_t> &sizes, int reps,
               std::vector<double> *xs, std::vector<double> *ts) {
    hipStream_t s = h2d ? m->pull_s : m->push_s;
    char *dev = m->ws + m->off_grads; // gradients are rewritten by every step
    const size_t dev_cap = m->n_params * sizeof(float);
    for (size_t sz : sizes) {
        size_t bytes = std::min({sz, dev_cap, m->probe_bytes});
        for (int r = 0; r <= reps; ++r) { // r = 0 warms up
            void *dst = h2d ? (void *)dev : (void *)m->probe_host;
            const void *src = h2d ? (const void *)m->probe_host : (const void *)dev;
            DC_TRY(transmit(m, dst, src, bytes, h2d ? hipMemcpyHostToDevice : hipMemcpyDeviceToHost, link,
                            m->slots() + 2 * m->L + 1, m->ev_pull_start[0], m->ev_pull_done[0], s));
            DC_HIP(hipEventSynchronize(m->ev_pull_done[0]));
            if (r == 0)
                continue;
            int64_t ns;
            DC_TRY(elapsed_ns(m->ev_pull_start[0], m->ev_pull_done[0], &ns));
            xs->push_back((double)bytes);
            ts->push_back((double)ns);
        }
    }
    return DC_OK;
}

// Handoff between streams: at a segment boundary one stream waits for an
// event of another (the forward waits for a pull, a push for the backward).
// The time from the awaited event to the waiting stream's next event is a
// fixed cost of every segment, which the cost model counts in Delta t with
// the transfer's own overhead.  Mean over reps of both directions, in ns.
int probe_handoff(dc_model *m, hipStream_t cs, int reps, double *ns) {
    double sum = 0;
    int n = 0;
    hipEvent_t e1 = m->ev_push_start[0], e2 = m->ev_push_done[0];
    for (int r = 0; r <= reps; ++r) { // r = 0 warms up
        for (int dir = 0; dir < 2; ++dir) {
            hipStream_t a = dir == 0 ? m->pull_s : cs, b = dir == 0 ? cs : m->push_s;
            DC_TRY(pace_mark(m->slots() + 2 * m->L, a));
            DC_HIP(hipEventRecord(e1, a));
            DC_HIP(hipStreamWaitEvent(b, e1, 0));
            DC_HIP(hipEventRecord(e2, b));
            DC_HIP(hipEventSynchronize(e2));
            if (r == 0)
                continue;
            int64_t d;
            DC_TRY(elapsed_ns(e1, e2, &d));
            sum += (double)std::max<int64_t>(d, 0);
            ++n;
        }
    }
    *ns = n ? sum / n : 0.0;
    return DC_OK;
}

} // namespace

extern "C" int dc_profile(dc_model *m, const dc_batch *b, const dc_link *link, int reps, void *stream,
                          dc_profile_t *out) {
    clear_error();
    if (!m || !out)
        return fail(DC_EINVAL, "model or out is NULL");
    if (!m->ws)
        return fail(DC_ESTATE, "no workspace bound");
    DC_TRY(check_batch(m, b));
    DC_TRY(check_link(link));
    if (reps < 1)
        return fail(DC_EINVAL, "reps must be >= 1");
    if (out->L != m->L || !out->pt_ns || !out->fc_ns || !out->bc_ns || !out->gt_ns)
        return fail(DC_EINVAL, "profile arrays must hold L=%d entries", m->L);
    const int L = m->L;
    hipStream_t cs = static_cast<hipStream_t>(stream);
    // the profile times whole layers; GEMM pass events are for dc_step only
    struct GemmTimingOff {
        dc_model *m;
        int saved;
        ~GemmTimingOff() { m->gemm_timing = saved; }
    } timing_off{m, m->gemm_timing};
    m->gemm_timing = 0;
    // every parameter on the device, then one untimed pass
    DC_HIP(hipMemcpyAsync(m->dparams(), m->ps_params, m->n_params * sizeof(float), hipMemcpyHostToDevice, cs));
    for (int l = 1; l <= L; ++l)
        DC_TRY(launch_forward_layer(m, l, b->x_dev, b->y_dev, cs));
    for (int l = L; l >= 1; --l)
        DC_TRY(launch_backward_layer(m, l, b->x_dev, cs));
    DC_HIP(hipStreamSynchronize(cs));
    std::vector<double> fsum(L + 1, 0.0), bsum(L + 1, 0.0);
    for (int r = 0; r < reps; ++r) {
        DC_HIP(hipEventRecord(m->ev_fwd_end[0], cs));
        for (int l = 1; l <= L; ++l) {
            DC_TRY(launch_forward_layer(m, l, b->x_dev, b->y_dev, cs));
            DC_HIP(hipEventRecord(m->ev_fwd_end[l], cs));
        }
        for (int l = L; l >= 1; --l) {
            DC_TRY(launch_backward_layer(m, l, b->x_dev, cs));
            DC_HIP(hipEventRecord(m->ev_bwd_end[l], cs));
        }
        DC_HIP(hipEventSynchronize(m->ev_bwd_end[1]));
        for (int l = 1; l <= L; ++l) {
            float ms;
            DC_HIP(hipEventElapsedTime(&ms, m->ev_fwd_end[l - 1], m->ev_fwd_end[l]));
            fsum[l] += ms;
            DC_HIP(hipEventElapsedTime(&ms, l == L ? m->ev_fwd_end[L] : m->ev_bwd_end[l + 1], m->ev_bwd_end[l]));
            bsum[l] += ms;
        }
    }
    for (int l = 1; l <= L; ++l) {
        out->fc_ns[l - 1] = std::max<int64_t>(0, (int64_t)llround(fsum[l] / reps * 1e6));
        out->bc_ns[l - 1] = std::max<int64_t>(0, (int64_t)llround(bsum[l] / reps * 1e6));
    }
    // transmission overhead and rate, per direction
    double a_h2d, b_h2d, a_d2h, b_d2h;
    std::vector<double> xs, ts;
    if (link->paced) {
        std::vector<size_t> sizes = {4096, 65536};
        double over[2] = {0, 0};
        for (int dir = 0; dir < 2; ++dir) {
            xs.clear();
            ts.clear();
            DC_TRY(probe_link(m, link, dir == 0, sizes, 3, &xs, &ts));
            double sum = 0;
            for (size_t i = 0; i < xs.size(); ++i)
                sum += ts[i] - xs[i] / link->bytes_per_s * 1e9;
            over[dir] = sum / xs.size();
        }
        a_h2d = over[0];
        a_d2h = over[1];
        b_h2d = b_d2h = 1e9 / link->bytes_per_s; // ns per byte
    } else {
        std::vector<size_t> sizes = {65536, 1 << 20, 4 << 20, 16 << 20};
        DC_TRY(probe_link(m, link, true, sizes, 3, &xs, &ts));
        fit_line(xs, ts, &a_h2d, &b_h2d);
        xs.clear();
        ts.clear();
        DC_TRY(probe_link(m, link, false, sizes, 3, &xs, &ts));
        fit_line(xs, ts, &a_d2h, &b_d2h);
        if (!(b_h2d > 0) || !(b_d2h > 0))
            return fail(DC_EHIP, "link probes gave a non-positive transfer rate");
    }
    for (int l = 1; l <= L; ++l) {
        double bytes = (double)m->layer_cnt[l] * sizeof(float);
        out->pt_ns[l - 1] = (int64_t)llround(bytes * b_h2d);
        out->gt_ns[l - 1] = (int64_t)llround(bytes * b_d2h);
    }
    double handoff = 0;
    DC_TRY(probe_handoff(m, cs, 5, &handoff));
    out->dt_ns = std::max<int64_t>(0, (int64_t)llround(0.5 * (a_h2d + a_d2h) + handoff));
    return DC_OK;
}
