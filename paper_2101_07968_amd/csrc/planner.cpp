// DynaComm's communication scheduler (Sec. IV-B) on the host.
//
// The forward decision comes from the Bellman equation of Eq. 8 solved
// bottom-up with the traceback of Algorithm 3, the backward decision from
// Eq. 9 and Algorithm 4.  All costs are int64 nanoseconds, so every sum is
// exact and independent of evaluation order; +infinity is INT64_MAX and
// never takes part in arithmetic.  Range sums come from prefix arrays
// (Sec. IV-B-4), giving O(L^3) time and O(L^2) space.  A table entry only
// changes when a candidate is strictly smaller, with k and then n scanned
// upwards, so ties keep the smallest split point and the fewest segments.
#include "dc_internal.h"

#include <algorithm>
#include <climits>
#include <vector>

namespace dc {
namespace {

constexpr int64_t INF = INT64_MAX;

bool add_ok(int64_t a, int64_t b, int64_t *out) { return !__builtin_add_overflow(a, b, out); }
bool mul_ok(int64_t a, int64_t b, int64_t *out) { return !__builtin_mul_overflow(a, b, out); }

// prefix[l] = v[0] + ... + v[l-1]; false on overflow or a negative entry.
bool prefix_sums(const int64_t *v, int L, std::vector<int64_t> &prefix) {
    prefix.assign(L + 1, 0);
    for (int l = 0; l < L; ++l) {
        if (v[l] < 0 || !add_ok(prefix[l], v[l], &prefix[l + 1]))
            return false;
    }
    return true;
}

// An upper bound on every finite table entry, checked once so that the inner
// loops can add without overflow tests: any schedule finishes by
// L*dt + sum(transfers) + sum(compute).
bool bound_ok(int L, int64_t dt, int64_t sum_a, int64_t sum_b) {
    int64_t t, u;
    return dt >= 0 && mul_ok((int64_t)L + 1, dt, &t) && add_ok(t, sum_a, &u) && add_ok(u, sum_b, &t) &&
           t < INF / 4;
}

} // namespace

int plan_forward(const int64_t *pt, const int64_t *fc, int64_t dt, int L, uint8_t *p, int64_t *t_fwd) {
    if (L < 1)
        return fail(DC_EINVAL, "L must be >= 1");
    std::vector<int64_t> PT, FC;
    if (!prefix_sums(pt, L, PT) || !prefix_sums(fc, L, FC))
        return fail(DC_EINVAL, "forward costs must be non-negative and their sums must fit in int64");
    if (!bound_ok(L, dt, PT[L], FC[L]))
        return fail(DC_EINVAL, "forward costs overflow int64 (or dt < 0)");
    const int W = L + 1;
    // F[m][n]: finishing time of the forward computation of layers 1..m when
    // their parameters arrive in n pull mini-procedures (Eq. 8).
    std::vector<int64_t> F((size_t)W * W, INF);
    std::vector<int32_t> Path((size_t)W * W, -1);
    F[0] = 0;
    for (int m = 1; m <= L; ++m) {
        for (int n = 1; n <= m; ++n) {
            int64_t best = INF;
            int32_t arg = -1;
            const int64_t arrive = (int64_t)n * dt + PT[m]; // the n-th pull ends
            for (int k = 0; k < m; ++k) {
                const int64_t prev = F[(size_t)k * W + (n - 1)];
                if (prev == INF)
                    continue;
                const int64_t start = prev > arrive ? prev : arrive;
                const int64_t cand = start + (FC[m] - FC[k]);
                if (best <= cand)
                    continue;
                best = cand;
                arg = k;
            }
            F[(size_t)m * W + n] = best;
            Path[(size_t)m * W + n] = arg;
        }
    }
    int64_t t = INF;
    int steps = -1;
    for (int k = 1; k <= L; ++k) {
        if (t <= F[(size_t)L * W + k])
            continue;
        t = F[(size_t)L * W + k];
        steps = k;
    }
    for (int l = 0; l < L - 1; ++l)
        p[l] = 0;
    int cl = L;
    for (int k = 1; k <= steps; ++k) {
        int tmp = Path[(size_t)cl * W + (steps - k + 1)];
        if (tmp >= 1 && tmp <= L - 1)
            p[tmp - 1] = 1;
        cl = tmp;
    }
    *t_fwd = t;
    return DC_OK;
}

int plan_backward(const int64_t *bc, const int64_t *gt, int64_t dt, int L, uint8_t *g, int64_t *t_bwd) {
    if (L < 1)
        return fail(DC_EINVAL, "L must be >= 1");
    std::vector<int64_t> BC, GT;
    if (!prefix_sums(bc, L, BC) || !prefix_sums(gt, L, GT))
        return fail(DC_EINVAL, "backward costs must be non-negative and their sums must fit in int64");
    if (!bound_ok(L, dt, BC[L], GT[L]))
        return fail(DC_EINVAL, "backward costs overflow int64 (or dt < 0)");
    const int W = L + 1;
    // B[m][n]: time at which the gradients of the last m layers have been
    // pushed in n push mini-procedures (Eq. 9).  The new segment holds layers
    // L-m+1..L-k and may start when backward has finished layer L-m+1.
    std::vector<int64_t> B((size_t)W * W, INF);
    std::vector<int32_t> Path((size_t)W * W, -1);
    B[0] = 0;
    for (int m = 1; m <= L; ++m) {
        const int64_t ready = BC[L] - BC[L - m]; // bc over layers L-m+1..L
        for (int n = 1; n <= m; ++n) {
            int64_t best = INF;
            int32_t arg = -1;
            for (int k = 0; k < m; ++k) {
                const int64_t prev = B[(size_t)k * W + (n - 1)];
                if (prev == INF)
                    continue;
                const int64_t start = prev > ready ? prev : ready;
                const int64_t cand = start + dt + (GT[L - k] - GT[L - m]); // gt over L-m+1..L-k
                if (best <= cand)
                    continue;
                best = cand;
                arg = k;
            }
            B[(size_t)m * W + n] = best;
            Path[(size_t)m * W + n] = arg;
        }
    }
    int64_t t = INF;
    int steps = -1;
    for (int k = 1; k <= L; ++k) {
        if (t <= B[(size_t)L * W + k])
            continue;
        t = B[(size_t)L * W + k];
        steps = k;
    }
    for (int l = 0; l < L - 1; ++l)
        g[l] = 0;
    int cl = 1;
    for (int k = 1; k <= steps; ++k) {
        int tmp = Path[(size_t)(L - cl + 1) * W + (steps - k + 1)];
        if (tmp >= 1 && tmp <= L - 1)
            g[tmp - 1] = 1;
        cl = L - tmp + 1;
    }
    *t_bwd = t;
    return DC_OK;
}

// iBatch, the greedy baseline the paper compares against (Sec. III-C,
// Algorithms 1 and 2).  Open cases are read as follows: the second position of
// Algorithm 1 is chosen, among the pairs sharing the selected first position,
// by the loop's least-slack rule; with no qualifying pair the model is one
// segment; with no qualifying position the forward loop sends the rest as one
// segment and the backward loop the single next layer; slack ties go to the
// position met first in the scan, candidate ties to the first candidate.
int plan_ibatch_forward(const int64_t *pt, const int64_t *fc, int64_t dt, int L, uint8_t *p) {
    std::vector<int64_t> PT, FC;
    if (L < 1 || !prefix_sums(pt, L, PT) || !prefix_sums(fc, L, FC) || !bound_ok(L, dt, PT[L], FC[L]))
        return fail(DC_EINVAL, "invalid forward costs");
    for (int l = 0; l < L - 1; ++l)
        p[l] = 0;
    if (L == 1)
        return DC_OK;
    // steps 1-4: the first two positions
    int d1 = -1;
    int64_t best_fc = -1, best_pull = INF;
    for (int a = 1; a < L; ++a) {
        bool any = false;
        for (int b = a + 1; b <= L && !any; ++b)
            any = dt + (PT[b] - PT[a]) >= FC[a];
        if (!any)
            continue;
        const int64_t f = FC[a], pull = dt + PT[a];
        if (f > best_fc || (f == best_fc && pull < best_pull)) {
            best_fc = f;
            best_pull = pull;
            d1 = a;
        }
    }
    if (d1 < 0)
        return DC_OK; // nothing qualifies: one segment
    int d2 = -1;
    int64_t best_slack = INF;
    for (int b = d1 + 1; b <= L; ++b) {
        const int64_t slack = dt + (PT[b] - PT[d1]) - FC[d1];
        if (slack >= 0 && slack < best_slack) {
            best_slack = slack;
            d2 = b;
        }
    }
    if (d1 <= L - 1)
        p[d1 - 1] = 1;
    int n = d1, m = d2;
    while (m != L) {
        p[m - 1] = 1;
        const int64_t need = FC[m] - FC[n];
        int j = L;
        int64_t bs = INF;
        for (int x = m + 1; x <= L; ++x) {
            const int64_t slack = dt + (PT[x] - PT[m]) - need;
            if (slack >= 0 && slack < bs) {
                bs = slack;
                j = x;
            }
        }
        n = m;
        m = j;
    }
    return DC_OK;
}

int plan_ibatch_backward(const int64_t *bc, const int64_t *gt, int64_t dt, int L, uint8_t *g, int64_t *t_bwd) {
    std::vector<int64_t> BC, GT;
    if (L < 1 || !prefix_sums(bc, L, BC) || !prefix_sums(gt, L, GT) || !bound_ok(L, dt, BC[L], GT[L]))
        return fail(DC_EINVAL, "invalid backward costs");
    std::vector<uint8_t> cand(L > 1 ? L - 1 : 1), best(L > 1 ? L - 1 : 1, 0);
    int64_t best_t = INF;
    if (L == 1) {
        *t_bwd = fm_backward(bc, gt, dt, L, best.data());
        return DC_OK;
    }
    for (int n = 2; n <= L; ++n) {
        std::fill(cand.begin(), cand.end(), 0);
        int m = n, k = 1;
        // position m (1 < m <= L) is the boundary between layer m and m-1: g_{L-m+1}
        for (;;) {
            cand[L - m] = 1;
            const int64_t pushed = (int64_t)k * dt + (GT[L] - GT[m - 1]);
            int j = m - 1;
            int64_t bs = INF;
            for (int x = 1; x < m; ++x) {
                const int64_t slack = pushed - (BC[m - 1] - BC[x - 1]);
                if (slack >= 0 && slack < bs) {
                    bs = slack;
                    j = x;
                }
            }
            m = j;
            ++k;
            if (m == 1)
                break;
        }
        const int64_t t = fm_backward(bc, gt, dt, L, cand.data());
        if (t < best_t) {
            best_t = t;
            best = cand;
        }
    }
    for (int l = 0; l < L - 1; ++l)
        g[l] = best[l];
    *t_bwd = best_t;
    return DC_OK;
}

// f_m, forward part: pulls back to back from time 0, each segment dt plus its
// layers' pt; a segment computes once it has arrived and its predecessor is done.
int64_t fm_forward(const int64_t *pt, const int64_t *fc, int64_t dt, int L, const uint8_t *p) {
    int64_t link = 0, done = 0;
    int lo = 1;
    for (int l = 1; l <= L; ++l) {
        if (l == L || p[l - 1]) {
            int64_t bytes_t = 0, comp = 0;
            for (int i = lo; i <= l; ++i) {
                bytes_t += pt[i - 1];
                comp += fc[i - 1];
            }
            link += dt + bytes_t;
            done = (done > link ? done : link) + comp;
            lo = l + 1;
        }
    }
    return done;
}

// f_m, backward part: segments top first; a segment starts when the link is
// free and backward has finished its lowest layer.
int64_t fm_backward(const int64_t *bc, const int64_t *gt, int64_t dt, int L, const uint8_t *g) {
    int64_t link = 0;
    int hi = L;
    for (int k = 1; k <= L; ++k) {
        if (k == L || g[k - 1]) {
            int lo = L - k + 1;
            int64_t ready = 0, xfer = 0;
            for (int i = lo; i <= L; ++i)
                ready += bc[i - 1];
            for (int i = lo; i <= hi; ++i)
                xfer += gt[i - 1];
            link = (link > ready ? link : ready) + dt + xfer;
            hi = lo - 1;
        }
    }
    return link;
}

} // namespace dc
