// The host planner under AddressSanitizer and UndefinedBehaviorSanitizer.
//
// Random profiles (a fixed xorshift stream), lengths 1..300 with every
// magnitude from a few ns to near the int64 limit, run through both DPs, both
// iBatch passes and the f_m evaluators.  Checks what optimality and the
// contract fix without a second implementation: the DP value equals f_m of the
// DP's own decision and is no larger than f_m of one segment, of one segment
// per layer and of iBatch's decision; inputs whose sums overflow int64 are
// refused with DC_EINVAL, never wrapped.  Built and run by test_host_pool.py.
#include "dc_internal.h"

#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <vector>

namespace dc {
// the error plumbing of the library, reduced to what the planner calls
int fail(int code, const char *, ...) { return code; }
int hip_fail(hipError_t, const char *) { return DC_EHIP; }
void clear_error() {}
} // namespace dc

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint64_t next() {
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 7;
    rng_state ^= rng_state << 17;
    return rng_state;
}
static int64_t draw(int64_t hi) { return hi <= 0 ? 0 : (int64_t)(next() % (uint64_t)(hi + 1)); }

#define CHECK(c)                                                                  \
    do {                                                                          \
        if (!(c)) {                                                               \
            std::fprintf(stderr, "check failed: %s (case %d, L %d)\n", #c, n, L); \
            return 1;                                                             \
        }                                                                         \
    } while (0)

int main(int argc, char **argv) {
    const int cases = argc > 1 ? std::atoi(argv[1]) : 3000;
    const int64_t his[] = {10, 1000, 1000000, 1000000000000LL, INT64_MAX / 400};
    for (int n = 0; n < cases; ++n) {
        const int L = n % 10 == 9 ? 100 + (int)draw(200) : 1 + (int)draw(40);
        const int64_t hi = his[n % 5];
        std::vector<int64_t> pt(L), fc(L), bc(L), gt(L);
        for (int l = 0; l < L; ++l) {
            pt[l] = draw(hi);
            fc[l] = draw(hi);
            bc[l] = draw(hi);
            gt[l] = draw(hi);
        }
        const int64_t dt = draw(hi / 2);
        const int m = L > 1 ? L - 1 : 1;
        std::vector<uint8_t> p(m, 0), g(m, 0), pi(m, 0), gi(m, 0), zero(m, 0), one(m, 1);
        int64_t tf = -1, tb = -1, tbi = -1;
        const int sf = dc::plan_forward(pt.data(), fc.data(), dt, L, p.data(), &tf);
        const int sb = dc::plan_backward(bc.data(), gt.data(), dt, L, g.data(), &tb);
        if (hi == INT64_MAX / 400 && L >= 100) {
            // sums of up to 300 values near 2^63 / 400 may overflow: refused or planned, never wrapped
            CHECK(sf == DC_OK || sf == DC_EINVAL);
            CHECK(sb == DC_OK || sb == DC_EINVAL);
            if (sf != DC_OK || sb != DC_OK)
                continue;
        }
        CHECK(sf == DC_OK && sb == DC_OK);
        CHECK(tf == dc::fm_forward(pt.data(), fc.data(), dt, L, p.data()));
        CHECK(tb == dc::fm_backward(bc.data(), gt.data(), dt, L, g.data()));
        CHECK(tf <= dc::fm_forward(pt.data(), fc.data(), dt, L, zero.data()));
        CHECK(tf <= dc::fm_forward(pt.data(), fc.data(), dt, L, one.data()));
        CHECK(tb <= dc::fm_backward(bc.data(), gt.data(), dt, L, zero.data()));
        CHECK(tb <= dc::fm_backward(bc.data(), gt.data(), dt, L, one.data()));
        CHECK(dc::plan_ibatch_forward(pt.data(), fc.data(), dt, L, pi.data()) == DC_OK);
        CHECK(dc::plan_ibatch_backward(bc.data(), gt.data(), dt, L, gi.data(), &tbi) == DC_OK);
        CHECK(tf <= dc::fm_forward(pt.data(), fc.data(), dt, L, pi.data()));
        CHECK(tb <= tbi && tbi == dc::fm_backward(bc.data(), gt.data(), dt, L, gi.data()));
    }
    // refused inputs
    {
        const int n = -1, L = 2;
        int64_t big[2] = {INT64_MAX, INT64_MAX}, one_[2] = {1, 1}, neg[2] = {1, -2}, t = 0;
        uint8_t d[1];
        CHECK(dc::plan_forward(big, one_, 0, 2, d, &t) == DC_EINVAL);
        CHECK(dc::plan_backward(one_, big, 0, 2, d, &t) == DC_EINVAL);
        CHECK(dc::plan_forward(neg, one_, 0, 2, d, &t) == DC_EINVAL);
        CHECK(dc::plan_forward(one_, one_, -1, 2, d, &t) == DC_EINVAL);
        CHECK(dc::plan_forward(one_, one_, 0, 0, d, &t) == DC_EINVAL);
    }
    std::printf("ok %d cases\n", cases);
    return 0;
}
