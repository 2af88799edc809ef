// Host check of the multiply-high division by an invariant integer that the
// kernels use for index arithmetic (dc::FDiv): against n / d for every
// divisor below 5000 and random divisors up to 2^31 - 1, at the boundary
// dividends (0, d - 1, d, d + 1, multiples of d, 2^31 - 1) and random ones.
#include "dc_internal.h"

#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

int main() {
    std::mt19937_64 rng(20210119);
    std::uniform_int_distribution<uint32_t> any(0, 0x7fffffffu), big(2, 0x7fffffffu);
    std::vector<uint32_t> divisors;
    for (uint32_t d = 1; d < 5000; ++d)
        divisors.push_back(d);
    for (int i = 0; i < 20000; ++i)
        divisors.push_back(big(rng));
    for (uint32_t d : {0x40000000u, 0x7fffffffu, 0x7ffffffeu, 65536u, 65537u, 3u * 224 * 224})
        divisors.push_back(d);
    long checked = 0;
    for (uint32_t d : divisors) {
        const dc::FDiv f = dc::make_fdiv(d);
        std::vector<uint32_t> ns = {0u, d - 1, d, d + 1, 2 * d - 1, 2 * d, 0x7fffffffu, 0x7ffffffeu};
        for (int i = 0; i < 64; ++i)
            ns.push_back(any(rng));
        const uint32_t q_top = 0x7fffffffu / d;
        ns.push_back(q_top * d);
        if (q_top * d > 0)
            ns.push_back(q_top * d - 1);
        for (uint32_t n : ns) {
            if (n > 0x7fffffffu)
                continue; // the kernels divide only n < 2^31
            if (f.div(n) != n / d) {
                std::printf("FAIL d=%u n=%u got %u want %u\n", d, n, f.div(n), n / d);
                return 1;
            }
            ++checked;
        }
    }
    std::printf("ok %ld\n", checked);
    return 0;
}
