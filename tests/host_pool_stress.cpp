// Stress driver for dc::HostPool (built with g++ by tests/test_host_pool.py).
// Many short jobs back to back, with a varying pause between them so that
// workers wake late, after the job they were signalled for has finished:
// every index of every job must run exactly once and nothing may crash.
#include "host_pool.h"

#include <atomic>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <vector>

int main(int argc, char **argv) {
    const int rounds = argc > 1 ? std::atoi(argv[1]) : 200000;
    dc::HostPool pool(8);
    std::vector<std::atomic<int>> hits(64);
    unsigned rng = 12345;
    for (int r = 0; r < rounds; ++r) {
        rng = rng * 1664525u + 1013904223u;
        const int n = 2 + (int)(rng >> 28) % 6; // 2..7 indices
        for (int i = 0; i < n; ++i)
            hits[i].store(0, std::memory_order_relaxed);
        pool.run(n, [&](int i, int m) {
            if (m != n || i < 0 || i >= n)
                std::abort();
            hits[i].fetch_add(1, std::memory_order_relaxed);
        });
        for (int i = 0; i < n; ++i)
            if (hits[i].load() != 1) {
                std::printf("round %d: index %d ran %d times\n", r, i, hits[i].load());
                return 1;
            }
        // pause 0-20 us so that late workers wake between jobs
        const auto t0 = std::chrono::steady_clock::now();
        const int us = (int)(rng >> 8) % 21;
        while (std::chrono::steady_clock::now() - t0 < std::chrono::microseconds(us)) {
        }
    }
    std::printf("ok %d rounds\n", rounds);
    return 0;
}
