// Launch plans chosen by measurement for the implicit-GEMM conv passes.
//
// The cost model in plan_core picks a tile and a split-K factor from an
// occupancy estimate.  For the shapes of the built-in workloads the library
// also carries the plan that timed fastest on gfx950 (plan_table.inc, written
// by paper_2101_07968_amd/tune.py, which times every candidate plan of every
// pass through the C ABI).  A shape is listed only where its best plan beat
// the cost model's choice by a clear margin.  Each process may further pin a
// plan per shape and pass (dc_conv2d_set_plan); pins take precedence over the
// table.  Plans only decide how the sums are tiled and split: a pass gives the
// same result to rounding whichever plan runs it.
#include "dc_internal.h"

#include <array>
#include <map>
#include <mutex>

namespace dc {
namespace {

struct Entry {
    int pass, n, h, w, c, k, r, s, st, pad, pad_w; // the pass and its dc_conv_shape
    int mt, nt, splits;                           // the measured plan
};

const Entry kTable[] = {
#include "plan_table.inc"
    {-1, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0}, // end
};

using Key = std::array<int, 11>;
using Plan = std::array<int, 3>;

Key key_of(const ConvGeom &g, int pass) {
    return {pass, g.N, g.H, g.W, g.C, g.K, g.R, g.S, g.st, g.pad, g.pad_w};
}

const std::map<Key, Plan> &table() {
    static const std::map<Key, Plan> m = [] {
        std::map<Key, Plan> t;
        for (const Entry &e : kTable)
            if (e.pass >= 0)
                t[{e.pass, e.n, e.h, e.w, e.c, e.k, e.r, e.s, e.st, e.pad, e.pad_w}] = {e.mt, e.nt, e.splits};
        return t;
    }();
    return m;
}

std::mutex g_pin_mu;
std::map<Key, Plan> g_pins; // mt == -1: the cost model's own choice

} // namespace

int lookup_plan(const ConvGeom &g, int pass, int out[3]) {
    const Key k = key_of(g, pass);
    {
        std::lock_guard<std::mutex> lk(g_pin_mu);
        auto it = g_pins.find(k);
        if (it != g_pins.end()) {
            if (it->second[0] < 0)
                return -1;
            for (int i = 0; i < 3; ++i)
                out[i] = it->second[i];
            return PLAN_PINNED;
        }
    }
    auto it = table().find(k);
    if (it == table().end())
        return PLAN_MODEL;
    for (int i = 0; i < 3; ++i)
        out[i] = it->second[i];
    return PLAN_TABLE;
}

void pin_plan(const ConvGeom &g, int pass, int mt, int nt, int splits) {
    const Key k = key_of(g, pass);
    std::lock_guard<std::mutex> lk(g_pin_mu);
    if (mt == 0)
        g_pins.erase(k);
    else
        g_pins[k] = {mt, nt, splits};
}

} // namespace dc
