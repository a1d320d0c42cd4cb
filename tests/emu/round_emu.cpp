// The bucketed insert's per-tensor hash rounds (bl_round, cut out of
// bloom.hip by the test that builds this file), checked over random item
// counts, capacities, planned rounds and hash counts: the rounds the host
// launches cover each tensor's hashes [0, k) exactly once and in order, and
// no round writes more position records than the tensor's region holds.
#include "hip/hip_runtime.h"
#include "dr_common.hpp"
#include <random>

namespace dr {
#include "ext_round.inc"
}  // namespace dr
using namespace dr;

int main(int argc, char **argv) {
    const uint32_t seed = argc > 1 ? atoi(argv[1]) : 1, cases = argc > 2 ? atoi(argv[2]) : 100000;
    std::mt19937_64 rng(seed);
    uint64_t bad = 0;
    for (uint32_t c = 0; c < cases; ++c) {
        TDesc td;
        memset(&td, 0, sizeof td);
        const uint32_t k = (uint32_t)(rng() % 33);                     // 0..32 hashes
        const uint64_t ncap = 1 + rng() % (c % 2 ? 40000000ull : 5000ull);
        const uint32_t hpr = (uint32_t)(1 + rng() % (k ? k : 1));    // the plan's hashes per round
        td.in.k = k;
        td.in.bl_poscap = ncap * hpr;
        td.n = (uint32_t)(rng() % 3 == 0 ? ncap : rng() % (ncap + 1));  // at most the planned items
        const uint32_t rounds = k ? (k + hpr - 1) / hpr : 1;            // what the launcher issues
        uint32_t next = 0;
        for (uint32_t r = 0; r < rounds; ++r) {
            uint32_t a, b;
            bl_round(td, r, hpr, &a, &b);
            if (a > b || b > k) ++bad;
            if (a < b && a != next) ++bad;                            // in order, no gap or overlap
            if ((uint64_t)td.n * (b - a) > td.in.bl_poscap) ++bad;    // the records fit the region
            if (a < b) next = b;
        }
        if (next != k) ++bad;  // every hash is inserted
    }
    printf("%s: %llu violations in %u cases\n", bad ? "FAIL" : "OK", (unsigned long long)bad, cases);
    return bad ? 1 : 0;
}
