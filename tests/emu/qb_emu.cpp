// Runs the receiver's bucketed query (the kernels' own source, extracted
// from bloom.hip by the test that builds this file) on the host, block by
// block, in the order the launcher issues them, and checks the positives
// bitmap against a direct query that uses the same hash code.  Built with
// AddressSanitizer and UBSan, so that any load or store outside a buffer
// (each is a separate heap allocation of exactly the planned size) stops
// the run.
#include "hip/hip_runtime.h"
#include "dr_common.hpp"
#include <functional>
#include <random>
#include <vector>

void emu_launch(uint32_t grid, uint32_t nt, const std::function<void()> &body);

namespace dr {
#include "ext_query.inc"
#include "ext_qb.inc"
}  // namespace dr
using namespace dr;

static uint64_t cdiv(uint64_t a, uint64_t b) { return (a + b - 1) / b; }

int main(int argc, char **argv) {
    if (argc < 6) {
        fprintf(stderr, "usage: d n m k layout [seed]\n");
        return 2;
    }
    const uint32_t d = atoi(argv[1]), n = atoi(argv[2]), m = atoi(argv[3]), k = atoi(argv[4]);
    const uint32_t layout = atoi(argv[5]);
    const uint32_t seed = argc > 6 ? atoi(argv[6]) : 1;
    const uint32_t ntiles = d ? (uint32_t)cdiv(d, TILE) : 1;
    // the filter of n random indices, with the device's own hash code
    std::mt19937 rng(seed);
    std::vector<uint8_t> insel(ntiles * TILE, 0);
    std::vector<uint32_t> S;
    while (S.size() < n) {
        const uint32_t i = rng() % d;
        if (!insel[i]) {
            insel[i] = 1;
            S.push_back(i);
        }
    }
    uint32_t ps[33];
    for (uint32_t j = 0; j <= k; ++j) ps[j] = (uint32_t)(((uint64_t)j * m) / k);
    const PosMap pm{m, layout == LAYOUT_PARTITIONED ? ps : nullptr};
    std::vector<uint32_t> filt(m / 32, 0);
    for (uint32_t i : S)
        for (uint32_t j = 0; j < k; ++j) {
            const uint32_t p = pm(mm3_key(i), j);
            filt[p >> 5] |= 1u << (p & 31);
        }
    std::vector<uint32_t> want(ntiles * TILE_WORDS, 0);
    for (uint32_t i = 0; i < d; ++i) {
        bool all = true;
        for (uint32_t j = 0; j < k && all; ++j) {
            const uint32_t p = pm(mm3_key(i), j);
            all = (filt[p >> 5] >> (p & 31)) & 1;
        }
        if (all) want[i >> 5] |= 1u << (i & 31);
    }
    // the record: a valid header (no values) and the filter
    std::vector<uint32_t> rec(16 + m / 32, 0);
    rec[H_MAGIC] = HDR_MAGIC;
    rec[H_BYTES] = HDR_BYTES;
    rec[H_D] = d;
    rec[H_MBITS] = m;
    rec[H_K] = k;
    rec[H_HASH] = layout == LAYOUT_PARTITIONED ? HASH_ID_PARTITIONED : HASH_ID_STANDARD;
    rec[H_B] = 1;
    memcpy(&rec[16], filt.data(), filt.size() * 4);
    // the plan's caps (api.hip plan_query_bucketed)
    const uint32_t nsl_cap = (uint32_t)cdiv(m, 1u << QB_SL), nch_cap = (uint32_t)cdiv(d, QB_CH),
                   nreg = (uint32_t)cdiv(d, 1u << QB_RL), ncol = std::max(nch_cap, nsl_cap);
    const uint64_t qcap = cdiv(d, 64) * 64, tab = (uint64_t)std::max(nsl_cap, nreg) * ncol,
                   rows = (uint64_t)(k + 1) * QB_MAX_BINS;
    std::vector<uint32_t> qlist(qcap, 0xA5A5A5A5u), qbkt(qcap, 0x5A5A5A5Au), qtab(tab, 0xDEADBEEFu),
        qrow(rows, 0xDEADBEEFu), pbits(ntiles * TILE_WORDS, 0xCCCCCCCCu), ttab(ntiles, 0);
    std::vector<TDesc> td(1);
    memset(&td[0], 0, sizeof(TDesc));
    TInit &in = td[0].in;
    in.d = d;
    in.ntiles = ntiles;
    in.k = k;
    in.layout = layout;
    in.rec = (uint8_t *)rec.data();
    in.rec_cap = rec.size() * 4;
    Work w{};
    w.td = td.data();
    w.ntensors = 1;
    w.ntiles_total = ntiles;
    w.slots = (uint64_t)ntiles * TILE;
    w.pbits = pbits.data();
    w.tile_tensor = ttab.data();
    w.qlist = qlist.data();
    w.qbkt = qbkt.data();
    w.qtab = qtab.data();
    w.qrow = qrow.data();
    w.qcap = qcap;
    const QbArgs a{0, k, 1024, nsl_cap, ncol};
    emu_launch(nch_cap, QB_THREADS, [&] { k_qb_count<Q_DECODE>(w, a); });
    for (uint32_t j = 0; j <= k; ++j) {
        emu_launch(j < k ? nsl_cap : nreg, QB_THREADS, [&] { k_qb_scan<Q_DECODE>(w, a, j); });
        emu_launch(ncol, QB_THREADS, [&] { k_qb_scatter<Q_DECODE>(w, a, j); });
        if (j < k) emu_launch(nsl_cap, QB_TEST_THREADS, [&] { k_qb_test<Q_DECODE>(w, a, j); });
    }
    emu_launch(nreg, QB_TEST_THREADS, [&] { k_qb_fill<Q_DECODE>(w, a); });
    if (!td[0].qb) {
        printf("FAIL: path not taken\n");
        return 1;
    }
    size_t bad = 0;
    for (size_t x = 0; x < want.size(); ++x) bad += pbits[x] != want[x];
    printf("%s: %zu of %zu words differ\n", bad ? "FAIL" : "OK", bad, want.size());
    return bad ? 1 : 0;
}
