// Runs the reorder-map packing (pack_sigma_words and the search it starts
// from: the kernel's own source, cut out of valuefit.hip by the test that
// builds this file) on the host, for every thread of a launch in turn, over
// tensors of random sizes (empty ones among them), and checks each tensor's
// words against a direct LSB-first packing of its b-bit entries.  Built with
// AddressSanitizer and UBSan: each tensor's output is a heap allocation of
// exactly its word count, so a store past a map stops the run.
#include "hip/hip_runtime.h"
#include "dr_common.hpp"
#include <random>
#include <vector>

namespace dr {
#include "ext_pack.inc"
}  // namespace dr
using namespace dr;

int main(int argc, char **argv) {
    if (argc < 5) {
        fprintf(stderr, "usage: seed ntensors max_nv threads\n");
        return 2;
    }
    const uint32_t seed = atoi(argv[1]), nt = atoi(argv[2]), max_nv = atoi(argv[3]), threads = atoi(argv[4]);
    std::mt19937 rng(seed);
    std::vector<TDesc> td(nt);
    std::vector<std::vector<uint32_t>> out(nt), want(nt);
    std::vector<uint32_t> nv(nt);
    uint64_t slots = 0, words = 0;
    for (uint32_t t = 0; t < nt; ++t) {
        // sizes over both of the packing's paths (b < 16 and b >= 16), and
        // empty tensors
        const uint32_t pick = rng() % 4;
        nv[t] = pick == 0 ? 0u : pick == 1 ? 1u + rng() % 300u : 1u + rng() % max_nv;
        slots += nv[t];
    }
    std::vector<uint32_t> sig(slots ? slots : 1);
    uint64_t slot = 0;
    for (uint32_t t = 0; t < nt; ++t) {
        memset(&td[t], 0, sizeof(TDesc));
        const uint32_t b = sigma_bits(nv[t]);
        const uint64_t nw = ((uint64_t)nv[t] * b + 31) / 32;
        td[t].nv = nv[t];
        td[t].b = b;
        td[t].sw0 = (uint32_t)words;
        td[t].in.slot = slot;
        out[t].assign(nw, 0xA5A5A5A5u);
        want[t].assign(nw, 0u);
        td[t].in.sigma = out[t].data();
        for (uint32_t q = 0; q < nv[t]; ++q) {
            const uint32_t e = (uint32_t)(rng() % nv[t]);  // a rank below nv: fits b bits
            sig[slot + q] = e;
            for (uint32_t x = 0; x < b; ++x)
                if ((e >> x) & 1u) {
                    const uint64_t bit = (uint64_t)q * b + x;
                    want[t][bit >> 5] |= 1u << (bit & 31);
                }
        }
        slot += nv[t];
        words += nw;
    }
    Glob glob{};
    glob.sigma_words = (uint32_t)words;
    Work w{};
    w.td = td.data();
    w.ntensors = nt;
    w.glob = &glob;
    w.sig = sig.data();
    for (uint32_t first = 0; first < threads; ++first) pack_sigma_words(w, first, threads);
    size_t bad = 0;
    for (uint32_t t = 0; t < nt; ++t)
        for (size_t x = 0; x < want[t].size(); ++x) bad += out[t][x] != want[t][x];
    printf("%s: %zu words differ of %llu (%u tensors)\n", bad ? "FAIL" : "OK", bad, (unsigned long long)words, nt);
    return bad ? 1 : 0;
}
