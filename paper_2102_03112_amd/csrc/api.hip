// api.hip -- the C ABI (include/deepreduce.h): argument checks, the
// per-tensor plan, the workspace carve, and the launch sequence of each
// entry point.  Everything here runs on the host; all arithmetic of the
// codec runs in the kernels.
#include <math.h>

#include <cmath>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "deepreduce.h"
#include "launch.hpp"

using namespace dr;
static_assert(POLICY_P0 == DR_POLICY_P0 && POLICY_RANDOM == DR_POLICY_RANDOM && POLICY_LEFTMOST == DR_POLICY_LEFTMOST &&
                  POLICY_MIDDLE == DR_POLICY_MIDDLE && POLICY_RIGHTMOST == DR_POLICY_RIGHTMOST,
              "index policy ids");
static_assert(SEG_EQUAL == DR_SEG_EQUAL && SEG_CHORD == DR_SEG_CHORD, "segmentation ids");
static_assert(FIT_POLY == DR_FIT_POLY && FIT_DEXP == DR_FIT_DEXP, "value model ids");
static_assert(VALUES_DENSE == DR_VALUES_DENSE && VALUES_SPARSE == DR_VALUES_SPARSE, "value source ids");
static_assert(LAYOUT_STANDARD == DR_FILTER_STANDARD && LAYOUT_PARTITIONED == DR_FILTER_PARTITIONED, "filter layouts");
static_assert(MAX_SEG == DR_MAX_SEGMENTS && MAX_DEG == DR_MAX_DEGREE, "limits of the header and the kernels");

namespace {

thread_local std::string g_err;

void trace_call(hipStream_t s);  // per-kernel timing, defined below

dr_status fail(dr_status st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

dr_status hip_fail(hipError_t e, const char *where) {
    return fail(DR_EDEVICE, "%s: %s", where, hipGetErrorString(e));
}

#define DR_HIP(call)                                       \
    do {                                                   \
        hipError_t e_ = (call);                            \
        if (e_ != hipSuccess) return hip_fail(e_, #call);  \
    } while (0)

uint64_t ceil_div(uint64_t a, uint64_t b) { return (a + b - 1) / b; }
uint64_t align_up(uint64_t a, uint64_t b) { return ceil_div(a, b) * b; }

// Remark 2 of Section 10.2, rounded (see deepreduce.h)
bool bloom_params_host(uint64_t n, double fpr, uint64_t *m, uint32_t *k) {
    if (!(fpr > 0.0 && fpr < 1.0)) return false;
    const double ln2 = log(2.0);
    long kr = lround(-log(fpr) / ln2);
    if (kr < 1) kr = 1;
    const double C = -log(fpr) / (ln2 * ln2);
    uint64_t mm = (uint64_t)ceil((double)n * C);
    mm = align_up(mm, 32);
    if (mm < 32) mm = 32;
    if (mm >= (1ull << 32) || kr > 32) return false;
    *m = mm;
    *k = (uint32_t)kr;
    return true;
}

uint32_t sigma_bits_host(uint64_t n) {
    uint32_t b = 1;
    while (b < 63 && (1ull << b) < n) ++b;
    return b;
}

int persist_grid(int per_cu) { return dr::device_cus() * per_cu; }

// Workspace regions, in carve order.  Element-sized regions have `slots`
// entries (padded elements); the last six are contiguous so the Bloom insert
// can borrow them for its position buffer before the value path needs them.
struct Carve {
    uint64_t slots = 0, ntiles = 0, ntensors = 0, hist_blocks = 0, redo_blocks = 0, fit_blocks = 0, btab = 0,
             bslices = 0, bnd = 0, segslots = 0;
    // bucketed query: list entries (the largest such tensor's size), count
    // table words and round-total words; both carves hold them
    uint64_t qb_entries = 0, qb_tab = 0, qb_rows = 0;
    // values the sender expects to code (r per top-r tensor, doubled for its
    // false positives; d for the support): sizes the reorder-map packing grid
    uint64_t vals_est = 0;
    bool query_only = false;  // descriptors, tile counts, the positives bitmap and the tile table only
    size_t bytes = 0;
    size_t o_td, o_glob, o_pstat, o_histA, o_shist, o_fcnt, o_tcnt, o_toff, o_ccnt, o_hist, o_sel, o_pbits, o_ckey, o_cidx, o_S, o_P,
        o_V, o_sstat, o_sdig, o_ttab, o_fit, o_btab, o_brow, o_keyA, o_keyB, o_valA, o_valB, o_sig, o_vs, o_bnd,
        o_segst, o_segpart, o_qlist, o_qbkt, o_qtab, o_qrow;

    void plan() {
        size_t at = 0;
        auto take = [&](size_t sz) {
            size_t r = at;
            at = align_up(at + sz, 256);
            return r;
        };
        const uint64_t all = query_only ? 0 : 1;  // regions the query alone does not use
        o_td = take(sizeof(TDesc) * ntensors);
        o_glob = take(sizeof(Glob));
        o_pstat = take(8ull * PSTAT_MAX);
        o_tcnt = take(4 * ntiles);
        o_toff = take(4 * ntiles);
        o_pbits = take(slots / 8);
        o_ttab = take(4ull * ntiles);
        o_qlist = take(4 * qb_entries);
        o_qbkt = take(4 * qb_entries);
        o_qtab = take(4 * qb_tab);
        o_qrow = take(4 * qb_rows);
        o_ccnt = take(all * 4 * ntiles);
        // the selection's counters, contiguous: k_init clears them as one range
        o_hist = take(all * 4ull * HIST1_BINS * ntensors);
        o_histA = take(all * 4ull * HISTA_BINS * HISTA_COPIES * ntensors);
        o_shist = take(all * 4ull * HIST1_BINS * SHIST_COPIES * ntensors);
        o_fcnt = take(all * 4ull * FCNT_COPIES * FCNT_W * ntensors);
        o_sel = take(all * slots / 8);
        o_ckey = take(all * 4 * slots);
        o_cidx = take(all * 4 * slots);
        o_S = take(all * 4 * slots);
        o_P = take(all * 4 * slots);
        o_V = take(all * 4 * slots);
        o_sstat = take(all * 8ull * 4 * SORT_BINS * ntiles);
        o_sdig = take(all * 4ull * 4 * SORT_BINS * ntensors);
        o_fit = take(all * 8ull * NMOM * fit_blocks);
        o_btab = take(all * 4 * btab);
        o_brow = take(all * 8 * bslices);
        o_bnd = take(all * 4 * bnd);
        o_segst = take(all * sizeof(SegState) * segslots);
        o_segpart = take(all * sizeof(SegPart) * SEG_GRID_BLOCKS * segslots);
        o_keyA = take(all * 4 * slots);
        o_keyB = take(all * 4 * slots);
        o_valA = take(all * 4 * slots);
        o_valB = take(all * 4 * slots);
        o_sig = take(all * 4 * slots);
        o_vs = take(all * 4 * slots);
        bytes = at;
    }

    Work view(uint8_t *ws) const {
        Work w{};
        w.td = (TDesc *)(ws + o_td);
        w.glob = (Glob *)(ws + o_glob);
        w.ntensors = (uint32_t)ntensors;
        w.ntiles_total = (uint32_t)ntiles;
        w.slots = slots;
        w.pstat = (uint64_t *)(ws + o_pstat);
        w.tcnt = (uint32_t *)(ws + o_tcnt);
        w.toff = (uint32_t *)(ws + o_toff);
        w.ccnt = (uint32_t *)(ws + o_ccnt);
        w.pbits = (uint32_t *)(ws + o_pbits);
        w.hist = (uint32_t *)(ws + o_hist);
        w.selbits = (uint32_t *)(ws + o_sel);
        w.cand_key = (uint32_t *)(ws + o_ckey);
        w.cand_idx = (uint32_t *)(ws + o_cidx);
        w.histA = (uint32_t *)(ws + o_histA);
        w.shist = (uint32_t *)(ws + o_shist);
        w.fcnt = (uint32_t *)(ws + o_fcnt);
        w.S = (uint32_t *)(ws + o_S);
        w.P = (uint32_t *)(ws + o_P);
        w.V = (float *)(ws + o_V);
        w.sub_key = (uint32_t *)(ws + o_P);  // short list of the top-r select, before P exists
        w.sub_idx = (uint32_t *)(ws + o_V);
        w.sstat = (uint64_t *)(ws + o_sstat);
        w.sdig = (uint32_t *)(ws + o_sdig);
        w.tile_tensor = (uint32_t *)(ws + o_ttab);
        w.fit_part = (double *)(ws + o_fit);
        w.fit_runs = (uint32_t)(fit_blocks / FIT_CHUNKS);
        w.btab = (uint32_t *)(ws + o_btab);
        w.brow = (uint32_t *)(ws + o_brow);
        w.bslices = (uint32_t)bslices;
        w.keyA = (uint32_t *)(ws + o_keyA);
        w.keyB = (uint32_t *)(ws + o_keyB);
        w.valA = (uint32_t *)(ws + o_valA);
        w.valB = (uint32_t *)(ws + o_valB);
        w.sig = (uint32_t *)(ws + o_sig);
        w.vsorted = (float *)(ws + o_vs);
        w.bpos = (uint32_t *)(ws + o_keyA);  // borrows keyA .. vsorted
        w.bounds = (uint32_t *)(ws + o_bnd);
        w.segst = (SegState *)(ws + o_segst);
        w.segpart = (SegPart *)(ws + o_segpart);
        w.qlist = (uint32_t *)(ws + o_qlist);
        w.qbkt = (uint32_t *)(ws + o_qbkt);
        w.qtab = (uint32_t *)(ws + o_qtab);
        w.qrow = (uint32_t *)(ws + o_qrow);
        w.qcap = qb_entries;
        return w;
    }

    uint64_t pos_capacity() const { return (o_vs + 4 * slots - o_keyA) / 4; }
};

// Tiles per top-r histogram block (1024 threads): about 256 blocks over the
// whole gradient, at least 16 tiles each (each block writes a partial
// histogram, so fewer blocks mean less to reduce).
uint64_t hist_tiles_per_block(uint64_t all_tiles) { return std::max<uint64_t>(16, ceil_div(all_tiles, 256)); }

// The first-digit histogram of a top-r tensor of d elements: exact (one
// read of the tensor before the filter pass reads it again), or, in a call
// of at least SAMPLE_MIN_TOTAL elements (`sample`), for a tensor of at least
// SAMPLE_MIN_D elements with r <= d / 16, from a sample:
// one SAMPLE_SEG-element segment in srate, srate the largest power of 2 that
// leaves at least max(2^18, 4096 ceil(d / r)) sampled elements (some 4096
// expected above the threshold).  The sample's ranks slo and shi bound the
// bracket the filter pass keeps as candidates.  hist_blocks counts the
// blocks of the first histogram pass and redo_blocks those of the exact
// redo of the sampled tensors.  Sampling costs launches of its own (the
// pick, and the redo passes, which have nothing to do unless a bracket
// missed), and the filter pass then reads the gradient from HBM rather than
// partly from the last-level cache the histogram pass filled: on a 25.6 M
// element gradient it measured no faster than the exact histogram, on a
// 138 M element one 3.5% faster for the whole round trip.
constexpr uint64_t SAMPLE_MIN_TOTAL = 1ull << 26;
void plan_topr_hist(TInit &in, uint64_t d, uint64_t r, uint64_t ht, bool sample, uint64_t &hist_blocks,
                    uint64_t &redo_blocks) {
    in.hb0 = (uint32_t)hist_blocks;
    in.rb0 = (uint32_t)redo_blocks;
    const uint64_t full = ceil_div(in.ntiles, ht);
    uint64_t rate = 0;
    if (sample && d >= SAMPLE_MIN_D && r >= 1 && r <= d / 16) {
        const uint64_t target = std::max<uint64_t>(1ull << 18, 4096ull * ceil_div(d, r));
        for (uint64_t q = d / target; q > 1; q >>= 1) rate = rate ? rate << 1 : 2;
    }
    if (rate >= 2) {
        const uint64_t nseg = ceil_div(d, SAMPLE_SEG), half = rate / 2;
        const uint64_t ns = (nseg - half - 1) / rate + 1;  // sampled segments (nseg > half here)
        const uint64_t last = (ns - 1) * rate + half;
        const uint64_t nsamp = (ns - 1) * SAMPLE_SEG + std::min<uint64_t>(SAMPLE_SEG, d - last * SAMPLE_SEG);
        const double rho = (double)r * (double)nsamp / (double)d, delta = 8.0 * std::sqrt(rho) + 64.0;
        uint64_t lo = rho - delta >= 1.0 ? (uint64_t)std::floor(rho - delta) : 1ull;
        uint64_t hi = std::min<uint64_t>(nsamp, (uint64_t)std::ceil(rho + delta));
        if (lo > hi) lo = hi;
        in.srate = (uint32_t)rate;
        in.nsamp = (uint32_t)nsamp;
        in.slo = (uint32_t)lo;
        in.shi = (uint32_t)hi;
        in.hbn = (uint32_t)ceil_div(ns, SAMPLE_SEGS_PER_BLOCK);
        in.rbn = (uint32_t)full;
    } else {
        in.hbn = (uint32_t)full;
        in.rbn = 0;
    }
    hist_blocks += in.hbn;
    redo_blocks += in.rbn;
}

// Generic bound used by dr_workspace_bytes: one fit block per element at most.
Carve bound_carve(uint64_t d, uint64_t n_tensors) {
    Carve c;
    c.ntensors = n_tensors;
    c.ntiles = ceil_div(d, TILE) + n_tensors;
    c.slots = c.ntiles * TILE;
    c.hist_blocks = c.ntiles / 16 + 2 * n_tensors;
    const uint64_t runs = n_tensors * (uint64_t)DR_MAX_SEGMENTS;
    c.fit_blocks = (runs < d + n_tensors ? runs : d + n_tensors) * FIT_CHUNKS;
    // chord run starts: at most (runs + 1) per tensor
    c.bnd = std::min<uint64_t>(n_tensors * (uint64_t)(DR_MAX_SEGMENTS + 1), d + 2 * n_tensors);
    c.segslots = n_tensors <= SEG_GRID_TENSORS ? n_tensors : 0;
    // Bloom table: per tensor (slices x chunks) with at most MAX_CHUNKS
    // chunks and at most ceil(m / 2^14) slices, where m <= 47 n + 32 (k <= 32
    // gives -ln(fpr) / (ln 2)^2 < 47 bits per item); plus one filter of
    // BL_MAX_SLICES for a standalone insert whose filter is larger than its
    // item count
    c.bslices = 47 * c.slots / (1u << SLICE_LOG2_MIN) + 2 * n_tensors + BL_MAX_SLICES;
    c.btab = c.bslices * MAX_CHUNKS;
    // the bucketed query of one tensor of at most d elements: at most
    // QB_MAX_BINS bins of max(ceil(d / QB_CH), slices) chunks each (slices
    // of 2^QB_SL bits of a filter of at most 47 n + 32 bits), rounds for
    // k <= 32
    c.qb_entries = c.slots;
    c.qb_tab = (uint64_t)QB_MAX_BINS *
               std::max<uint64_t>(c.slots / QB_CH + 1,
                                  std::min<uint64_t>(QB_MAX_BINS, (47 * c.slots + 32) / (1ull << QB_SL) + 1));
    c.qb_rows = 33ull * QB_MAX_BINS;
    c.plan();
    return c;
}

struct Plan {
    std::vector<TInit> t;
    std::vector<uint64_t> bl_ncap;  // Bloom items reserved per tensor
    Carve carve;
    uint32_t bl_chunks = 0, bl_slices = 0, max_slices = 0, hash_per_round = 1, kmax = 0;
    uint64_t bl_items = 0;
    std::vector<uint64_t> bl_mcap;  // planned filter bits per tensor
    std::vector<QbTensor> qb;       // tensors given the bucketed query
    uint32_t qb_min_bits = 0, qb_k = 0;
    bool any_topr = false;
    bool direct = false;  // every filter small enough for the direct insert
    bool segment = false; // some tensor needs the segmentation pass (chord, or the heuristic count)
    bool dexp = false;    // some tensor fits double exponentials
    uint32_t dir_blocks = 0, dir_slices = 0;
    uint32_t seg_grid_req = 0;  // most runs requested of a tensor segmented over the grid
    bool seg_block_pass = false;  // some tensor needs the one-block segmentation pass
};

// Per-tensor Bloom insert layout for at most n_cap items and m_cap_bits:
// at most MAX_CHUNKS chunks of items, each a run of bitmap tiles (at least
// CHUNK_TILES) or of list entries (at least 1024).

void plan_bloom(TInit &in, uint64_t n_cap, uint64_t m_cap_bits, bool from_bitmap, Plan &p) {
    p.bl_ncap.push_back(n_cap);
    p.bl_mcap.push_back(m_cap_bits);
    if (from_bitmap) {
        const uint64_t chunk = std::max<uint64_t>(CHUNK_TILES, ceil_div(in.ntiles, MAX_CHUNKS));
        in.bl_chunk = (uint32_t)chunk;
        in.bl_nchunks = (uint32_t)ceil_div(in.ntiles, chunk);
    } else {
        const uint64_t chunk = std::max<uint64_t>(1024, ceil_div(n_cap, MAX_CHUNKS));
        in.bl_chunk = (uint32_t)chunk;
        in.bl_nchunks = (uint32_t)(n_cap ? ceil_div(n_cap, chunk) : 0);
    }
    // About 256 slices (of 2^14 to 2^20 bits): enough fill blocks, and runs
    // of about 64 records per slice in each of the scatter's groups
    uint32_t sl2 = SLICE_LOG2_MIN;
    while (sl2 < SLICE_LOG2_MAX && ceil_div(m_cap_bits, 1ull << sl2) > 256) ++sl2;
    in.slice_log2 = sl2;
    in.bl_nslices = (uint32_t)ceil_div(m_cap_bits, 1ull << in.slice_log2);
    in.bl_chunk0 = p.bl_chunks;
    in.bl_slice0 = p.bl_slices;
    in.bl_tab0 = p.carve.btab;
    p.bl_chunks += in.bl_nchunks;
    p.bl_slices += in.bl_nslices;
    p.carve.bslices += in.bl_nslices;
    p.carve.btab += (uint64_t)in.bl_nchunks * in.bl_nslices;
    p.bl_items += n_cap;
    if (in.bl_nslices > p.max_slices) p.max_slices = in.bl_nslices;
}

// After the carve: how many hash functions one insert round can bucket (the
// position buffer holds n_cap positions per hash per tensor), and each
// tensor's place in that buffer.
void plan_bloom_rounds(Plan &p, uint32_t k) {
    p.kmax = k;
    const uint64_t cap = p.carve.pos_capacity();
    uint64_t h = p.bl_items ? cap / p.bl_items : k;
    if (h < 1) h = 1;
    if (h > k) h = k;
    // a tensor's records are addressed with 32-bit offsets
    uint64_t ncap_max = 0;
    for (uint64_t n : p.bl_ncap) ncap_max = std::max(ncap_max, n);
    while (h > 1 && ncap_max * h >= (1ull << 31)) --h;
    p.hash_per_round = (uint32_t)h;
    uint64_t at = 0;
    for (size_t i = 0; i < p.t.size(); ++i) {
        p.t[i].bl_pos0 = at;
        p.t[i].bl_poscap = p.bl_ncap[i] * h;
        at += p.bl_ncap[i] * h;
    }
}

// The direct insert, when every planned filter has at most DIR_MAX_BITS bits
// and the partial slices fit in the position buffer: G item chunks per
// slice, about 1024 blocks in all (at most 64 chunks).
void plan_bloom_direct(Plan &p, bool from_bitmap) {
    p.direct = false;
    uint64_t nsl_all = 0;
    for (uint64_t m : p.bl_mcap) {
        if (m > DIR_MAX_BITS) return;
        nsl_all += ceil_div(m / 32, DIR_SLICE_WORDS);
    }
    if (nsl_all == 0) return;
    uint64_t G = std::max<uint64_t>(1, std::min<uint64_t>(64, 1024 / nsl_all));
    auto words = [&](uint64_t g) {
        uint64_t tot = 0;
        for (uint64_t m : p.bl_mcap) tot += ceil_div(m / 32, DIR_SLICE_WORDS) * g * std::min<uint64_t>(DIR_SLICE_WORDS, m / 32);
        return tot;
    };
    const uint64_t cap_words = p.carve.pos_capacity();  // the position buffer, in 32-bit words
    while (G > 1 && words(G) > cap_words) G /= 2;
    if (words(G) > cap_words) return;
    uint64_t blk = 0, sl = 0, pb = 0;
    for (size_t i = 0; i < p.t.size(); ++i) {
        TInit &in = p.t[i];
        const uint64_t mw = p.bl_mcap[i] / 32;
        in.dir_nsl = (uint32_t)ceil_div(mw, DIR_SLICE_WORDS);
        in.dir_g = (uint32_t)G;
        in.dir_sw = (uint32_t)std::min<uint64_t>(DIR_SLICE_WORDS, mw);
        in.dir_blk0 = (uint32_t)blk;
        in.dir_sl0 = (uint32_t)sl;
        in.dir_pb = pb;
        in.dir_per = from_bitmap ? (uint32_t)ceil_div(in.ntiles, G)
                                 : (uint32_t)std::max<uint64_t>(1, ceil_div(p.bl_ncap[i], G));
        blk += (uint64_t)in.dir_nsl * G;
        sl += in.dir_nsl;
        pb += (uint64_t)in.dir_nsl * G * in.dir_sw;
    }
    p.direct = true;
    p.dir_blocks = (uint32_t)blk;
    p.dir_slices = (uint32_t)sl;
}

// The receiver's bucketed query, for tensors whose filter may be larger
// than an XCD's L2: those of at most QB_MAX_D elements whose largest filter (m for their
// n_cap items) has at least qb_min_bits() bits, the first QB_MAX_TENSORS of
// them.  The kernels check the actual filter against the same threshold and
// leave smaller ones to the probe pass.  The environment variable
// DR_QUERY_BUCKET_MIN_BITS replaces the threshold (the tests lower it to
// run the path on small tensors).
constexpr uint64_t QB_MIN_BITS_DEFAULT = 1ull << 25;  // 4 MiB, an XCD's L2
constexpr size_t QB_MAX_TENSORS = 16;

uint64_t qb_min_bits() {
    const char *e = getenv("DR_QUERY_BUCKET_MIN_BITS");
    if (!e || !*e) return QB_MIN_BITS_DEFAULT;
    char *end = nullptr;
    const unsigned long long v = strtoull(e, &end, 10);
    return (end && *end == 0) ? std::min<uint64_t>(v, 0xffffffffull) : QB_MIN_BITS_DEFAULT;
}

void plan_query_bucketed(Plan &p, bool allow) {
    p.qb.clear();
    p.carve.qb_entries = p.carve.qb_tab = p.carve.qb_rows = 0;
    if (!allow) return;
    const uint64_t mb = qb_min_bits();
    uint64_t ent = 0, tab = 0;
    uint32_t k = 0;
    for (size_t t = 0; t < p.t.size() && p.qb.size() < QB_MAX_TENSORS; ++t) {
        const TInit &in = p.t[t];
        const uint64_t m = p.bl_mcap[t];
        if (in.k < 1 || m < mb || in.d < 1 || in.d > QB_MAX_D) continue;
        QbTensor q;
        q.t = (uint32_t)t;
        q.nsl_cap = (uint32_t)ceil_div(m, 1ull << QB_SL);
        q.nch_cap = (uint32_t)ceil_div(in.d, QB_CH);
        q.nreg = (uint32_t)ceil_div(in.d, 1ull << QB_RL);
        if (q.nsl_cap > QB_MAX_BINS || q.nreg > QB_MAX_BINS) continue;
        // round 0's chunks are QB_CH indices, later rounds' the slices
        q.ncol = std::max(q.nch_cap, q.nsl_cap);
        p.qb.push_back(q);
        ent = std::max<uint64_t>(ent, in.d);
        tab = std::max<uint64_t>(tab, (uint64_t)std::max(q.nsl_cap, q.nreg) * q.ncol);
        k = in.k;
    }
    if (p.qb.empty()) return;
    p.qb_min_bits = (uint32_t)mb;
    p.qb_k = k;
    p.carve.qb_entries = align_up(ent, 64);
    p.carve.qb_tab = tab;
    p.carve.qb_rows = (uint64_t)(k + 1) * QB_MAX_BINS;
}

dr_status check_cfg(const dr_config *cfg) {
    if (!cfg) return fail(DR_EINVAL, "cfg is null");
    if (cfg->n_tensors < 1 || cfg->n_tensors > DR_MAX_TENSORS) return fail(DR_EINVAL, "n_tensors out of range");
    if (!cfg->offsets_h) return fail(DR_EINVAL, "offsets_h is null");
    if (cfg->offsets_h[0] != 0) return fail(DR_EINVAL, "offsets_h[0] must be 0");
    for (uint64_t t = 0; t < cfg->n_tensors; ++t) {
        if (cfg->offsets_h[t + 1] < cfg->offsets_h[t]) return fail(DR_EINVAL, "offsets_h must be nondecreasing");
        if (cfg->offsets_h[t + 1] - cfg->offsets_h[t] >= (1ull << 32))
            return fail(DR_EINVAL, "tensor %llu has 2^32 or more elements", (unsigned long long)t);
    }
    if (cfg->ratio_num != DR_R_NONZERO) {
        if (cfg->ratio_den == 0 || cfg->ratio_den >= (1ull << 32) || cfg->ratio_num > cfg->ratio_den)
            return fail(DR_EINVAL, "ratio must satisfy 0 <= num <= den < 2^32");
    }
    if (!(cfg->fpr > 0.0 && cfg->fpr < 1.0)) return fail(DR_EINVAL, "fpr must be in (0, 1)");
    if (cfg->degree > DR_MAX_DEGREE) return fail(DR_EINVAL, "degree > %d", DR_MAX_DEGREE);
    if (cfg->n_seg > DR_MAX_SEGMENTS) return fail(DR_EINVAL, "n_seg out of range");
    if (cfg->segmentation > DR_SEG_CHORD) return fail(DR_EINVAL, "unknown segmentation %u", cfg->segmentation);
    if (cfg->fit_model > DR_FIT_DEXP) return fail(DR_EINVAL, "unknown value model %u", cfg->fit_model);
    if (cfg->policy > DR_POLICY_RIGHTMOST) return fail(DR_EINVAL, "unknown index policy %u", cfg->policy);
    if (cfg->value_source > DR_VALUES_SPARSE) return fail(DR_EINVAL, "unknown value source %u", cfg->value_source);
    if (cfg->filter_layout > DR_FILTER_PARTITIONED)
        return fail(DR_EINVAL, "unknown filter layout %u", cfg->filter_layout);
    return DR_OK;
}

// Most runs a tensor of d elements can be fitted with: the requested count
// (or, for the heuristic, the most segments), never more than one per D+1
// values.
uint64_t runs_cap(uint64_t d, uint32_t degree, uint32_t nseg) {
    const uint64_t req = nseg ? nseg : (uint64_t)DR_MAX_SEGMENTS;
    return std::min<uint64_t>(req, std::max<uint64_t>(1, d / (degree + 1)));
}

uint64_t record_capacity(uint64_t d, uint64_t n_cap, double fpr, uint32_t degree, uint64_t runs, bool knots) {
    uint64_t m = 0;
    uint32_t k = 0;
    bloom_params_host(n_cap, fpr, &m, &k);
    const uint64_t sig_words = ceil_div(d * sigma_bits_host(d ? d : 1), 32);
    return HDR_BYTES + m / 8 + 4ull * runs * (degree + 1) + (knots ? 4ull * runs : 0) + 4 * sig_words;
}

// The per-tensor plan of a round trip (sender and receiver use the same one).
dr_status plan_config(const dr_config *cfg, Plan &p, std::vector<uint64_t> &rec_off, bool allow_qb = true) {
    dr_status st = check_cfg(cfg);
    if (st != DR_OK) return st;
    const uint64_t T = cfg->n_tensors;
    const bool nz = cfg->ratio_num == DR_R_NONZERO;
    const double ln2 = log(2.0);
    const double mC = -log(cfg->fpr) / (ln2 * ln2);
    uint64_t m_any = 0;
    uint32_t k = 0;
    if (!bloom_params_host(1, cfg->fpr, &m_any, &k)) return fail(DR_EINVAL, "fpr gives more than 32 hashes");
    p.t.resize(T);
    rec_off.assign(T + 1, 0);
    uint64_t tiles = 0, hist_blocks = 0, redo_blocks = 0, fit_blocks = 0, bnd = 0;
    p.carve = Carve();
    uint64_t all_tiles = 0;
    for (uint64_t t = 0; t < T; ++t) {
        const uint64_t d = cfg->offsets_h[t + 1] - cfg->offsets_h[t];
        all_tiles += d ? ceil_div(d, TILE) : 1;
    }
    const uint64_t ht = hist_tiles_per_block(all_tiles);
    for (uint64_t t = 0; t < T; ++t) {
        TInit &in = p.t[t];
        memset(&in, 0, sizeof in);
        const uint64_t d = cfg->offsets_h[t + 1] - cfg->offsets_h[t];
        const uint64_t r = nz ? 0 : ceil_div(d * cfg->ratio_num, cfg->ratio_den);
        const uint64_t n_cap = nz ? d : r;
        p.carve.vals_est += nz ? d : std::min<uint64_t>(d, 2 * r + TILE);
        uint64_t m_cap = 0;
        uint32_t kk = 0;
        if (!bloom_params_host(n_cap, cfg->fpr, &m_cap, &kk))
            return fail(DR_ENOTSUP, "tensor %llu: filter of %llu items needs 2^32 bits or more",
                        (unsigned long long)t, (unsigned long long)n_cap);
        if (ceil_div(m_cap, 1ull << SLICE_LOG2_MAX) > BL_MAX_SLICES)
            return fail(DR_ENOTSUP, "tensor %llu: filter larger than 2^30 bits", (unsigned long long)t);
        in.off = cfg->offsets_h[t];
        in.d = (uint32_t)d;
        in.r = nz ? R_NONZERO : (uint32_t)r;
        in.ntiles = (uint32_t)(d ? ceil_div(d, TILE) : 1);
        in.tile0 = (uint32_t)tiles;
        in.slot = tiles * TILE;
        tiles += in.ntiles;
        in.k = kk;
        // the double exponential has four parameters per run, the row of a
        // cubic
        const uint32_t degree = cfg->fit_model == DR_FIT_DEXP ? 3u : cfg->degree;
        in.degree = degree;
        in.fit_model = cfg->fit_model;
        in.nseg = cfg->n_seg;
        in.policy = cfg->policy;
        in.seed = cfg->seed;
        in.seg_mode = cfg->segmentation;
        in.value_src = cfg->value_source;
        in.layout = cfg->filter_layout;
        in.mC = mC;
        // top-r: |S| = r is known, so the filter size is too
        in.m_words_in = nz ? 0u : (uint32_t)(m_cap / 32);
        const uint64_t runs = runs_cap(d, degree, cfg->n_seg);
        in.fit_blk0 = (uint32_t)fit_blocks;
        fit_blocks += runs * FIT_CHUNKS;
        in.seg_slot = NO_SEG_SLOT;
        if (cfg->segmentation == DR_SEG_CHORD) {
            in.bnd0 = (uint32_t)bnd;
            bnd += runs + 1;
            // a requested run count of at most SEG_GRID_RUNS, for a few
            // tensors: the splits are evaluated over the whole grid
            if (T <= SEG_GRID_TENSORS && cfg->n_seg >= 1 && cfg->n_seg <= SEG_GRID_RUNS) {
                in.seg_slot = (uint32_t)p.carve.segslots++;
                p.seg_grid_req = std::max(p.seg_grid_req, cfg->n_seg);
            }
        }
        const bool seg = cfg->segmentation == DR_SEG_CHORD || cfg->n_seg == 0;
        p.segment |= seg;
        p.seg_block_pass |= seg && in.seg_slot == NO_SEG_SLOT;
        p.dexp |= cfg->fit_model == DR_FIT_DEXP;
        if (!nz) {
            plan_topr_hist(in, d, r, ht, cfg->offsets_h[T] >= SAMPLE_MIN_TOTAL, hist_blocks, redo_blocks);
        } else {
            in.hb0 = (uint32_t)hist_blocks;
            in.hbn = 0;
            in.rb0 = (uint32_t)redo_blocks;
            in.rbn = 0;
        }
        plan_bloom(in, n_cap, m_cap, true, p);
        rec_off[t + 1] = rec_off[t] + align_up(record_capacity(d, n_cap, cfg->fpr, degree, runs,
                                                               cfg->segmentation == DR_SEG_CHORD),
                                               256);
    }
    p.any_topr = !nz;
    p.carve.ntensors = T;
    p.carve.ntiles = tiles;
    p.carve.slots = tiles * TILE;
    p.carve.hist_blocks = hist_blocks;
    p.carve.redo_blocks = redo_blocks;
    p.carve.fit_blocks = fit_blocks;
    p.carve.bnd = bnd;
    plan_query_bucketed(p, allow_qb);
    p.carve.plan();
    plan_bloom_rounds(p, k);
    plan_bloom_direct(p, true);
    return DR_OK;
}

// Descriptors and the zeroed regions; a query-only work has no histogram or
// sort regions, and `extra` (words) is a caller's buffer to clear as well.
hipError_t run_init(const Work &w, const std::vector<TInit> &t, hipStream_t s, bool query_only = false,
                    ZeroRange extra = {nullptr, 0}) {
    ZeroArgs z;
    memset(&z, 0, sizeof z);
    z.z[0] = {w.glob, sizeof(Glob) / 4};
    z.z[1] = {w.pstat, 2ull * PSTAT_MAX};
    z.n = 2;
    if (!query_only) {
        z.z[z.n++] = {w.sdig, 4ull * SORT_BINS * w.ntensors};
        // hist, histA, shist and fcnt (carved one after the other)
        z.z[z.n++] = {w.hist, (uint64_t)(((uint8_t *)w.fcnt - (uint8_t *)w.hist) / 4) +
                                  (uint64_t)FCNT_COPIES * FCNT_W * w.ntensors};
    }
    if (extra.p && extra.words) z.z[z.n++] = extra;
    for (size_t f = 0; f < t.size(); f += INIT_CHUNK) {
        InitArgs a;
        memset(&a, 0, sizeof a);
        a.first = (uint32_t)f;
        a.count = (uint32_t)std::min<size_t>(INIT_CHUNK, t.size() - f);
        for (uint32_t i = 0; i < a.count; ++i) a.t[i] = t[f + i];
        hipError_t e = launch_init(w, a, z, s);
        if (e != hipSuccess) return e;
        z.n = 0;  // cleared once
    }
    return hipSuccess;
}

bool ws_ok(void *ws, size_t ws_bytes, size_t need) {
    return ws && ws_bytes >= need && ((uintptr_t)ws & 255u) == 0;
}

// The sender in two halves: select, insert, query and the values' layout
// (front), then sort, segmentation, fit and reorder map (back).
struct Encode {
    Plan p;
    std::vector<uint64_t> rec_off;
    Work w;
};

dr_status encode_prepare(const float *g, const dr_config *cfg, uint8_t *payload, size_t payload_bytes,
                         uint64_t *counts_out, void *ws, size_t ws_bytes, Encode &e, bool allow_qb = true) {
    dr_status st = plan_config(cfg, e.p, e.rec_off, allow_qb);
    if (st != DR_OK) return st;
    if (!g && cfg->offsets_h[cfg->n_tensors] > 0) return fail(DR_EINVAL, "g is null");
    if (!payload || payload_bytes < e.rec_off.back()) return fail(DR_EINVAL, "payload buffer too small");
    if (!ws_ok(ws, ws_bytes, e.p.carve.bytes))
        return fail(DR_EINVAL, "workspace too small or not 256-byte aligned (need %zu)", e.p.carve.bytes);
    for (size_t t = 0; t < e.p.t.size(); ++t) {
        e.p.t[t].rec_off = e.rec_off[t];
        e.p.t[t].rec_cap = e.rec_off[t + 1] - e.rec_off[t];
        e.p.t[t].rec = payload + e.rec_off[t];
        e.p.t[t].bits = (uint32_t *)(payload + e.rec_off[t] + HDR_BYTES);
        e.p.t[t].coef = nullptr;
        e.p.t[t].sigma = nullptr;
    }
    e.w = e.p.carve.view((uint8_t *)ws);
    e.w.counts_out = counts_out;
    return DR_OK;
}

// after_probe, if given, is recorded once the records' headers and filters
// are written (the receiver's probe pass needs nothing more)
dr_status encode_front(Encode &e, const float *g, uint64_t *counts_out, hipStream_t s,
                       hipEvent_t after_probe = nullptr) {
    const Plan &p = e.p;
    const Work &w = e.w;
    // counts_out starts as zeros (its flags words are OR-ed)
    DR_HIP(run_init(w, p.t, s, false, {counts_out, counts_out ? 8ull * w.ntensors : 0}));
    if (p.any_topr)
        DR_HIP(launch_topr(w, g, (uint32_t)p.carve.hist_blocks, (uint32_t)p.carve.redo_blocks, true, s));
    else
        DR_HIP(launch_nonzero(w, g, persist_grid(8), s));
    if (p.direct)
        DR_HIP(launch_bloom_direct(w, true, p.dir_blocks, p.dir_slices, s));
    else
        DR_HIP(launch_bloom_insert(w, true, p.bl_chunks, p.bl_slices, p.max_slices, p.hash_per_round, p.kmax, s));
    DR_HIP(launch_query_encode(w, g, persist_grid(4), counts_out, s, after_probe));
    return DR_OK;
}

dr_status encode_back(Encode &e, hipStream_t s) {
    const Plan &p = e.p;
    const Work &w = e.w;
    DR_HIP(launch_sort(w, (uint32_t)p.carve.ntiles, s));
    if (p.segment) DR_HIP(launch_segment(w, p.seg_grid_req, p.seg_block_pass, s));
    DR_HIP(launch_fit(w, (uint32_t)p.carve.fit_blocks, p.carve.vals_est, p.dexp, s));
    return DR_OK;
}

dr_status encode_impl(const float *g, const dr_config *cfg, uint8_t *payload, size_t payload_bytes,
                      uint64_t *counts_out, void *ws, size_t ws_bytes, hipStream_t s) {
    Encode e;
    dr_status st = encode_prepare(g, cfg, payload, payload_bytes, counts_out, ws, ws_bytes, e);
    if (st != DR_OK) return st;
    trace_call(s);
    st = encode_front(e, g, counts_out, s);
    if (st != DR_OK) return st;
    return encode_back(e, s);
}

// The receiver: its own descriptors over the payload's records, in the
// workspace at byte offset ws_off (a query-only carve there if query_only).
struct Decode {
    Plan p;
    std::vector<uint64_t> rec_off;
    Work w;
    float *dense_out;
    uint32_t *idx_out;
    float *val_out;
    uint64_t *counts_out;
    bool general;  // chord runs or the double exponential: the emit pass that handles them
};

dr_status decode_prepare(const uint8_t *payload, const dr_config *cfg, float *dense_out, uint32_t *idx_out,
                         float *val_out, uint64_t *counts_out, void *ws, size_t ws_bytes, Decode &dd,
                         bool allow_qb = true) {
    dr_status st = plan_config(cfg, dd.p, dd.rec_off, allow_qb);
    if (st != DR_OK) return st;
    if (!payload) return fail(DR_EINVAL, "payload is null");
    if (!dense_out && cfg->offsets_h[cfg->n_tensors] > 0) return fail(DR_EINVAL, "dense_out is null");
    if (!ws_ok(ws, ws_bytes, dd.p.carve.bytes))
        return fail(DR_EINVAL, "workspace too small or not 256-byte aligned (need %zu)", dd.p.carve.bytes);
    for (size_t t = 0; t < dd.p.t.size(); ++t) {
        dd.p.t[t].rec_off = dd.rec_off[t];
        dd.p.t[t].rec_cap = dd.rec_off[t + 1] - dd.rec_off[t];
        dd.p.t[t].rec = const_cast<uint8_t *>(payload) + dd.rec_off[t];
        dd.p.t[t].bits = nullptr;
    }
    dd.w = dd.p.carve.view((uint8_t *)ws);
    dd.dense_out = dense_out;
    dd.idx_out = idx_out;
    dd.val_out = val_out;
    dd.counts_out = counts_out;
    dd.general = cfg->segmentation != DR_SEG_EQUAL || cfg->fit_model != DR_FIT_POLY;
    return DR_OK;
}

// Bytes of a receiver's query-only work for the plan's layout (with or
// without regions of its own for the bucketed query).
Carve query_carve(const Plan &p, bool with_qb = true) {
    Carve c;
    c.query_only = true;
    c.ntensors = p.carve.ntensors;
    c.ntiles = p.carve.ntiles;
    c.slots = p.carve.slots;
    if (with_qb) {
        c.qb_entries = p.carve.qb_entries;
        c.qb_tab = p.carve.qb_tab;
        c.qb_rows = p.carve.qb_rows;
    }
    c.plan();
    return c;
}

dr_status decode_init(Decode &dd, bool query_only, hipStream_t s) {
    DR_HIP(run_init(dd.w, dd.p.t, s, query_only));
    return DR_OK;
}

dr_status decode_probe(Decode &dd, uint32_t max_probe_blocks, hipStream_t s) {
    for (const QbTensor &q : dd.p.qb) DR_HIP(launch_query_bucketed(dd.w, q, dd.p.qb_k, dd.p.qb_min_bits, s));
    DR_HIP(launch_probe_decode(dd.w, dd.dense_out, dd.counts_out, max_probe_blocks, s));
    return DR_OK;
}

dr_status decode_front(Decode &dd, uint32_t max_probe_blocks, bool query_only, hipStream_t s) {
    dr_status st = decode_init(dd, query_only, s);
    if (st != DR_OK) return st;
    return decode_probe(dd, max_probe_blocks, s);
}

dr_status decode_back(Decode &dd, hipStream_t s) {
    DR_HIP(launch_emit_decode(dd.w, dd.dense_out, dd.idx_out, dd.val_out, dd.counts_out, dd.general, s));
    return DR_OK;
}

dr_status decode_impl(const uint8_t *payload, const dr_config *cfg, float *dense_out, uint32_t *idx_out,
                      float *val_out, uint64_t *counts_out, void *ws, size_t ws_bytes, hipStream_t s) {
    Decode dd;
    dr_status st = decode_prepare(payload, cfg, dense_out, idx_out, val_out, counts_out, ws, ws_bytes, dd);
    if (st != DR_OK) return st;
    trace_call(s);
    st = decode_front(dd, 0xffffffffu, false, s);
    if (st != DR_OK) return st;
    return decode_back(dd, s);
}

// A second stream per device for the round trip's overlap, with the two
// events that fork and join it; created on first use, kept until exit.
struct SideStream {
    hipStream_t s = nullptr;
    hipEvent_t start = nullptr, fork = nullptr, join = nullptr;
};
std::mutex g_side_mu;  // guards creation and each fork/join sequence
SideStream g_side[64];

// the current device's side stream; call with g_side_mu held
bool side_stream(SideStream **out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return false;
    SideStream &ss = g_side[dev];
    if (!ss.s) {
        if (hipStreamCreateWithFlags(&ss.s, hipStreamNonBlocking) != hipSuccess) return false;
        if (hipEventCreateWithFlags(&ss.start, hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&ss.fork, hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&ss.join, hipEventDisableTiming) != hipSuccess) {
            ss.s = nullptr;
            return false;
        }
    }
    *out = &ss;
    return true;
}

// dr_roundtrip: the receiver's probe pass needs only the payload's header
// and filter, which the sender's probe pass has written (it sets each
// tensor's run shape and header where it learns |P|), so it runs on a
// second stream while the sender emits, sorts and fits its values (the
// probe is bound by L2 request throughput and loses little when some CUs
// are left to the sender).  The receiver then
// uses its own query-only work after the sender's in the workspace; without
// room for it, or with segmentation passes that rewrite the header after
// the sort, the two sides run one after the other.
dr_status roundtrip_impl(const float *g, const dr_config *cfg, uint8_t *payload, size_t payload_bytes,
                         float *dense_out, uint32_t *idx_out, float *val_out, uint64_t *counts_out, void *ws,
                         size_t ws_bytes, hipStream_t s) {
    Encode e;
    dr_status st = encode_prepare(g, cfg, payload, payload_bytes, counts_out, ws, ws_bytes, e);
    if (st != DR_OK) return st;
    Decode dd;
    st = decode_prepare(payload, cfg, dense_out, idx_out, val_out, counts_out, ws, ws_bytes, dd);
    if (st != DR_OK) return st;
    // the receiver's bucketed query borrows the sender's lists and tables,
    // which the sender does not use
    const Carve qc = query_carve(dd.p, false);
    const size_t qoff = align_up(e.p.carve.bytes, 256);
    // one fork/join sequence at a time per process, so that the two events
    // are not re-recorded by another thread between a record and its wait
    std::unique_lock<std::mutex> lock(g_side_mu);
    SideStream *ss = nullptr;
    const bool overlap = !e.p.segment && qoff + qc.bytes <= ws_bytes && side_stream(&ss);
    if (!overlap) lock.unlock();
    trace_call(s);
    if (overlap) {
        // the receiver's set-up needs nothing from the sender: the side
        // stream runs it (once the caller's earlier work on s is done) while
        // the sender selects
        dd.w = qc.view((uint8_t *)ws + qoff);
        dd.w.qlist = e.w.qlist;
        dd.w.qbkt = e.w.qbkt;
        dd.w.qtab = e.w.qtab;
        dd.w.qrow = e.w.qrow;
        dd.w.qcap = e.w.qcap;
        DR_HIP(hipEventRecord(ss->start, s));
        DR_HIP(hipStreamWaitEvent(ss->s, ss->start, 0));
        trace_call(ss->s);  // per-kernel timing: the side stream's kernels count from here
        st = decode_init(dd, true, ss->s);
        if (st != DR_OK) return st;
    }
    // the fork: once the sender's probe pass has written the records'
    // headers and filters, the receiver's probe pass can run beside the
    // sender's emit pass and value stage
    st = encode_front(e, g, counts_out, s, overlap ? ss->fork : nullptr);
    if (st != DR_OK) return st;
    if (!overlap) {
        st = encode_back(e, s);
        if (st != DR_OK) return st;
        st = decode_front(dd, 0xffffffffu, false, s);
        if (st != DR_OK) return st;
        return decode_back(dd, s);
    }
    DR_HIP(hipStreamWaitEvent(ss->s, ss->fork, 0));
    trace_call(ss->s);  // per-kernel timing: the wait for the fork is idle time
    // CUs left to the sender: a multiple of the 32 shader engines (8 XCDs of
    // 4).  Workgroups are dealt to the engines in turn, so a kernel launched
    // beside the probe pass needs a free CU in every engine: with fewer than
    // 32 left, its workgroups dealt to a full engine wait for the probe pass
    // to end, and the sender's value stage runs after it instead of beside
    // it (seen with 8, 16 and 24 left).  A top-r gradient codes about r
    // values, a small sort beside a long probe pass: one CU per engine.  An
    // inherently sparse one codes every nonzero (19 M values for the NCF
    // workload), and its sort needs more of the chip than the probe pass
    // loses: four per engine (measured on ncf_32m: 7.96 ms with 32 left,
    // 7.72 with 64, 7.66 with 96, 7.56 with 128; resnet50_25m gets slower
    // with each step above 32).
    const uint32_t reserve = e.p.any_topr ? 32u : 128u;
    st = decode_probe(dd, (uint32_t)std::max(1, dr::device_cus() - (int)reserve), ss->s);
    if (st != DR_OK) return st;
    DR_HIP(hipEventRecord(ss->join, ss->s));
    st = encode_back(e, s);
    if (st != DR_OK) return st;
    DR_HIP(hipStreamWaitEvent(s, ss->join, 0));
    trace_call(s);  // per-kernel timing: the wait for the join is idle time
    return decode_back(dd, s);
}

// ---------------------------------------------------------------------------
// The round trip for callers that cannot allocate: its scratch is a static
// device array of the library, one per GPU, held until the process ends.
// ---------------------------------------------------------------------------
static __device__ __align__(256) uint8_t scratch[DR_STATIC_SCRATCH_BYTES];

std::mutex g_scratch_mu;       // guards the first lookup on each device
void *g_scratch_ptr[64] = {};  // scratch's device address, per device

// The device address of `scratch` on the current device, looked up once per
// device (each GPU holds its own copy of the array).  In host code the
// array's name is a host-side stand-in, never a device address.
dr_status static_scratch(void **out) {
    int dev = 0;
    DR_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= 64) return fail(DR_ENOTSUP, "device %d: at most 64 devices", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "hipGetSymbolAddress");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return DR_OK;
}

// dr_roundtrip's sender then receiver, one after the other on `s`, in the
// static scratch: no second stream, no event, no allocation.
dr_status roundtrip_static_impl(const float *g, const dr_config *cfg, uint8_t *payload, size_t payload_bytes,
                                float *dense_out, uint32_t *idx_out, float *val_out, uint64_t *counts_out,
                                hipStream_t s) {
    {
        Plan p;
        std::vector<uint64_t> rec_off;
        dr_status st = plan_config(cfg, p, rec_off, false);
        if (st != DR_OK) return st;
        if (p.carve.bytes > DR_STATIC_SCRATCH_BYTES)
            return fail(DR_ECAPACITY, "this gradient needs %zu bytes of scratch; the static scratch holds %zu "
                        "(use dr_roundtrip with a workspace)", p.carve.bytes, (size_t)DR_STATIC_SCRATCH_BYTES);
    }
    void *ws = nullptr;
    dr_status st = static_scratch(&ws);
    if (st != DR_OK) return st;
    Encode e;
    // without the bucketed query, whose lists would take scratch the array
    // does not have
    st = encode_prepare(g, cfg, payload, payload_bytes, counts_out, ws, DR_STATIC_SCRATCH_BYTES, e, false);
    if (st != DR_OK) return st;
    Decode dd;
    st = decode_prepare(payload, cfg, dense_out, idx_out, val_out, counts_out, ws, DR_STATIC_SCRATCH_BYTES, dd,
                        false);
    if (st != DR_OK) return st;
    trace_call(s);
    st = encode_front(e, g, counts_out, s);
    if (st != DR_OK) return st;
    st = encode_back(e, s);
    if (st != DR_OK) return st;
    st = decode_front(dd, 0xffffffffu, false, s);
    if (st != DR_OK) return st;
    return decode_back(dd, s);
}

dr_status decode_sum_impl(const uint8_t *const *payloads, uint32_t npay, const dr_config *cfg, float scale,
                          float *dense_out, uint64_t *counts_out, void *ws, size_t ws_bytes, hipStream_t s) {
    Plan p;
    std::vector<uint64_t> rec_off;
    dr_status st = plan_config(cfg, p, rec_off);
    if (st != DR_OK) return st;
    if (npay < 1 || npay > DR_MAX_SUM_PAYLOADS) return fail(DR_EINVAL, "n_payloads must be in [1, %d]", DR_MAX_SUM_PAYLOADS);
    if (!payloads) return fail(DR_EINVAL, "payloads_h is null");
    for (uint32_t q = 0; q < npay; ++q)
        if (!payloads[q]) return fail(DR_EINVAL, "payloads_h[%u] is null", q);
    const uint64_t T = cfg->n_tensors, d = cfg->offsets_h[T];
    if (!dense_out && d > 0) return fail(DR_EINVAL, "dense_out is null");
    if (!std::isfinite(scale)) return fail(DR_EINVAL, "scale is not finite");
    const uint64_t ntiles1 = p.carve.ntiles;
    if (ntiles1 * npay >= (1ull << 32) || T * npay > (1ull << 32)) return fail(DR_ENOTSUP, "too many tiles");
    // tensor t of payload q is descriptor q * T + t, its tiles follow payload q - 1's
    std::vector<TInit> vt;
    vt.reserve(T * npay);
    for (uint32_t q = 0; q < npay; ++q)
        for (uint64_t t = 0; t < T; ++t) {
            TInit in = p.t[t];
            in.tile0 = (uint32_t)(q * ntiles1 + in.tile0);
            in.slot = q * ntiles1 * TILE + in.slot;
            in.rec_off = rec_off[t];
            in.rec_cap = rec_off[t + 1] - rec_off[t];
            in.rec = const_cast<uint8_t *>(payloads[q]) + rec_off[t];
            in.bits = nullptr;
            vt.push_back(in);
        }
    Carve c;
    c.query_only = true;
    c.ntensors = T * npay;
    c.ntiles = ntiles1 * npay;
    c.slots = c.ntiles * TILE;
    c.plan();
    if (!ws_ok(ws, ws_bytes, c.bytes))
        return fail(DR_EINVAL, "workspace too small or not 256-byte aligned (need %zu)", c.bytes);
    const Work w = c.view((uint8_t *)ws);
    trace_call(s);
    DR_HIP(run_init(w, vt, s, true, {counts_out, counts_out ? 8 * T * npay : 0}));
    DR_HIP(launch_query_decode_sum(w, npay, (uint32_t)T, (uint32_t)ntiles1, scale, dense_out, counts_out, s));
    return DR_OK;
}

// A single-tensor plan for the standalone calls.
Plan single_plan(uint64_t d) {
    Plan p;
    p.t.resize(1);
    TInit &in = p.t[0];
    memset(&in, 0, sizeof in);
    in.seg_slot = NO_SEG_SLOT;
    in.d = (uint32_t)d;
    in.ntiles = (uint32_t)(d ? ceil_div(d, TILE) : 1);
    in.tile0 = 0;
    in.slot = 0;
    p.carve.ntensors = 1;
    p.carve.ntiles = in.ntiles;
    p.carve.slots = (uint64_t)in.ntiles * TILE;
    p.carve.vals_est = d;
    return p;
}

// ---------------------------------------------------------------------------
// Host-side range check: the kernels' index arithmetic (ranges.hpp) replayed
// over every chunk, slice, block and sort tile a configuration plans.
// ---------------------------------------------------------------------------
struct RangeCheck {
    uint64_t bad = 0;
    std::string first;
    void fail_if(bool cond, const char *fmt, ...) {
        if (!cond) return;
        if (bad++ == 0) {
            char buf[512];
            va_list ap;
            va_start(ap, fmt);
            vsnprintf(buf, sizeof buf, fmt, ap);
            va_end(ap);
            first = buf;
        }
    }
};

// The direct insert of a plan: every (slice, chunk) block's bitmap window
// or list window, and its partial slice in the position buffer.
void check_direct(const Plan &p, bool from_bitmap, const std::vector<uint64_t> &list_n, RangeCheck &rc) {
    const Carve &c = p.carve;
    const uint64_t sel_words = c.slots / 32, pos_cap = c.pos_capacity();
    for (size_t t = 0; t < p.t.size(); ++t) {
        const TInit &in = p.t[t];
        const uint32_t G = in.dir_g, per = in.dir_per;
        const uint64_t m_words = p.bl_mcap[t] / 32;
        rc.fail_if(G == 0 || per == 0, "tensor %zu: direct insert with %u chunks of %u", t, G, per);
        for (uint32_t ch = 0; ch < G; ++ch) {
            if (from_bitmap) {
                const Range32 cw = dir_bitmap_chunk(in.ntiles, per, ch, TILE_WORDS);
                // the kernel's view and loop run over hi - lo words (32-bit)
                rc.fail_if(cw.lo > cw.hi || (uint32_t)(cw.hi - cw.lo) > (uint64_t)per * TILE_WORDS,
                           "tensor %zu chunk %u: bitmap words [%u, %u)", t, ch, cw.lo, cw.hi);
                rc.fail_if(cw.hi > (uint64_t)in.ntiles * TILE_WORDS,
                           "tensor %zu chunk %u: bitmap words end %u past the tensor's %u tiles", t, ch, cw.hi,
                           in.ntiles);
                rc.fail_if((in.slot >> 5) + cw.hi > sel_words, "tensor %zu chunk %u: bitmap words past the bitmap",
                           t, ch);
            } else {
                for (uint64_t n : list_n) {
                    const Range32 cq = dir_list_chunk((uint32_t)n, per, ch);
                    rc.fail_if(cq.hi > n || cq.lo > cq.hi || (uint32_t)(cq.hi - cq.lo) > per,
                               "tensor %zu chunk %u: items [%u, %u) of %llu", t, ch,
                               cq.lo, cq.hi, (unsigned long long)n);
                }
                // every item below the capacity falls in some chunk
                rc.fail_if((uint64_t)G * per < p.bl_ncap[t], "tensor %zu: %u chunks of %u cover fewer than %llu items",
                           t, G, per, (unsigned long long)p.bl_ncap[t]);
            }
            for (uint32_t sl = 0; sl < in.dir_nsl; ++sl) {
                const uint64_t w0 = (uint64_t)sl * DIR_SLICE_WORDS;
                if (w0 >= m_words) continue;
                const uint64_t nw = std::min<uint64_t>(DIR_SLICE_WORDS, m_words - w0);
                const uint64_t local = (uint64_t)sl * G + ch;
                rc.fail_if(nw > in.dir_sw, "tensor %zu slice %u: %llu words in a %u-word partial", t, sl,
                           (unsigned long long)nw, in.dir_sw);
                rc.fail_if(in.dir_pb + local * in.dir_sw + nw > pos_cap,
                           "tensor %zu slice %u chunk %u: partial slice past the position buffer", t, sl, ch);
                rc.fail_if(in.dir_blk0 + local >= p.dir_blocks, "tensor %zu: block %llu past the grid", t,
                           (unsigned long long)(in.dir_blk0 + local));
            }
        }
        // the OR pass: slice sl's partials are G consecutive runs of dir_sw words
        rc.fail_if(in.dir_sl0 + in.dir_nsl > p.dir_slices, "tensor %zu: slices past the OR grid", t);
    }
}

// The bucketed insert's regions of a plan.
void check_bucketed(const Plan &p, RangeCheck &rc) {
    const Carve &c = p.carve;
    const uint64_t pos_cap = c.pos_capacity();
    for (size_t t = 0; t < p.t.size(); ++t) {
        const TInit &in = p.t[t];
        rc.fail_if(in.bl_pos0 + in.bl_poscap > pos_cap, "tensor %zu: position records past the buffer", t);
        rc.fail_if(in.bl_tab0 + (uint64_t)in.bl_nchunks * in.bl_nslices > c.btab, "tensor %zu: count table overrun",
                   t);
        rc.fail_if((uint64_t)in.bl_nslices << in.slice_log2 < p.bl_mcap[t], "tensor %zu: slices cover too few bits",
                   t);
    }
}

// The probe pass's block ranges for several grid sizes: contiguous, in
// block order, covering every tile once.
void check_probe_blocks(uint32_t ntiles, RangeCheck &rc) {
    const uint32_t grids[] = {1u, 2u, 3u, 7u, 32u, 224u, 255u, 256u, 1024u, PSTAT_MAX};
    for (uint32_t grid : grids) {
        uint32_t next = 0;
        for (uint32_t b = 0; b < grid; ++b) {
            const Range32 r = probe_block_tiles(ntiles, grid, b);
            rc.fail_if(r.lo > r.hi || r.hi > ntiles, "grid %u block %u: tiles [%u, %u) of %u", grid, b, r.lo, r.hi,
                       ntiles);
            if (r.lo < r.hi) {
                rc.fail_if(r.lo != next, "grid %u block %u: starts at tile %u, not %u", grid, b, r.lo, next);
                next = r.hi;
            }
        }
        rc.fail_if(next != ntiles, "grid %u: blocks cover %u of %u tiles", grid, next, ntiles);
    }
}

// The value sort's tiles for value counts from 0 to d per tensor (the count
// is known only on the device): each tile's view lies inside the tensor's
// slot and below the count, and the tiles of all tensors fit the look-back
// status rows (one per tile of the gradient).
void check_sort_tiles(const Plan &p, RangeCheck &rc) {
    const Carve &c = p.carve;
    uint64_t max_tiles = 0;
    for (size_t t = 0; t < p.t.size(); ++t) {
        const TInit &in = p.t[t];
        const uint64_t d = in.d;
        const uint64_t cand[] = {0, 1, TILE - 1, TILE, TILE + 1, 2 * TILE + 7, d / 2, d > 0 ? d - 1 : 0, d};
        uint64_t most = 0;
        for (uint64_t nv : cand) {
            if (nv > d) continue;
            const uint32_t ntl = (uint32_t)((nv + TILE - 1) / TILE);
            for (uint32_t lt = 0; lt <= ntl; ++lt) {  // one past the last, as a block past the end computes it
                const Range32 r = sort_tile_values((uint32_t)nv, lt, TILE);
                rc.fail_if(r.lo > r.hi || r.hi > nv || r.hi - r.lo > TILE,
                           "tensor %zu, %llu values, tile %u: values [%u, %u)", t, (unsigned long long)nv, lt, r.lo,
                           r.hi);
                rc.fail_if(in.slot + r.hi > c.slots, "tensor %zu, %llu values, tile %u: past the work arrays", t,
                           (unsigned long long)nv, lt);
            }
            most = std::max<uint64_t>(most, ntl);
        }
        max_tiles += most;
    }
    rc.fail_if(max_tiles > c.ntiles, "sort tiles %llu exceed the %llu look-back rows", (unsigned long long)max_tiles,
               (unsigned long long)c.ntiles);
}

dr_status check_ranges_impl(const dr_config *cfg, uint64_t *violations) {
    if (!violations) return fail(DR_EINVAL, "violations_h is null");
    Plan p;
    std::vector<uint64_t> rec_off;
    dr_status st = plan_config(cfg, p, rec_off);
    if (st != DR_OK) return st;
    RangeCheck rc;
    // the round trip's plan: items from the selection bitmap
    if (p.direct)
        check_direct(p, true, {}, rc);
    else
        check_bucketed(p, rc);
    check_probe_blocks((uint32_t)p.carve.ntiles, rc);
    check_sort_tiles(p, rc);
    // the standalone insert of each tensor's selection (dr_bloom_encode's
    // plan: items from a list of n_cap entries)
    for (size_t t = 0; t < p.t.size(); ++t) {
        const uint64_t n_cap = p.bl_ncap[t];
        Plan q = single_plan(n_cap);
        TInit &in = q.t[0];
        in.k = p.t[t].k;
        in.m_words_in = (uint32_t)(p.bl_mcap[t] / 32);
        plan_bloom(in, n_cap, p.bl_mcap[t], false, q);
        q.carve.plan();
        plan_bloom_rounds(q, in.k);
        plan_bloom_direct(q, false);
        if (q.direct)
            check_direct(q, false, {0, 1, n_cap / 2, n_cap}, rc);
        else
            check_bucketed(q, rc);
    }
    *violations = rc.bad;
    if (rc.bad) return fail(DR_OK, "%llu range violations; first: %s", (unsigned long long)rc.bad, rc.first.c_str());
    g_err.clear();
    return DR_OK;
}

// ---------------------------------------------------------------------------
// Opt-in per-kernel timing
// ---------------------------------------------------------------------------
struct TraceMark {
    const char *name;  // null: boundary at the start of an entry point (its interval is idle time)
    hipEvent_t ev;
    hipStream_t s;     // a kernel's time runs from the previous mark on the same stream
};
struct Tracer {
    bool on = false;
    std::vector<TraceMark> marks;
    std::vector<hipEvent_t> pool;
};
thread_local Tracer g_trace;

void trace_record(hipStream_t s, const char *name) {
    if (!g_trace.on) return;
    hipEvent_t ev;
    if (!g_trace.pool.empty()) {
        ev = g_trace.pool.back();
        g_trace.pool.pop_back();
    } else if (hipEventCreate(&ev) != hipSuccess) {
        return;
    }
    if (hipEventRecord(ev, s) != hipSuccess) {
        g_trace.pool.push_back(ev);
        return;
    }
    g_trace.marks.push_back({name, ev, s});
}

// every entry point that launches work marks its start
void trace_call(hipStream_t s) { trace_record(s, nullptr); }


}  // namespace

namespace dr {
// Compute units of the current device (cached per device).
int device_cus() {
    static int cus[64] = {0};
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
    const int slot = dev < 64 ? dev : 63;
    if (cus[slot] == 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
            cus[slot] = v;
        else
            cus[slot] = 256;
    }
    return cus[slot];
}
void trace_mark(hipStream_t s, const char *kernel) { trace_record(s, kernel); }

int blocks_per_cu(const void *kernel, int threads) {
    static std::mutex mu;
    static std::map<std::tuple<const void *, int, int>, int> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
    const auto key = std::make_tuple(kernel, threads, dev);
    std::lock_guard<std::mutex> lock(mu);
    auto it = cache.find(key);
    if (it != cache.end()) return it->second;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) != hipSuccess || n < 1) n = 1;
    cache[key] = n;
    return n;
}
}  // namespace dr

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

const char *dr_last_error(void) { return g_err.c_str(); }

dr_status dr_trace_begin(void *stream) {
    if (g_trace.on) return fail(DR_EINVAL, "tracing already begun on this thread");
    g_trace.on = true;
    g_trace.marks.clear();
    trace_record((hipStream_t)stream, nullptr);
    return DR_OK;
}

dr_status dr_trace_end(char *buf_h, size_t buf_bytes) {
    if (!g_trace.on) return fail(DR_EINVAL, "tracing was not begun on this thread");
    g_trace.on = false;
    std::vector<std::string> names;
    std::vector<double> total;
    std::vector<uint64_t> count;
    dr_status st = DR_OK;
    if (!g_trace.marks.empty()) {
        hipError_t e = hipEventSynchronize(g_trace.marks.back().ev);
        if (e != hipSuccess) st = hip_fail(e, "hipEventSynchronize");
    }
    for (size_t i = 1; st == DR_OK && i < g_trace.marks.size(); ++i) {
        if (!g_trace.marks[i].name) continue;
        size_t p = i - 1;  // the previous mark on the kernel's stream
        while (p > 0 && g_trace.marks[p].s != g_trace.marks[i].s) --p;
        if (g_trace.marks[p].s != g_trace.marks[i].s) continue;
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, g_trace.marks[p].ev, g_trace.marks[i].ev) != hipSuccess) continue;
        size_t j = 0;
        while (j < names.size() && names[j] != g_trace.marks[i].name) ++j;
        if (j == names.size()) {
            names.push_back(g_trace.marks[i].name);
            total.push_back(0.0);
            count.push_back(0);
        }
        total[j] += ms;
        count[j] += 1;
    }
    for (const TraceMark &m : g_trace.marks) g_trace.pool.push_back(m.ev);
    g_trace.marks.clear();
    std::string out;
    char line[256];
    for (size_t j = 0; j < names.size(); ++j) {
        snprintf(line, sizeof line, "%s %llu %.6f\n", names[j].c_str(), (unsigned long long)count[j], total[j]);
        out += line;
    }
    if (buf_h && buf_bytes) {
        const size_t n = std::min(out.size(), buf_bytes - 1);
        memcpy(buf_h, out.data(), n);
        buf_h[n] = 0;
    }
    return st;
}

dr_status dr_check_ranges(const dr_config *cfg_h, uint64_t *violations_h) {
    return check_ranges_impl(cfg_h, violations_h);
}

dr_status dr_bloom_params(uint64_t n_items, double fpr, uint64_t *m_bits_h, uint32_t *k_h) {
    if (!m_bits_h || !k_h) return fail(DR_EINVAL, "null output pointer");
    if (!bloom_params_host(n_items, fpr, m_bits_h, k_h)) return fail(DR_EINVAL, "fpr outside (0, 1) or m >= 2^32");
    return DR_OK;
}

uint32_t dr_sigma_bits(uint64_t n) { return sigma_bits_host(n); }

size_t dr_workspace_bytes(uint64_t d, uint64_t n_tensors) {
    if (n_tensors < 1) n_tensors = 1;
    return bound_carve(d, n_tensors).bytes;
}

size_t dr_payload_layout(const dr_config *cfg_h, uint64_t *rec_off_h) {
    Plan p;
    std::vector<uint64_t> rec_off;
    if (plan_config(cfg_h, p, rec_off) != DR_OK) return 0;
    if (rec_off_h)
        for (size_t i = 0; i < rec_off.size(); ++i) rec_off_h[i] = rec_off[i];
    return rec_off.back();
}

dr_status dr_payload_encode(const float *g, const dr_config *cfg_h, uint8_t *payload, size_t payload_bytes,
                            uint64_t *counts_out, void *ws, size_t ws_bytes, void *stream) {
    return encode_impl(g, cfg_h, payload, payload_bytes, counts_out, ws, ws_bytes, (hipStream_t)stream);
}

dr_status dr_payload_decode(const uint8_t *payload, const dr_config *cfg_h, float *dense_out, uint32_t *idx_out,
                            float *val_out, uint64_t *counts_out, void *ws, size_t ws_bytes, void *stream) {
    return decode_impl(payload, cfg_h, dense_out, idx_out, val_out, counts_out, ws, ws_bytes, (hipStream_t)stream);
}

dr_status dr_payload_decode_sum(const uint8_t *const *payloads_h, uint32_t n_payloads, const dr_config *cfg_h,
                                float scale, float *dense_out, uint64_t *counts_out, void *ws, size_t ws_bytes,
                                void *stream) {
    return decode_sum_impl(payloads_h, n_payloads, cfg_h, scale, dense_out, counts_out, ws, ws_bytes,
                           (hipStream_t)stream);
}

dr_status dr_roundtrip(const float *g, const dr_config *cfg_h, uint8_t *payload, size_t payload_bytes,
                       float *dense_out, uint32_t *idx_out, float *val_out, uint64_t *counts_out, void *ws,
                       size_t ws_bytes, void *stream) {
    return roundtrip_impl(g, cfg_h, payload, payload_bytes, dense_out, idx_out, val_out, counts_out, ws, ws_bytes,
                          (hipStream_t)stream);
}

dr_status dr_roundtrip_static(const float *g, const dr_config *cfg_h, uint8_t *payload, size_t payload_bytes,
                              float *dense_out, uint32_t *idx_out, float *val_out, uint64_t *counts_out,
                              void *stream) {
    return roundtrip_static_impl(g, cfg_h, payload, payload_bytes, dense_out, idx_out, val_out, counts_out,
                                 (hipStream_t)stream);
}

dr_status dr_sparsify_topr(const float *g, uint64_t d, uint64_t r, uint32_t *idx_out, float *val_out,
                           uint64_t *n_out, void *ws, size_t ws_bytes, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (d >= (1ull << 32)) return fail(DR_EINVAL, "d >= 2^32");
    const bool nz = r == DR_R_NONZERO;
    if (!nz && r > d) return fail(DR_EINVAL, "r > d");
    if ((!g && d) || !n_out || (!idx_out && (nz ? d : r) > 0)) return fail(DR_EINVAL, "null pointer");
    Plan p = single_plan(d);
    TInit &in = p.t[0];
    in.r = nz ? R_NONZERO : (uint32_t)r;
    if (!nz) {
        uint64_t hb = 0, rb = 0;
        plan_topr_hist(in, d, r, hist_tiles_per_block(in.ntiles), d >= SAMPLE_MIN_TOTAL, hb, rb);
        p.carve.hist_blocks = hb;
        p.carve.redo_blocks = rb;
    }
    p.carve.plan();
    if (!ws_ok(ws, ws_bytes, p.carve.bytes))
        return fail(DR_EINVAL, "workspace too small or not 256-byte aligned (need %zu)", p.carve.bytes);
    Work w = p.carve.view((uint8_t *)ws);
    w.S = idx_out;  // single tensor: slot 0 is the caller's list
    trace_call(s);
    DR_HIP(run_init(w, p.t, s));
    if (!nz)
        DR_HIP(launch_topr(w, g, (uint32_t)p.carve.hist_blocks, (uint32_t)p.carve.redo_blocks, true, s));
    else
        DR_HIP(launch_nonzero(w, g, persist_grid(8), s));
    DR_HIP(launch_compact_selection(w, g, val_out, persist_grid(8), s));
    DR_HIP(launch_export_n(w, n_out, 0, s));
    return DR_OK;
}

dr_status dr_bloom_encode(const uint32_t *idx, const uint64_t *n, uint64_t n_cap, uint64_t m_bits, uint32_t k,
                          uint32_t *bits_out, uint64_t *flags_out, void *ws, size_t ws_bytes, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (!n || !bits_out || (!idx && n_cap)) return fail(DR_EINVAL, "null pointer");
    if (m_bits < 32 || (m_bits & 31) || m_bits >= (1ull << 32)) return fail(DR_EINVAL, "bad m_bits");
    if (k < 1 || k > 32) return fail(DR_EINVAL, "k must be in [1, 32]");
    if (n_cap >= (1ull << 32)) return fail(DR_EINVAL, "n_cap >= 2^32");
    if (ceil_div(m_bits, 1ull << SLICE_LOG2_MAX) > BL_MAX_SLICES) return fail(DR_ENOTSUP, "filter larger than 2^30 bits");
    Plan p = single_plan(n_cap);
    TInit &in = p.t[0];
    in.k = k;
    in.m_words_in = (uint32_t)(m_bits / 32);
    in.bits = bits_out;
    plan_bloom(in, n_cap, m_bits, false, p);
    p.carve.plan();
    plan_bloom_rounds(p, k);
    plan_bloom_direct(p, false);
    if (!ws_ok(ws, ws_bytes, p.carve.bytes))
        return fail(DR_EINVAL, "workspace too small or not 256-byte aligned (need %zu)", p.carve.bytes);
    Work w = p.carve.view((uint8_t *)ws);
    w.S = const_cast<uint32_t *>(idx);
    trace_call(s);
    DR_HIP(run_init(w, p.t, s));
    DR_HIP(launch_import_n(w, n, n_cap, flags_out, s));
    if (p.direct)
        DR_HIP(launch_bloom_direct(w, false, p.dir_blocks, p.dir_slices, s));
    else
        DR_HIP(launch_bloom_insert(w, false, p.bl_chunks, p.bl_slices, p.max_slices, p.hash_per_round, p.kmax, s));
    return DR_OK;
}

dr_status dr_bloom_decode(const uint32_t *bits, uint64_t m_bits, uint32_t k, uint64_t d, uint32_t *idx_out,
                          uint64_t cap, uint64_t *n_out, void *ws, size_t ws_bytes, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (!bits || !n_out || (!idx_out && cap)) return fail(DR_EINVAL, "null pointer");
    if (m_bits < 32 || (m_bits & 31) || m_bits >= (1ull << 32)) return fail(DR_EINVAL, "bad m_bits");
    if (k < 1 || k > 32) return fail(DR_EINVAL, "k must be in [1, 32]");
    if (d >= (1ull << 32)) return fail(DR_EINVAL, "d >= 2^32");
    Plan p = single_plan(d);
    TInit &in = p.t[0];
    in.k = k;
    in.m_words_in = (uint32_t)(m_bits / 32);
    in.bits = const_cast<uint32_t *>(bits);
    p.carve.plan();
    if (!ws_ok(ws, ws_bytes, p.carve.bytes))
        return fail(DR_EINVAL, "workspace too small or not 256-byte aligned (need %zu)", p.carve.bytes);
    const Work w = p.carve.view((uint8_t *)ws);
    trace_call(s);
    DR_HIP(run_init(w, p.t, s));
    DR_HIP(launch_query_plain(w, idx_out, cap, n_out, persist_grid(4), s));
    return DR_OK;
}

dr_status dr_curvefit_encode(const float *vals, const uint64_t *n, uint64_t n_cap, uint32_t degree, uint32_t n_seg,
                             float *coef_out, uint32_t *sigma_out, uint64_t *flags_out, void *ws, size_t ws_bytes,
                             void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (!n || !coef_out || ((!vals || !sigma_out) && n_cap)) return fail(DR_EINVAL, "null pointer");
    if (degree > DR_MAX_DEGREE) return fail(DR_EINVAL, "degree > %d", DR_MAX_DEGREE);
    if (n_seg < 1 || n_seg > DR_MAX_SEGMENTS) return fail(DR_EINVAL, "n_seg out of range");
    if (n_cap >= (1ull << 32)) return fail(DR_EINVAL, "n_cap >= 2^32");
    Plan p = single_plan(n_cap);
    TInit &in = p.t[0];
    in.degree = degree;
    in.nseg = n_seg;
    in.coef = coef_out;
    in.coef_stride = degree + 1;
    in.sigma = sigma_out;
    in.fit_blk0 = 0;
    p.carve.fit_blocks = (uint64_t)n_seg * FIT_CHUNKS;
    p.carve.plan();
    if (!ws_ok(ws, ws_bytes, p.carve.bytes))
        return fail(DR_EINVAL, "workspace too small or not 256-byte aligned (need %zu)", p.carve.bytes);
    const Work w = p.carve.view((uint8_t *)ws);
    trace_call(s);
    DR_HIP(run_init(w, p.t, s));
    DR_HIP(launch_keygen(w, vals, n, n_cap, flags_out, persist_grid(4), s));
    DR_HIP(launch_value_setup(w, false, nullptr, s));
    DR_HIP(launch_sort(w, (uint32_t)p.carve.ntiles, s));
    DR_HIP(launch_fit(w, (uint32_t)p.carve.fit_blocks, p.carve.vals_est, p.dexp, s));
    return DR_OK;
}

dr_status dr_curvefit_decode(const float *coef, const uint32_t *sigma, const uint64_t *n, uint64_t n_cap,
                             uint32_t degree, uint32_t n_seg, float *vals_out, uint64_t *flags_out, void *ws,
                             size_t ws_bytes, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (!n || ((!coef || !sigma || !vals_out) && n_cap)) return fail(DR_EINVAL, "null pointer");
    if (degree > DR_MAX_DEGREE) return fail(DR_EINVAL, "degree > %d", DR_MAX_DEGREE);
    if (n_seg < 1 || n_seg > DR_MAX_SEGMENTS) return fail(DR_EINVAL, "n_seg out of range");
    if (n_cap >= (1ull << 32)) return fail(DR_EINVAL, "n_cap >= 2^32");
    Plan p = single_plan(0);
    TInit &in = p.t[0];
    in.degree = degree;
    in.nseg = n_seg;
    p.carve.plan();
    if (!ws_ok(ws, ws_bytes, p.carve.bytes))
        return fail(DR_EINVAL, "workspace too small or not 256-byte aligned (need %zu)", p.carve.bytes);
    const Work w = p.carve.view((uint8_t *)ws);
    trace_call(s);
    DR_HIP(run_init(w, p.t, s));
    DR_HIP(launch_curvefit_decode(w, coef, sigma, n, n_cap, vals_out, flags_out, persist_grid(4), s));
    return DR_OK;
}

}  // extern "C"
