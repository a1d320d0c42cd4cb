// valuefit.hip -- curve-fitting value compression (Section 5) and the
// reorder map (Section 5.1).
//
//  * Sort: the values of each tensor are sorted in descending order by an
//    LSD radix sort (four 8-bit digits) of the order-preserving u32 image,
//    complemented so that ascending order of the key is descending order of
//    the value.  One pass counts all four digits; each digit pass is then a
//    single kernel whose tiles chain their offsets by decoupled look-back.
//    Each pass is stable (ranks within a tile come from wave ballots in
//    element order), so equal values keep their original order.
//  * Fit: each run of equal count is fitted by least squares in double: the
//    normal-equation sums are accumulated per block and reduced in a fixed
//    order, then a Gaussian elimination with partial pivoting solves the
//    (D+1) x (D+1) system.  No MFMA: this is a small reduction.
//  * Reorder map: sigma[q] = sorted rank of value q, packed b bits per entry.
#include "launch.hpp"
#include "value_setup.hpp"

namespace dr {

// standalone value path: keys from the caller's values
__global__ __launch_bounds__(NTHREADS) void k_keygen(Work w, const float *__restrict__ vals, const uint64_t *n,
                                                     uint64_t n_cap, uint64_t *flags_out) {
    const uint64_t n64 = *n;
    const uint32_t nv = (uint32_t)(n64 < n_cap ? n64 : n_cap);
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        w.td[0].nv = nv;
        w.td[0].npos = nv;
        if (n64 > n_cap) atomicOr(&w.td[0].flags, FLAG_CAPACITY);
        if (flags_out) *flags_out = n64 > n_cap ? FLAG_CAPACITY : 0u;
    }
    for (uint32_t q = blockIdx.x * NTHREADS + threadIdx.x; q < nv; q += gridDim.x * NTHREADS) {
        w.keyA[q] = ~order_key(vals[q]);
        w.valA[q] = q;
    }
}

hipError_t launch_keygen(const Work &w, const float *vals, const uint64_t *n, uint64_t n_cap, uint64_t *flags_out,
                         int grid_persist, hipStream_t s) {
    k_keygen<<<grid_persist, NTHREADS, 0, s>>>(w, vals, n, n_cap, flags_out);
    trace_mark(s, "k_keygen");
    return hipGetLastError();
}

// After |P| is known: run shape, reorder-map width, sort tiling, record
// layout and header (value_setup_block).
constexpr uint32_t SETUP_THREADS = 1024;

__global__ __launch_bounds__(SETUP_THREADS) void k_value_setup(Work w, int payload, uint64_t *counts_out) {
    value_setup_block<SETUP_THREADS>(w, payload, counts_out);
}

hipError_t launch_value_setup(const Work &w, bool payload, uint64_t *counts_out, hipStream_t s) {
    k_value_setup<<<1, SETUP_THREADS, 0, s>>>(w, payload ? 1 : 0, counts_out);
    trace_mark(s, "k_value_setup");
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// LSD radix sort, segmented by tensor
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t tensor_of_stile(const Work &w, uint32_t g) {
    uint32_t lo = 0, hi = w.ntensors;
    while (hi - lo > 1) {
        uint32_t mid = (lo + hi) >> 1;
        if (w.td[mid].stile0 <= g)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

// Before the passes: each tensor's totals of all four digits, and the
// look-back status of every sort tile cleared.  Blocks own contiguous tile
// ranges and add their LDS counts to the tensor's totals when the tensor
// changes and at the end.
__global__ __launch_bounds__(NTHREADS) void k_sort_upfront(Work w, const uint32_t *__restrict__ keys) {
    __shared__ uint32_t h[4][SORT_BINS];
    const uint32_t total = w.glob->sort_tiles;
    const uint32_t per = (total + gridDim.x - 1) / gridDim.x;
    const uint32_t g0 = min(total, blockIdx.x * per), g1 = min(total, g0 + per);
    uint32_t cur = 0xffffffffu;
    for (uint32_t gt = g0; gt < g1; ++gt) {
        const uint32_t t = tensor_of_stile(w, gt);
        if (t != cur) {
            if (cur != 0xffffffffu) {
                __syncthreads();
                for (uint32_t p = 0; p < 4; ++p)
                    if (h[p][threadIdx.x]) atomicAdd(&w.sdig[(cur * 4 + p) * SORT_BINS + threadIdx.x], h[p][threadIdx.x]);
            }
            __syncthreads();
            for (uint32_t p = 0; p < 4; ++p) h[p][threadIdx.x] = 0;
            __syncthreads();
            cur = t;
        }
        const TDesc &td = w.td[t];
        const uint32_t lt = gt - td.stile0;
        const Range32 sr = sort_tile_values(td.nv, lt, TILE);
        const uint32_t q0 = sr.lo, nq = sr.hi - sr.lo;
        const __amdgpu_buffer_rsrc_t kv = buffer_view(keys + td.in.slot + q0, 4u * nq);
        uint32_t k16[TILE / NTHREADS];
#pragma unroll
        for (uint32_t c = 0; c < TILE / NTHREADS; ++c) k16[c] = buffer_u32(kv, 4u * (c * NTHREADS + threadIdx.x));
        asm volatile("" ::: "memory");
#pragma unroll
        for (uint32_t c = 0; c < TILE / NTHREADS; ++c) {
            if (c * NTHREADS + threadIdx.x < nq) {
#pragma unroll
                for (uint32_t p = 0; p < 4; ++p) atomicAdd(&h[p][(k16[c] >> (8 * p)) & 255u], 1u);
            }
        }
        uint64_t *st = w.sstat + (uint64_t)gt * SORT_BINS;
        for (uint32_t p = 0; p < 4; ++p) st[(uint64_t)p * w.ntiles_total * SORT_BINS + threadIdx.x] = 0;
    }
    if (cur != 0xffffffffu) {
        __syncthreads();
        for (uint32_t p = 0; p < 4; ++p)
            if (h[p][threadIdx.x]) atomicAdd(&w.sdig[(cur * 4 + p) * SORT_BINS + threadIdx.x], h[p][threadIdx.x]);
    }
}

// One stable pass of the digit at bits [8 pass, 8 pass + 8): tiles are
// taken in ticket order, so a tile only ever waits for tiles that running
// blocks hold.  A tile
//  1. reads its keys and values (wave w holds elements [1024 w, 1024 w +
//     1024) of the tile, 64 consecutive per step) and counts its digits in
//     LDS;
//  2. publishes the counts at once and starts reading the counts of the
//     tensor's earlier tiles (decoupled look-back, LB_WIN tiles per read
//     round; a tile that already knows its inclusive prefix ends the walk);
//  3. while those reads are in flight, ranks its elements: lanes with equal
//     digits find each other with 8 ballots, and each wave keeps running
//     per-digit counts, so ranks follow element order (a stable pass);
//  4. finishes the look-back, publishes its inclusive prefix, and scatters.
constexpr uint64_t ST_AGG = 1ull << 32, ST_INC = 2ull << 32;
constexpr uint32_t SPIN_LIMIT = 1u << 20;
constexpr uint32_t LB_WIN = 8;  // look-back window (tiles read together)
constexpr uint32_t SORT_STEPS = TILE / NTHREADS;  // 16 keys per thread

// At most 168 VGPRs (three blocks per CU; 233 without the bound, which
// left the 32 CUs the round trip gives the sender 64 block slots for a
// 25.6 M-element gradient's 69 tiles, so 5 tiles waited for a second round).
__global__ __launch_bounds__(NTHREADS) __attribute__((amdgpu_waves_per_eu(3))) void k_sort_pass(Work w, const uint32_t *__restrict__ kin,
                                                        const uint32_t *__restrict__ vin,
                                                        uint32_t *__restrict__ kout, uint32_t *__restrict__ vout,
                                                        uint32_t pass) {
    __shared__ uint32_t hist[SORT_BINS];
    __shared__ uint32_t run[NWAVES][SORT_BINS];  // per-wave running counts, then per-wave bases
    __shared__ uint32_t goff[SORT_BINS];
    __shared__ uint32_t scratch[NWAVES + 1];
    __shared__ uint32_t ticket;
    const uint32_t lane = threadIdx.x & 63u, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t total = w.glob->sort_tiles;
    if (blockIdx.x >= total) return;
    const uint32_t shift = 8u * pass;
    uint64_t *stat = w.sstat + (uint64_t)pass * w.ntiles_total * SORT_BINS;
    for (;;) {
        if (threadIdx.x == 0) ticket = atomicAdd(&w.glob->sort_ticket[pass], 1u);
        hist[threadIdx.x] = 0;
#pragma unroll
        for (uint32_t q = 0; q < NWAVES; ++q) run[q][threadIdx.x] = 0;
        __syncthreads();
        const uint32_t gt = ticket;
        if (gt >= total) break;
        const uint32_t t = tensor_of_stile(w, gt);
        TDesc &td = w.td[t];
        // descriptor fields in registers: the scatter's stores could alias
        // them for all the compiler knows, which would reload them per store
        const uint32_t stile0 = td.stile0;
        const uint32_t lt = gt - stile0;
        const uint32_t nv = td.nv;
        const uint64_t slot = td.in.slot;
        const Range32 sr = sort_tile_values(nv, lt, TILE);
        const uint32_t q0 = sr.lo, nq = sr.hi - sr.lo;
        const __amdgpu_buffer_rsrc_t kv = buffer_view(kin + slot + q0, 4u * nq);
        const __amdgpu_buffer_rsrc_t vv = buffer_view(vin + slot + q0, 4u * nq);
        const uint32_t ebase = wv * (SORT_STEPS * 64) + lane;  // element of step c: ebase + 64 c
        // keys and values read together and held until the scatter: one
        // round trip to memory per tile
        uint32_t key[SORT_STEPS], val[SORT_STEPS];
#pragma unroll
        for (uint32_t c = 0; c < SORT_STEPS; ++c) {
            key[c] = buffer_u32(kv, 4u * (ebase + 64 * c));
            val[c] = buffer_u32(vv, 4u * (ebase + 64 * c));
        }
        asm volatile("" ::: "memory");
        // the tensor's base of each digit of this pass
        uint32_t dtot;
        const uint32_t dbase = block_excl_scan(w.sdig[(t * 4 + pass) * SORT_BINS + threadIdx.x], scratch, &dtot);
        // 1. the tile's digit counts
#pragma unroll
        for (uint32_t c = 0; c < SORT_STEPS; ++c)
            if (ebase + 64 * c < nq) atomicAdd(&hist[(key[c] >> shift) & 255u], 1u);
        __syncthreads();
        // 2. publish; first look-back window in flight
        const uint32_t dg = threadIdx.x;
        const uint32_t agg = hist[dg];
        uint64_t *me = stat + (uint64_t)gt * SORT_BINS + dg;
        __hip_atomic_store(me, (lt == 0 ? ST_INC : ST_AGG) | agg, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        uint32_t j = gt - 1;  // next earlier tile to read (valid while lt > 0)
        uint32_t nwin = lt == 0 ? 0u : min(LB_WIN, j - stile0 + 1);
        uint64_t sv[LB_WIN];
#pragma unroll
        for (uint32_t u = 0; u < LB_WIN; ++u)
            sv[u] = u < nwin ? __hip_atomic_load(stat + (uint64_t)(j - u) * SORT_BINS + dg, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT)
                             : 0ull;
        // 3. ranks within the wave, in element order
        uint32_t rk[SORT_STEPS / 2];  // two 16-bit ranks per word
#pragma unroll
        for (uint32_t c = 0; c < SORT_STEPS / 2; ++c) rk[c] = 0;
#pragma unroll
        for (uint32_t c = 0; c < SORT_STEPS; ++c) {
            const bool valid = ebase + 64 * c < nq;
            const uint32_t d8 = (key[c] >> shift) & 255u;
            uint64_t peers = ballot(valid);
#pragma unroll
            for (int bb = 0; bb < 8; ++bb) {
                const bool bit = (d8 >> bb) & 1u;
                const uint64_t m = ballot(bit);
                peers &= bit ? m : ~m;
            }
            const uint32_t leader = (uint32_t)__ffsll((unsigned long long)peers) - 1u;
            uint32_t r0 = 0;
            if (valid && lane == leader) {
                r0 = run[wv][d8];
                run[wv][d8] = r0 + popc64(peers);
            }
            r0 = __shfl(r0, leader, 64);
            rk[c >> 1] |= (r0 + lanes_below(peers)) << (16 * (c & 1));
        }
        __syncthreads();
        // per-wave bases of each digit (waves in element order)
        {
            uint32_t acc = 0;
#pragma unroll
            for (uint32_t q = 0; q < NWAVES; ++q) {
                const uint32_t x = run[q][dg];
                run[q][dg] = acc;
                acc += x;
            }
        }
        // 4. finish the look-back: a tile that has not published yet ends
        // the window, and the next window starts at it
        uint32_t excl = 0;
        if (lt > 0) {
            uint32_t rounds = 0;
            for (;;) {
                uint32_t used = nwin;
                bool inc = false;
#pragma unroll
                for (uint32_t u = 0; u < LB_WIN; ++u) {
                    if (u < used && !inc) {
                        if ((sv[u] >> 32) == 0) {
                            used = u;  // not published yet
                        } else {
                            excl += (uint32_t)sv[u];
                            inc = (sv[u] & ST_INC) != 0;
                        }
                    }
                }
                if (inc || (used == nwin && j - stile0 + 1 == nwin)) break;  // prefix complete
                j -= used;
                if (used == 0) {
                    if (++rounds >= SPIN_LIMIT) {  // cannot happen; never hang the device on a bug
                        atomicOr(&td.flags, FLAG_STALLED);
                        if (w.counts_out) atomicOr((unsigned long long *)&w.counts_out[4 * t + 3], FLAG_STALLED);
                        break;
                    }
                    __builtin_amdgcn_s_sleep(1);
                }
                nwin = min(LB_WIN, j - stile0 + 1);
#pragma unroll
                for (uint32_t u = 0; u < LB_WIN; ++u)
                    sv[u] = u < nwin ? __hip_atomic_load(stat + (uint64_t)(j - u) * SORT_BINS + dg, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_AGENT)
                                     : 0ull;
            }
            __hip_atomic_store(me, ST_INC | (uint64_t)(excl + agg), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        goff[dg] = dbase + excl;
        __syncthreads();
#pragma unroll
        for (uint32_t c = 0; c < SORT_STEPS; ++c) {
            const uint32_t d8 = (key[c] >> shift) & 255u;
            const uint32_t pos = goff[d8] + run[wv][d8] + ((rk[c >> 1] >> (16 * (c & 1))) & 0xffffu);
            if (ebase + 64 * c < nq && pos < nv && val[c] < nv) {
                if (pass == 3) {
                    w.sig[slot + val[c]] = pos;  // reorder map: value q has rank pos
                    w.vsorted[slot + pos] = order_key_inv(~key[c]);
                } else {
                    kout[slot + pos] = key[c];
                    vout[slot + pos] = val[c];
                }
            }
        }
        __syncthreads();  // hist, run, goff and ticket are rewritten by the next tile
    }
}

hipError_t launch_sort(const Work &w, uint32_t cap_tiles, hipStream_t s) {
    const uint32_t cus = (uint32_t)device_cus();
    k_sort_upfront<<<cus, NTHREADS, 0, s>>>(w, w.keyA);
    trace_mark(s, "k_sort_upfront");
    const int grid = (int)std::max(1u, std::min(cap_tiles, cus * 4u));
    uint32_t *kin = w.keyA, *vin = w.valA, *kout = w.keyB, *vout = w.valB;
    for (uint32_t p = 0; p < 4; ++p) {
        k_sort_pass<<<grid, NTHREADS, 0, s>>>(w, kin, vin, kout, vout, p);
        trace_mark(s, "k_sort_pass");
        uint32_t *tk = kin, *tv = vin;
        kin = kout;
        vin = vout;
        kout = tk;
        vout = tv;
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Segmentation of the sorted values (Section 5, "Piece-wise approximation")
// ---------------------------------------------------------------------------
// One block per tensor, after the sort.  Equal-count runs need nothing here
// unless their number comes from the heuristic.  Chord segmentation keeps
// the run starts and each run's farthest allowed split point in LDS and
// splits greedily; each split costs one block-wide arg-max over the two new
// runs.  Distances are evaluated as in the oracle's definition, one
// rounding per double operation (no contraction), so both take the same
// decisions.
constexpr uint32_t SEG_THREADS = 1024;
constexpr uint32_t SEG_BATCH = 8;

__device__ __forceinline__ double chord_dist(double ca, double m, uint32_t a, uint32_t i, float ci) {
#pragma clang fp contract(off)
    const double y = ca + m * (double)(i - a);
    return fabs(y - (double)ci);
}

// farthest allowed split point of run [a, e) for degree D, block-wide; the
// returned distance is 0 when no split is allowed (then *i_out is unset)
__device__ double seg_candidate(const float *C, uint32_t a, uint32_t e, uint32_t D, uint32_t *i_out, double *rd,
                                uint32_t *ri) {
#pragma clang fp contract(off)
    const uint32_t minpts = D + 1u;
    double best = 0.0;
    uint32_t bi = 0xffffffffu;
    if (e - a >= 2u * minpts) {
        const uint32_t z = e - 1u;
        const double ca = (double)C[a];
        const double m = ((double)C[z] - ca) / (double)(z - a);
        const uint32_t i0 = a + D, i1 = z - D;  // split points [i0, i1)
        // SEG_BATCH reads in flight per thread; each thread's points are
        // visited in increasing order, so a strict compare keeps the
        // smallest rank among equal distances
        for (uint32_t ib = i0; ib < i1; ib += SEG_THREADS * SEG_BATCH) {
            float v[SEG_BATCH];
#pragma unroll
            for (uint32_t u = 0; u < SEG_BATCH; ++u) {
                const uint32_t i = ib + u * SEG_THREADS + threadIdx.x;
                v[u] = i < i1 ? C[i] : 0.0f;
            }
#pragma unroll
            for (uint32_t u = 0; u < SEG_BATCH; ++u) {
                const uint32_t i = ib + u * SEG_THREADS + threadIdx.x;
                if (i < i1) {
                    const double dd = chord_dist(ca, m, a, i, v[u]);
                    if (dd > best) {
                        best = dd;
                        bi = i;
                    }
                }
            }
        }
    }
    // arg-max over the block: larger distance, then smaller rank
    for (uint32_t off = 32; off > 0; off >>= 1) {
        const double od = __shfl_down(best, off);
        const uint32_t oi = __shfl_down(bi, off);
        if (od > best || (od == best && oi < bi)) {
            best = od;
            bi = oi;
        }
    }
    const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
    __syncthreads();  // rd and ri are free
    if (lane == 0) {
        rd[wv] = best;
        ri[wv] = bi;
    }
    __syncthreads();
    best = rd[0];
    bi = ri[0];
    for (uint32_t q = 1; q < SEG_THREADS / 64; ++q)
        if (rd[q] > best || (rd[q] == best && ri[q] < bi)) {
            best = rd[q];
            bi = ri[q];
        }
    if (best > 0.0) *i_out = bi;
    return best;
}

// segments for the heuristic (p + 1 pieces): p = ceil(2 sqrt(M)) for degree
// >= 1, ceil(M / sqrt(2) - 1) for degree 0, M from the first and last
// differences of the sorted curve; each ceiling found by the smallest p with
// p^2 >= 4M, resp. 2 (p+1)^2 >= M^2
__device__ uint32_t seg_heuristic(const float *C, uint32_t n, uint32_t D) {
#pragma clang fp contract(off)
    double M = 0.0;
    if (n >= 2) M = fabs(((double)C[0] - (double)C[1]) - ((double)C[n - 2] - (double)C[n - 1]));
    uint32_t p = 0;
    if (D == 0) {
        const double M2 = M * M;
        while (p + 1 < MAX_SEG && 2.0 * (double)(p + 1) * (double)(p + 1) < M2) ++p;
    } else {
        const double M4 = 4.0 * M;
        while (p + 1 < MAX_SEG && (double)p * (double)p < M4) ++p;
    }
    return p + 1;
}

// The record's layout once the run count seff is known: the knots (chord
// runs: the seff - 1 interior starts st[1..seff-1]) and the header fields
// that follow from the count.  Block-wide, NT threads.
template <uint32_t NT>
__device__ void seg_finish(TDesc &td, uint32_t seff, bool chord, const uint32_t *st) {
    const uint32_t deff = td.deff;
    const uint32_t nkn = chord && seff > 1 ? seff - 1 : 0u;
    if (td.in.rec) {
        const uint32_t kn_off = td.coef_off + 4u * seff * (deff + 1u);
        uint32_t *kn = (uint32_t *)(td.in.rec + kn_off);
        for (uint32_t x = threadIdx.x; x < nkn; x += NT) kn[x] = st[x + 1];
        if (threadIdx.x == 0) {
            td.seff = seff;
            td.sigma_off = kn_off + 4u * nkn;
            td.rec_bytes = td.sigma_off + 4u * td.swords;
            uint32_t *h = (uint32_t *)td.in.rec;
            h[H_SEFF] = seff;
            h[H_RECBYTES] = td.rec_bytes;
        }
    } else if (threadIdx.x == 0) {
        td.seff = seff;
    }
}

// values with the sign bit clear come first in the sorted order: their count
__device__ __forceinline__ uint32_t sign_split(const float *C, uint32_t n) {
    uint32_t lo = 0, hi = n;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (!(__float_as_uint(C[mid]) >> 31))
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

// Chord segmentation over the whole grid, for tensors with a state slot.
// k_seg_init makes the sign split and marks the first runs for evaluation.
// In each k_seg_step every block evaluates its share of the marked runs'
// allowed split points (the runs' ranges laid end to end), and the last
// block to finish a tensor reduces the blocks' results, picks the run to
// split (farthest candidate, then the leftmost run), splits it after its
// candidate and marks the two new runs.  The host launches one step per
// split that may be needed; steps after the last split return at once.
// The decisions are those of the one-block loop in k_segment: the same
// distances, evaluated the same way, and the same tie rules.
constexpr uint32_t SEGG_THREADS = 256;
static_assert(SEG_GRID_BLOCKS <= SEGG_THREADS, "the last block reduces one result per thread");

__global__ __launch_bounds__(SEGG_THREADS) void k_seg_init(Work w) {
    __shared__ uint32_t st[3];
    TDesc &td = w.td[blockIdx.x];
    if (td.in.seg_slot == NO_SEG_SLOT) return;
    SegState &ss = w.segst[td.in.seg_slot];
    const uint32_t n = td.nv, D = td.in.degree, req = td.in.nseg;
    const float *C = w.vsorted + td.in.slot;
    // the sign split, by a 256-way search: the values with the sign bit
    // clear are a prefix of the sorted order
    uint32_t lo = 0, hi = n;  // the first value with the sign bit set is in [lo, hi]
    while (hi - lo > SEGG_THREADS) {
        const uint32_t x = lo + (uint32_t)((uint64_t)(hi - lo) * threadIdx.x / SEGG_THREADS);
        const uint32_t c = (uint32_t)__syncthreads_count(!(__float_as_uint(C[x]) >> 31));
        // the first c probes hold values with the sign bit clear
        const uint32_t nlo = c == 0 ? lo : lo + (uint32_t)((uint64_t)(hi - lo) * (c - 1) / SEGG_THREADS) + 1u;
        const uint32_t nhi = c == SEGG_THREADS ? hi : lo + (uint32_t)((uint64_t)(hi - lo) * c / SEGG_THREADS);
        lo = nlo;
        hi = c == 0 ? lo : nhi;
    }
    {
        const uint32_t x = lo + threadIdx.x;
        lo += (uint32_t)__syncthreads_count(x < hi && !(__float_as_uint(C[x]) >> 31));
    }
    uint32_t count = 0;
    if (threadIdx.x == 0) {
        st[0] = 0;
        st[1] = n;
        if (n > 0) {
            count = 1;
            if (req >= 2 && lo >= D + 1 && n - lo >= D + 1) {
                st[1] = lo;
                st[2] = n;
                count = 2;
            }
        }
        uint32_t *stw = w.bounds + td.in.bnd0;
        for (uint32_t x = 0; x <= count && n > 0; ++x) stw[x] = st[x];
        ss.count = count;
        ss.req = req;
        ss.done = n == 0 || count >= req;
        ss.pend = 0;
        ss.npend = count;
        ss.arrive = 0;
    }
    count = __shfl(count, 0, 64);  // wave 0 holds it; the other waves are done
    if (threadIdx.x < 64 && n > 0 && count >= req) seg_finish<64>(td, count, true, st);
}

// arg-max of (distance, rank) pairs over a wave: larger distance, then the
// smaller rank
__device__ __forceinline__ void argmax_wave(double *d, uint32_t *i) {
    for (uint32_t off = 32; off > 0; off >>= 1) {
        const double od = __shfl_down(*d, off);
        const uint32_t oi = __shfl_down(*i, off);
        if (od > *d || (od == *d && oi < *i)) {
            *d = od;
            *i = oi;
        }
    }
}

__global__ __launch_bounds__(SEGG_THREADS) void k_seg_step(Work w) {
    __shared__ double rd[2][SEGG_THREADS / 64];
    __shared__ uint32_t ri[2][SEGG_THREADS / 64];
    __shared__ uint32_t last, s_nc, s_done;
    __shared__ uint32_t lst[SEG_GRID_RUNS + 1];
    __shared__ double lcd[SEG_GRID_RUNS];
    __shared__ uint32_t lci[SEG_GRID_RUNS];
    const uint32_t G = gridDim.x, lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
    for (uint32_t t = 0; t < w.ntensors; ++t) {
        TDesc &td = w.td[t];
        const uint32_t slot = td.in.seg_slot;
        if (slot == NO_SEG_SLOT) continue;
        SegState &ss = w.segst[slot];
        if (ss.done) continue;
        const uint32_t D = td.in.degree;
        const float *C = w.vsorted + td.in.slot;
        const uint32_t *st = w.bounds + td.in.bnd0;
        const uint32_t p0 = ss.pend, np = ss.npend;
        // run q: split points [a + D, z - D), z = e - 1, when it holds at
        // least 2 (D + 1) points; its chord through (a, C[a]) and (z, C[z])
        uint32_t a[2] = {0, 0}, L[2] = {0, 0};
        double ca[2] = {0.0, 0.0}, m[2] = {0.0, 0.0};
#pragma unroll
        for (uint32_t q = 0; q < 2; ++q) {
            if (q < np) {
                const uint32_t aq = st[p0 + q], eq = st[p0 + q + 1];
                if (eq - aq >= 2u * (D + 1u)) {
                    const uint32_t z = eq - 1u;
                    a[q] = aq;
                    L[q] = (z - D) - (aq + D);
                    ca[q] = (double)C[aq];
                    m[q] = ((double)C[z] - ca[q]) / (double)(z - aq);
                }
            }
        }
        const uint32_t tot = L[0] + L[1];
        const uint32_t c0 = (uint32_t)((uint64_t)tot * blockIdx.x / G);
        const uint32_t c1 = (uint32_t)((uint64_t)tot * (blockIdx.x + 1) / G);
        double best[2] = {0.0, 0.0};
        uint32_t bi[2] = {0xffffffffu, 0xffffffffu};
        // SEG_BATCH reads in flight per thread; a thread's points come in
        // increasing rank, so a strict compare keeps the smallest rank
        for (uint32_t xb = c0; xb < c1; xb += SEGG_THREADS * SEG_BATCH) {
            float v[SEG_BATCH];
#pragma unroll
            for (uint32_t u = 0; u < SEG_BATCH; ++u) {
                const uint32_t x = xb + u * SEGG_THREADS + threadIdx.x;
                const uint32_t i = x < L[0] ? a[0] + D + x : a[1] + D + (x - L[0]);
                v[u] = x < c1 ? C[i] : 0.0f;
            }
#pragma unroll
            for (uint32_t u = 0; u < SEG_BATCH; ++u) {
                const uint32_t x = xb + u * SEGG_THREADS + threadIdx.x;
                if (x < c1) {
                    const uint32_t q = x < L[0] ? 0u : 1u;
                    const uint32_t i = q ? a[1] + D + (x - L[0]) : a[0] + D + x;
                    const double dd = chord_dist(ca[q], m[q], a[q], i, v[u]);
                    if (dd > best[q]) {
                        best[q] = dd;
                        bi[q] = i;
                    }
                }
            }
        }
#pragma unroll
        for (uint32_t q = 0; q < 2; ++q) {
            argmax_wave(&best[q], &bi[q]);
            if (lane == 0) {
                rd[q][wv] = best[q];
                ri[q][wv] = bi[q];
            }
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            SegPart part;
#pragma unroll
            for (uint32_t q = 0; q < 2; ++q) {
                double b = rd[q][0];
                uint32_t k = ri[q][0];
                for (uint32_t x = 1; x < SEGG_THREADS / 64; ++x)
                    if (rd[q][x] > b || (rd[q][x] == b && ri[q][x] < k)) {
                        b = rd[q][x];
                        k = ri[q][x];
                    }
                part.d[q] = b;
                part.i[q] = k;
            }
            w.segpart[(uint64_t)slot * SEG_GRID_BLOCKS + blockIdx.x] = part;
            __threadfence();
            last = atomicAdd(&ss.arrive, 1u) == G - 1u;
        }
        __syncthreads();
        if (last) {
            // the last block: every block's result, then the split, made on
            // an LDS copy of the tensor's runs
            __threadfence();
#pragma unroll
            for (uint32_t q = 0; q < 2; ++q) {
                double b = 0.0;
                uint32_t k = 0xffffffffu;
                if (threadIdx.x < G) {
                    const SegPart &pp = w.segpart[(uint64_t)slot * SEG_GRID_BLOCKS + threadIdx.x];
                    b = pp.d[q];
                    k = pp.i[q];
                }
                argmax_wave(&b, &k);
                if (lane == 0) {
                    rd[q][wv] = b;
                    ri[q][wv] = k;
                }
            }
            uint32_t *stw = w.bounds + td.in.bnd0;
            const uint32_t count = ss.count;
            for (uint32_t x = threadIdx.x; x <= count; x += SEGG_THREADS) lst[x] = stw[x];
            for (uint32_t x = threadIdx.x; x < count; x += SEGG_THREADS) {
                lcd[x] = ss.cd[x];
                lci[x] = ss.ci[x];
            }
            __syncthreads();
            if (threadIdx.x == 0) {
                for (uint32_t q = 0; q < np; ++q) {
                    double b = rd[q][0];
                    uint32_t k = ri[q][0];
                    for (uint32_t x = 1; x < SEGG_THREADS / 64; ++x)
                        if (rd[q][x] > b || (rd[q][x] == b && ri[q][x] < k)) {
                            b = rd[q][x];
                            k = ri[q][x];
                        }
                    lcd[p0 + q] = b;
                    lci[p0 + q] = b > 0.0 ? k : 0u;
                }
                // the run to split: farthest candidate, then the leftmost run
                double b = 0.0;
                uint32_t k = 0xffffffffu;
                for (uint32_t x = 0; x < count; ++x)
                    if (lcd[x] > b) {
                        b = lcd[x];
                        k = x;
                    }
                uint32_t nc = count;
                if (k != 0xffffffffu) {
                    // a start after run k: runs k+1.. move one place right
                    for (uint32_t x = count; x >= k + 1u; --x) lst[x + 1] = lst[x];
                    for (uint32_t x = count - 1u; x >= k + 1u && x < count; --x) {
                        lcd[x + 1] = lcd[x];
                        lci[x + 1] = lci[x];
                    }
                    lst[k + 1] = lci[k] + 1u;
                    nc = count + 1u;
                }
                s_nc = nc;
                s_done = k == 0xffffffffu || nc >= ss.req;  // no split left, or enough runs
                ss.count = nc;
                ss.done = s_done;
                ss.pend = k;
                ss.npend = 2;
                ss.arrive = 0;
            }
            __syncthreads();
            const uint32_t nc = s_nc;
            for (uint32_t x = threadIdx.x; x <= nc; x += SEGG_THREADS) stw[x] = lst[x];
            for (uint32_t x = threadIdx.x; x < nc; x += SEGG_THREADS) {
                ss.cd[x] = lcd[x];
                ss.ci[x] = lci[x];
            }
            if (s_done) seg_finish<SEGG_THREADS>(td, nc, true, lst);
        }
        __syncthreads();  // rd, ri and last are reused for the next tensor
    }
}

__global__ __launch_bounds__(SEG_THREADS) void k_segment(Work w) {
    TDesc &td = w.td[blockIdx.x];
    const bool chord = td.in.seg_mode == SEG_CHORD;
    const uint32_t n = td.nv;
    if ((!chord && td.in.nseg != 0) || n == 0) return;
    __shared__ uint32_t st[MAX_SEG + 1];  // run starts, st[count] = n
    __shared__ double cd[MAX_SEG];        // each run's farthest allowed split distance (0: none)
    __shared__ uint32_t ci[MAX_SEG];      // and the rank that would end its left part
    __shared__ double rd[SEG_THREADS / 64];
    __shared__ uint32_t ri[SEG_THREADS / 64];
    __shared__ uint32_t sh_req, sh_count, sh_pick;
    const uint32_t D = td.in.degree;
    const float *C = w.vsorted + td.in.slot;
    if (td.in.seg_slot != NO_SEG_SLOT) return;  // segmented over the grid, layout written
    if (threadIdx.x == 0) {
        const uint32_t req = td.in.nseg ? td.in.nseg : seg_heuristic(C, n, D);
        sh_req = req;
        uint32_t count = 1;
        st[0] = 0;
        st[1] = n;
        if (chord) {
            const uint32_t lo = sign_split(C, n);
            if (req >= 2 && lo >= D + 1 && n - lo >= D + 1) {
                st[1] = lo;
                st[2] = n;
                count = 2;
            }
        }
        sh_count = count;
    }
    __syncthreads();
    uint32_t count = sh_count;
    const uint32_t req = sh_req;
    if (chord) {
        for (uint32_t k = 0; k < count; ++k) {
            uint32_t i = 0;
            const double dd = seg_candidate(C, st[k], st[k + 1], D, &i, rd, ri);
            if (threadIdx.x == 0) {
                cd[k] = dd;
                ci[k] = i;
            }
        }
        __syncthreads();
        while (count < req) {
            // the run to split: farthest candidate, then the leftmost run
            double best = 0.0;
            uint32_t bk = 0xffffffffu;
            for (uint32_t k = threadIdx.x; k < count; k += SEG_THREADS)
                if (cd[k] > best) {
                    best = cd[k];
                    bk = k;
                }
            for (uint32_t off = 32; off > 0; off >>= 1) {
                const double od = __shfl_down(best, off);
                const uint32_t ok = __shfl_down(bk, off);
                if (od > best || (od == best && ok < bk)) {
                    best = od;
                    bk = ok;
                }
            }
            const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
            if (lane == 0) {
                rd[wv] = best;
                ri[wv] = bk;
            }
            __syncthreads();
            if (threadIdx.x == 0) {
                double b = rd[0];
                uint32_t k = ri[0];
                for (uint32_t q = 1; q < SEG_THREADS / 64; ++q)
                    if (rd[q] > b || (rd[q] == b && ri[q] < k)) {
                        b = rd[q];
                        k = ri[q];
                    }
                sh_pick = b > 0.0 ? k : 0xffffffffu;
            }
            __syncthreads();
            const uint32_t k = sh_pick;
            if (k == 0xffffffffu) break;
            // insert a start after run k: entries k+1..count move one place
            // right, in chunks from the top so that no chunk reads what
            // another has written
            for (int64_t top = count; top >= (int64_t)k + 1; top -= SEG_THREADS) {
                const int64_t xx = top - (int64_t)threadIdx.x;
                const bool mv = xx >= (int64_t)k + 1;
                uint32_t s_v = 0, c_i = 0;
                double c_d = 0.0;
                if (mv) {
                    s_v = st[xx];
                    if (xx < count) {
                        c_d = cd[xx];
                        c_i = ci[xx];
                    }
                }
                __syncthreads();
                if (mv) {
                    st[xx + 1] = s_v;
                    if (xx < count) {
                        cd[xx + 1] = c_d;
                        ci[xx + 1] = c_i;
                    }
                }
                __syncthreads();
            }
            if (threadIdx.x == 0) st[k + 1] = ci[k] + 1u;
            ++count;
            __syncthreads();
            for (uint32_t kk = k; kk <= k + 1; ++kk) {
                uint32_t i = 0;
                const double dd = seg_candidate(C, st[kk], st[kk + 1], D, &i, rd, ri);
                if (threadIdx.x == 0) {
                    cd[kk] = dd;
                    ci[kk] = i;
                }
            }
            __syncthreads();
        }
    }
    // the record's layout now that the run count is known
    const uint32_t seff = chord ? count : (req < max(1u, n / (D + 1u)) ? req : max(1u, n / (D + 1u)));
    if (chord)
        for (uint32_t x = threadIdx.x; x <= seff; x += SEG_THREADS) w.bounds[td.in.bnd0 + x] = st[x];
    seg_finish<SEG_THREADS>(td, seff, chord, st);
}

// grid_req: the most runs requested of a tensor with a state slot (0: none);
// block_pass: some tensor has no state slot and is segmented by k_segment
hipError_t launch_segment(const Work &w, uint32_t grid_req, bool block_pass, hipStream_t s) {
    if (grid_req > 0) {
        k_seg_init<<<w.ntensors, SEGG_THREADS, 0, s>>>(w);
        trace_mark(s, "k_seg_init");
        for (uint32_t q = 1; q < grid_req; ++q) {
            k_seg_step<<<SEG_GRID_BLOCKS, SEGG_THREADS, 0, s>>>(w);
            trace_mark(s, "k_seg_step");
        }
    }
    if (!block_pass) return hipGetLastError();
    k_segment<<<w.ntensors, SEG_THREADS, 0, s>>>(w);
    trace_mark(s, "k_segment");
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Least-squares fit of each run
// ---------------------------------------------------------------------------
// The double-exponential fit's state per run, after DEXP_PARTS x 15 partial
// sums in the run's share of the fit partials (FIT_CHUNKS x NMOM doubles,
// free once the polynomial fit has read them).
constexpr uint32_t DEXP_PARTS = 8;  // blocks per run and pass
struct DexpState {
    double th[4];    // current point (a, b, c, d)
    double tt[4];    // trial point
    double cur[15];  // sums at the current point
    double lambda;
    int it;          // steps taken
    uint32_t done;   // the fit has ended and the row is written
    uint32_t arrive; // blocks done with this pass
    uint32_t pad;
};
static_assert(DEXP_PARTS * 15 * 8 + sizeof(DexpState) <= FIT_CHUNKS * NMOM * 8, "state fits in the run's partials");
__device__ __forceinline__ DexpState *dexp_state(const Work &w, uint32_t run) {
    return (DexpState *)(w.fit_part + (uint64_t)run * FIT_CHUNKS * NMOM + DEXP_PARTS * 15);
}
// sorted ranks [lo, hi) of run s
__device__ __forceinline__ void run_range(const Work &w, const TDesc &td, uint32_t s, uint64_t *lo, uint64_t *hi) {
    if (td.in.seg_mode == SEG_CHORD) {
        *lo = w.bounds[td.in.bnd0 + s];
        *hi = w.bounds[td.in.bnd0 + s + 1];
    } else {
        const uint64_t nv = td.nv, S = td.seff;
        *lo = s * nv / S;
        *hi = (s + 1) * nv / S;
    }
}
__device__ __forceinline__ uint32_t tensor_of_fit_block(const Work &w, uint32_t b) {
    uint32_t lo = 0, hi = w.ntensors;
    while (hi - lo > 1) {
        uint32_t mid = (lo + hi) >> 1;
        if (w.td[mid].in.fit_blk0 <= b)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

// Moments of one chunk of a run: sums of t^e (e <= 2D) and t^e y (e <= D)
// over local ranks [j0, j1) of a run of ns points starting at lo_run.
// Each thread reads FIT_BATCH values before it uses any.  Blocks of four
// waves: beside the receiver's probe pass the launch has 32 CUs, and
// 1024-thread blocks (one per CU at 120 VGPRs) left them idle between
// rounds of blocks; at 256 threads (146 VGPRs, three blocks per CU) the
// launch took resnet50_25m 33 -> 22 us, vgg16_138m 73 -> 31 us and
// transformer_355m_x24 600 -> 391 us.  Long runs get fewer threads
// (FIT_CHUNKS blocks each): ncf_32m's launch went from 0.22 to 0.48 ms,
// inside the slack its sender's branch has beside the receiver's query.
constexpr uint32_t FIT_THREADS = 256;
constexpr uint32_t FIT_BATCH = 8;

// Chunks a run of ns points is cut into: at most FIT_CHUNKS, each at least
// a batch per thread.  A block reduces its 3 D + 2 sums over all its waves
// whatever its chunk's size, so many chunks of a short run would be mostly
// reductions.  The blocks of unused chunks write zero partials.
constexpr uint64_t FIT_MIN_CHUNK = (uint64_t)FIT_THREADS * FIT_BATCH;
__device__ __forceinline__ uint32_t fit_chunks(uint64_t ns) {
    const uint64_t c = (ns + FIT_MIN_CHUNK - 1) / FIT_MIN_CHUNK;
    return (uint32_t)(c < 1 ? 1 : (c > FIT_CHUNKS ? FIT_CHUNKS : c));
}

template <int D>
__device__ void fit_moments_body(const float *y, uint64_t lo_run, uint64_t ns, uint64_t j0, uint64_t j1,
                                 double *out) {
    constexpr int NP = 2 * D + 1;
    double pw[NP], rh[D + 1];
#pragma unroll
    for (int e = 0; e < NP; ++e) pw[e] = 0.0;
#pragma unroll
    for (int e = 0; e <= D; ++e) rh[e] = 0.0;
    const double inv = ns > 1 ? 1.0 / (double)(ns - 1) : 0.0;
    const double off = (double)(ns - 1);
    for (uint64_t jb = j0; jb < j1; jb += (uint64_t)FIT_THREADS * FIT_BATCH) {
        float v[FIT_BATCH];
#pragma unroll
        for (uint32_t u = 0; u < FIT_BATCH; ++u) {
            const uint64_t j = jb + (uint64_t)u * FIT_THREADS + threadIdx.x;
            v[u] = j < j1 ? y[lo_run + j] : 0.0f;
        }
        asm volatile("" ::: "memory");
#pragma unroll
        for (uint32_t u = 0; u < FIT_BATCH; ++u) {
            const uint64_t j = jb + (uint64_t)u * FIT_THREADS + threadIdx.x;
            if (j >= j1) break;
            const double t = ((double)(2 * j) - off) * inv;
            const double yv = (double)v[u];
            double tp = 1.0;
#pragma unroll
            for (int e = 0; e < NP; ++e) {
                pw[e] += tp;
                if (e <= D) rh[e] += tp * yv;
                tp *= t;
            }
        }
    }
    constexpr uint32_t NW = FIT_THREADS / 64;
    __shared__ double red[NW][NP + D + 1];
    const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
#pragma unroll
    for (int e = 0; e < NP; ++e) {
        const double s = wave_sum_f64(pw[e]);
        if (lane == 0) red[wv][e] = s;
    }
#pragma unroll
    for (int e = 0; e <= D; ++e) {
        const double s = wave_sum_f64(rh[e]);
        if (lane == 0) red[wv][NP + e] = s;
    }
    __syncthreads();
    if (threadIdx.x < (uint32_t)(NP + D + 1)) {
        double s = 0.0;
        for (uint32_t q = 0; q < NW; ++q) s += red[q][threadIdx.x];
        out[threadIdx.x < (uint32_t)NP ? threadIdx.x : (2 * MAX_DEG + 1) + (threadIdx.x - NP)] = s;
    }
}

__device__ void solve_run(const TDesc &td, uint32_t s, const double *mom);

__device__ void pack_sigma_words(const Work &w, uint32_t first, uint32_t stride);

// Moments of one chunk of one run (blocks [0, fit_blocks)); the blocks
// after them pack the reorder map, which needs only the sort.
__global__ __launch_bounds__(FIT_THREADS) void k_fit_moments(Work w, uint32_t fit_blocks) {
    if (blockIdx.x >= fit_blocks) {
        pack_sigma_words(w, (blockIdx.x - fit_blocks) * FIT_THREADS + threadIdx.x,
                         (gridDim.x - fit_blocks) * FIT_THREADS);
        return;
    }
    const uint32_t t = tensor_of_fit_block(w, blockIdx.x);
    const TDesc &td = w.td[t];
    const uint32_t local = blockIdx.x - td.in.fit_blk0;
    const uint32_t s = local / FIT_CHUNKS, ch = local % FIT_CHUNKS;
    if (s >= td.seff || td.model == FIT_DEXP) return;
    uint64_t lo, hi;
    run_range(w, td, s, &lo, &hi);
    const uint64_t ns = hi - lo;
    const uint32_t nch = fit_chunks(ns);
    double *out = w.fit_part + (uint64_t)blockIdx.x * NMOM;
    if (ch >= nch) {  // block-uniform: the run has fewer chunks; this one adds nothing
        if (threadIdx.x < NMOM) out[threadIdx.x] = 0.0;
        return;
    }
    const uint64_t j0 = ns * ch / nch, j1 = ns * (ch + 1) / nch;
    const float *y = w.vsorted + td.in.slot;
    switch (td.deff) {
        case 0: fit_moments_body<0>(y, lo, ns, j0, j1, out); break;
        case 1: fit_moments_body<1>(y, lo, ns, j0, j1, out); break;
        case 2: fit_moments_body<2>(y, lo, ns, j0, j1, out); break;
        case 3: fit_moments_body<3>(y, lo, ns, j0, j1, out); break;
        case 4: fit_moments_body<4>(y, lo, ns, j0, j1, out); break;
        case 5: fit_moments_body<5>(y, lo, ns, j0, j1, out); break;
        case 6: fit_moments_body<6>(y, lo, ns, j0, j1, out); break;
        default: fit_moments_body<7>(y, lo, ns, j0, j1, out); break;
    }
}

// One run per block: its chunks' moments summed in chunk order, then the
// solve (one thread; the system is at most 8 x 8).  Caller-owned
// coefficient rows past the fitted runs are zeroed.
__global__ __launch_bounds__(64) void k_fit_solve(Work w) {
    const uint32_t blk = blockIdx.x * FIT_CHUNKS;
    const uint32_t t = tensor_of_fit_block(w, blk);
    const TDesc &td = w.td[t];
    const uint32_t s = (blk - td.in.fit_blk0) / FIT_CHUNKS;
    if (s >= td.seff) {
        if (td.in.coef && s < td.in.nseg && threadIdx.x < td.in.coef_stride)
            td.in.coef[(uint64_t)s * td.in.coef_stride + threadIdx.x] = 0.0f;
        return;
    }
    if (td.model == FIT_DEXP) {  // fitted by k_dexp_pass: its state starts cleared
        if (threadIdx.x < sizeof(DexpState) / 4)
            ((uint32_t *)dexp_state(w, blockIdx.x))[threadIdx.x] = 0u;
        return;
    }
    __shared__ double mom[NMOM];
    if (threadIdx.x < NMOM) {
        const double *part = w.fit_part + (uint64_t)blk * NMOM;
        double acc = 0.0;
        for (uint32_t c = 0; c < FIT_CHUNKS; ++c) acc += part[c * NMOM + threadIdx.x];
        mom[threadIdx.x] = acc;
    }
    __syncthreads();
    if (threadIdx.x == 0) solve_run(td, s, mom);
}

// Normal equations of degree D from the summed moments, solved by Gaussian
// elimination with partial pivoting; the system lives in registers.
template <int D>
__device__ void solve_normal(const double *mom, float *row) {
    constexpr int N = D + 1;
    double A[N][N + 1];
#pragma unroll
    for (int p = 0; p < N; ++p) {
#pragma unroll
        for (int q = 0; q < N; ++q) A[p][q] = mom[p + q];
        A[p][N] = mom[2 * MAX_DEG + 1 + p];
    }
    bool ok = true;
#pragma unroll
    for (int col = 0; col < N; ++col) {
        int piv = col;
#pragma unroll
        for (int r = col + 1; r < N; ++r)
            if (fabs(A[r][col]) > fabs(A[piv][col])) piv = r;
        if (A[piv][col] == 0.0) ok = false;
        // swap rows col and piv without dynamic register indexing
#pragma unroll
        for (int r = col + 1; r < N; ++r) {
            if (r == piv) {
#pragma unroll
                for (int c = 0; c <= N; ++c) {
                    const double tmp = A[col][c];
                    A[col][c] = A[r][c];
                    A[r][c] = tmp;
                }
            }
        }
        if (A[col][col] != 0.0) {
#pragma unroll
            for (int r = col + 1; r < N; ++r) {
                const double f = A[r][col] / A[col][col];
#pragma unroll
                for (int c = col; c <= N; ++c) A[r][c] -= f * A[col][c];
            }
        }
    }
    double x[N];
#pragma unroll
    for (int p = N - 1; p >= 0; --p) {
        double acc = A[p][N];
#pragma unroll
        for (int q = p + 1; q < N; ++q) acc -= A[p][q] * x[q];
        x[p] = ok ? acc / A[p][p] : 0.0;
    }
#pragma unroll
    for (int p = 0; p < N; ++p) row[p] = (float)x[p];
}

// Solve run s of a tensor and write its coefficient row (fp32).
__device__ void solve_run(const TDesc &td, uint32_t s, const double *mom) {
    const uint32_t D = td.deff, N = D + 1;
    float *row;
    if (td.in.coef) {
        row = td.in.coef + (uint64_t)s * td.in.coef_stride;
        for (uint32_t p = N; p < td.in.coef_stride; ++p) row[p] = 0.0f;
    } else {
        row = (float *)(td.in.rec + td.coef_off) + (uint64_t)s * N;
    }
    double m[NMOM];
    for (uint32_t e = 0; e < NMOM; ++e) m[e] = mom[e];
    switch (D) {
        case 0: solve_normal<0>(m, row); break;
        case 1: solve_normal<1>(m, row); break;
        case 2: solve_normal<2>(m, row); break;
        case 3: solve_normal<3>(m, row); break;
        case 4: solve_normal<4>(m, row); break;
        case 5: solve_normal<5>(m, row); break;
        case 6: solve_normal<6>(m, row); break;
        default: solve_normal<7>(m, row); break;
    }
}

// ---------------------------------------------------------------------------
// Double-exponential fit (Section 5, "Nonlinear regression"):
// Levenberg-Marquardt on y ~ a e^(bt) + c e^(dt) with the same steps as the
// oracle (start at rates (1, -1) with the amplitudes of the linear problem;
// DEXP_ITERS steps, rates clamped to [-40, 40], lambda from 1e-3, x10 on a
// reject, /10 on an accept).  Each step is one pass over the run: the 15
// sums of J^T J, J^T r and r^T r at the trial point.  A pass is one launch
// of k_dexp_pass, with DEXP_PARTS blocks per run; each block sums its part
// of the run and the last block to finish (a counter) adds the parts in a
// fixed order, takes the step's decision and solves the 4 x 4 system for
// the next trial point.  The solver's state stays in the run's share of
// the fit partials, which the polynomial fit no longer needs.  A thread
// takes a contiguous range of points: the abscissae are equally spaced, so
// e^(b t) advances by one multiplication per point from one exp() at the
// range's start (relative drift ~1e-15 over a range, far below the fit's
// tolerance).
// ---------------------------------------------------------------------------
constexpr uint32_t DEXP_THREADS = 256;
constexpr int DEXP_ITERS = 40;
constexpr uint32_t DEXP_BATCH = 8;
constexpr double DEXP_RATE_MAX = 40.0;

// sums over the block, in wave order, into tot[0..N) (LDS); the block is
// synchronised on return
template <int N>
__device__ void block_sums(const double *v, double (*red)[15], double *tot) {
    const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
#pragma unroll
    for (int e = 0; e < N; ++e) {
        const double sm = wave_sum_f64(v[e]);
        if (lane == 0) red[wv][e] = sm;
    }
    __syncthreads();
    if (threadIdx.x < (uint32_t)N) {
        double acc = 0.0;
        for (uint32_t q = 0; q < DEXP_THREADS / 64; ++q) acc += red[q][threadIdx.x];
        tot[threadIdx.x] = acc;
    }
    __syncthreads();
}

// solve A x = rhs (4 x 4, augmented) by elimination with partial pivoting;
// false if a pivot is zero
// (every index is a compile-time constant once unrolled, so A stays in
// registers: the pivot row is swapped in by selects)
__device__ __forceinline__ bool solve4(double A[4][5], double *x) {
#pragma unroll
    for (int col = 0; col < 4; ++col) {
        int piv = col;
        double best = fabs(A[col][col]);
#pragma unroll
        for (int row = col + 1; row < 4; ++row)
            if (fabs(A[row][col]) > best) {
                best = fabs(A[row][col]);
                piv = row;
            }
        if (best == 0.0) return false;
#pragma unroll
        for (int row = col + 1; row < 4; ++row) {
            const bool sw = row == piv;
#pragma unroll
            for (int c = 0; c <= 4; ++c) {
                const double a = A[col][c], b = A[row][c];
                A[col][c] = sw ? b : a;
                A[row][c] = sw ? a : b;
            }
        }
#pragma unroll
        for (int row = col + 1; row < 4; ++row) {
            const double f = A[row][col] / A[col][col];
#pragma unroll
            for (int c = col; c <= 4; ++c) A[row][c] -= f * A[col][c];
        }
    }
#pragma unroll
    for (int p = 3; p >= 0; --p) {
        double s = A[p][4];
#pragma unroll
        for (int q = p + 1; q < 4; ++q) s -= A[p][q] * x[q];
        x[p] = s / A[p][p];
    }
    return true;
}

// one pass over block `part`'s share of run [lo, lo + ns) at (a, b, c, dd):
// init: the 6 sums of the linear start; else the 15 sums of the step
__device__ void dexp_part_sums(const float *y, uint64_t ns, uint32_t part, bool init, const double th[4],
                               double (*red)[15], double *tot) {
    const double inv = ns > 1 ? 1.0 / (double)(ns - 1) : 0.0;
    const double off = (double)(ns - 1);
    const double step = 2.0 * inv;
    const uint64_t b0 = ns * part / DEXP_PARTS, b1 = ns * (part + 1) / DEXP_PARTS;
    const uint64_t per = (b1 - b0 + DEXP_THREADS - 1) / DEXP_THREADS;
    const uint64_t j0 = min(b1, b0 + threadIdx.x * per), j1 = min(b1, j0 + per);
    double v[15];
#pragma unroll
    for (int e = 0; e < 15; ++e) v[e] = 0.0;
    if (init) {
        if (j0 < j1) {
            const double t0 = ((double)(2 * j0) - off) * inv;
            double e1 = exp(t0), e2 = exp(-t0);
            const double r1 = exp(step), r2 = exp(-step);
            for (uint64_t jb = j0; jb < j1; jb += DEXP_BATCH) {
                float yv[DEXP_BATCH];
#pragma unroll
                for (uint32_t u = 0; u < DEXP_BATCH; ++u) yv[u] = jb + u < j1 ? y[jb + u] : 0.0f;
#pragma unroll
                for (uint32_t u = 0; u < DEXP_BATCH; ++u) {
                    if (jb + u >= j1) break;
                    const double yj = (double)yv[u];
                    v[0] += e1 * e1;
                    v[1] += e1 * e2;
                    v[2] += e2 * e2;
                    v[3] += yj * e1;
                    v[4] += yj * e2;
                    v[5] += yj;
                    e1 *= r1;
                    e2 *= r2;
                }
            }
        }
        block_sums<6>(v, red, tot);
        return;
    }
    const double a = th[0], b = th[1], c = th[2], dd = th[3];
    if (j0 < j1) {
        const double t0 = ((double)(2 * j0) - off) * inv;
        double eb = exp(b * t0), ed = exp(dd * t0);
        const double rb = exp(b * step), rd = exp(dd * step);
        for (uint64_t jb = j0; jb < j1; jb += DEXP_BATCH) {
            float yv[DEXP_BATCH];
#pragma unroll
            for (uint32_t u = 0; u < DEXP_BATCH; ++u) yv[u] = jb + u < j1 ? y[jb + u] : 0.0f;
#pragma unroll
            for (uint32_t u = 0; u < DEXP_BATCH; ++u) {
                const uint64_t j = jb + u;
                if (j >= j1) break;
                const double tj = ((double)(2 * j) - off) * inv, yj = (double)yv[u];
                const double J[4] = {eb, a * tj * eb, ed, c * tj * ed};
                const double r = yj - (a * eb + c * ed);
                int e = 0;
#pragma unroll
                for (int p = 0; p < 4; ++p)
#pragma unroll
                    for (int q = p; q < 4; ++q) v[e++] += J[p] * J[q];
#pragma unroll
                for (int p = 0; p < 4; ++p) v[10 + p] += J[p] * r;
                v[14] += r * r;
                eb *= rb;
                ed *= rd;
            }
        }
    }
    block_sums<15>(v, red, tot);
}

// Pass `pass` of every double-exponential run: 0 sums the linear start,
// 1 evaluates the start, each later pass a trial point.  Launched
// 2 + DEXP_ITERS times; a run whose fit has ended returns at once.
__global__ __launch_bounds__(DEXP_THREADS) void k_dexp_pass(Work w, uint32_t pass) {
    const uint32_t run = blockIdx.x / DEXP_PARTS, part = blockIdx.x % DEXP_PARTS;
    const uint32_t blk = run * FIT_CHUNKS;
    const uint32_t t = tensor_of_fit_block(w, blk);
    const TDesc &td = w.td[t];
    const uint32_t s = (blk - td.in.fit_blk0) / FIT_CHUNKS;
    if (td.model != FIT_DEXP || s >= td.seff) return;
    DexpState &st = *dexp_state(w, run);
    if (st.done) return;
    __shared__ double red[DEXP_THREADS / 64][15];
    __shared__ double tot[15];
    __shared__ uint32_t last;
    uint64_t lo, hi;
    run_range(w, td, s, &lo, &hi);
    const uint64_t ns = hi - lo;
    const float *y = w.vsorted + td.in.slot + lo;
    double th[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) th[p] = st.tt[p];
    dexp_part_sums(y, ns, part, pass == 0, th, red, tot);
    double *parts = w.fit_part + (uint64_t)blk * NMOM;  // DEXP_PARTS x 15 sums
    if (threadIdx.x < 15) parts[part * 15 + threadIdx.x] = tot[threadIdx.x];
    __syncthreads();
    if (threadIdx.x == 0) {
        __threadfence();
        last = atomicAdd(&st.arrive, 1u) == DEXP_PARTS - 1u;
    }
    __syncthreads();
    if (!last) return;
    // the last block: the run's sums (parts in order) and the solver's state
    // into LDS, read in parallel; then thread 0 takes the step's decision
    __threadfence();
    __shared__ double sum[15], cur[15], sth[4], stt[4], slam;
    __shared__ int sit;
    if (threadIdx.x < 15) {
        double acc = 0.0;
        for (uint32_t q = 0; q < DEXP_PARTS; ++q) acc += parts[q * 15 + threadIdx.x];
        sum[threadIdx.x] = acc;
        cur[threadIdx.x] = st.cur[threadIdx.x];
    } else if (threadIdx.x < 19) {
        sth[threadIdx.x - 15] = st.th[threadIdx.x - 15];
        stt[threadIdx.x - 15] = st.tt[threadIdx.x - 15];
    } else if (threadIdx.x == 19) {
        slam = st.lambda;
        sit = st.it;
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    st.arrive = 0;
    if (pass == 0) {
        // start: rates (1, -1), amplitudes from the 2 x 2 linear problem
        const double det = sum[0] * sum[2] - sum[1] * sum[1];
        double th0, th2;
        if (det != 0.0) {
            th0 = (sum[3] * sum[2] - sum[4] * sum[1]) / det;
            th2 = (sum[4] * sum[0] - sum[3] * sum[1]) / det;
        } else {
            th0 = sum[5] / (double)ns;
            th2 = 0.0;
        }
        const double th4[4] = {th0, 1.0, th2, -1.0};
        for (int p = 0; p < 4; ++p) {
            st.th[p] = th4[p];
            st.tt[p] = th4[p];
        }
        st.lambda = 1e-3;
        st.it = 0;
        return;
    }
    double lambda = slam;
    if (pass == 1) {
        for (int e = 0; e < 15; ++e) cur[e] = sum[e];
    } else if (sum[14] < cur[14]) {
        for (int p = 0; p < 4; ++p) sth[p] = stt[p];
        for (int e = 0; e < 15; ++e) cur[e] = sum[e];
        lambda /= 10.0;
    } else {
        lambda *= 10.0;
    }
    // the next trial point; a singular system uses up a step
    int it = sit;
    bool go = false;
    while (it < DEXP_ITERS) {
        ++it;
        double A[4][5];
        int e = 0;
        for (int p = 0; p < 4; ++p)
            for (int q = p; q < 4; ++q) {
                A[p][q] = cur[e];
                A[q][p] = cur[e];
                ++e;
            }
        for (int p = 0; p < 4; ++p) {
            A[p][p] += lambda * A[p][p];
            A[p][4] = cur[10 + p];
        }
        double delta[4];
        if (!solve4(A, delta)) {
            lambda *= 10.0;
            continue;
        }
        for (int p = 0; p < 4; ++p) stt[p] = sth[p] + delta[p];
        for (int p = 1; p < 4; p += 2)
            stt[p] = stt[p] > DEXP_RATE_MAX ? DEXP_RATE_MAX : (stt[p] < -DEXP_RATE_MAX ? -DEXP_RATE_MAX : stt[p]);
        go = true;
        break;
    }
    for (int p = 0; p < 4; ++p) {
        st.th[p] = sth[p];
        st.tt[p] = stt[p];
    }
    for (int e = 0; e < 15; ++e) st.cur[e] = cur[e];
    st.lambda = lambda;
    st.it = it;
    if (!go) {
        // the fit has ended: the run's row
        st.done = 1;
        float *row = td.in.coef ? td.in.coef + (uint64_t)s * td.in.coef_stride
                                : (float *)(td.in.rec + td.coef_off) + (uint64_t)s * 4u;
        for (int p = 0; p < 4; ++p) row[p] = (float)sth[p];
    }
}

hipError_t launch_fit(const Work &w, uint32_t fit_blocks, uint64_t vals_est, bool dexp, hipStream_t s) {
    // the fit's chunk blocks, then blocks packing the reorder maps: one per
    // PACK_PER_BLOCK of the values the plan expects (each takes at most 32
    // bits, so as many words), at least 8 and at most 512.  Sized by the
    // work's slots instead (one per 32 Ki, at most 1024), resnet50_25m
    // launched 780 blocks for 166 K words; with the words found by a cursor
    // instead of a search per word, ncf_32m's launch went from 0.45 to 0.25 ms.
    // (At most 512 Ki threads instead of 512 blocks, as many threads as
    // before the fit's blocks shrank to 256, changed no workload's step.)
    constexpr uint64_t PACK_PER_BLOCK = 4ull * FIT_THREADS;
    const uint32_t pack_blocks =
        (uint32_t)std::min<uint64_t>(512, std::max<uint64_t>(8, (vals_est + PACK_PER_BLOCK - 1) / PACK_PER_BLOCK));
    k_fit_moments<<<fit_blocks + pack_blocks, FIT_THREADS, 0, s>>>(w, fit_blocks);
    trace_mark(s, "k_fit_moments");
    if (fit_blocks == 0) return hipGetLastError();
    k_fit_solve<<<fit_blocks / FIT_CHUNKS, 64, 0, s>>>(w);
    trace_mark(s, "k_fit_solve");
    if (dexp) {
        for (uint32_t pass = 0; pass < 2u + (uint32_t)DEXP_ITERS; ++pass) {
            k_dexp_pass<<<(fit_blocks / FIT_CHUNKS) * DEXP_PARTS, DEXP_THREADS, 0, s>>>(w, pass);
            trace_mark(s, "k_dexp_pass");
        }
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Reorder map packing: each output word gathers the entries it overlaps.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t tensor_of_sword(const Work &w, uint32_t g) {
    uint32_t lo = 0, hi = w.ntensors;
    while (hi - lo > 1) {
        uint32_t mid = (lo + hi) >> 1;
        if (w.td[mid].sw0 <= g)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

// Words first, first + stride, ... of the reorder maps of all tensors.  A
// thread's words ascend, so its tensor only moves forward: the tensor's
// fields are read when it changes, not per word.  Words of a tensor with
// b >= 16 overlap at most three entries; four such words have all their
// entries' reads in flight together.
__device__ void pack_sigma_words(const Work &w, uint32_t first, uint32_t stride) {
    constexpr uint32_t U = 4;
    const uint32_t total = w.glob->sigma_words;
    if (first >= total) return;
    uint32_t t = tensor_of_sword(w, first);
    uint32_t sw0 = 0, swn = 0, b = 0, nv = 0;
    const uint32_t *sg = nullptr;
    uint32_t *out = nullptr;
    auto enter = [&]() {  // tensor t's fields
        const TDesc &td = w.td[t];
        sw0 = td.sw0;
        swn = t + 1 < w.ntensors ? w.td[t + 1].sw0 : total;
        b = td.b;
        nv = td.nv;
        sg = w.sig + td.in.slot;
        out = td.in.sigma ? td.in.sigma : (uint32_t *)(td.in.rec + td.sigma_off);
    };
    enter();
    // floor(bit0 / b) in double: exact, since bit0 < 2^53 and a quotient that
    // is not an integer lies at least 1/b from one
    auto first_entry = [&](uint64_t bit0) { return (uint64_t)floor((double)bit0 / (double)b); };
    // one word from its entries qa..qb, all read here
    auto word_of = [&](uint32_t wl) {
        const uint64_t bit0 = (uint64_t)wl * 32u;
        const uint64_t qa = first_entry(bit0);
        uint64_t qb = first_entry(bit0 + 31u);
        if (qb > nv - 1u) qb = nv - 1u;
        uint32_t v = 0;
        for (uint64_t q = qa; q <= qb; ++q) {
            const int64_t sh = (int64_t)(q * b) - (int64_t)bit0;
            const uint64_t e = sg[q];
            v |= sh >= 0 ? (uint32_t)(e << sh) : (uint32_t)(e >> (-sh));
        }
        return v;
    };
    for (uint32_t g0 = first; g0 < total; g0 += U * stride) {
        while (g0 >= swn) {  // the thread's next word lies in a later tensor
            ++t;
            enter();
        }
        const uint32_t glast = (uint32_t)min<uint64_t>((uint64_t)g0 + (U - 1) * (uint64_t)stride, total - 1u);
        if (glast < swn && b >= 16u) {
            // U words of tensor t (the last ones may lie past the maps' end)
            uint32_t e[U][3], wl[U];
            int32_t sh[U];
#pragma unroll
            for (uint32_t u = 0; u < U; ++u) {
                const uint64_t gw = (uint64_t)g0 + u * (uint64_t)stride;
                wl[u] = gw < total ? (uint32_t)(gw - sw0) : 0u;
                const uint64_t bit0 = (uint64_t)wl[u] * 32u;
                const uint64_t qa = first_entry(bit0);
                sh[u] = (int32_t)((int64_t)(qa * b) - (int64_t)bit0);  // in (-b, 0]
#pragma unroll
                for (uint32_t k = 0; k < 3; ++k) {
                    // an entry past the map's last is 0 (the last word's
                    // bits past the map are clear)
                    const bool in = gw < total && qa + k < nv;
                    const uint32_t x = sg[in ? qa + k : 0u];
                    e[u][k] = in ? x : 0u;
                }
            }
#pragma unroll
            for (uint32_t u = 0; u < U; ++u) {
                if ((uint64_t)g0 + u * (uint64_t)stride >= total) break;
                const int32_t s0 = sh[u];
                uint32_t v = (uint32_t)(e[u][0] >> (uint32_t)(-s0));
                const int32_t s1 = s0 + (int32_t)b, s2 = s1 + (int32_t)b;
                v |= s1 < 32 ? e[u][1] << (uint32_t)s1 : 0u;
                v |= s2 < 32 ? e[u][2] << (uint32_t)s2 : 0u;
                out[wl[u]] = v;
            }
        } else {
            for (uint32_t u = 0; u < U; ++u) {
                const uint64_t gw = (uint64_t)g0 + u * (uint64_t)stride;
                if (gw >= total) break;
                while (gw >= swn) {
                    ++t;
                    enter();
                }
                out[gw - sw0] = word_of((uint32_t)(gw - sw0));
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Standalone value decode: sigma and coefficients in the caller's layout
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NTHREADS) void k_curvefit_decode(Work w, const float *__restrict__ coef,
                                                              const uint32_t *__restrict__ sigma,
                                                              const uint64_t *n, uint64_t n_cap,
                                                              float *__restrict__ out, uint64_t *flags_out) {
    const TDesc &td = w.td[0];
    const uint64_t n64 = *n;
    const uint32_t nv = (uint32_t)(n64 < n_cap ? n64 : n_cap);
    if (flags_out && blockIdx.x == 0 && threadIdx.x == 0) *flags_out = n64 > n_cap ? FLAG_CAPACITY : 0u;
    uint32_t seff, deff;
    fit_shape(nv, td.in.degree, td.in.nseg, &seff, &deff);
    const uint32_t b = sigma_bits(nv);
    const uint32_t stride = td.in.degree + 1u;
    for (uint32_t q = blockIdx.x * NTHREADS + threadIdx.x; q < nv; q += gridDim.x * NTHREADS) {
        const uint64_t bit = (uint64_t)q * b;
        const uint32_t w0 = sigma[bit >> 5], sh = (uint32_t)(bit & 31u);
        uint64_t v = w0 >> sh;
        if (sh + b > 32u) v |= (uint64_t)sigma[(bit >> 5) + 1] << (32u - sh);
        const uint32_t rank = (uint32_t)(v & ((1ull << b) - 1ull));
        float y = __uint_as_float(0x7fc00000u);  // NaN for an out-of-range rank
        if (rank < nv) {
            uint32_t s, lo, ns;
            run_of_rank(rank, nv, seff, &s, &lo, &ns);
            y = horner(coef + (uint64_t)s * stride, deff, abscissa(rank - lo, ns));
        }
        out[q] = y;
    }
}

hipError_t launch_curvefit_decode(const Work &w, const float *coef, const uint32_t *sigma, const uint64_t *n,
                                  uint64_t n_cap, float *vals_out, uint64_t *flags_out, int grid_persist,
                                  hipStream_t s) {
    k_curvefit_decode<<<grid_persist, NTHREADS, 0, s>>>(w, coef, sigma, n, n_cap, vals_out, flags_out);
    trace_mark(s, "k_curvefit_decode");
    return hipGetLastError();
}

__global__ void k_import_n(Work w, const uint64_t *n, uint64_t n_cap, uint64_t *flags_out) {
    const uint64_t v = *n;
    w.td[0].n = (uint32_t)(v < n_cap ? v : n_cap);
    if (v > n_cap) w.td[0].flags |= FLAG_CAPACITY;
    if (flags_out) *flags_out = v > n_cap ? FLAG_CAPACITY : 0u;
}

__global__ void k_export_n(Work w, uint64_t *n_out, int field) {
    const TDesc &td = w.td[0];
    *n_out = field == 0 ? td.n : td.nv;
}

hipError_t launch_import_n(const Work &w, const uint64_t *n, uint64_t n_cap, uint64_t *flags_out, hipStream_t s) {
    k_import_n<<<1, 1, 0, s>>>(w, n, n_cap, flags_out);
    trace_mark(s, "k_import_n");
    return hipGetLastError();
}

hipError_t launch_export_n(const Work &w, uint64_t *n_out, int field, hipStream_t s) {
    k_export_n<<<1, 1, 0, s>>>(w, n_out, field);
    trace_mark(s, "k_export_n");
    return hipGetLastError();
}

}  // namespace dr
