// select.hip -- set-up, top-r and support selection, and ordered compaction
// of the selection bitmap into index lists.
//
// Top-r (Section 2 "Sparsification"; Section 10.2: the r entries of largest
// magnitude, ties to the smaller index) is an exact radix select on the
// 31-bit magnitude key (IEEE bits with the sign cleared):
//   1. histogram of key bits 30..20 over the tensor (per-block partial
//      histograms, reduced without global atomics), pick the bin b1 that
//      holds the r-th largest key;
//   2. one pass over the tensor marks every element above b1 in the
//      selection bitmap (the d-bit string B of Section 3) and compacts the
//      elements of bin b1 into an index-ordered candidate list;
//   3. one block per tensor finishes the select on the candidates' low 20
//      key bits and resolves ties at the threshold by index order.
// The support of an inherently sparse gradient (Section 3) is the bitmap of
// nonzeros, written by the same pass.
#include "launch.hpp"

namespace dr {

__global__ __launch_bounds__(NTHREADS) void k_init(Work w, InitArgs a) {
    uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= a.count) return;
    TDesc &t = w.td[a.first + i];
    t.in = a.t[i];
    t.n = 0;
    t.m_words = 0;
    t.nv = 0;
    t.nv_dec = 0;
    t.seff = 0;
    t.deff = 0;
    t.b = 0;
    t.flags = 0;
    t.b1 = 0;
    t.need1 = 0;
    t.ncand = 0;
    t.T = 0;
    t.needT = 0;
    t.ntie = 0;
    t.idx_star = 0;
    t.stile0 = 0;
    t.sntiles = 0;
    t.sw0 = 0;
    t.swords = 0;
    t.coef_off = 0;
    t.sigma_off = 0;
    t.rec_bytes = 0;
}

__global__ __launch_bounds__(NTHREADS) void k_zero(ZeroArgs a) {
    uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint32_t r = 0; r < a.n; ++r) {
        uint32_t *p = (uint32_t *)a.z[r].p;
        for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < a.z[r].words; i += stride) p[i] = 0u;
    }
}

hipError_t launch_init(const Work &w, const InitArgs &a, hipStream_t s) {
    k_init<<<1, INIT_CHUNK <= NTHREADS ? NTHREADS : INIT_CHUNK, 0, s>>>(w, a);
    return hipGetLastError();
}

hipError_t launch_zero(const ZeroArgs &a, hipStream_t s) {
    k_zero<<<1024, NTHREADS, 0, s>>>(a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// top-r step 1: first-digit histogram
// ---------------------------------------------------------------------------

// histogram block -> tensor (hb0 ascending over top-r tensors)
__device__ __forceinline__ int tensor_of_hist_block(const Work &w, uint32_t b) {
    uint32_t lo = 0, hi = w.ntensors;
    while (hi - lo > 1) {
        uint32_t mid = (lo + hi) >> 1;
        if (w.td[mid].in.hb0 <= b)
            lo = mid;
        else
            hi = mid;
    }
    const TInit &in = w.td[lo].in;
    if (in.hbn == 0 || b < in.hb0 || b >= in.hb0 + in.hbn) return -1;
    return (int)lo;
}

__global__ __launch_bounds__(NTHREADS) void k_topr_hist(Work w, const float *__restrict__ g) {
    __shared__ uint32_t h[HIST1_BINS];
    __shared__ uint32_t bad;
    for (uint32_t i = threadIdx.x; i < HIST1_BINS; i += NTHREADS) h[i] = 0;
    if (threadIdx.x == 0) bad = 0;
    __syncthreads();
    const int t = tensor_of_hist_block(w, blockIdx.x);
    if (t < 0) return;
    const TInit &in = w.td[t].in;
    const uint32_t lb = blockIdx.x - in.hb0;
    const uint64_t span = (uint64_t)((in.ntiles + in.hbn - 1) / in.hbn) * TILE;
    const uint64_t lo = lb * span;
    const uint64_t hi = lo + span < in.d ? lo + span : in.d;
    const float *gt = g + in.off;
    uint32_t nonfinite = 0;
    for (uint64_t i = lo + threadIdx.x; i < hi; i += NTHREADS) {
        uint32_t key = mag_key(gt[i]);
        nonfinite |= key >= 0x7f800000u;
        atomicAdd(&h[key >> HIST1_SHIFT], 1u);
    }
    if (nonfinite) bad = 1;
    __syncthreads();
    uint32_t *out = w.hist_part + (uint64_t)blockIdx.x * HIST1_BINS;
    for (uint32_t i = threadIdx.x; i < HIST1_BINS; i += NTHREADS) out[i] = h[i];
    if (threadIdx.x == 0 && bad) atomicOr(&w.td[t].flags, FLAG_NONFINITE);
}

// Find, scanning bins from the top, the bin where the running count reaches
// `need` (1 <= need <= total).  `cnt(i)` is the count of bin i; bins
// [0, nbins), one bin per thread or several.  Returns the bin and the count
// strictly above it.  Block-wide; all threads get the result.
template <uint32_t NB, uint32_t NT>
__device__ void find_from_top(const uint32_t *cnt, uint32_t need, uint32_t *res_bin, uint32_t *res_above,
                              uint32_t *scratch /* NT/64 + 1 */) {
    constexpr uint32_t PER = NB / NT;  // bins per thread, taken from the top
    const uint32_t tid = threadIdx.x;
    uint32_t sum = 0;
#pragma unroll
    for (uint32_t q = 0; q < PER; ++q) sum += cnt[NB - 1 - (tid * PER + q)];
    // exclusive scan over threads (descending bins)
    const uint32_t lane = tid & 63u, wv = tid >> 6;
    uint32_t inc = wave_incl_scan(sum);
    if (lane == 63) scratch[wv] = inc;
    __syncthreads();
    if (tid == 0) {
        uint32_t s = 0;
        for (uint32_t i = 0; i < NT / 64; ++i) {
            uint32_t x = scratch[i];
            scratch[i] = s;
            s += x;
        }
    }
    __syncthreads();
    uint32_t excl = scratch[wv] + inc - sum;
    if (excl < need && need <= excl + sum) {
        uint32_t run = excl;
        for (uint32_t q = 0; q < PER; ++q) {
            uint32_t bin = NB - 1 - (tid * PER + q);
            uint32_t c = cnt[bin];
            if (run + c >= need) {
                *res_bin = bin;
                *res_above = run;
                break;
            }
            run += c;
        }
    }
    __syncthreads();
}

// Sum the partial histograms; the last block of each tensor picks b1.
__global__ __launch_bounds__(NTHREADS) void k_topr_reduce(Work w) {
    const uint32_t t = blockIdx.x / (HIST1_BINS / NTHREADS);
    const uint32_t part = blockIdx.x % (HIST1_BINS / NTHREADS);
    TDesc &td = w.td[t];
    if (td.in.r == R_NONZERO) return;
    const uint32_t bin = part * NTHREADS + threadIdx.x;
    uint32_t s = 0;
    for (uint32_t q = 0; q < td.in.hbn; ++q) s += w.hist_part[(uint64_t)(td.in.hb0 + q) * HIST1_BINS + bin];
    uint32_t *hist = w.hist + (uint64_t)t * HIST1_BINS;
    hist[bin] = s;
    __threadfence();
    __shared__ uint32_t ticket, res_bin, res_above;
    __shared__ uint32_t scratch[NWAVES + 1];
    __syncthreads();
    if (threadIdx.x == 0) ticket = atomicAdd(&w.done[t], 1u);
    __syncthreads();
    if (ticket != HIST1_BINS / NTHREADS - 1) return;
    __threadfence();
    const uint32_t r = td.in.r;
    if (r == 0) {
        if (threadIdx.x == 0) {
            td.b1 = HIST1_BINS;  // nothing above, nothing in the bin
            td.need1 = 0;
            td.ncand = 0;
        }
        return;
    }
    if (threadIdx.x == 0) {
        res_bin = 0;
        res_above = 0;
    }
    __syncthreads();
    find_from_top<HIST1_BINS, NTHREADS>(hist, r, &res_bin, &res_above, scratch);
    if (threadIdx.x == 0) {
        td.b1 = res_bin;
        td.need1 = r - res_above;
        td.ncand = hist[res_bin];
    }
}

// ---------------------------------------------------------------------------
// top-r step 2 / support: bitmap of definite selections + ordered candidates
// ---------------------------------------------------------------------------
// Elements of a tile are visited as e = j * 256 + threadIdx.x (j = 0..15):
// each load instruction reads 256 consecutive floats, and one wave ballot
// covers 64 consecutive elements, i.e. two whole bitmap words.
__global__ __launch_bounds__(NTHREADS) void k_select_filter(Work w, const float *__restrict__ g) {
    __shared__ uint32_t tkt;
    __shared__ uint32_t wcnt[16 * NWAVES];
    __shared__ uint32_t woff[16 * NWAVES];
    __shared__ uint32_t tile_excl, bad;
    const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
    if (threadIdx.x == 0) bad = 0;
    for (;;) {
        const uint32_t tile = next_ticket(&w.tickets[0], &tkt);
        if (tile >= w.ntiles_total) break;
        const uint32_t t = tensor_of_tile(w.td, w.ntensors, tile);
        TDesc &td = w.td[t];
        const uint32_t lt = tile - td.in.tile0;
        const uint32_t base = lt * TILE;
        const bool nz = td.in.r == R_NONZERO;
        const uint32_t b1 = nz ? 0u : td.b1;
        const float *gt = g + td.in.off;
        uint32_t keys[16];
        uint64_t cmask[16];
        uint32_t nonfinite = 0;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const uint32_t i = base + j * NTHREADS + threadIdx.x;
            const bool valid = i < td.in.d;
            const uint32_t key = valid ? mag_key(gt[i]) : 0u;
            nonfinite |= key >= 0x7f800000u;
            const uint32_t bin = key >> HIST1_SHIFT;
            const bool def = valid && (nz ? key != 0u : bin > b1);
            const bool cand = valid && !nz && bin == b1;
            const uint64_t dm = ballot(def);
            cmask[j] = ballot(cand);
            keys[j] = key;
            if (lane == 0 || lane == 32) {
                const uint32_t word = (uint32_t)((td.in.slot + base + j * NTHREADS + wv * 64 + lane) >> 5);
                w.selbits[word] = lane == 0 ? (uint32_t)dm : (uint32_t)(dm >> 32);
            }
            if (lane == 0) wcnt[j * NWAVES + wv] = popc64(cmask[j]);
        }
        if (nonfinite) bad = 1;
        __syncthreads();
        if (threadIdx.x < 64) {
            // (j, wave) counts in element order -> exclusive offsets
            uint32_t c = wcnt[threadIdx.x];
            uint32_t inc = wave_incl_scan(c);
            woff[threadIdx.x] = inc - c;
            if (threadIdx.x == 63) tile_excl = (uint32_t)lookback(w.lb0, tile, td.in.tile0, inc);
        }
        __syncthreads();
        if (threadIdx.x == 0 && bad) {
            atomicOr(&td.flags, FLAG_NONFINITE);
            bad = 0;
        }
        const uint64_t cbase = td.in.slot + tile_excl;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            if ((cmask[j] >> lane) & 1ull) {
                const uint64_t q = cbase + woff[j * NWAVES + wv] + lanes_below(cmask[j]);
                w.cand_key[q] = keys[j];
                w.cand_idx[q] = base + j * NTHREADS + threadIdx.x;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// top-r step 3: exact select among the candidates, one block per tensor
// ---------------------------------------------------------------------------
constexpr uint32_t SEL_THREADS = 1024;

__global__ __launch_bounds__(SEL_THREADS) void k_topr_select(Work w) {
    TDesc &td = w.td[blockIdx.x];
    if (td.in.r == R_NONZERO || td.ncand == 0) return;
    __shared__ uint32_t h[1024];
    __shared__ uint32_t scratch[SEL_THREADS / 64 + 1];
    __shared__ uint32_t res_bin, res_above, found, run_total;
    const uint32_t nc = td.ncand, need1 = td.need1;
    const uint32_t *ck = w.cand_key + td.in.slot;
    const uint32_t *ci = w.cand_idx + td.in.slot;
    uint32_t T, needT, ntie, idx_star = 0xFFFFFFFFu;
    if (threadIdx.x == 0) {
        res_bin = 0;
        res_above = 0;
    }
    __syncthreads();
    if (need1 == nc) {
        // the whole bin is taken: every candidate is selected
        T = td.b1 << HIST1_SHIFT;
        needT = 0;
        ntie = 0;
    } else {
        // digit A: key bits 19..10
        h[threadIdx.x] = 0;
        __syncthreads();
        for (uint32_t q = threadIdx.x; q < nc; q += SEL_THREADS) atomicAdd(&h[(ck[q] >> 10) & 1023u], 1u);
        __syncthreads();
        find_from_top<1024, SEL_THREADS>(h, need1, &res_bin, &res_above, scratch);
        const uint32_t bA = res_bin, needA = need1 - res_above;
        // digit B: key bits 9..0 among candidates in bin bA
        h[threadIdx.x] = 0;
        __syncthreads();
        for (uint32_t q = threadIdx.x; q < nc; q += SEL_THREADS) {
            uint32_t k = ck[q];
            if (((k >> 10) & 1023u) == bA) atomicAdd(&h[k & 1023u], 1u);
        }
        __syncthreads();
        find_from_top<1024, SEL_THREADS>(h, needA, &res_bin, &res_above, scratch);
        const uint32_t bB = res_bin;
        needT = needA - res_above;
        ntie = h[bB];
        T = (td.b1 << HIST1_SHIFT) | (bA << 10) | bB;
        if (needT < ntie) {
            // ties split: take the needT smallest indices among key == T;
            // the list is in index order, so find the needT-th such entry
            if (threadIdx.x == 0) {
                found = 0xFFFFFFFFu;
                run_total = 0;
            }
            __syncthreads();
            for (uint32_t q0 = 0; q0 < nc; q0 += SEL_THREADS) {
                const uint32_t q = q0 + threadIdx.x;
                const uint32_t f = (q < nc && ck[q] == T) ? 1u : 0u;
                uint32_t tot;
                const uint32_t before = run_total;
                const uint32_t ex = block_excl_scan_n<SEL_THREADS>(f, scratch, &tot);
                if (f && before + ex + 1 == needT) found = ci[q];
                __syncthreads();
                if (threadIdx.x == 0) run_total = before + tot;
                __syncthreads();
                if (found != 0xFFFFFFFFu) break;
            }
            idx_star = found;
        }
    }
    // mark the selected candidates in the bitmap
    uint32_t *sb = w.selbits + (td.in.slot >> 5);
    for (uint32_t q = threadIdx.x; q < nc; q += SEL_THREADS) {
        const uint32_t k = ck[q], i = ci[q];
        const bool sel = k > T || (k == T && (needT == ntie || i <= idx_star));
        if (sel) atomicOr(&sb[i >> 5], 1u << (i & 31u));
    }
    if (threadIdx.x == 0) {
        td.T = T;
        td.needT = needT;
        td.ntie = ntie;
        td.idx_star = idx_star;
    }
}

hipError_t launch_topr(const Work &w, const float *g, uint32_t hist_blocks, int grid_persist, bool any_topr,
                       hipStream_t s) {
    if (any_topr) {
        k_topr_hist<<<hist_blocks, NTHREADS, 0, s>>>(w, g);
        k_topr_reduce<<<w.ntensors * (HIST1_BINS / NTHREADS), NTHREADS, 0, s>>>(w);
    }
    k_select_filter<<<grid_persist, NTHREADS, 0, s>>>(w, g);
    if (any_topr) k_topr_select<<<w.ntensors, SEL_THREADS, 0, s>>>(w);
    return hipGetLastError();
}

hipError_t launch_nonzero(const Work &w, const float *g, int grid_persist, hipStream_t s) {
    k_select_filter<<<grid_persist, NTHREADS, 0, s>>>(w, g);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Ordered compaction of the selection bitmap into S (ascending indices).
// Threads 0..127 of a block own one bitmap word of the tile each.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NTHREADS) void k_compact_selection(Work w, const float *__restrict__ g,
                                                                float *__restrict__ val_out) {
    __shared__ uint32_t tkt;
    __shared__ uint32_t scratch[NWAVES + 1];
    __shared__ uint32_t tile_excl;
    for (;;) {
        const uint32_t tile = next_ticket(&w.tickets[1], &tkt);
        if (tile >= w.ntiles_total) break;
        const uint32_t t = tensor_of_tile(w.td, w.ntensors, tile);
        TDesc &td = w.td[t];
        const uint32_t lt = tile - td.in.tile0;
        uint32_t word = 0;
        if (threadIdx.x < TILE_WORDS) word = w.selbits[((td.in.slot + (uint64_t)lt * TILE) >> 5) + threadIdx.x];
        uint32_t tot;
        uint32_t ex = block_excl_scan(__popc(word), scratch, &tot);
        if (threadIdx.x == 0) tile_excl = (uint32_t)lookback(w.lb1, tile, td.in.tile0, tot);
        __syncthreads();
        // output capacity: r entries for top-r, d for the support
        const uint32_t cap = td.in.r != R_NONZERO ? td.in.r : td.in.d;
        uint32_t rank = tile_excl + ex;
        const uint32_t i0 = lt * TILE + threadIdx.x * 32;
        while (word) {
            const uint32_t b = __ffs(word) - 1;
            word &= word - 1;
            const uint32_t i = i0 + b;
            if (rank < cap) {
                w.S[td.in.slot + rank] = i;
                if (val_out) val_out[td.in.slot + rank] = g[td.in.off + i];
            }
            ++rank;
        }
        if (threadIdx.x == 0 && lt == td.in.ntiles - 1) {
            const uint32_t n = tile_excl + tot;
            td.n = n < cap ? n : cap;
            if (td.in.r != R_NONZERO && n != td.in.r) atomicOr(&td.flags, FLAG_COUNT);
        }
        __syncthreads();
    }
}

hipError_t launch_compact_selection(const Work &w, const float *g, float *val_out, int grid_persist,
                                    hipStream_t s) {
    k_compact_selection<<<grid_persist, NTHREADS, 0, s>>>(w, g, val_out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Per-tensor Bloom parameters from |S| (Remark 2 of Section 10.2).
// ---------------------------------------------------------------------------
__global__ void k_params(Work w) {
    const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= w.ntensors) return;
    TDesc &td = w.td[t];
    uint32_t mw = td.in.m_words_in;
    if (mw == 0) {
        const double raw = ceil((double)td.n * td.in.mC);
        uint64_t words = ((uint64_t)raw + 31u) / 32u;
        if (words < 1) words = 1;
        const uint64_t cap = (uint64_t)td.in.bl_nslices * SLICE_WORDS;
        if (words > cap) {
            atomicOr(&td.flags, FLAG_CAPACITY);
            words = cap;
        }
        mw = (uint32_t)words;
    }
    td.m_words = mw;
}

hipError_t launch_params(const Work &w, hipStream_t s) {
    k_params<<<(w.ntensors + 255) / 256, 256, 0, s>>>(w);
    return hipGetLastError();
}

}  // namespace dr
