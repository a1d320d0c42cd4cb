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
//      selection bitmap (the d-bit string B of Section 3), compacts the
//      elements of bin b1 into an index-ordered candidate list and counts
//      them by key bits 19..10;
//   3. the select finishes on the candidates' low 20 key bits and resolves
//      ties at the threshold by index order.
// The support of an inherently sparse gradient (Section 3) is the bitmap of
// nonzeros, written by the same pass.
#include "launch.hpp"

namespace dr {

// Set-up: block 0 writes the tensor descriptors of this chunk (the
// device-produced fields start at zero); every block clears its share of
// the zero ranges.
__global__ __launch_bounds__(NTHREADS) void k_init(Work w, InitArgs a, ZeroArgs z) {
    if (blockIdx.x == 0 && threadIdx.x < a.count) {
        TDesc &t = w.td[a.first + threadIdx.x];
        uint32_t *dev = (uint32_t *)&t + sizeof(TInit) / 4;
        for (uint32_t q = 0; q < (sizeof(TDesc) - sizeof(TInit)) / 4; ++q) dev[q] = 0u;
        t.in = a.t[threadIdx.x];
        // known before any data is seen: |S| = r for top-r, and a filter size
        // given by the caller or computed on the host from r
        if (t.in.r != R_NONZERO) t.n = t.in.r;
        t.m_words = t.in.m_words_in;
    }
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint32_t c = 0; c < a.count; ++c) {
        const TInit &in = a.t[c];
        for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < in.ntiles; i += stride)
            w.tile_tensor[in.tile0 + i] = a.first + c;
    }
    for (uint32_t r = 0; r < z.n; ++r) {
        uint32_t *p = (uint32_t *)z.z[r].p;
        for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < z.z[r].words; i += stride) p[i] = 0u;
    }
}

hipError_t launch_init(const Work &w, const InitArgs &a, const ZeroArgs &z, hipStream_t s) {
    uint64_t words = 0;
    for (uint32_t r = 0; r < z.n; ++r) words += z.z[r].words;
    const uint64_t blocks = words / (NTHREADS * 8) + 1;
    k_init<<<blocks < 1024 ? (uint32_t)blocks : 1024u, NTHREADS, 0, s>>>(w, a, z);
    trace_mark(s, "k_init");
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// top-r step 1: first-digit histogram
// ---------------------------------------------------------------------------

// histogram block -> tensor: PHASE 0 blocks by hb0/hbn (exact histograms
// and samples), PHASE 1 (redo) blocks by rb0/rbn; both ascending over the
// tensors
template <int PHASE>
__device__ __forceinline__ int tensor_of_hist_block(const Work &w, uint32_t b) {
    uint32_t lo = 0, hi = w.ntensors;
    while (hi - lo > 1) {
        uint32_t mid = (lo + hi) >> 1;
        if ((PHASE == 0 ? w.td[mid].in.hb0 : w.td[mid].in.rb0) <= b)
            lo = mid;
        else
            hi = mid;
    }
    const TInit &in = w.td[lo].in;
    const uint32_t b0 = PHASE == 0 ? in.hb0 : in.rb0, bn = PHASE == 0 ? in.hbn : in.rbn;
    if (bn == 0 || b < b0 || b >= b0 + bn) return -1;
    return (int)lo;
}

// The filter pass's exact counts of sampled top-r tensor t: elements above
// the bracket, and candidates in each bracket bin.
__device__ __forceinline__ void filter_counts(const Work &w, uint32_t t, uint32_t *above, uint32_t inb[NBR]) {
    const uint32_t *c = w.fcnt + (uint64_t)t * FCNT_COPIES * FCNT_W;
    uint32_t a = 0;
#pragma unroll
    for (uint32_t x = 0; x < NBR; ++x) inb[x] = 0;
    for (uint32_t q = 0; q < FCNT_COPIES; ++q) {
        a += c[q * FCNT_W];
#pragma unroll
        for (uint32_t x = 0; x < NBR; ++x) inb[x] += c[q * FCNT_W + 1 + x];
    }
    *above = a;
}

// A sampled tensor's first filter pass missed the threshold: its exact
// counts put the r-th largest magnitude above or below the bracket.
__device__ __forceinline__ bool bracket_missed(const Work &w, uint32_t t) {
    const TInit &in = w.td[t].in;
    if (in.srate == 0 || in.r == 0 || in.r == R_NONZERO) return false;
    uint32_t above, inb[NBR];
    filter_counts(w, t, &above, inb);
    uint64_t tot = above;
#pragma unroll
    for (uint32_t x = 0; x < NBR; ++x) tot += inb[x];
    return above >= in.r || tot < in.r;
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

// The filter pass's blocks: 512 threads, 8 elements of a tile each, and at
// most 80 VGPRs so that three blocks (six waves per SIMD) fit on a CU.
// Measured against 256 threads and 16 elements (120 VGPRs, four waves per
// SIMD): 40 µs against 44 per pass over 25.6 M elements; seven or eight
// waves per SIMD spill enough to be slower.
constexpr uint32_t FILTER_THREADS = 512;
constexpr uint32_t FILTER_WAVES = FILTER_THREADS / 64;
constexpr uint32_t FILTER_STEPS = TILE / FILTER_THREADS;  // elements per thread per tile

struct PickLds {
    uint32_t res_bin, res_above;
    uint32_t scratch[1024 / 64 + 1];  // block scans of up to 1024 threads
};

// The bracket of an exact top-r tensor: bL = bH = the bin b1 holding the
// r-th largest magnitude, from the tensor's full histogram (block-wide,
// every thread gets it; r = 0: an empty bracket past the last bin).  The
// recording block also writes how many to take from b1 and its size.
template <uint32_t NT>
__device__ uint32_t pick_b1(const Work &w, uint32_t t, bool record, PickLds &l) {
    TDesc &td = w.td[t];
    const uint32_t r = td.in.r;
    if (r == 0) {
        if (record && threadIdx.x == 0) {
            td.bL = td.bH = HIST1_BINS;
            td.need1 = td.ncand = 0;
        }
        return HIST1_BINS;
    }
    if (threadIdx.x == 0) {
        l.res_bin = 0;
        l.res_above = 0;
    }
    __syncthreads();
    const uint32_t *hist = w.hist + (uint64_t)t * HIST1_BINS;
    find_from_top<HIST1_BINS, NT>(hist, r, &l.res_bin, &l.res_above, l.scratch);
    const uint32_t b1 = l.res_bin;
    if (record && threadIdx.x == 0) {
        td.bL = td.bH = b1;
        td.need1 = r - l.res_above;
        td.ncand = hist[b1];
    }
    __syncthreads();  // l is reused
    return b1;
}

// The bracket of a sampled tensor from the sample's histogram hs (summed
// over its copies into LDS): with rho = r nsamp / d the threshold's
// expected rank in the sample and delta = 8 sqrt(rho) + 64, bH is the bin
// holding the sample's (rho - delta)-th largest and bL the one holding its
// (rho + delta)-th (slo and shi), so that the r-th largest of the tensor
// lies in [bL, bH] unless the sample is off by more than eight binomial
// standard deviations (plus a margin for correlated values).  At most NBR
// bins: a wider bracket keeps its top NBR bins (and the counts decide).
template <uint32_t NT>
__device__ void pick_sampled(const Work &w, uint32_t t, bool record, PickLds &l, uint32_t *hs, uint32_t *bL,
                             uint32_t *bH) {
    TDesc &td = w.td[t];
    const uint32_t *sh = w.shist + (uint64_t)t * SHIST_COPIES * HIST1_BINS;
    for (uint32_t b = threadIdx.x; b < HIST1_BINS; b += NT) {
        uint32_t c = 0;
#pragma unroll
        for (uint32_t q = 0; q < SHIST_COPIES; ++q) c += sh[q * HIST1_BINS + b];
        hs[b] = c;
    }
    if (threadIdx.x == 0) {
        l.res_bin = 0;
        l.res_above = 0;
    }
    __syncthreads();
    find_from_top<HIST1_BINS, NT>(hs, td.in.slo, &l.res_bin, &l.res_above, l.scratch);
    const uint32_t hi = l.res_bin;
    __syncthreads();  // every thread has read the result
    if (threadIdx.x == 0) {
        l.res_bin = 0;
        l.res_above = 0;
    }
    __syncthreads();
    find_from_top<HIST1_BINS, NT>(hs, td.in.shi, &l.res_bin, &l.res_above, l.scratch);
    uint32_t lo = l.res_bin;
    if (lo > hi) lo = hi;  // cannot happen: slo <= shi
    if (hi - lo >= NBR) lo = hi - (NBR - 1u);
    if (record && threadIdx.x == 0) {
        td.bL = lo;
        td.bH = hi;
    }
    __syncthreads();  // l and hs are reused
    *bL = lo;
    *bH = hi;
}

constexpr uint32_t HIST_THREADS = 1024;
constexpr uint32_t HIST_SUB = 4;  // sub-histograms, to spread LDS atomics on popular bins

// PHASE 0: the histogram of key bits 30..20 of each exact top-r tensor, and
// of the sample of each sampled one.  PHASE 1: the full histogram of each
// sampled tensor whose bracket missed (the tensor is marked, and the
// candidate histogram the redo's filter pass adds to is cleared); the
// blocks of other tensors return at once.
template <int PHASE>
__global__ __launch_bounds__(HIST_THREADS) void k_topr_hist(Work w, const float *__restrict__ g) {
    __shared__ uint32_t h[HIST_SUB][HIST1_BINS];
    __shared__ uint32_t bad, miss;
    const int t = tensor_of_hist_block<PHASE>(w, blockIdx.x);
    if (t < 0) return;  // block-uniform
    TDesc &td = w.td[t];
    const TInit &in = td.in;
    const uint32_t lb = blockIdx.x - (PHASE == 0 ? in.hb0 : in.rb0);
    const uint32_t nb = PHASE == 0 ? in.hbn : in.rbn;
    if (PHASE == 1) {
        if (threadIdx.x == 0) miss = bracket_missed(w, t) ? 1u : 0u;
        __syncthreads();
        if (!miss) return;  // block-uniform
        if (threadIdx.x == 0) w.glob->redo = 1u;  // the redo's filter pass has work
        // this block's share of the candidate histogram, cleared for the redo
        uint32_t *ha = w.histA + (uint64_t)t * HISTA_COPIES * HISTA_BINS;
        constexpr uint32_t NW = HISTA_COPIES * HISTA_BINS;
        const uint32_t per = (NW + nb - 1) / nb;
        for (uint32_t i = lb * per + threadIdx.x; i < min(NW, (lb + 1) * per); i += HIST_THREADS) ha[i] = 0;
        if (lb == 0 && threadIdx.x == 0) td.sfail = 1;
    }
    for (uint32_t i = threadIdx.x; i < HIST_SUB * HIST1_BINS; i += HIST_THREADS) (&h[0][0])[i] = 0;
    if (threadIdx.x == 0) bad = 0;
    __syncthreads();
    const float *gt = g + in.off;
    uint32_t *mine = h[(threadIdx.x >> 6) % HIST_SUB];
    uint32_t nonfinite = 0;
    const bool sample = PHASE == 0 && in.srate != 0;
    if (sample) {
        // sampled segments [lb SAMPLE_SEGS_PER_BLOCK, +SAMPLE_SEGS_PER_BLOCK):
        // wave q reads segments q, q + 16, ... of the block's share, one
        // element per lane, all its reads in flight together
        constexpr uint32_t WAVES = HIST_THREADS / 64, PER_WAVE = SAMPLE_SEGS_PER_BLOCK / WAVES;
        static_assert(PER_WAVE * WAVES == SAMPLE_SEGS_PER_BLOCK, "whole segments per wave");
        const uint32_t lane = threadIdx.x & 63u, wq = threadIdx.x >> 6;
        const uint64_t nseg = ((uint64_t)in.d + SAMPLE_SEG - 1) / SAMPLE_SEG;
        uint32_t v[PER_WAVE];
        bool in_s[PER_WAVE];
#pragma unroll
        for (uint32_t u = 0; u < PER_WAVE; ++u) {
            const uint64_t j = (uint64_t)lb * SAMPLE_SEGS_PER_BLOCK + u * WAVES + wq;  // sampled segment
            const uint64_t seg = j * in.srate + in.srate / 2;
            const uint64_t e = seg * SAMPLE_SEG + lane;
            in_s[u] = seg < nseg && e < in.d;
            v[u] = in_s[u] ? __float_as_uint(gt[e]) : 0u;
        }
#pragma unroll
        for (uint32_t u = 0; u < PER_WAVE; ++u) {
            if (in_s[u]) {
                const uint32_t key = mag_key(__uint_as_float(v[u]));
                nonfinite |= key >= 0x7f800000u;
                atomicAdd(&mine[key >> HIST1_SHIFT], 1u);
            }
        }
    } else {
        const uint64_t span = (uint64_t)((in.ntiles + nb - 1) / nb) * TILE;
        const uint64_t lo = lb * span;
        const uint64_t hi = lo + span < in.d ? lo + span : in.d;
        // 8 values per thread per step; the next step's values are in flight
        // while this step's are counted.  Reads past the block's range return
        // 0 through the buffer view and are not counted.
        constexpr uint32_t STEP = 8 * HIST_THREADS;
        const uint32_t n = (uint32_t)(hi > lo ? hi - lo : 0);
        const __amdgpu_buffer_rsrc_t gv = buffer_view(gt + lo, 4u * n);
        uint32_t vn[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) vn[u] = buffer_u32(gv, 4u * (u * HIST_THREADS + threadIdx.x));
        for (uint32_t b0 = 0; b0 < n; b0 += STEP) {
            uint32_t v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = vn[u];
            if (b0 + STEP < n) {
#pragma unroll
                for (int u = 0; u < 8; ++u) vn[u] = buffer_u32(gv, 4u * (b0 + STEP + u * HIST_THREADS + threadIdx.x));
            }
            asm volatile("" ::: "memory");
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const uint32_t i = b0 + u * HIST_THREADS + threadIdx.x;
                if (i < n) {
                    const uint32_t key = mag_key(__uint_as_float(v[u]));
                    nonfinite |= key >= 0x7f800000u;
                    atomicAdd(&mine[key >> HIST1_SHIFT], 1u);
                }
            }
        }
    }
    if (nonfinite) bad = 1;
    __syncthreads();
    // the tensor's histogram (the sample's: one of SHIST_COPIES copies):
    // integer sums, so the order of the adds does not matter
    uint32_t *out = sample ? w.shist + ((uint64_t)t * SHIST_COPIES + lb % SHIST_COPIES) * HIST1_BINS
                           : w.hist + (uint64_t)t * HIST1_BINS;
    for (uint32_t i = threadIdx.x; i < HIST1_BINS; i += HIST_THREADS) {
        const uint32_t c = h[0][i] + h[1][i] + h[2][i] + h[3][i];
        if (c) atomicAdd(&out[i], c);
    }
    if (threadIdx.x == 0 && bad) atomicOr(&td.flags, FLAG_NONFINITE);
}

// The filter pass's bracket of each top-r tensor, one block per tensor,
// from the exact histogram or the sample's (the redo's filter pass picks
// the exact bin of a tensor whose sampled bracket missed itself).  (A separate
// launch: inside the filter pass its registers would spill the
// classification's, and making the histogram pass's last block pick needs
// device-wide fences that cost more than the launch.)
__global__ __launch_bounds__(HIST_THREADS) void k_topr_pick(Work w) {
    __shared__ uint32_t hs[HIST1_BINS];
    __shared__ PickLds pl;
    const uint32_t t = blockIdx.x;
    const TDesc &td = w.td[t];
    if (td.in.r == R_NONZERO) return;  // block-uniform
    if (td.in.srate != 0 && td.in.r != 0) {
        uint32_t bL, bH;
        pick_sampled<HIST_THREADS>(w, t, true, pl, hs, &bL, &bH);
    } else {
        pick_b1<HIST_THREADS>(w, t, true, pl);
    }
}

// ---------------------------------------------------------------------------
// top-r step 2 / support: bitmap of definite selections + per-tile candidates
// ---------------------------------------------------------------------------
// Each wave owns whole tiles (a run of consecutive ones), so the pass has
// no block barriers: a tile is 64 steps of 64 consecutive elements, read 8
// steps at a time with the next 8 in flight.
// Top-r elements above the tensor's bracket [bL, bH] are selected; those in
// it are candidates, written in index order (a running count and the
// lanes below in the step's ballot) to the tile's own stretch of the
// candidate arrays (their number in ccnt[tile]) and counted in the
// candidate histogram by (bin - bL, key bits 19..10).  Lane s keeps step
// s's 64-bit ballot, so the tile's 128 bitmap words leave in one coalesced
// 8-byte store per lane.  For the support, tcnt[tile] receives the number
// of selected elements.
// The calls with a sampled tensor use it.  PHASE 0 is the first pass over
// every tile, with the brackets of the pick kernel; it adds each wave's
// exact counts per tensor (above the bracket, in each bracket bin) to copy
// (wave mod FCNT_COPIES).  PHASE 1 redoes the tiles of the sampled tensors
// whose bracket missed; each wave picks the exact bin b1 itself from the
// histogram.
struct FilterTile {
    uint32_t t, base, d;
    uint64_t slot, off;
    bool nz;
};

__device__ __forceinline__ FilterTile filter_tile(const Work &w, uint32_t tile) {
    FilterTile f;
    f.t = tensor_of_tile(w, tile);
    const TDesc &td = w.td[f.t];
    f.base = (tile - td.in.tile0) * TILE;
    f.d = td.in.d;
    f.slot = td.in.slot;
    f.off = td.in.off;
    f.nz = td.in.r == R_NONZERO;
    return f;
}

constexpr uint32_t SF_THREADS = 256;                         // filter blocks: 4 waves, each on tiles of its own
constexpr uint32_t SF_GROUP = 8;                             // steps of 64 elements read together
constexpr uint32_t SF_STEPS = TILE / 64;                     // 64 steps per tile: one per lane
constexpr uint32_t SF_GROUPS = SF_STEPS / SF_GROUP;
static_assert(SF_STEPS == 64, "lane s keeps the ballot of step s");

// A lane's values of steps [grp SF_GROUP, +SF_GROUP) of a tile, read
// through a raw buffer view (reads past the tensor's end return 0 and touch
// no memory).
__device__ __forceinline__ void sf_load(const float *g, const FilterTile &f, uint32_t grp, float x[SF_GROUP]) {
    const __amdgpu_buffer_rsrc_t gv = buffer_view(g + f.off + f.base, 4u * min(TILE, f.d - min(f.d, f.base)));
    const uint32_t lane = threadIdx.x & 63u;
#pragma unroll
    for (uint32_t u = 0; u < SF_GROUP; ++u)
        x[u] = __uint_as_float(buffer_u32(gv, 4u * ((grp * SF_GROUP + u) * 64u + lane)));
}

// The exact bin b1 of top-r tensor t for one wave (every lane gets it):
// lane l sums the 32 bins [2016 - 32 l, 2047 - 32 l] (from the top), a
// wave scan finds the lane whose bins hold the r-th largest magnitude, and
// that lane walks them.  The recording wave writes the bracket, how many to
// take from b1 and its size.
__device__ __noinline__ uint32_t wave_pick_b1(const Work &w, uint32_t t, bool record) {
    TDesc &td = w.td[t];
    const uint32_t r = td.in.r, lane = threadIdx.x & 63u;
    if (r == 0) {
        if (record && lane == 0) {
            td.bL = td.bH = HIST1_BINS;  // nothing above, nothing in the bracket
            td.need1 = td.ncand = 0;
        }
        return HIST1_BINS;
    }
    constexpr uint32_t PER = HIST1_BINS / 64;
    const uint32_t *hist = w.hist + (uint64_t)t * HIST1_BINS;
    uint32_t sum = 0;
#pragma unroll 8
    for (uint32_t q = 0; q < PER; ++q) sum += hist[HIST1_BINS - 1 - (lane * PER + q)];
    const uint32_t incl = wave_incl_scan(sum), excl = incl - sum;
    const bool mine = excl < r && r <= incl;
    uint32_t bin = 0, above = 0;
    if (mine) {
        uint32_t run = excl;
        for (uint32_t q = 0; q < PER; ++q) {
            const uint32_t b = HIST1_BINS - 1 - (lane * PER + q);
            const uint32_t c = hist[b];
            if (run + c >= r) {
                bin = b;
                above = run;
                break;
            }
            run += c;
        }
    }
    const uint64_t m = ballot(mine);
    const int src = m ? __ffsll((unsigned long long)m) - 1 : 0;  // one lane (r <= d: the counts reach r)
    bin = __shfl(bin, src, 64);
    above = __shfl(above, src, 64);
    if (record && lane == 0) {
        td.bL = td.bH = bin;
        td.need1 = r - above;
        td.ncand = hist[bin];
    }
    return bin;
}

constexpr uint32_t NO_TENSOR = 0xffffffffu;

template <int PHASE>
__global__ __launch_bounds__(SF_THREADS) void k_select_filter_wave(Work w, const float *__restrict__ g) {
    constexpr bool COUNT = PHASE == 0;  // brackets from the pick kernel; exact counts
    static_assert(NBR * 16 <= 64, "a lane's bracket-bin counts fit one 64-bit word");
    const uint32_t lane = threadIdx.x & 63u;
    const uint32_t gw = blockIdx.x * (SF_THREADS / 64) + (threadIdx.x >> 6);  // this wave, over the grid
    const uint32_t nw = gridDim.x * (SF_THREADS / 64);
    const uint32_t hcopy = gw % HISTA_COPIES, ccopy = gw % FCNT_COPIES;
    if (PHASE == 1 && !w.glob->redo) return;  // no tensor missed its bracket
    uint32_t cur_t = NO_TENSOR, bL = 0, bH = 0;  // tensor whose bracket the wave holds, and the bracket
    // COUNT: the wave's count above the bracket of tensor cur_t, and each
    // lane's count per bracket bin (16-bit fields, bin bL + x in bits
    // [16 x, 16 x + 16)); a lane adds at most 64 per tile, so the fields
    // are emptied at least every FLUSH_TILES tiles
    constexpr uint32_t FLUSH_TILES = 1000;
    uint32_t acc_def = 0, since = 0;
    uint64_t acc_x = 0;
    auto flush = [&]() {
        if (COUNT && cur_t != NO_TENSOR) {
            uint32_t cx[NBR];
#pragma unroll
            for (uint32_t x = 0; x < NBR; ++x) cx[x] = wave_sum((uint32_t)(acc_x >> (16 * x)) & 0xffffu);
            if (lane == 0) {
                uint32_t *c = w.fcnt + ((uint64_t)cur_t * FCNT_COPIES + ccopy) * FCNT_W;
                if (acc_def) atomicAdd(&c[0], acc_def);
#pragma unroll
                for (uint32_t x = 0; x < NBR; ++x)
                    if (cx[x]) atomicAdd(&c[1 + x], cx[x]);
            }
        }
        acc_def = 0;
        acc_x = 0;
        since = 0;
    };
    // PHASE 0 reads the next tile's first values while it classifies a
    // tile's last ones; the redo reads a tile only once it knows the tile's
    // tensor was redone
    // wave gw takes tiles [t_lo, t_hi), consecutive ones.  Measured against
    // tiles gw, gw + waves, ... (and runs of 4 or 16 tiles taken that way):
    // transformer_355m_x24 350 against 427 us (384, 437), vgg16_138m 168
    // against 159 us (163, 163)
    const uint32_t per = (w.ntiles_total + nw - 1) / nw;
    const uint32_t t_lo = min(w.ntiles_total, gw * per), t_hi = min(w.ntiles_total, t_lo + per);
    float xn[SF_GROUP];
    FilterTile fn{};
    if (PHASE == 0 && t_lo < t_hi) {
        fn = filter_tile(w, t_lo);
        sf_load(g, fn, 0, xn);
    }
    for (uint32_t tile = t_lo; tile < t_hi; ++tile) {
        const FilterTile f = PHASE == 0 ? fn : filter_tile(w, tile);
        if (PHASE == 1) {
            if (!w.td[f.t].sfail) continue;  // wave-uniform
            sf_load(g, f, 0, xn);
        }
        if (!f.nz && (f.t != cur_t || (COUNT && since == FLUSH_TILES))) {  // wave-uniform
            flush();
            if (f.t != cur_t) {
                cur_t = f.t;
                if constexpr (COUNT) {
                    bL = w.td[f.t].bL;
                    bH = w.td[f.t].bH;
                } else {
                    bL = bH = wave_pick_b1(w, f.t, f.base == 0);
                }
            }
        }
        // the tile's fields are wave-uniform: saying so keeps them, and the
        // addresses below, in scalar registers
        const uint32_t base = __builtin_amdgcn_readfirstlane(f.base);
        const uint32_t lim = __builtin_amdgcn_readfirstlane(f.d) - base;  // elements of the tensor here (> 0)
        const uint32_t span = bH - bL;
        const uint64_t cb = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(f.slot >> 32)) << 32) |
                            __builtin_amdgcn_readfirstlane((uint32_t)f.slot);
        uint32_t *const ckey = w.cand_key + cb + base;  // the tile's stretch of the candidate arrays
        uint32_t *const cidx = w.cand_idx + cb + base;
        uint32_t *const histA =
            w.histA + ((uint64_t)__builtin_amdgcn_readfirstlane(f.t) * HISTA_COPIES + hcopy) * HISTA_BINS;
        uint32_t run = 0, ndef = 0, kmax = 0;
        uint32_t wlo = 0, whi = 0;  // lane s: the ballot of step s
        // one step of 64 elements; MODE 0: top-r, whole tile; 1: top-r, the
        // tensor's last (partial) tile; 2: support (no candidates).  A value
        // past the tensor's end reads as 0, so only a bracket reaching bin 0
        // needs the lane mask.
        auto step = [&](auto MODE, uint32_t st, float xv) {
            const uint32_t key = mag_key(xv);
            kmax = max(kmax, key);
            const uint32_t bin = key >> HIST1_SHIFT;
            uint64_t dm, cm = 0;
            if constexpr (MODE() == 2) {
                dm = __builtin_amdgcn_ballot_w64(key != 0u);
            } else {
                dm = __builtin_amdgcn_ballot_w64(bin > bH);
                // unsigned: bL <= bin <= bH
                const bool c = bin - bL <= span && (MODE() == 0 || st * 64u + lane < lim);
                cm = __builtin_amdgcn_ballot_w64(c);
                if (cm) {  // wave-uniform
                    if (c) {
                        const uint32_t q = __builtin_amdgcn_mbcnt_hi((uint32_t)(cm >> 32),
                                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)cm, run));
                        const uint32_t xb = bin - bL;  // < NBR: the candidate lies in the bracket
                        ckey[q] = key;
                        cidx[q] = base + st * 64u + lane;
                        atomicAdd(&histA[(xb << 10) | ((key >> 10) & 1023u)], 1u);
                        if (COUNT) acc_x += 1ull << (xb << 4);
                    }
                    run += popc64(cm);
                }
            }
            ndef += popc64(dm);
            // lane st of wlo / whi takes the ballot's halves (wave-uniform
            // operands: the ballot and the lane number)
            uint32_t lo = wlo, hi = whi;
            asm("v_writelane_b32 %0, %1, m0" : "+v"(lo) : "s"((uint32_t)dm), "{m0}"(st));
            asm("v_writelane_b32 %0, %1, m0" : "+v"(hi) : "s"((uint32_t)(dm >> 32)), "{m0}"(st));
            wlo = lo;
            whi = hi;
        };
        auto steps = [&](auto MODE) {
            for (uint32_t grp = 0; grp < SF_GROUPS; ++grp) {
                float x[SF_GROUP];
#pragma unroll
                for (uint32_t u = 0; u < SF_GROUP; ++u) x[u] = xn[u];
                if (grp + 1 < SF_GROUPS) {
                    sf_load(g, f, grp + 1, xn);
                } else if (PHASE == 0 && tile + 1 < t_hi) {
                    fn = filter_tile(w, tile + 1);
                    sf_load(g, fn, 0, xn);
                }
                // keeps the scheduler from sinking the loads next to their uses
                asm volatile("" ::: "memory");
#pragma unroll
                for (uint32_t u = 0; u < SF_GROUP; ++u) step(MODE, grp * SF_GROUP + u, x[u]);
            }
        };
        if (f.nz)
            steps(std::integral_constant<int, 2>());
        else if (lim >= TILE)
            steps(std::integral_constant<int, 0>());
        else
            steps(std::integral_constant<int, 1>());
        // slot + base is a multiple of TILE, so the tile's words are 8-byte aligned
        uint2 *sb = (uint2 *)(w.selbits + ((f.slot + base) >> 5));
        sb[lane] = make_uint2(wlo, whi);
        if (lane == 0) {
            w.ccnt[tile] = run;
            w.tcnt[tile] = ndef;
        }
        if (COUNT && !f.nz) {
            acc_def += ndef;
            ++since;
        }
        if (__builtin_amdgcn_ballot_w64(kmax >= 0x7f800000u) && lane == 0) atomicOr(&w.td[f.t].flags, FLAG_NONFINITE);
    }
    flush();
}

// The block-wide form of the filter pass: a tile per block at a time, 512
// threads of 8 elements each; each block finds the exact bin b1 itself.
// The exact calls use it: with few tiles per wave, the wave-per-tile form
// above leaves its waves' reads exposed (normal_1m: 19 against 11 µs;
// resnet50_25m: 46 against 44), where the sampled calls' many tiles
// amortise them (transformer_355m_x24: 437 against 517 µs).
// The FILTER_STEPS values of a thread for a tile, read through a raw buffer
// view (reads past the tensor's end return 0 and touch no memory).
__device__ __forceinline__ void filter_load(const float *g, const FilterTile &f, float x[FILTER_STEPS]) {
    const __amdgpu_buffer_rsrc_t gv = buffer_view(g + f.off + f.base, 4u * min(TILE, f.d - min(f.d, f.base)));
#pragma unroll
    for (uint32_t j = 0; j < FILTER_STEPS; ++j)
        x[j] = __uint_as_float(buffer_u32(gv, 4u * (j * FILTER_THREADS + threadIdx.x)));
}

__global__ __launch_bounds__(FILTER_THREADS) __attribute__((amdgpu_waves_per_eu(6))) void k_select_filter_blk(Work w, const float *__restrict__ g) {
    static_assert(FILTER_STEPS * FILTER_WAVES == 64, "one wave scans the (step, wave) candidate counts");
    __shared__ uint32_t wcnt[FILTER_STEPS * FILTER_WAVES];
    __shared__ uint32_t woff[FILTER_STEPS * FILTER_WAVES];
    __shared__ uint32_t dcnt[FILTER_WAVES];
    __shared__ uint32_t sbw[TILE_WORDS];
    __shared__ uint32_t bad;
    __shared__ PickLds pl;
    const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
    const uint32_t hcopy = blockIdx.x % HISTA_COPIES;
    if (threadIdx.x == 0) bad = 0;
    __syncthreads();
    uint32_t cur_t = NO_TENSOR, b1 = 0;  // tensor whose bin b1 the block holds, and b1
    // classify one tile's values
    auto classify = [&](uint32_t tile, const FilterTile &f, const float (&x)[FILTER_STEPS]) {
        if (!f.nz && f.t != cur_t) {  // block-uniform
            cur_t = f.t;
            b1 = pick_b1<FILTER_THREADS>(w, f.t, f.base == 0, pl);
        }
        // the tile's fields are block-uniform: saying so keeps them in
        // scalar registers
        const uint32_t base = __builtin_amdgcn_readfirstlane(f.base);
        const uint32_t lim = __builtin_amdgcn_readfirstlane(f.d) - base;  // elements of the tensor here (> 0)
        const uint64_t slot = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(f.slot >> 32)) << 32) |
                              __builtin_amdgcn_readfirstlane((uint32_t)f.slot);
        uint32_t keys[FILTER_STEPS];
        uint64_t cmask[FILTER_STEPS];
        uint32_t kmax = 0, ndef = 0;
        // lane 2j + h ends up holding half h of step j's bitmap ballot, and
        // lane j the candidate count of step j (lane writes of wave-uniform
        // values)
        uint32_t myword = 0, mycand = 0;
        // MODE 0: top-r, whole tile; 1: top-r, the tensor's last (partial)
        // tile; 2: support.  A value past the tensor's end reads as 0, so
        // only a bin b1 of 0 needs the lane mask.
        auto steps = [&](auto MODE) {
#pragma unroll
            for (uint32_t j = 0; j < FILTER_STEPS; ++j) {
                const uint32_t key = mag_key(x[j]);
                kmax = max(kmax, key);
                const uint32_t bin = key >> HIST1_SHIFT;
                uint64_t dm, cm = 0;
                if constexpr (MODE() == 2) {
                    dm = __builtin_amdgcn_ballot_w64(key != 0u);
                } else {
                    dm = __builtin_amdgcn_ballot_w64(bin > b1);
                    cm = __builtin_amdgcn_ballot_w64(bin == b1 &&
                                                     (MODE() == 0 || j * FILTER_THREADS + threadIdx.x < lim));
                }
                cmask[j] = cm;
                keys[j] = key;
                ndef += popc64(dm);
                uint32_t mw = myword, mc = mycand;
                asm("v_writelane_b32 %0, %1, m0" : "+v"(mw) : "s"((uint32_t)dm), "{m0}"(2u * j));
                asm("v_writelane_b32 %0, %1, m0" : "+v"(mw) : "s"((uint32_t)(dm >> 32)), "{m0}"(2u * j + 1u));
                asm("v_writelane_b32 %0, %1, m0" : "+v"(mc) : "s"(popc64(cm)), "{m0}"(j));
                myword = mw;
                mycand = mc;
            }
        };
        if (f.nz)
            steps(std::integral_constant<int, 2>());
        else if (lim >= TILE)
            steps(std::integral_constant<int, 0>());
        else
            steps(std::integral_constant<int, 1>());
        const bool nonfinite = kmax >= 0x7f800000u;
        // the tile's bitmap words are staged in LDS and written by one
        // coalesced store after the barrier (two-lane stores per step cost a
        // third of the pass's read bandwidth)
        if (lane < 2 * FILTER_STEPS) sbw[(lane >> 1) * (FILTER_THREADS / 32) + wv * 2 + (lane & 1)] = myword;
        if (lane < FILTER_STEPS) wcnt[lane * FILTER_WAVES + wv] = mycand;
        if (nonfinite) bad = 1;
        if (lane == 0) dcnt[wv] = ndef;
        __syncthreads();
        if (threadIdx.x < 64) {
            // (j, wave) candidate counts in element order -> exclusive offsets
            const uint32_t c = wcnt[threadIdx.x];
            const uint32_t inc = wave_incl_scan(c);
            woff[threadIdx.x] = inc - c;
            if (threadIdx.x == 63) {
                w.ccnt[tile] = inc;
                uint32_t nd = 0;
                for (uint32_t q = 0; q < FILTER_WAVES; ++q) nd += dcnt[q];
                w.tcnt[tile] = nd;
            }
        }
        __syncthreads();
        if (threadIdx.x == 0 && bad) {
            atomicOr(&w.td[f.t].flags, FLAG_NONFINITE);
            bad = 0;
        }
        if (threadIdx.x < TILE_WORDS) w.selbits[((slot + base) >> 5) + threadIdx.x] = sbw[threadIdx.x];
        const uint64_t cbase = slot + base;
        uint32_t *histA = w.histA + ((uint64_t)f.t * HISTA_COPIES + hcopy) * HISTA_BINS;
#pragma unroll
        for (uint32_t j = 0; j < FILTER_STEPS; ++j) {
            if (cmask[j] && ((cmask[j] >> lane) & 1ull)) {  // the first test is wave-uniform
                const uint64_t q = cbase + woff[j * FILTER_WAVES + wv] + lanes_below(cmask[j]);
                w.cand_key[q] = keys[j];
                w.cand_idx[q] = base + j * FILTER_THREADS + threadIdx.x;
                atomicAdd(&histA[(keys[j] >> 10) & 1023u], 1u);  // bracket bin 0
            }
        }
        __syncthreads();
    };
    // the next tile's values are in flight while this tile is classified
    float xn[FILTER_STEPS];
    FilterTile fn{};
    if (blockIdx.x < w.ntiles_total) {
        fn = filter_tile(w, blockIdx.x);
        filter_load(g, fn, xn);
    }
    for (uint32_t tile = blockIdx.x; tile < w.ntiles_total; tile += gridDim.x) {
        const FilterTile f = fn;
        const bool more = tile + gridDim.x < w.ntiles_total;
        if (more) fn = filter_tile(w, tile + gridDim.x);
        float x[FILTER_STEPS];
#pragma unroll
        for (uint32_t j = 0; j < FILTER_STEPS; ++j) x[j] = xn[j];
        if (more) filter_load(g, fn, xn);
        // keeps the scheduler from sinking the loads next to their uses
        asm volatile("" ::: "memory");
        classify(tile, f, x);
    }
}

// ---------------------------------------------------------------------------
// top-r step 3: finish the select on the candidates' low 20 key bits.
//  a. each block of the candidate pass picks, for the tensors of its tiles,
//     the bin bA of key bits 19..10 from the histograms the filter pass
//     built (the block holding a tensor's first tile records it);
//  b. that pass marks the candidates above bA and gathers those in bA
//     (usually a few dozen) into a short list;
//  c. one block per tensor finishes on the short list: bin of bits 9..0,
//     then, if equal keys straddle the cut, the smallest indices among them.
// ---------------------------------------------------------------------------
constexpr uint32_t SEL_THREADS = 1024;
constexpr uint32_t ALL_OF_B1 = 0xFFFFFFFFu;  // bA when the whole bin b1 is taken

// Candidates above bin bA are selected; those in bA go to the short list.
// A block takes CP_TILES tiles at a time and treats their candidates as one
// flat range (a scan of the tiles' counts), so the work per thread does not
// depend on how the candidates fall into tiles; each thread handles
// CP_BATCH of them with all their reads in flight.
constexpr uint32_t CP_BATCH = 4;
constexpr uint32_t CP_TILES = 32;

// Where the threshold of top-r tensor t lies among its candidates: the
// bracket bin x (from the bottom of the bracket) that holds the r-th largest
// magnitude, the bin bA of key bits 19..10 within it (ALL_OF_B1: the whole
// bin x is taken) and how many to take from bA; from the filter pass's
// exact counts (the redo's, if the tensor was redone) and its candidate
// histogram.  x = NBR takes no candidate.  Block-wide; the block that
// records also writes the tensor's first-digit bin b1 = bL + x for the
// final step.
struct Thr {
    uint32_t x, bA, needA;
};

__device__ Thr pick_thr(const Work &w, uint32_t t, uint32_t *hsum, PickLds &l, bool record) {
    TDesc &td = w.td[t];
    const uint32_t r = td.in.r;
    uint32_t above = 0, inb[NBR] = {0, 0, 0, 0};
    static_assert(NBR == 4, "initialiser");
    if (td.in.srate == 0 || td.sfail) {
        // exact bracket (bin b1): from the histogram, through the pick
        above = r - td.need1;
        inb[0] = td.ncand;
    } else {
        filter_counts(w, t, &above, inb);
    }
    uint64_t tot = above;
#pragma unroll
    for (uint32_t x = 0; x < NBR; ++x) tot += inb[x];
    Thr th{NBR, ALL_OF_B1, 0};
    if (r == 0 || above >= r || tot < r) {
        // r = 0, or counts that contradict the bracket, which the redo
        // rules out: the selection count then differs from r and says so
        if (r != 0 && record && threadIdx.x == 0) atomicOr(&td.flags, FLAG_COUNT);
        return th;
    }
    uint32_t need = r - above;
    uint32_t x = NBR - 1;
    while (need > inb[x]) {  // ends at x >= 0: the bins hold at least `need`
        need -= inb[x];
        --x;
    }
    th.x = x;
    if (record && threadIdx.x == 0) {
        td.b1 = td.bL + x;
        td.ncand = inb[x];
    }
    if (need == inb[x]) return th;  // the whole bin (bA = ALL_OF_B1)
    const uint32_t *histA = w.histA + (uint64_t)t * HISTA_COPIES * HISTA_BINS + x * 1024u;
    for (uint32_t b = threadIdx.x; b < 1024u; b += NTHREADS) {
        uint32_t c = 0;
#pragma unroll
        for (uint32_t q = 0; q < HISTA_COPIES; ++q) c += histA[q * HISTA_BINS + b];
        hsum[b] = c;
    }
    if (threadIdx.x == 0) {
        l.res_bin = 0;
        l.res_above = 0;
    }
    __syncthreads();
    find_from_top<1024, NTHREADS>(hsum, need, &l.res_bin, &l.res_above, l.scratch);
    th.bA = l.res_bin;
    th.needA = need - l.res_above;
    __syncthreads();  // hsum and l are reused
    return th;
}

__global__ __launch_bounds__(NTHREADS) void k_topr_candpass(Work w) {
    __shared__ uint32_t pre[CP_TILES];
    __shared__ uint32_t tten[CP_TILES];
    __shared__ uint64_t tbase[CP_TILES];  // workspace offset of the tile's first candidate
    __shared__ uint32_t tbA[CP_TILES], tx[CP_TILES], tbL[CP_TILES];  // the tile's tensor's pick and bracket
    __shared__ uint32_t tpk[CP_TILES];    // the tile's entry in the group's tensor list
    __shared__ uint32_t gten[CP_TILES], gbA[CP_TILES], gx[CP_TILES], gbL[CP_TILES];  // the group's tensors, in tile order, and their picks
    __shared__ uint32_t gtot, ngten;
    __shared__ uint32_t hsum[1024];
    __shared__ PickLds pl;
    uint32_t last_t = 0xFFFFFFFFu;  // the block's most recent pick
    Thr last{NBR, ALL_OF_B1, 0};
    for (uint32_t g0 = blockIdx.x * CP_TILES; g0 < w.ntiles_total; g0 += gridDim.x * CP_TILES) {
        if (threadIdx.x < 64) {  // the first wave scans the group's counts and lists its tensors
            const uint32_t tile = g0 + threadIdx.x;
            const bool in = threadIdx.x < CP_TILES && tile < w.ntiles_total;
            uint32_t c = 0, t = 0xFFFFFFFFu;
            if (in) {
                t = tensor_of_tile(w, tile);
                const TDesc &td = w.td[t];
                c = td.in.r == R_NONZERO ? 0u : w.ccnt[tile];
                tbase[threadIdx.x] = td.in.slot + (uint64_t)(tile - td.in.tile0) * TILE;
            }
            const uint32_t inc = wave_incl_scan(c);
            // tiles are in tensor order: a tile whose tensor differs from the
            // previous tile's starts the next entry of the group's list
            const uint32_t tprev = __shfl_up(t, 1, 64);
            const bool fresh = in && (threadIdx.x == 0 || t != tprev);
            const uint64_t fm = ballot(fresh);
            const uint32_t ord = lanes_below(fm) + (fresh ? 1u : 0u);  // list entries up to this tile
            if (fresh) gten[ord - 1] = t;
            if (threadIdx.x < CP_TILES) {  // past the last tile: an empty tile (pre = total)
                pre[threadIdx.x] = inc - c;
                tten[threadIdx.x] = t;
                tpk[threadIdx.x] = in ? ord - 1 : 0u;
            }
            if (threadIdx.x == 63) {
                gtot = inc;
                ngten = popc64(fm);
            }
        }
        __syncthreads();
        const uint32_t ng = ngten;
        for (uint32_t q = 0; q < ng; ++q) {  // block-uniform
            const uint32_t t = gten[q];
            if (t != last_t) {
                TDesc &td = w.td[t];
                Thr th{NBR, ALL_OF_B1, 0};
                if (td.in.r != R_NONZERO) {
                    // the group holding the tensor's first tile records the
                    // pick for the final step
                    const bool record = td.in.tile0 >= g0;
                    th = pick_thr(w, t, hsum, pl, record);
                    if (record && threadIdx.x == 0) {
                        td.bA = th.bA;
                        td.needA = th.needA;
                    }
                }
                last_t = t;
                last = th;
            }
            if (threadIdx.x == 0) {
                gbA[q] = last.bA;
                gx[q] = last.x;
                gbL[q] = w.td[t].bL;
            }
        }
        __syncthreads();
        if (threadIdx.x < CP_TILES && g0 + threadIdx.x < w.ntiles_total) {
            const uint32_t e = tpk[threadIdx.x];
            tbA[threadIdx.x] = gbA[e];
            tx[threadIdx.x] = gx[e];
            tbL[threadIdx.x] = gbL[e];
        }
        __syncthreads();
        const uint32_t tot = gtot;
        for (uint32_t e0 = 0; e0 < tot; e0 += NTHREADS * CP_BATCH) {
            uint32_t key[CP_BATCH], idx[CP_BATCH], tix[CP_BATCH];
#pragma unroll
            for (uint32_t u = 0; u < CP_BATCH; ++u) {
                const uint32_t e = e0 + u * NTHREADS + threadIdx.x;
                // the tile holding flat candidate e: the last x with pre[x] <= e
                uint32_t lo = 0, hi = CP_TILES;
                while (hi - lo > 1) {
                    const uint32_t mid = (lo + hi) >> 1;
                    if (pre[mid] <= e)
                        lo = mid;
                    else
                        hi = mid;
                }
                tix[u] = lo;
                const uint64_t at = e < tot ? tbase[lo] + (e - pre[lo]) : 0u;  // past the end: any valid slot
                key[u] = w.cand_key[at];
                idx[u] = w.cand_idx[at];
            }
            asm volatile("" ::: "memory");
#pragma unroll
            for (uint32_t u = 0; u < CP_BATCH; ++u) {
                const uint32_t e = e0 + u * NTHREADS + threadIdx.x;
                const bool act = e < tot;
                const uint32_t x = tix[u];
                const uint32_t bA = tbA[x], k = key[u], i = idx[u];
                // the candidate's bracket bin (from the bracket's bottom) and
                // key bits 19..10
                const uint32_t xb = (k >> HIST1_SHIFT) - tbL[x], xt = tx[x];
                const uint32_t dA = (k >> 10) & 1023u;
                const bool take = act && (xb > xt || (xb == xt && (bA == ALL_OF_B1 || dA > bA)));
                const bool sub = act && xb == xt && bA != ALL_OF_B1 && dA == bA;
                // i lies in tile x, whose first element sits at slot tbase[x]
                if (take) atomicOr(&w.selbits[(tbase[x] + (i % TILE)) >> 5], 1u << (i & 31u));
                if (sub) {
                    // appends to the tensor's short list; a wave's lanes of
                    // one tensor share one atomic
                    const uint32_t tt = tten[x];
                    TDesc &td = w.td[tt];
                    const uint64_t m = ballot(sub);
                    const uint32_t first = (uint32_t)__ffsll((unsigned long long)m) - 1;
                    const uint32_t t_first = __shfl(tt, first, 64);
                    const uint64_t same = ballot(tt == t_first) & m;
                    uint32_t at0;
                    uint64_t q;
                    if (tt == t_first) {
                        at0 = 0;
                        if (lane_id() == first) at0 = atomicAdd(&td.nsub, popc64(same));
                        at0 = __shfl(at0, first, 64);
                        q = td.in.slot + at0 + lanes_below(same);
                    } else {
                        at0 = atomicAdd(&td.nsub, 1u);
                        q = td.in.slot + at0;
                    }
                    w.sub_key[q] = k;
                    w.sub_idx[q] = i;
                }
            }
        }
        __syncthreads();  // the group's tables are rewritten by the next group
    }
}

// Among the short list (unordered), take the needA largest by key, ties to
// the smaller index; set their bits.
__global__ __launch_bounds__(SEL_THREADS) void k_topr_final(Work w) {
    TDesc &td = w.td[blockIdx.x];
    if (td.in.r == R_NONZERO || td.ncand == 0 || td.bA == ALL_OF_B1) return;
    __shared__ uint32_t h[2048];
    __shared__ uint32_t scratch[SEL_THREADS / 64 + 1];
    __shared__ uint32_t res_bin, res_above;
    const uint32_t ns = td.nsub, needA = td.needA;
    const uint32_t *sk = w.sub_key + td.in.slot;
    const uint32_t *si = w.sub_idx + td.in.slot;
    // bits 9..0 of the key
    h[threadIdx.x] = 0;
    if (threadIdx.x == 0) {
        res_bin = 0;
        res_above = 0;
    }
    __syncthreads();
    for (uint32_t q = threadIdx.x; q < ns; q += SEL_THREADS) atomicAdd(&h[sk[q] & 1023u], 1u);
    __syncthreads();
    find_from_top<1024, SEL_THREADS>(h, needA, &res_bin, &res_above, scratch);
    const uint32_t bB = res_bin;
    const uint32_t needT = needA - res_above, ntie = h[bB];
    const uint32_t T = (td.b1 << HIST1_SHIFT) | (td.bA << 10) | bB;
    __syncthreads();
    uint32_t idx_star = 0xFFFFFFFFu;
    if (needT < ntie) {
        // the needT smallest indices among key == T: radix select on the
        // index, 11 + 11 + 10 bits, counting from the bottom
        uint32_t prefix = 0, need = needT;
        for (int pass = 0; pass < 3; ++pass) {
            const uint32_t shift = pass == 0 ? 21u : (pass == 1 ? 10u : 0u);
            const uint32_t nb = pass == 2 ? 1024u : 2048u;
            for (uint32_t i = threadIdx.x; i < 2048; i += SEL_THREADS) h[i] = 0;
            __syncthreads();
            for (uint32_t q = threadIdx.x; q < ns; q += SEL_THREADS) {
                const uint32_t ix = si[q];
                const bool match = sk[q] == T && (pass == 0 || (ix >> (shift + (pass == 1 ? 11u : 10u))) == prefix);
                if (match) atomicAdd(&h[(ix >> shift) & (nb - 1u)], 1u);
            }
            __syncthreads();
            // find from the bottom: the bin where the running count reaches `need`
            const uint32_t per = nb / SEL_THREADS;  // 2 or 1 bins per thread
            uint32_t sum = 0;
            for (uint32_t u = 0; u < per; ++u) sum += h[threadIdx.x * per + u];
            uint32_t tot;
            const uint32_t ex = block_excl_scan_n<SEL_THREADS>(sum, scratch, &tot);
            if (ex < need && need <= ex + sum) {
                uint32_t run = ex;
                for (uint32_t u = 0; u < per; ++u) {
                    const uint32_t bin = threadIdx.x * per + u;
                    if (run + h[bin] >= need) {
                        res_bin = bin;
                        res_above = run;
                        break;
                    }
                    run += h[bin];
                }
            }
            __syncthreads();
            prefix = (prefix << (pass == 2 ? 10u : 11u)) | res_bin;
            need -= res_above;
            __syncthreads();
        }
        idx_star = prefix;
    }
    uint32_t *sb = w.selbits + (td.in.slot >> 5);
    for (uint32_t q = threadIdx.x; q < ns; q += SEL_THREADS) {
        const uint32_t k = sk[q], i = si[q];
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

hipError_t launch_topr(const Work &w, const float *g, uint32_t hist_blocks, uint32_t redo_blocks, bool any_topr,
                       hipStream_t s) {
    const bool sampled = redo_blocks > 0;
    // the wave-per-tile form: at least 8 tiles per wave (vgg16_138m: 193
    // against 206 µs with a wave per tile; a 16-tile floor was slower again)
    const int fgrid = resident_grid(k_select_filter_wave<0>, SF_THREADS, (w.ntiles_total + 31) / 32);
    if (any_topr && hist_blocks > 0) {
        k_topr_hist<0><<<hist_blocks, HIST_THREADS, 0, s>>>(w, g);
        trace_mark(s, "k_topr_hist");
    }
    if (any_topr && sampled) {
        k_topr_pick<<<w.ntensors, HIST_THREADS, 0, s>>>(w);
        trace_mark(s, "k_topr_pick");
        k_select_filter_wave<0><<<fgrid, SF_THREADS, 0, s>>>(w, g);
    } else {
        k_select_filter_blk<<<resident_grid(k_select_filter_blk, FILTER_THREADS, w.ntiles_total),
                                         FILTER_THREADS, 0, s>>>(w, g);
    }
    trace_mark(s, "k_select_filter");
    if (any_topr) {
        if (sampled) {
            // the exact redo of sampled brackets that missed (blocks of other
            // tensors return at once)
            k_topr_hist<1><<<redo_blocks, HIST_THREADS, 0, s>>>(w, g);
            trace_mark(s, "k_topr_hist_redo");
            k_select_filter_wave<1><<<fgrid, SF_THREADS, 0, s>>>(w, g);
            trace_mark(s, "k_select_filter_redo");
        }
        k_topr_candpass<<<resident_grid(k_topr_candpass, NTHREADS, (w.ntiles_total + CP_TILES - 1) / CP_TILES), NTHREADS, 0, s>>>(w);
        trace_mark(s, "k_topr_candpass");
        k_topr_final<<<w.ntensors, SEL_THREADS, 0, s>>>(w);
        trace_mark(s, "k_topr_final");
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Ordered passes: per-tile counts -> per-tensor offsets -> emit in order
// ---------------------------------------------------------------------------
// tcnt[tile] = set bits of the tile's words of `bits`
__global__ __launch_bounds__(NTHREADS) void k_tile_popc(Work w, const uint32_t *__restrict__ bits) {
    __shared__ uint32_t part[NWAVES];
    for (uint32_t tile = blockIdx.x; tile < w.ntiles_total; tile += gridDim.x) {
        uint32_t c = 0;
        if (threadIdx.x < TILE_WORDS) c = __popc(bits[(uint64_t)tile * TILE_WORDS + threadIdx.x]);
        c = wave_sum(c);
        if ((threadIdx.x & 63u) == 0) part[threadIdx.x >> 6] = c;
        __syncthreads();
        if (threadIdx.x == 0) w.tcnt[tile] = part[0] + part[1] + part[2] + part[3];
        __syncthreads();
    }
}

// toff = exclusive scan of the selection's tcnt over the tiles of each
// tensor; the total is |S| (the queries scan their counts in the probe pass)
constexpr uint32_t TSCAN_THREADS = 1024;
constexpr uint32_t TSCAN_PER = 8;  // counts per thread per step, loaded together

__global__ __launch_bounds__(TSCAN_THREADS) void k_tile_scan(Work w) {
    TDesc &td = w.td[blockIdx.x];
    __shared__ uint32_t scratch[TSCAN_THREADS / 64 + 1];
    const uint32_t nt = td.in.ntiles;
    const __amdgpu_buffer_rsrc_t cv = buffer_view(w.tcnt + td.in.tile0, 4u * nt);  // past the end: 0
    uint32_t *off = w.toff + td.in.tile0;
    uint32_t carry = 0;
    // thread x owns counts [x * PER, (x+1) * PER) of each step of PER * 1024
    for (uint32_t q0 = 0; q0 < nt; q0 += TSCAN_THREADS * TSCAN_PER) {
        uint32_t v[TSCAN_PER];
        const uint32_t b = q0 + threadIdx.x * TSCAN_PER;
#pragma unroll
        for (uint32_t u = 0; u < TSCAN_PER; ++u) v[u] = buffer_u32(cv, 4u * (b + u));
        uint32_t sum = 0;
#pragma unroll
        for (uint32_t u = 0; u < TSCAN_PER; ++u) sum += v[u];
        uint32_t tot;
        uint32_t run = carry + block_excl_scan_n<TSCAN_THREADS>(sum, scratch, &tot);
#pragma unroll
        for (uint32_t u = 0; u < TSCAN_PER; ++u) {
            if (b + u < nt) off[b + u] = run;
            run += v[u];
        }
        carry += tot;
    }
    if (threadIdx.x == 0) {
        const uint32_t cap = td.in.r != R_NONZERO ? td.in.r : td.in.d;
        td.n = carry < cap ? carry : cap;
        if (td.in.r != R_NONZERO && carry != td.in.r) atomicOr(&td.flags, FLAG_COUNT);
        td.m_words = filter_words(td);
    }
}

hipError_t launch_tile_popc(const Work &w, const uint32_t *bits, int grid_persist, hipStream_t s) {
    k_tile_popc<<<grid_persist, NTHREADS, 0, s>>>(w, bits);
    trace_mark(s, "k_tile_popc");
    return hipGetLastError();
}


// S = the selection bitmap's set bits in ascending order (val_out: g there).
// Threads 0..127 of a block own one bitmap word of the tile each.
__global__ __launch_bounds__(NTHREADS) void k_compact_selection(Work w, const float *__restrict__ g,
                                                                float *__restrict__ val_out) {
    __shared__ uint32_t scratch[NWAVES + 1];
    for (uint32_t tile = blockIdx.x; tile < w.ntiles_total; tile += gridDim.x) {
        const uint32_t t = tensor_of_tile(w, tile);
        const TDesc &td = w.td[t];
        const uint32_t lt = tile - td.in.tile0;
        uint32_t word = 0;
        if (threadIdx.x < TILE_WORDS) word = w.selbits[(uint64_t)tile * TILE_WORDS + threadIdx.x];
        uint32_t tot;
        const uint32_t ex = block_excl_scan(__popc(word), scratch, &tot);
        const uint32_t cap = td.in.r != R_NONZERO ? td.in.r : td.in.d;
        uint32_t rank = w.toff[tile] + ex;
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
    }
}

hipError_t launch_compact_selection(const Work &w, const float *g, float *val_out, int grid_persist,
                                    hipStream_t s) {
    k_tile_popc<<<grid_persist, NTHREADS, 0, s>>>(w, w.selbits);
    trace_mark(s, "k_tile_popc");
    k_tile_scan<<<w.ntensors, TSCAN_THREADS, 0, s>>>(w);
    trace_mark(s, "k_tile_scan");
    k_compact_selection<<<grid_persist, NTHREADS, 0, s>>>(w, g, val_out);
    trace_mark(s, "k_compact_selection");
    return hipGetLastError();
}

hipError_t launch_nonzero(const Work &w, const float *g, int grid_persist, hipStream_t s) {
    (void)grid_persist;
    k_select_filter_blk<<<resident_grid(k_select_filter_blk, FILTER_THREADS, w.ntiles_total),
                                     FILTER_THREADS, 0, s>>>(w, g);
    trace_mark(s, "k_select_filter");
    // |S| from the per-tile counts of the filter pass
    k_tile_scan<<<w.ntensors, TSCAN_THREADS, 0, s>>>(w);
    trace_mark(s, "k_tile_scan");
    return hipGetLastError();
}

}  // namespace dr
