// bloom.hip -- Bloom-filter index compression (Sections 2 and 4).
//
// Insert: every selected index s sets bits h_j(s), j < k.  Device-wide
// atomics into a filter larger than a CU's LDS are slow on this GPU, so the
// insert buckets the k n bit positions by slice of the filter (2^14 or
// 2^16 bits; count, scan, scatter), and one block per slice then sets its
// bits in LDS and writes the slice out whole.  OR is commutative, so the
// filter does not depend on the order of any of this.
//
// Query (policy P0, Section 4): every i of the tensor's index range whose k
// bits are all set is a positive, reported in ascending order.  Each wave
// owns 1024 consecutive indices and tests them probe by probe: after probe
// j only the indices still alive are kept, compacted into an LDS queue in
// index order (ballot + mbcnt), so lanes do not idle while a few indices
// need many probes.  The key-dependent half of MurmurHash3 is computed once
// per index.  The probe kernel writes a positives bitmap and per-tile
// counts; after a per-tensor scan of the counts, the emit kernel writes the
// positives in order.
#include "launch.hpp"
#include "value_setup.hpp"

namespace dr {

// ---------------------------------------------------------------------------
// Insert
// ---------------------------------------------------------------------------
// The items come either from the selection bitmap (the round trip: chunk c
// of a tensor is its bitmap tiles [c * bl_chunk, (c+1) * bl_chunk)) or from
// a list of indices (chunk c is items [c * bl_chunk, (c+1) * bl_chunk)).

__device__ __forceinline__ uint32_t tensor_of_chunk(const Work &w, uint32_t c) {
    uint32_t lo = 0, hi = w.ntensors;
    while (hi - lo > 1) {
        uint32_t mid = (lo + hi) >> 1;
        if (w.td[mid].in.bl_chunk0 <= c)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

__device__ __forceinline__ uint32_t tensor_of_slice(const Work &w, uint32_t s) {
    uint32_t lo = 0, hi = w.ntensors;
    while (hi - lo > 1) {
        uint32_t mid = (lo + hi) >> 1;
        if (w.td[mid].in.bl_slice0 <= s)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

// Calls f(index) for every item of chunk c of tensor td (strided over the
// block's NT threads).
template <bool FROM_BITMAP, uint32_t NT, typename F>
__device__ __forceinline__ void for_chunk_items(const Work &w, const TDesc &td, uint32_t c, F f) {
    if (FROM_BITMAP) {
        const uint32_t w0 = c * td.in.bl_chunk * TILE_WORDS;
        const uint32_t w1 = min(td.in.ntiles * TILE_WORDS, w0 + td.in.bl_chunk * TILE_WORDS);
        const uint32_t *sb = w.selbits + (td.in.slot >> 5);
        for (uint32_t x = w0 + threadIdx.x; x < w1; x += NT) {
            uint32_t word = sb[x];
            while (word) {
                const uint32_t b = __ffs(word) - 1;
                word &= word - 1;
                f(x * 32u + b);
            }
        }
    } else {
        const uint32_t n = td.n, chunk = td.in.bl_chunk;
        const uint32_t q0 = c * chunk, q1 = min(n, q0 + chunk);
        const uint32_t *S = w.S + td.in.slot;
        for (uint32_t q = q0 + threadIdx.x; q < q1; q += NT) f(S[q]);
    }
}

__device__ __forceinline__ uint32_t active_chunks(const TDesc &td, bool from_bitmap) {
    if (from_bitmap) return td.in.bl_nchunks;
    return (td.n + td.in.bl_chunk - 1) / td.in.bl_chunk;
}

// The hashes [*a, *b) of tensor td in round r of the bucketed insert.  The
// plan gives rounds of hpr hashes, for the most items a tensor may have;
// a tensor with fewer (a support's count is known only on the device) takes
// as many hashes per round as its position region holds, so that it may
// finish in fewer rounds, and the later rounds' kernels skip it (ncf_32m,
// 13 hashes: two rounds of 10 and 3 instead of three of 6, 6 and 1).
__device__ __forceinline__ void bl_round(const TDesc &td, uint32_t r, uint32_t hpr, uint32_t *a, uint32_t *b) {
    const uint32_t k = td.in.k;
    uint64_t h = td.n ? td.in.bl_poscap / td.n : k;
    if (h < hpr) h = hpr;
    if (h > k) h = k;
    const uint64_t a64 = (uint64_t)r * h;
    *a = (uint32_t)(a64 < k ? a64 : k);
    *b = (uint32_t)min<uint64_t>(k, (uint64_t)*a + h);
}

// The bucketed insert's kernels run 1024 threads per block: a chunk's
// items are hashed one after another per thread, and the LDS atomics of the
// count and scatter passes need many waves in flight to hide their latency.
// Each takes round r of hpr planned hashes per round.
constexpr uint32_t BL_THREADS = 1024;

template <bool FROM_BITMAP>
__global__ __launch_bounds__(BL_THREADS) void k_bloom_count(Work w, uint32_t r, uint32_t hpr) {
    extern __shared__ uint32_t lh[];
    const uint32_t t = tensor_of_chunk(w, blockIdx.x);
    const TDesc &td = w.td[t];
    const uint32_t c = blockIdx.x - td.in.bl_chunk0;
    if (c >= td.in.bl_nchunks || c >= active_chunks(td, FROM_BITMAP)) return;
    uint32_t j0, je;
    bl_round(td, r, hpr, &j0, &je);
    if (j0 >= je) return;  // the tensor has had all its hashes
    const uint32_t m_bits = td.m_words * 32u;
    const uint32_t sl2 = td.in.slice_log2;
    const uint32_t nsl = (m_bits + (1u << sl2) - 1) >> sl2;
    __shared__ uint32_t ps[33];
    const bool part = td.in.layout == LAYOUT_PARTITIONED;
    if (part) fill_part_starts(ps, m_bits, td.in.k);
    const PosMap pm{m_bits, part ? ps : nullptr};
    for (uint32_t s = threadIdx.x; s < nsl; s += BL_THREADS) lh[s] = 0;
    __syncthreads();
    for_chunk_items<FROM_BITMAP, BL_THREADS>(w, td, c, [&](uint32_t x) {
        const uint32_t km = mm3_key(x);
        for (uint32_t j = j0; j < je; ++j) atomicAdd(&lh[pm(km, j) >> sl2], 1u);
    });
    __syncthreads();
    uint32_t *tab = w.btab + td.in.bl_tab0;
    for (uint32_t s = threadIdx.x; s < nsl; s += BL_THREADS) tab[(uint64_t)s * td.in.bl_nchunks + c] = lh[s];
}

// Row scan: for slice s of a tensor (one block each), offsets of its chunks
// within the slice's bucket, and the bucket's size.
__global__ __launch_bounds__(NTHREADS) void k_bloom_rowscan(Work w, uint32_t r, uint32_t hpr, int from_bitmap) {
    __shared__ uint32_t scratch[NWAVES + 1];
    const uint32_t t = tensor_of_slice(w, blockIdx.x);
    const TDesc &td = w.td[t];
    const uint32_t s = blockIdx.x - td.in.bl_slice0;
    uint32_t j0, je;
    bl_round(td, r, hpr, &j0, &je);
    if (s >= td.in.bl_nslices || j0 >= je) return;
    const uint32_t sl2 = td.in.slice_log2;
    const uint32_t nsl = (td.m_words * 32u + (1u << sl2) - 1) >> sl2;
    if (s >= nsl) return;
    const uint32_t nact = active_chunks(td, from_bitmap != 0);
    uint32_t *row = w.btab + td.in.bl_tab0 + (uint64_t)s * td.in.bl_nchunks;
    uint32_t carry = 0;
    for (uint32_t c0 = 0; c0 < nact; c0 += NTHREADS) {
        const uint32_t c = c0 + threadIdx.x;
        const uint32_t v = c < nact ? row[c] : 0u;
        uint32_t tot;
        const uint32_t ex = block_excl_scan(v, scratch, &tot);
        if (c < nact) row[c] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) w.brow[blockIdx.x] = carry;
}

constexpr uint32_t SCAN_THREADS = 1024;

// per tensor: start of each slice's bucket; the end of the last goes to bl_end
__global__ __launch_bounds__(SCAN_THREADS) void k_bloom_rowbase(Work w, uint32_t r, uint32_t hpr) {
    TDesc &td = w.td[blockIdx.x];
    uint32_t j0, je;
    bl_round(td, r, hpr, &j0, &je);
    if (j0 >= je) return;
    __shared__ uint32_t scratch[SCAN_THREADS / 64 + 1];
    const uint32_t sl2 = td.in.slice_log2;
    const uint32_t nsl = (td.m_words * 32u + (1u << sl2) - 1) >> sl2;
    const uint32_t *tot = w.brow + td.in.bl_slice0;
    uint32_t *base = w.brow + w.bslices + td.in.bl_slice0;
    uint32_t carry = 0;
    for (uint32_t q0 = 0; q0 < nsl; q0 += SCAN_THREADS) {
        const uint32_t q = q0 + threadIdx.x;
        const uint32_t v = q < nsl ? tot[q] : 0u;
        uint32_t sum;
        const uint32_t ex = block_excl_scan_n<SCAN_THREADS>(v, scratch, &sum);
        if (q < nsl) base[q] = carry + ex;
        carry += sum;
    }
    if (threadIdx.x == 0) td.bl_end = carry;
}

// Scatter: each position goes to its slice's bucket, after the chunk's
// offset within that bucket, as a 32-bit offset within the slice.  A block
// takes its chunk's items 4096 at a time and their positions two hashes at
// a time (8 K positions), groups them by slice in LDS (a counting sort:
// ranks from LDS atomics, a scan of the counts, then the placement), and
// writes each slice's run with consecutive lanes on consecutive addresses.
// Stored straight from the hashing lanes, each 4-byte record was an L2
// request of its own, and the pass ran at the L2 request rate.  Two blocks
// share a CU (76 KiB of LDS and at most 64 VGPRs each; four hashes per
// group and one block per CU took 0.68 ms on ncf_32m, two 0.585 ms).
constexpr uint32_t SC_ITEMS = 4096;                      // items per batch
constexpr uint32_t SC_HASHES = 2;                        // hashes per group
constexpr uint32_t SC_PER = SC_ITEMS / BL_THREADS;       // items per thread
constexpr uint32_t SC_STAGE = SC_ITEMS * SC_HASHES;      // positions per group

template <bool FROM_BITMAP>
__global__ __launch_bounds__(BL_THREADS) __attribute__((amdgpu_waves_per_eu(8))) void k_bloom_scatter(Work w, uint32_t r,
                                                                                                     uint32_t hpr) {
    __shared__ uint32_t gcur[BL_MAX_SLICES];  // next record of this chunk in each slice's bucket
    __shared__ uint32_t cnt[BL_MAX_SLICES];   // the group's positions per slice
    __shared__ uint32_t off[BL_MAX_SLICES];   // their start in the staging area
    __shared__ uint32_t items[SC_ITEMS];
    __shared__ uint32_t stage[SC_STAGE];
    __shared__ uint16_t sbkt[SC_STAGE];
    __shared__ uint32_t scratch[BL_THREADS / 64 + 1];
    __shared__ uint32_t s_nitems;
    const uint32_t t = tensor_of_chunk(w, blockIdx.x);
    TDesc &td = w.td[t];
    const uint32_t c = blockIdx.x - td.in.bl_chunk0;
    if (c >= td.in.bl_nchunks || c >= active_chunks(td, FROM_BITMAP)) return;
    uint32_t j0, je;
    bl_round(td, r, hpr, &j0, &je);
    if (je <= j0) return;
    const uint32_t m_bits = td.m_words * 32u;
    __shared__ uint32_t ps[33];
    const bool part = td.in.layout == LAYOUT_PARTITIONED;
    if (part) fill_part_starts(ps, m_bits, td.in.k);  // read after the barrier below
    const PosMap pm{m_bits, part ? ps : nullptr};
    const uint32_t sl2 = td.in.slice_log2;
    const uint32_t nsl = (m_bits + (1u << sl2) - 1) >> sl2;
    if (nsl > BL_MAX_SLICES) {  // excluded by the plan
        if (threadIdx.x == 0) atomicOr(&td.flags, FLAG_CAPACITY);
        return;
    }
    const uint32_t *tab = w.btab + td.in.bl_tab0;
    const uint32_t *base = w.brow + w.bslices + td.in.bl_slice0;
    for (uint32_t s = threadIdx.x; s < nsl; s += BL_THREADS) {
        gcur[s] = base[s] + tab[(uint64_t)s * td.in.bl_nchunks + c];
        cnt[s] = 0;
    }
    uint32_t *pos = w.bpos + td.in.bl_pos0;
    const uint64_t poscap = td.in.bl_poscap;
    const uint32_t mask = (1u << sl2) - 1;
    // the chunk's items: bitmap words [x0, x1) or list entries [x0, x1)
    uint32_t x0, x1;
    const uint32_t *src;
    if (FROM_BITMAP) {
        x0 = c * td.in.bl_chunk * TILE_WORDS;
        x1 = min(td.in.ntiles * TILE_WORDS, x0 + td.in.bl_chunk * TILE_WORDS);
        src = w.selbits + (td.in.slot >> 5);
    } else {
        x0 = c * td.in.bl_chunk;
        x1 = min(td.n, x0 + td.in.bl_chunk);
        src = w.S + td.in.slot;
    }
    __syncthreads();
    while (x0 < x1) {
        // 1. the batch's items into LDS
        uint32_t nitems;
        if (FROM_BITMAP) {
            // the longest run of words from x0 whose items fit (one word at least)
            const uint32_t x = x0 + threadIdx.x;
            const uint32_t word = x < x1 ? src[x] : 0u;
            const uint32_t pc = __popc(word);
            uint32_t tot;
            const uint32_t ex = block_excl_scan_n<BL_THREADS, true>(pc, scratch, &tot);
            const bool take = ex + pc <= SC_ITEMS;  // a prefix of the threads
            if (take) {
                uint32_t wd = word, e = ex;
                while (wd) {
                    items[e++] = x * 32u + (uint32_t)(__ffs(wd) - 1);
                    wd &= wd - 1;
                }
            }
            const uint32_t ntake = (uint32_t)__syncthreads_count(take);
            if (take && threadIdx.x == ntake - 1) s_nitems = ex + pc;
            __syncthreads();
            nitems = s_nitems;
            x0 += ntake;
        } else {
            nitems = min(SC_ITEMS, x1 - x0);
#pragma unroll
            for (uint32_t u = 0; u < SC_PER; ++u) {
                const uint32_t i = u * BL_THREADS + threadIdx.x;
                if (i < nitems) items[i] = src[x0 + i];
            }
            x0 += nitems;
            __syncthreads();
        }
        uint32_t km[SC_PER];
#pragma unroll
        for (uint32_t u = 0; u < SC_PER; ++u) {
            const uint32_t i = u * BL_THREADS + threadIdx.x;
            km[u] = i < nitems ? mm3_key(items[i]) : 0u;
        }
        for (uint32_t jg = j0; jg < je; jg += SC_HASHES) {
            // 2. positions, and their ranks within their slice's group
            uint32_t pr[SC_PER * SC_HASHES], br[SC_PER * SC_HASHES];
#pragma unroll
            for (uint32_t u = 0; u < SC_PER; ++u) {
                const bool iv = u * BL_THREADS + threadIdx.x < nitems;
#pragma unroll
                for (uint32_t v = 0; v < SC_HASHES; ++v) {
                    const uint32_t q = u * SC_HASHES + v;
                    br[q] = 0xffffffffu;
                    pr[q] = 0;
                    if (iv && jg + v < je) {
                        const uint32_t p = pm(km[u], jg + v);
                        const uint32_t b = p >> sl2;
                        br[q] = (b << 16) | atomicAdd(&cnt[b], 1u);
                        pr[q] = p & mask;
                    }
                }
            }
            lds_barrier();
            // 3. each slice's place in the staging area
            uint32_t tot;
            const uint32_t ex = block_excl_scan_n<BL_THREADS, true>(threadIdx.x < nsl ? cnt[threadIdx.x] : 0u, scratch,
                                                                    &tot);
            if (threadIdx.x < nsl) off[threadIdx.x] = ex;
            lds_barrier();
#pragma unroll
            for (uint32_t q = 0; q < SC_PER * SC_HASHES; ++q) {
                if (br[q] != 0xffffffffu) {
                    const uint32_t b = br[q] >> 16;
                    const uint32_t at = off[b] + (br[q] & 0xffffu);
                    stage[at] = pr[q];
                    sbkt[at] = (uint16_t)b;
                }
            }
            lds_barrier();
            // 4. each slice's run, coalesced, after the chunk's earlier records
            for (uint32_t i = threadIdx.x; i < tot; i += BL_THREADS) {
                const uint32_t b = sbkt[i];
                const uint32_t g = gcur[b] + (i - off[b]);
                if (g < poscap) pos[g] = stage[i];
            }
            lds_barrier();
            for (uint32_t s = threadIdx.x; s < nsl; s += BL_THREADS) {
                gcur[s] += cnt[s];
                cnt[s] = 0;
            }
            lds_barrier();
        }
    }
}

// Fill: one block per slice sets its bucket's bits in an LDS copy of the
// slice (up to 128 KiB) and writes the slice out.
__global__ __launch_bounds__(BL_THREADS) void k_bloom_fill(Work w, uint32_t r, uint32_t hpr) {
    __shared__ uint32_t words[SLICE_WORDS_MAX];
    const uint32_t t = tensor_of_slice(w, blockIdx.x);
    const TDesc &td = w.td[t];
    const uint32_t s = blockIdx.x - td.in.bl_slice0;
    if (s >= td.in.bl_nslices) return;
    uint32_t j0, je;
    bl_round(td, r, hpr, &j0, &je);
    // a round past the tensor's last leaves its filter alone; round 0 of a
    // tensor with no hashes (k = 0) still writes its empty slices
    if (r > 0 && j0 >= je) return;
    const uint32_t m_words = td.m_words;
    const uint32_t m_bits = m_words * 32u;
    const uint32_t sl2 = td.in.slice_log2;
    const uint32_t slice_words = (1u << sl2) / 32u;
    const uint32_t nsl = (m_bits + (1u << sl2) - 1) >> sl2;
    if (s >= nsl) return;
    uint32_t *out = td.in.bits + (uint64_t)s * slice_words;
    const uint32_t lim = min(slice_words, m_words - s * slice_words);
    // the first round starts from an empty slice, later rounds add to it
    for (uint32_t i = threadIdx.x; i < slice_words; i += BL_THREADS) words[i] = (r > 0 && i < lim) ? out[i] : 0u;
    __syncthreads();
    if (je > j0) {
        const uint32_t start = w.brow[w.bslices + blockIdx.x];
        uint32_t end = start + w.brow[blockIdx.x];
        if (end > td.in.bl_poscap) end = (uint32_t)td.in.bl_poscap;
        const uint32_t *pos = w.bpos + td.in.bl_pos0;
        if (td.in.bl_nchunks > 0) {
            // eight loads in flight per thread before their bits are set
            constexpr uint32_t U = 8;
            for (uint32_t q0 = start; q0 < end; q0 += U * BL_THREADS) {
                uint32_t p[U];
#pragma unroll
                for (uint32_t u = 0; u < U; ++u) {
                    const uint32_t q = q0 + u * BL_THREADS + threadIdx.x;
                    p[u] = q < end ? pos[q] : 0xffffffffu;
                }
#pragma unroll
                for (uint32_t u = 0; u < U; ++u)
                    if (p[u] != 0xffffffffu) atomicOr(&words[p[u] >> 5], 1u << (p[u] & 31u));
            }
        }
    }
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < lim; i += BL_THREADS) out[i] = words[i];
}

// ---------------------------------------------------------------------------
// Direct insert, for filters of at most DIR_MAX_BITS bits: block (s, c) of
// a tensor hashes the items of chunk c, sets the bits that fall in slice s
// in a 128 KiB LDS copy, and writes that copy to its own partial slice; a
// second kernel ORs each slice's partials.  OR is commutative, so the
// filter is the same as any other insertion order gives.  Two launches and
// no position buffer: the hashing is repeated once per slice, which is
// cheap for the few slices such filters have.
// ---------------------------------------------------------------------------
constexpr uint32_t DIR_THREADS = 1024;

__device__ __forceinline__ uint32_t tensor_of_dir_block(const Work &w, uint32_t b) {
    uint32_t lo = 0, hi = w.ntensors;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (w.td[mid].in.dir_blk0 <= b)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

__device__ __forceinline__ uint32_t tensor_of_dir_slice(const Work &w, uint32_t s) {
    uint32_t lo = 0, hi = w.ntensors;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (w.td[mid].in.dir_sl0 <= s)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

template <bool FROM_BITMAP>
__global__ __launch_bounds__(DIR_THREADS) void k_bloom_direct(Work w) {
    __shared__ __attribute__((aligned(16))) uint32_t sl[DIR_SLICE_WORDS];
    __shared__ uint32_t queue[DIR_THREADS / 64][128];  // per wave: selected indices waiting to be hashed
    const uint32_t t = tensor_of_dir_block(w, blockIdx.x);
    const TDesc &td = w.td[t];
    const uint32_t local = blockIdx.x - td.in.dir_blk0;
    const uint32_t G = td.in.dir_g;
    if (local >= td.in.dir_nsl * G) return;
    const uint32_t s = local / G, c = local % G;
    const uint32_t m_words = td.m_words, m_bits = m_words * 32u, k = td.in.k;
    const uint32_t w0 = s * DIR_SLICE_WORDS;
    if (w0 >= m_words) return;  // past the filter this call built
    const uint32_t nw = min(DIR_SLICE_WORDS, m_words - w0);
    const uint32_t b0 = w0 * 32u, nb = nw * 32u;
    const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
    __shared__ uint32_t ps[33];
    const bool parts = td.in.layout == LAYOUT_PARTITIONED;
    if (parts) fill_part_starts(ps, m_bits, k);
    const PosMap pm{m_bits, parts ? ps : nullptr};
    for (uint32_t i = threadIdx.x; i < DIR_SLICE_WORDS / 4; i += DIR_THREADS) ((uint4 *)sl)[i] = make_uint4(0, 0, 0, 0);
    __syncthreads();
    // the hashes that can land in this slice: all, or (partitioned) those
    // whose part meets [b0, b0 + nb)
    uint32_t jlo = 0, jhi = k;
    if (parts) {
        while (jlo < k && ps[jlo + 1] <= b0) ++jlo;
        jhi = jlo;
        while (jhi < k && ps[jhi] < b0 + nb) ++jhi;
    }
    auto add = [&](uint32_t x) {
        const uint32_t km = mm3_key(x);
        for (uint32_t j = jlo; j < jhi; ++j) {
            const uint32_t p = pm(km, j) - b0;  // wraps for positions below the slice
            if (p < nb) atomicOr(&sl[p >> 5], 1u << (p & 31u));
        }
    };
    if (FROM_BITMAP) {
        // chunk c's bitmap words [wa, wb); chunks past the tensor's tiles
        // (more chunks than tiles) are empty
        const Range32 cw = dir_bitmap_chunk(td.in.ntiles, td.in.dir_per, c, TILE_WORDS);
        const uint32_t wa = cw.lo, wb = cw.hi;
        // eight bitmap words per thread in flight, read through a buffer
        // view of the chunk (reads past it return 0).  A wave's selected
        // indices go through its queue, and are hashed 64 at a time, so all
        // lanes work however sparse the bitmap is.
        const __amdgpu_buffer_rsrc_t sv = buffer_view(w.selbits + (td.in.slot >> 5) + wa, 4u * (wb - wa));
        uint32_t *q = queue[wv];
        uint32_t qn = 0;
        for (uint32_t x0 = 0; x0 < wb - wa; x0 += 8 * DIR_THREADS) {
            uint32_t wd[8];
#pragma unroll
            for (uint32_t u = 0; u < 8; ++u) wd[u] = buffer_u32(sv, 4u * (x0 + u * DIR_THREADS + threadIdx.x));
#pragma unroll
            for (uint32_t u = 0; u < 8; ++u) {
                uint32_t word = wd[u];
                const uint32_t base = (wa + x0 + u * DIR_THREADS + threadIdx.x) * 32u;
                while (ballot(word != 0u)) {
                    const bool has = word != 0u;
                    const uint32_t item = base + (has ? (uint32_t)(__ffs(word) - 1) : 0u);
                    word &= word - 1u;
                    const uint64_t m = ballot(has);
                    if (has) q[qn + lanes_below(m)] = item;
                    qn += popc64(m);
                    __builtin_amdgcn_wave_barrier();
                    if (qn >= 64) {  // the last 64 entries, one per lane
                        const uint32_t x = q[qn - 64 + lane];
                        __builtin_amdgcn_wave_barrier();
                        qn -= 64;
                        add(x);
                    }
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        if (lane < qn) add(q[lane]);
    } else {
        const Range32 cq = dir_list_chunk(td.n, td.in.dir_per, c);
        const uint32_t qa = cq.lo, qb = cq.hi;
        const __amdgpu_buffer_rsrc_t iv = buffer_view(w.S + td.in.slot + qa, 4u * (qb - qa));
        for (uint32_t x0 = 0; qa + x0 < qb; x0 += 8 * DIR_THREADS) {
            uint32_t it[8];
#pragma unroll
            for (uint32_t u = 0; u < 8; ++u) it[u] = buffer_u32(iv, 4u * (x0 + u * DIR_THREADS + threadIdx.x));
#pragma unroll
            for (uint32_t u = 0; u < 8; ++u)
                if (qa + x0 + u * DIR_THREADS + threadIdx.x < qb) add(it[u]);
        }
    }
    __syncthreads();
    uint32_t *part = w.bpos + td.in.dir_pb + (uint64_t)local * td.in.dir_sw;
    if ((((uintptr_t)part) & 15u) == 0) {
        for (uint32_t i = threadIdx.x; i < nw / 4; i += DIR_THREADS) ((uint4 *)part)[i] = ((const uint4 *)sl)[i];
        for (uint32_t i = (nw & ~3u) + threadIdx.x; i < nw; i += DIR_THREADS) part[i] = sl[i];
    } else {
        for (uint32_t i = threadIdx.x; i < nw; i += DIR_THREADS) part[i] = sl[i];
    }
}

// One thread per filter word: the OR of the word's partials, in chunk order.
__global__ __launch_bounds__(DIR_THREADS) void k_bloom_direct_or(Work w) {
    const uint32_t gs = blockIdx.x / (DIR_SLICE_WORDS / DIR_THREADS);  // slice over all tensors
    const uint32_t part_of_slice = blockIdx.x % (DIR_SLICE_WORDS / DIR_THREADS);
    const uint32_t t = tensor_of_dir_slice(w, gs);
    const TDesc &td = w.td[t];
    const uint32_t s = gs - td.in.dir_sl0;
    if (s >= td.in.dir_nsl) return;
    const uint32_t wi = part_of_slice * DIR_THREADS + threadIdx.x;  // word within the slice
    const uint32_t m_words = td.m_words;
    const uint32_t w0 = s * DIR_SLICE_WORDS;
    if (w0 >= m_words || wi >= min(DIR_SLICE_WORDS, m_words - w0)) return;
    const uint32_t G = td.in.dir_g, sw = td.in.dir_sw;
    const uint32_t *part = w.bpos + td.in.dir_pb + (uint64_t)s * G * sw + wi;
    uint32_t acc = 0;
    uint32_t c = 0;
    for (; c + 8 <= G; c += 8) {  // eight partials in flight
        uint32_t v[8];
#pragma unroll
        for (uint32_t u = 0; u < 8; ++u) v[u] = part[(uint64_t)(c + u) * sw];
#pragma unroll
        for (uint32_t u = 0; u < 8; ++u) acc |= v[u];
    }
    for (; c < G; ++c) acc |= part[(uint64_t)c * sw];
    td.in.bits[w0 + wi] = acc;
}

hipError_t launch_bloom_direct(const Work &w, bool from_bitmap, uint32_t blocks, uint32_t slices, hipStream_t s) {
    if (blocks == 0) return hipSuccess;
    if (from_bitmap)
        k_bloom_direct<true><<<blocks, DIR_THREADS, 0, s>>>(w);
    else
        k_bloom_direct<false><<<blocks, DIR_THREADS, 0, s>>>(w);
    trace_mark(s, "k_bloom_direct");
    k_bloom_direct_or<<<slices * (DIR_SLICE_WORDS / DIR_THREADS), DIR_THREADS, 0, s>>>(w);
    trace_mark(s, "k_bloom_direct_or");
    return hipGetLastError();
}

hipError_t launch_bloom_insert(const Work &w, bool from_bitmap, uint32_t total_chunks, uint32_t total_slices,
                               uint32_t max_slices, uint32_t hash_per_round, uint32_t kmax, hipStream_t s) {
    // LDS for one counter per slice of the largest filter
    const size_t lds = (size_t)max_slices * 4u;
    // the rounds the plan needs; a tensor with fewer items than planned may
    // need fewer (bl_round), and later rounds' kernels skip it
    const uint32_t hpr = std::max<uint32_t>(1, hash_per_round);
    const uint32_t rounds = std::max<uint32_t>(1, (kmax + hpr - 1) / hpr);
    for (uint32_t r = 0; r < rounds; ++r) {
        if (total_chunks) {
            if (from_bitmap)
                k_bloom_count<true><<<total_chunks, BL_THREADS, lds, s>>>(w, r, hpr);
            else
                k_bloom_count<false><<<total_chunks, BL_THREADS, lds, s>>>(w, r, hpr);
            trace_mark(s, "k_bloom_count");
            k_bloom_rowscan<<<total_slices, NTHREADS, 0, s>>>(w, r, hpr, from_bitmap ? 1 : 0);
            trace_mark(s, "k_bloom_rowscan");
            k_bloom_rowbase<<<w.ntensors, SCAN_THREADS, 0, s>>>(w, r, hpr);
            trace_mark(s, "k_bloom_rowbase");
            if (from_bitmap)
                k_bloom_scatter<true><<<total_chunks, BL_THREADS, 0, s>>>(w, r, hpr);
            else
                k_bloom_scatter<false><<<total_chunks, BL_THREADS, 0, s>>>(w, r, hpr);
            trace_mark(s, "k_bloom_scatter");
        }
        k_bloom_fill<<<total_slices, BL_THREADS, 0, s>>>(w, r, hpr);
        trace_mark(s, "k_bloom_fill");
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Full-range query
// ---------------------------------------------------------------------------
// Q_SUM probes like Q_DECODE but leaves the dense output to the summing
// emit pass.
enum QueryMode { Q_ENCODE = 0, Q_PLAIN = 1, Q_DECODE = 2, Q_SUM = 3 };

struct QueryOut {
    const float *g;         // encode: dense gradient (values of the positives)
    uint32_t *idx_out;      // plain: output list; decode: optional positives
    uint64_t cap;           // plain: output capacity
    uint64_t *n_out;        // plain: device count
    float *dense_out;       // decode: dense gradient
    float *val_out;         // decode: optional values
    uint64_t *counts_out;   // decode: optional per-tensor counts (flags word)
    float scale;            // sum: factor applied to the sum
    uint32_t npay;          // sum: payloads
    uint32_t ntens;         // sum: tensors per payload
    uint32_t ntiles1;       // sum: tiles per payload
    int setup;              // encode: block 0 of the emit pass also runs the value set-up
};

struct RecordView {
    const uint32_t *bits;
    const float *coef;
    const uint32_t *knots;  // chord segmentation: the seff - 1 interior run starts
    const uint32_t *sigma;
    uint32_t m_bits, k, npos, nv, policy, seed, deff, seff, b, segmode, model;
    uint32_t layout;  // LAYOUT_* of the filter (from the record's hash id)
};

// A record's fields, and a tensor's, are the same in every lane of a block:
// readfirstlane states it, so that a loop over many tiles keeps them in
// scalar registers rather than in a vector register each.
__device__ __forceinline__ uint32_t uni(uint32_t x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ uint64_t uni(uint64_t x) {
    return ((uint64_t)uni((uint32_t)(x >> 32)) << 32) | uni((uint32_t)x);
}
template <typename T>
__device__ __forceinline__ T *uni(T *p) {
    return (T *)uni((uint64_t)p);
}
__device__ __forceinline__ void uniform_record(RecordView &v) {
    v.bits = uni(v.bits);
    v.coef = uni(v.coef);
    v.knots = uni(v.knots);
    v.sigma = uni(v.sigma);
    v.m_bits = uni(v.m_bits);
    v.k = uni(v.k);
    v.npos = uni(v.npos);
    v.nv = uni(v.nv);
    v.policy = uni(v.policy);
    v.seed = uni(v.seed);
    v.deff = uni(v.deff);
    v.seff = uni(v.seff);
    v.b = uni(v.b);
    v.segmode = uni(v.segmode);
    v.model = uni(v.model);
    v.layout = uni(v.layout);
}

// Reads a record header and checks it against the record's capacity and
// the tensor's size; an invalid record decodes as empty (k = 0) and is
// flagged, so a damaged payload cannot send reads past its record.
__device__ __forceinline__ RecordView read_record(const uint8_t *rec, uint64_t cap, uint32_t d, bool *ok) {
    RecordView v;
    const uint32_t *h = (const uint32_t *)rec;
    const uint64_t m_bits = h[H_MBITS];
    v.m_bits = (uint32_t)m_bits;
    v.npos = h[H_NPOS];
    v.nv = h[H_NVAL];
    v.policy = h[H_POLICY];
    v.seed = h[H_SEED];
    v.k = h[H_K];
    const uint32_t hash_id = h[H_HASH];
    v.layout = hash_id == HASH_ID_PARTITIONED ? LAYOUT_PARTITIONED : LAYOUT_STANDARD;
    v.deff = h[H_DEFF];
    v.seff = h[H_SEFF];
    v.b = h[H_B];
    const uint32_t hw15 = h[H_SEGMODE];  // segmentation | value model << 8 | value source << 16
    v.segmode = hw15 & 0xffu;
    v.model = (hw15 >> 8) & 0xffu;
    const uint32_t vsrc = (hw15 >> 16) & 0xffu;
    v.bits = (const uint32_t *)(rec + HDR_BYTES);
    const uint32_t coef_off = HDR_BYTES + (v.m_bits / 32u) * 4u;
    v.coef = (const float *)(rec + coef_off);
    const uint32_t nknots = v.segmode == SEG_CHORD && v.seff > 1 ? v.seff - 1 : 0u;
    const uint64_t need = (uint64_t)HDR_BYTES + m_bits / 8u + 4ull * v.seff * (v.deff + 1ull) + 4ull * nknots +
                          4ull * (((uint64_t)v.nv * v.b + 31u) / 32u);
    *ok = h[H_MAGIC] == HDR_MAGIC && h[H_BYTES] == HDR_BYTES && m_bits >= 32 && (m_bits & 31u) == 0 && v.k >= 1 &&
          (hash_id == HASH_ID_STANDARD || hash_id == HASH_ID_PARTITIONED) &&
          v.k <= 32 && v.deff <= MAX_DEG && v.b >= 1 && v.b <= 32 && v.npos <= d && v.nv <= v.npos &&
          v.policy <= POLICY_RIGHTMOST && (v.policy != POLICY_P0 || v.nv == v.npos) && v.segmode <= SEG_CHORD &&
          (hw15 >> 24) == 0 && vsrc <= VALUES_SPARSE && v.model <= FIT_DEXP && (v.model != FIT_DEXP || v.deff == 3) &&
          (v.nv == 0 || (v.seff >= 1 && v.seff <= v.nv && v.seff <= MAX_SEG && v.b >= sigma_bits(v.nv))) &&
          need <= cap;
    if (!*ok) {  // nothing of an invalid record is read past its first filter word
        v.k = 0;
        v.layout = LAYOUT_STANDARD;
        v.npos = 0;
        v.nv = 0;
        v.policy = POLICY_P0;
        v.segmode = SEG_EQUAL;
        v.model = FIT_POLY;
        v.m_bits = 32;
        v.seff = 0;
        v.deff = 0;
        v.b = 1;
        v.coef = (const float *)(rec + HDR_BYTES + 4);
    }
    v.knots = (const uint32_t *)((const uint8_t *)v.coef + v.seff * (v.deff + 1u) * 4u);
    v.sigma = v.knots + (*ok ? nknots : 0u);
    return v;
}

// the b-bit entry at bit offset `bit` of a packed LSB-first stream (b <= 32)
__device__ __forceinline__ uint32_t sigma_get(const uint32_t *sig, uint64_t bit, uint32_t b) {
    const uint32_t w0 = sig[bit >> 5], sh = (uint32_t)(bit & 31u);
    uint64_t v = w0 >> sh;
    if (sh + b > 32u) v |= (uint64_t)sig[(bit >> 5) + 1] << (32u - sh);
    return b == 32u ? (uint32_t)v : (uint32_t)(v & ((1ull << b) - 1ull));
}

constexpr uint32_t QWAVE = 512;              // indices per wave per step (an eighth of a tile)
constexpr uint32_t PB_THREADS = 1024;        // probe block: 16 waves, one block per CU
constexpr uint32_t PB_WAVES = PB_THREADS / 64;
constexpr uint32_t PB_TILES = PB_WAVES * QWAVE / TILE;  // tiles one block probes per step
constexpr uint32_t FC_WORDS = 35840;         // filter words kept in LDS (140 KiB)

// The filter a tile is probed against: the sender's freshly built filter,
// the caller's (plain decode), or the payload record's (receiver).
__device__ __forceinline__ RecordView query_filter(const Work &w, const QueryOut &o, TDesc &td, int mode, bool *ok) {
    RecordView rv;
    *ok = true;
    if (mode == Q_DECODE || mode == Q_SUM) {
        rv = read_record(td.in.rec, td.in.rec_cap, td.in.d, ok);
    } else {
        rv.bits = td.in.bits;
        rv.m_bits = td.m_words * 32u;
        rv.k = td.in.k;
        rv.layout = td.in.layout;
    }
    return rv;
}

// One filter word: from the LDS copy of the filter's first `fcw` words, else
// from global memory (an L2 hit: the filter is small and read by every CU).
// A lane that is not `live` (an empty queue slot) makes no memory request.
__device__ __forceinline__ uint32_t filter_word(const uint32_t *fc, uint32_t fcw, __amdgpu_buffer_rsrc_t rs,
                                                uint32_t wi, bool live = true) {
    const bool in_lds = wi < fcw;
    const uint32_t l = fc[in_lds ? wi : 0u];
    // the offset of a word held in LDS, or of a dead lane, lies past the
    // view: no memory access
    const uint32_t g = buffer_u32(rs, (in_lds || !live) ? 0xfffffff0u : wi * 4u);
    return in_lds ? l : g;
}

// Probe pass: the positives of each tile as a bitmap (pbits) and a count
// (tcnt).  The sender already knows that its selected indices are
// positives (S is a subset of P, Section 4), so it skips probing them.
//
// The random filter reads are this kernel's cost: they are L2 hits, and
// the L2-to-CU line transfers bound it.  One 1024-thread block runs per CU
// and keeps the first 140 KiB of the current tensor's filter in LDS, so
// that share of the probes never leaves the CU (all of them for filters up
// to 1,146,880 bits).  Each block owns a contiguous range of tiles, cut into
// runs that stay inside one tensor; the LDS copy is reloaded only when a
// run enters a new tensor.  Inside a run, waves take eighths of a tile (512
// indices) from a shared counter, so they stay busy until the run ends.
// The step is an eighth rather than a quarter so that the waves' survivor
// queues leave LDS room for 20 KiB more of the filter (measured: 3% faster;
// a sixteenth, for 9 KiB more, was slower).
//
// Each probe round costs a wave one L2 round trip.  Once a step's
// survivors fit in one 64-lane group (mostly positives, which take every
// probe), the round trips, not the reads, are the cost: the next TAIL_PROBES
// probes are then read together.  A survivor that fails the first of them
// costs one read it did not need.
constexpr uint32_t RUN_TILES = 512;  // most tiles per run (LDS tile counters)
constexpr uint32_t TAIL_PROBES = 2;  // probes per round once the survivors fit one group

// The tensor totals of the probe pass: the sender's |P| and values coded,
// the plain query's count, or the receiver's |P| (checked against the
// record's header).
template <int MODE>
__device__ void probe_total(const Work &w, const QueryOut &o, uint32_t t, uint32_t total) {
    TDesc &td = w.td[t];
    if (MODE == Q_ENCODE) {
        // the policy codes every positive (P0) or r of them
        td.npos = total;
        td.nv = td.in.policy == POLICY_P0 ? total : min(td.n, total);
        // the record's header is complete here, so the receiver's probe
        // pass can start as soon as this pass ends
        value_setup_tensor(w, t, 1, o.counts_out);
    } else if (MODE == Q_PLAIN) {
        if (o.n_out) *o.n_out = total;  // one tensor
    } else {
        td.nv_dec = total;
        if (o.counts_out) {
            o.counts_out[4 * t + 2] = total;
            if (total != ((const uint32_t *)td.in.rec)[H_NPOS])
                atomicOr((unsigned long long *)&o.counts_out[4 * t + 3], FLAG_DEC_MISMATCH);
        }
    }
}

// The tile scan, at the end of the probe pass: toff = each tile's exclusive
// count within its tensor, and each tensor's total where its last tile
// lies.  Blocks own contiguous tile ranges in block order.  A block
//  1. sums its trailing segment (its tiles of the tensor of its last tile)
//     and publishes it: as inclusive if the block holds that tensor's first
//     tile, else as an aggregate;
//  2. if its first tile continues a tensor that began in an earlier block,
//     wave 0 walks back over the preceding blocks, 64 at a time, adding
//     aggregates until an inclusive entry (decoupled look-back); a block
//     whose range lies inside that tensor then publishes its inclusive sum;
//  3. scans its tiles, segmented at tensor starts.
// A block waits only for blocks with smaller indices, which start first, so
// every wait ends; the wait is bounded anyway and flags the tensor if it
// gives up.  `lds` is the filter copy's LDS, free at this point.
constexpr uint64_t PS_AGG = 1ull << 62, PS_INC = 2ull << 62;
constexpr uint32_t PS_SPIN_LIMIT = 1u << 20;

template <int MODE>
__device__ void probe_scan(const Work &w, const QueryOut &o, uint32_t t_begin, uint32_t t_end, uint32_t *lds) {
    if (t_end <= t_begin) return;  // block-uniform
    const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
    const uint32_t t_first = tensor_of_tile(w, t_begin), t_last = tensor_of_tile(w, t_end - 1);
    const uint32_t tile0_first = w.td[t_first].in.tile0;
    const uint32_t trail0 = max(t_begin, w.td[t_last].in.tile0);
    const bool cont = t_begin > tile0_first;  // the first tensor began in an earlier block
    // 1. the trailing segment's sum
    uint32_t s = 0;
    for (uint32_t t = trail0 + threadIdx.x; t < t_end; t += PB_THREADS) s += w.tcnt[t];
    s = wave_sum(s);
    if (lane == 0) lds[wv] = s;
    __syncthreads();
    s = 0;
    for (uint32_t q = 0; q < PB_WAVES; ++q) s += lds[q];
    uint64_t *st = w.pstat;
    const bool trail_inc = trail0 > t_begin || !cont;
    if (threadIdx.x == 0)
        __hip_atomic_store(&st[blockIdx.x], (trail_inc ? PS_INC : PS_AGG) | s, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();  // lds is rewritten below
    // 2. look-back
    if (cont && wv == 0) {
        uint32_t excl = 0, j = blockIdx.x, rounds = 0;  // next window: blocks j - 1, j - 2, ...
        for (;;) {
            const uint32_t nwin = min(64u, j);
            const bool inw = lane < nwin;
            const uint64_t v = inw ? __hip_atomic_load(&st[j - 1 - lane], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                   : 0ull;
            const uint64_t unpub = ballot(inw && (v >> 62) == 0);
            const uint64_t inc = ballot(inw && (v >> 62) == 2);
            const uint32_t first_unpub = unpub ? (uint32_t)__ffsll((unsigned long long)unpub) - 1 : 64u;
            const uint32_t first_inc = inc ? (uint32_t)__ffsll((unsigned long long)inc) - 1 : 64u;
            if (first_inc < first_unpub) {  // the nearest entries up to an inclusive one are all published
                excl += wave_sum(lane <= first_inc ? (uint32_t)v : 0u);
                break;
            }
            const uint32_t upto = min(first_unpub, nwin);  // published aggregates nearest first
            excl += wave_sum(lane < upto ? (uint32_t)v : 0u);
            j -= upto;
            if (j == 0) break;  // cannot happen: block 0 holds the first tensor's start
            if (upto == 0) {
                if (++rounds >= PS_SPIN_LIMIT) {  // never hang the device on a bug
                    if (lane == 0) {
                        atomicOr(&w.td[t_first].flags, FLAG_STALLED);
                        if (o.counts_out)
                            atomicOr((unsigned long long *)&o.counts_out[4 * t_first + 3], FLAG_STALLED);
                    }
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        if (lane == 0) {
            lds[0] = excl;
            if (t_first == t_last)
                __hip_atomic_store(&st[blockIdx.x], PS_INC | (uint64_t)(excl + s), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    __syncthreads();
    uint32_t carry = cont ? lds[0] : 0u;  // the running count of the segment entering the chunk
    __syncthreads();
    // 3. segmented exclusive scan, PB_THREADS tiles at a time
    for (uint32_t c0 = t_begin; c0 < t_end; c0 += PB_THREADS) {
        const uint32_t t = c0 + threadIdx.x;
        const bool in = t < t_end;
        uint32_t v = 0, tt = 0;
        bool f = false, last = false;
        if (in) {
            v = w.tcnt[t];
            tt = tensor_of_tile(w, t);
            const TInit &ti = w.td[tt].in;
            f = t == ti.tile0;  // a tensor starts here
            last = t + 1 == ti.tile0 + ti.ntiles;
        }
        uint32_t sv = v, sf = f ? 1u : 0u;  // inclusive within the wave: (segment started, sum)
#pragma unroll
        for (uint32_t d = 1; d < 64; d <<= 1) {
            const uint32_t pv = __shfl_up(sv, d, 64), pf = __shfl_up(sf, d, 64);
            if (lane >= d) {
                if (!sf) sv += pv;
                sf |= pf;
            }
        }
        if (lane == 63) {
            lds[wv] = sv;
            lds[PB_WAVES + wv] = sf;
        }
        __syncthreads();
        uint32_t pre = carry;
        for (uint32_t q = 0; q < wv; ++q) pre = lds[PB_WAVES + q] ? lds[q] : pre + lds[q];
        const uint32_t incl = sf ? sv : pre + sv;
        if (in) {
            w.toff[t] = incl - v;
            if (last) probe_total<MODE>(w, o, tt, incl);
        }
        for (uint32_t q = 0; q < PB_WAVES; ++q) carry = lds[PB_WAVES + q] ? lds[q] : carry + lds[q];
        __syncthreads();  // lds is rewritten by the next chunk
    }
}

template <int MODE>
__global__ __launch_bounds__(PB_THREADS) void k_probe(Work w, QueryOut o) {
    __shared__ uint32_t fc[FC_WORDS];
    __shared__ uint16_t qe[PB_WAVES][QWAVE];
    __shared__ uint32_t lw[PB_WAVES][QWAVE / 32];
    __shared__ uint32_t tcl[RUN_TILES];
    __shared__ uint32_t next;
    __shared__ uint32_t ps[33];  // part starts of a partitioned filter
    // the wave index is uniform across the wave; saying so keeps everything
    // derived from it in scalar registers
    const uint32_t lane = threadIdx.x & 63u, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    constexpr uint32_t QPT = TILE / QWAVE;  // steps per tile
    const Range32 own = probe_block_tiles(w.ntiles_total, gridDim.x, blockIdx.x);
    const uint32_t t_begin = own.lo, t_end = own.hi;
    uint32_t cached = 0xffffffffu, fcw = 0;
    for (uint32_t rb = t_begin; rb < t_end;) {
        const uint32_t t = tensor_of_tile(w, rb);
        TDesc &td = w.td[t];
        const uint32_t re = min(min(t_end, td.in.tile0 + td.in.ntiles), rb + RUN_TILES);
        const uint32_t nq = (re - rb) * QPT;
        bool ok;
        const RecordView rv = query_filter(w, o, td, MODE, &ok);
        // a tensor the bucketed query has done: its positives bitmap is
        // written, and the pass only counts it
        const bool pre = __builtin_amdgcn_readfirstlane(td.qb) != 0u;
        // The sender knows its own selection to be positives.  Where it is
        // dense (an inherently sparse gradient's support, or r >= d / 8),
        // the step reads its selection bits first and skips the filter
        // reads of those indices (ncf_32m, 60% selected: 0.76 -> 0.45 ms);
        // where it is sparse the extra dependency costs more than the few
        // reads it saves (resnet50_25m 167 -> 171 us, transformer 1.25 ->
        // 1.40 ms), and the selection bits are read beside the filter's
        const bool dense_sel =
            MODE == Q_ENCODE &&
            __builtin_amdgcn_readfirstlane(td.in.r == R_NONZERO || 8ull * td.in.r >= td.in.d ? 1u : 0u) != 0u;
        __syncthreads();  // the previous run is finished with fc, tcl and next
        if (t != cached) {
            fcw = pre ? 0u : min(rv.m_bits / 32u, FC_WORDS);
            for (uint32_t x = threadIdx.x; x < fcw; x += PB_THREADS) fc[x] = rv.bits[x];
            if (rv.layout == LAYOUT_PARTITIONED) fill_part_starts(ps, rv.m_bits, rv.k);
            cached = t;
        }
        for (uint32_t x = threadIdx.x; x < re - rb; x += PB_THREADS) tcl[x] = 0;
        if (threadIdx.x == 0) {
            next = 0;
            if ((MODE == Q_DECODE || MODE == Q_SUM) && !ok) {
                atomicOr(&td.flags, FLAG_DEC_MISMATCH);
                if (o.counts_out) atomicOr((unsigned long long *)&o.counts_out[4 * t + 3], FLAG_DEC_MISMATCH);
            }
        }
        __syncthreads();
        const uint32_t m_bits = rv.m_bits, k = rv.k, d = td.in.d;
        const __amdgpu_buffer_rsrc_t bits = buffer_view(rv.bits, m_bits / 8u);
        // with the partitioned layout the first parts, those of the first
        // probes, are the ones held in LDS
        const PosMap pm{m_bits, rv.layout == LAYOUT_PARTITIONED ? ps : nullptr};
        uint16_t *me = qe[wv];
        uint32_t *mw = lw[wv];
        for (;;) {
            uint32_t qi = 0;
            if (lane == 0) qi = atomicAdd(&next, 1u);
            qi = __builtin_amdgcn_readfirstlane(qi);
            if (qi >= nq) break;
            const uint32_t tile = rb + qi / QPT;
            const uint32_t wbase = (tile - td.in.tile0) * TILE + (qi % QPT) * QWAVE;  // first index
            if (MODE == Q_DECODE) {
                // the receiver's dense output starts as zeros here, written
                // while the filter reads (an L2-bound loop) are in flight;
                // the emit pass then stores only the positives.  The zeros
                // are stored non-temporally: they are not read again here,
                // and the filter's lines keep the L2 to themselves
                // (resnet50_25m: 192 -> 187.5 us)
                float *dz = o.dense_out + td.in.off + wbase;
                if (wbase + QWAVE <= d && ((uintptr_t)dz & 15u) == 0) {
                    typedef float f4 __attribute__((ext_vector_type(4)));
                    const f4 zero4 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                    for (uint32_t u = 0; u < QWAVE / 256; ++u)
                        __builtin_nontemporal_store(zero4, &((f4 *)dz)[u * 64 + lane]);
                } else {
                    for (uint32_t e = lane; e < QWAVE; e += 64)
                        if (wbase + e < d) dz[e] = 0.0f;
                }
            }
            if (pre) {
                const uint32_t pw =
                    lane < QWAVE / 32 ? w.pbits[(uint64_t)tile * TILE_WORDS + (qi % QPT) * (QWAVE / 32) + lane] : 0u;
                const uint32_t pc = wave_sum(__popc(pw));
                if (lane == 0) atomicAdd(&tcl[qi / QPT], pc);
                // the wave reconverges here, before the next step's ticket:
                // without it the compiler merged this lane-0 branch with
                // the ticket's (also lane 0), so that lanes 1..63 reached
                // the ticket's readfirstlane without lane 0, read step 0
                // from it again and again, and the pass never ended
                __builtin_amdgcn_wave_barrier();
                continue;
            }
            if (lane < QWAVE / 32) mw[lane] = 0;
            __builtin_amdgcn_wave_barrier();
            // probe 0 over the step's 512 indices: 8 per lane, all reads
            // in flight before any is tested
            uint32_t cnt = 0, known = 0;
            uint32_t wrd[QWAVE / 64], sel[QWAVE / 64];
            if (dense_sel) {
                // the selection bits first; no filter read for an index of
                // the selection or past the tensor's end
#pragma unroll
                for (uint32_t c = 0; c < QWAVE / 64; ++c) {
                    const uint32_t i = wbase + c * 64 + lane;
                    sel[c] = i < d ? w.selbits[(td.in.slot + i) >> 5] : 0u;
                }
#pragma unroll
                for (uint32_t c = 0; c < QWAVE / 64; ++c) {
                    const uint32_t i = wbase + c * 64 + lane;
                    const uint32_t p = pm(mm3_key(i), 0);
                    const bool need = i < d && !((sel[c] >> (lane & 31u)) & 1u);
                    const uint32_t word = filter_word(fc, fcw, bits, p >> 5, need) >> (p & 31u);
                    wrd[c] = (i < d && k > 0) ? word : 0u;
                }
            } else {
#pragma unroll
                for (uint32_t c = 0; c < QWAVE / 64; ++c) {
                    const uint32_t i = wbase + c * 64 + lane;
                    const uint32_t p = pm(mm3_key(i), 0);
                    // p < m_bits always, so the read is in bounds; i past the
                    // tensor's end stays inside its slot and is masked below
                    const uint32_t word = filter_word(fc, fcw, bits, p >> 5) >> (p & 31u);
                    wrd[c] = (i < d && k > 0) ? word : 0u;
                    if (MODE == Q_ENCODE) {
                        const uint32_t sw = w.selbits[(td.in.slot + i) >> 5];
                        sel[c] = i < d ? sw : 0u;
                    }
                }
            }
#pragma unroll
            for (uint32_t c = 0; c < QWAVE / 64; ++c) {
                const uint32_t e = c * 64 + lane;
                bool in_s = false;
                if (MODE == Q_ENCODE) in_s = (sel[c] >> (e & 31u)) & 1u;
                const bool hit = !in_s && (wrd[c] & 1u);
                if (MODE == Q_ENCODE) {
                    const uint64_t sm = ballot(in_s);
                    if (lane < 2) mw[c * 2 + lane] |= (uint32_t)(sm >> (32 * lane));
                    known += popc64(sm);
                }
                const uint64_t mask = ballot(hit);
                if (hit) me[cnt + lanes_below(mask)] = (uint16_t)e;
                cnt += popc64(mask);
            }
            // probes 1..k-1 over the survivors, compacted in place in index
            // order; four groups of 64 queue entries have their reads in
            // flight together
            constexpr uint32_t G = 4;
            for (uint32_t j = 1; j < k && cnt > 0; ++j) {
                __builtin_amdgcn_wave_barrier();
                const uint32_t L = cnt;
                if (L <= 64) {
                    // survivor x in lane x; probes j .. j + S - 1 in flight together
                    const uint32_t S = min(k - j, TAIL_PROBES);
                    const bool act = lane < L;
                    const uint32_t e = act ? me[lane] : 0u;
                    const uint32_t key = mm3_key(wbase + e);
                    uint32_t all = 1u;
#pragma unroll
                    for (uint32_t u = 0; u < TAIL_PROBES; ++u) {
                        if (u < S) {
                            const uint32_t p = pm(key, j + u);
                            all &= filter_word(fc, fcw, bits, p >> 5, act) >> (p & 31u);
                        }
                    }
                    const bool hit = act && (all & 1u);
                    __builtin_amdgcn_wave_barrier();
                    const uint64_t mask = ballot(hit);
                    if (hit) me[lanes_below(mask)] = (uint16_t)e;
                    cnt = popc64(mask);
                    j += S - 1;
                    continue;
                }
                cnt = 0;
                for (uint32_t b0 = 0; b0 < L; b0 += 64 * G) {
                    uint32_t ev[G], bw[G];
#pragma unroll
                    for (uint32_t u = 0; u < G; ++u) {
                        const uint32_t x = b0 + u * 64 + lane;
                        ev[u] = x < L ? me[x] : 0u;
                        bw[u] = 0u;
                    }
#pragma unroll
                    for (uint32_t u = 0; u < G; ++u) {
                        if (b0 + u * 64 >= L) break;  // this group and the ones after it are empty
                        const bool live = b0 + u * 64 + lane < L;
                        const uint32_t p = pm(mm3_key(wbase + ev[u]), j);
                        const uint32_t word = filter_word(fc, fcw, bits, p >> 5, live) >> (p & 31u);
                        bw[u] = live ? word : 0u;
                    }
                    __builtin_amdgcn_wave_barrier();
#pragma unroll
                    for (uint32_t u = 0; u < G; ++u) {
                        if (b0 + u * 64 >= L) break;
                        const bool hit = bw[u] & 1u;
                        const uint64_t mask = ballot(hit);
                        if (hit) me[cnt + lanes_below(mask)] = (uint16_t)ev[u];
                        cnt += popc64(mask);
                    }
                    __builtin_amdgcn_wave_barrier();
                }
            }
            __builtin_amdgcn_wave_barrier();
            for (uint32_t x = lane; x < cnt; x += 64) {
                const uint32_t e = me[x];
                atomicOr(&mw[e >> 5], 1u << (e & 31u));
            }
            __builtin_amdgcn_wave_barrier();
            if (lane < QWAVE / 32) w.pbits[(uint64_t)tile * TILE_WORDS + (qi % QPT) * (QWAVE / 32) + lane] = mw[lane];
            if (lane == 0) atomicAdd(&tcl[qi / QPT], cnt + known);
            __builtin_amdgcn_wave_barrier();
        }
        __syncthreads();
        for (uint32_t x = threadIdx.x; x < re - rb; x += PB_THREADS) w.tcnt[rb + x] = tcl[x];
        rb = re;
    }
    __syncthreads();  // the block's tile counts are written; fc is free
    probe_scan<MODE>(w, o, t_begin, t_end, fc);
}

// ---------------------------------------------------------------------------
// Bucketed query
// ---------------------------------------------------------------------------
// For a filter larger than an XCD's L2, every probe of the probe pass is a
// random read from the last-level cache, and the pass runs at the fabric's
// rate for such reads (ncf_32m: the receiver's 273 M probes of a 46 MB
// filter, most of them the k probes of each of its 19 M positives).  The
// receiver's bucketed query takes the probes one hash at a time and brings
// them to the filter instead:
//  * round j < k: the live indices (round 0: all of the tensor's) are
//    counted per chunk of the list and per bin, the bin being the filter
//    slice (2^QB_SL bits) that hash j's bit falls in; a scan of the counts
//    gives each (bin, chunk) its place, and a scatter writes the indices
//    bin by bin (qbkt).  One block per slice then loads its slice into LDS
//    and tests its bin's indices, writing each index, or QB_DEAD where its
//    bit is clear, to the same place of qlist: the next round's list.  In
//    round 0 the chunks are QB_CH consecutive indices and a count pass
//    counts them; in later rounds chunk s is what test block s wrote, and
//    that block counts its survivors by their next bin itself (a count
//    pass per round cost about 0.85 ms on ncf_32m);
//  * round k: the survivors, which are the positives, are bucketed the same
//    way by index region (2^QB_RL indices), and one block per region sets
//    their bits in an LDS copy of the region's bitmap and writes it out.
// The probe pass then only counts that bitmap.  Every global access is a
// stream; the random ones go to LDS.  The kernels are launched per tensor
// and decide alike, from the record's header, whether the tensor is theirs
// (k as planned, a filter of at least min_bits that the work has room
// for); one that is not is left to the probe pass.  The sender keeps its
// probe pass: it skips its own selection, so it probes far fewer indices,
// most of them once, and the rounds' fixed costs outweigh what they save
// there (ncf_32m: 1.17 ms in rounds against 0.76 ms).
struct QbArgs {
    uint32_t t;         // tensor
    uint32_t k;         // hashes planned on the host
    uint32_t min_bits;  // smallest filter taken this way
    uint32_t nsl_cap;   // slices the work has room for
    uint32_t ncol;      // columns of qtab: at least round 0's chunks and nsl_cap
};

constexpr uint32_t QB_TEST_THREADS = 512;

__device__ __forceinline__ uint32_t qb_slices(uint32_t m_bits) {
    return (uint32_t)(((uint64_t)m_bits + (1u << QB_SL) - 1) >> QB_SL);
}
__device__ __forceinline__ uint32_t qb_regions(uint32_t d) {
    return (uint32_t)(((uint64_t)d + (1u << QB_RL) - 1) >> QB_RL);
}

__device__ __forceinline__ bool qb_usable(const RecordView &rv, bool ok, const TDesc &td, const QbArgs &a) {
    return ok && rv.k >= 1 && rv.k == a.k && rv.m_bits >= a.min_bits && qb_slices(rv.m_bits) <= a.nsl_cap &&
           td.in.d >= 1 && td.in.d <= QB_MAX_D;
}

// v[0] + ... + v[n-1], for every thread of the block (NT threads)
template <uint32_t NT>
__device__ __forceinline__ uint32_t qb_sum(const uint32_t *v, uint32_t n, uint32_t *scratch) {
    uint32_t s = 0;
    for (uint32_t b = threadIdx.x; b < n; b += NT) s += v[b];
    s = wave_sum(s);
    __syncthreads();  // scratch is free
    if ((threadIdx.x & 63u) == 0) scratch[threadIdx.x >> 6] = s;
    __syncthreads();
    uint32_t tot = 0;
#pragma unroll
    for (uint32_t q = 0; q < NT / 64; ++q) tot += scratch[q];
    __syncthreads();  // every thread has read scratch
    return tot;
}

// Entries [b0, b0 + QB_SUB) of round j's list, QB_PER per thread; QB_DEAD
// at and past `len` and for an index that failed a probe.
__device__ __forceinline__ void qb_load(const Work &w, uint32_t j, uint32_t b0, uint32_t len, uint32_t *e) {
    const uint32_t x0 = b0 + threadIdx.x;
    if (j == 0) {
#pragma unroll
        for (uint32_t u = 0; u < QB_PER; ++u) {
            const uint32_t x = x0 + u * QB_THREADS;
            e[u] = x < len ? x : QB_DEAD;
        }
    } else {
#pragma unroll
        for (uint32_t u = 0; u < QB_PER; ++u) {
            const uint32_t x = x0 + u * QB_THREADS;
            e[u] = x < len ? w.qlist[x] : QB_DEAD;
        }
    }
}

// bin of index i in round j: the slice of hash j's bit, or (last round) the
// index region
__device__ __forceinline__ uint32_t qb_key(const PosMap &pm, uint32_t i, uint32_t j, bool fin) {
    return fin ? (i >> QB_RL) : (pm(mm3_key(i), j) >> QB_SL);
}

// Round 0: counts of chunk c's indices (QB_CH consecutive ones) per bin:
// column c of qtab.  The first block marks the tensor as taken this way.
template <int MODE>
__global__ __launch_bounds__(QB_THREADS) void k_qb_count(Work w, QbArgs a) {
    __shared__ uint32_t h[QB_MAX_BINS];
    __shared__ uint32_t ps[33];
    TDesc &td = w.td[a.t];
    const QueryOut o{};
    bool ok;
    const RecordView rv = query_filter(w, o, td, MODE, &ok);
    if (!qb_usable(rv, ok, td, a)) return;
    if (blockIdx.x == 0 && threadIdx.x == 0) td.qb = 1u;
    const uint32_t d = td.in.d, nb = qb_slices(rv.m_bits);
    const uint32_t c = blockIdx.x;
    if ((uint64_t)c * QB_CH >= d) return;
    const bool part = rv.layout == LAYOUT_PARTITIONED;
    if (part) fill_part_starts(ps, rv.m_bits, rv.k);
    for (uint32_t b = threadIdx.x; b < nb; b += QB_THREADS) h[b] = 0;
    __syncthreads();
    const PosMap pm{rv.m_bits, part ? ps : nullptr};
    for (uint32_t b0 = c * QB_CH; b0 < min(d, (c + 1) * QB_CH); b0 += QB_SUB) {
        uint32_t e[QB_PER];
        qb_load(w, 0, b0, d, e);
#pragma unroll
        for (uint32_t u = 0; u < QB_PER; ++u) {
            if (e[u] != QB_DEAD) {
                const uint32_t b = qb_key(pm, e[u], 0, false);
                if (b < nb) atomicAdd(&h[b], 1u);
            }
        }
    }
    __syncthreads();
    for (uint32_t b = threadIdx.x; b < nb; b += QB_THREADS) w.qtab[(uint64_t)b * a.ncol + c] = h[b];
}

// Round j's chunks: QB_CH consecutive indices in round 0, else the buckets
// of round j - 1 (chunk s: the places test block s wrote in qlist).
__device__ __forceinline__ uint32_t qb_chunks(const TDesc &td, uint32_t j, uint32_t nsl) {
    return j == 0 ? (td.in.d + QB_CH - 1) / QB_CH : nsl;
}

// One block per bin: its row of qtab becomes each chunk's offset within the
// bin's bucket, and the bin's total goes to qrow.
template <int MODE>
__global__ __launch_bounds__(QB_THREADS) void k_qb_scan(Work w, QbArgs a, uint32_t j) {
    __shared__ uint32_t scratch[QB_THREADS / 64 + 1];
    TDesc &td = w.td[a.t];
    if (!td.qb) return;
    const QueryOut o{};
    bool ok;
    const RecordView rv = query_filter(w, o, td, MODE, &ok);
    const uint32_t d = td.in.d, nsl = qb_slices(rv.m_bits);
    const uint32_t nb = j == rv.k ? qb_regions(d) : nsl;
    const uint32_t b = blockIdx.x;
    if (b >= nb) return;
    const uint32_t nch = qb_chunks(td, j, nsl);
    uint32_t *row = w.qtab + (uint64_t)b * a.ncol;
    uint32_t carry = 0;
    for (uint32_t c0 = 0; c0 < nch; c0 += QB_THREADS) {
        const uint32_t c = c0 + threadIdx.x;
        const uint32_t v = c < nch ? row[c] : 0u;
        uint32_t tot;
        const uint32_t ex = block_excl_scan_n<QB_THREADS>(v, scratch, &tot);
        if (c < nch) row[c] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) w.qrow[j * QB_MAX_BINS + b] = carry;
}

// Chunk c's entries into their bins' buckets (qbkt), QB_SUB at a time:
// grouped by bin in LDS (ranks from LDS atomics, a scan of the bins'
// counts, the placement), then written bin by bin, so that consecutive
// lanes store to consecutive addresses.  The order within a bucket does not
// matter: a bucket's indices are tested independently, and the positives
// end up in a bitmap.  Two blocks per CU (78 KiB of LDS and at most 64
// VGPRs each): while one waits at a barrier the other's loads and stores
// are in flight (ncf_32m: 1.57 ms against 2.11 with one block of twice the
// staging).  Nine entries per thread rather than eight fill what LDS two
// blocks leave (ncf_32m: 5.53 to 5.47 ms for the round trip).
template <int MODE>
__global__ __launch_bounds__(QB_THREADS) __attribute__((amdgpu_waves_per_eu(8))) void k_qb_scatter(Work w, QbArgs a,
                                                                                                  uint32_t j) {
    __shared__ uint32_t bst[QB_MAX_BINS];  // where the chunk's entries of each bin go
    __shared__ uint32_t lc[QB_MAX_BINS];   // the chunk's entries per bin
    __shared__ uint32_t lo[QB_MAX_BINS];   // their first place in the staging area
    __shared__ uint32_t stage[QB_SUB];
    __shared__ uint16_t sb[QB_SUB];
    __shared__ uint32_t ps[33];
    __shared__ uint32_t scratch[QB_THREADS / 64 + 1];
    static_assert(QB_MAX_BINS <= 65536, "bins are staged as 16-bit numbers");
    TDesc &td = w.td[a.t];
    if (!td.qb) return;
    const QueryOut o{};
    bool ok;
    const RecordView rv = query_filter(w, o, td, MODE, &ok);
    const uint32_t d = td.in.d, nsl = qb_slices(rv.m_bits);
    const bool fin = j == rv.k;
    const uint32_t nb = fin ? qb_regions(d) : nsl;
    const uint32_t c = blockIdx.x;
    if (c >= qb_chunks(td, j, nsl)) return;
    // the chunk's places [xa, xb) in round j's list
    uint32_t xa, xb;
    if (j == 0) {
        xa = c * QB_CH;
        xb = min(d, xa + QB_CH);
    } else {
        const uint32_t *prev = w.qrow + (j - 1) * QB_MAX_BINS;
        xa = qb_sum<QB_THREADS>(prev, c, scratch);
        xb = xa + prev[c];
    }
    const bool part = rv.layout == LAYOUT_PARTITIONED;
    if (part) fill_part_starts(ps, rv.m_bits, rv.k);
    // bucket starts (exclusive scan of the round's bin totals), each plus
    // this chunk's offset within the bucket
    const uint32_t *rowj = w.qrow + j * QB_MAX_BINS;
    uint32_t carry = 0;
    for (uint32_t b0 = 0; b0 < nb; b0 += QB_THREADS) {
        const uint32_t b = b0 + threadIdx.x;
        const uint32_t v = b < nb ? rowj[b] : 0u;
        uint32_t tot;
        const uint32_t ex = block_excl_scan_n<QB_THREADS>(v, scratch, &tot);
        if (b < nb) bst[b] = carry + ex + w.qtab[(uint64_t)b * a.ncol + c];
        carry += tot;
    }
    const PosMap pm{rv.m_bits, part ? ps : nullptr};
    for (uint32_t x0 = xa; x0 < xb; x0 += QB_SUB) {
        for (uint32_t b = threadIdx.x; b < nb; b += QB_THREADS) lc[b] = 0;
        uint32_t e[QB_PER];
        qb_load(w, j, x0, xb, e);
        __syncthreads();  // lc is clear (and, the first time, bst and ps are set)
        uint32_t key[QB_PER], rk[QB_PER];
#pragma unroll
        for (uint32_t u = 0; u < QB_PER; ++u) {
            key[u] = QB_DEAD;
            rk[u] = 0;
            if (e[u] != QB_DEAD) {
                const uint32_t b = qb_key(pm, e[u], j, fin);
                if (b < nb) {
                    key[u] = b;
                    rk[u] = atomicAdd(&lc[b], 1u);
                }
            }
        }
        __syncthreads();
        carry = 0;
        for (uint32_t b0 = 0; b0 < nb; b0 += QB_THREADS) {
            const uint32_t b = b0 + threadIdx.x;
            const uint32_t v = b < nb ? lc[b] : 0u;
            uint32_t tot;
            const uint32_t ex = block_excl_scan_n<QB_THREADS>(v, scratch, &tot);
            if (b < nb) lo[b] = carry + ex;
            carry += tot;
        }
        const uint32_t total = carry;
        __syncthreads();
#pragma unroll
        for (uint32_t u = 0; u < QB_PER; ++u) {
            if (key[u] != QB_DEAD) {
                const uint32_t q = lo[key[u]] + rk[u];
                stage[q] = e[u];
                sb[q] = (uint16_t)key[u];
            }
        }
        __syncthreads();
        for (uint32_t q = threadIdx.x; q < total; q += QB_THREADS) {
            const uint32_t b = sb[q];
            const uint32_t dst = bst[b] + (q - lo[b]);
            if (dst < w.qcap) w.qbkt[dst] = stage[q];
        }
        __syncthreads();  // the stores have read bst, lo, sb and stage
        // the next batch's entries of each bin go after this batch's
        for (uint32_t b = threadIdx.x; b < nb; b += QB_THREADS) bst[b] += lc[b];
    }
}

// Round j's test: block s loads filter slice s into LDS and tests hash j of
// the indices in its bucket; each goes back to its place in qlist, or
// QB_DEAD if its bit is clear.  The block also counts its survivors by
// their bin in round j + 1 (the slice of hash j + 1, or after the last hash
// the index region): column s of qtab, for round j + 1's chunk s.
template <int MODE>
__global__ __launch_bounds__(QB_TEST_THREADS) void k_qb_test(Work w, QbArgs a, uint32_t j) {
    __shared__ uint32_t sl[QB_SW];
    __shared__ uint32_t h[QB_MAX_BINS];
    __shared__ uint32_t ps[33];
    __shared__ uint32_t scratch[QB_TEST_THREADS / 64 + 1];
    TDesc &td = w.td[a.t];
    if (!td.qb) return;
    const QueryOut o{};
    bool ok;
    const RecordView rv = query_filter(w, o, td, MODE, &ok);
    const uint32_t nsl = qb_slices(rv.m_bits);
    const uint32_t s = blockIdx.x;
    if (s >= nsl) return;
    const uint32_t *rowj = w.qrow + j * QB_MAX_BINS;
    const uint32_t start = qb_sum<QB_TEST_THREADS>(rowj, s, scratch), end = start + rowj[s];
    const uint32_t w0 = s * QB_SW, nw = min(QB_SW, rv.m_bits / 32u - w0);
    for (uint32_t q = threadIdx.x; q < nw; q += QB_TEST_THREADS) sl[q] = rv.bits[w0 + q];
    const bool fin = j + 1 == rv.k;  // round j + 1 bins by index region
    const uint32_t nb = fin ? qb_regions(td.in.d) : nsl;
    for (uint32_t b = threadIdx.x; b < nb; b += QB_TEST_THREADS) h[b] = 0;
    const bool part = rv.layout == LAYOUT_PARTITIONED;
    if (part) fill_part_starts(ps, rv.m_bits, rv.k);
    __syncthreads();
    const PosMap pm{rv.m_bits, part ? ps : nullptr};
    const uint32_t p0 = s << QB_SL, nbits = nw * 32u;
    for (uint32_t x0 = start + threadIdx.x; x0 < end; x0 += QB_TEST_THREADS * QB_PER) {
        uint32_t e[QB_PER];
#pragma unroll
        for (uint32_t u = 0; u < QB_PER; ++u) {
            const uint32_t x = x0 + u * QB_TEST_THREADS;
            e[u] = x < end ? w.qbkt[x] : QB_DEAD;
        }
#pragma unroll
        for (uint32_t u = 0; u < QB_PER; ++u) {
            const uint32_t x = x0 + u * QB_TEST_THREADS;
            if (x < end) {
                const uint32_t key = mm3_key(e[u]);
                const uint32_t p = pm(key, j) - p0;  // wraps for a bit below the slice
                const bool alive = p < nbits && ((sl[p >> 5] >> (p & 31u)) & 1u);
                if (x < w.qcap) w.qlist[x] = alive ? e[u] : QB_DEAD;
                if (alive) {
                    const uint32_t b = fin ? e[u] >> QB_RL : pm(key, j + 1) >> QB_SL;
                    if (b < nb) atomicAdd(&h[b], 1u);
                }
            }
        }
    }
    __syncthreads();
    for (uint32_t b = threadIdx.x; b < nb; b += QB_TEST_THREADS) w.qtab[(uint64_t)b * a.ncol + s] = h[b];
}

// Last step: block r sets the bits of the positives in index region r in an
// LDS copy of the region's bitmap and writes the region's words of pbits.
template <int MODE>
__global__ __launch_bounds__(QB_TEST_THREADS) void k_qb_fill(Work w, QbArgs a) {
    __shared__ uint32_t bm[QB_RW];
    __shared__ uint32_t scratch[QB_TEST_THREADS / 64 + 1];
    TDesc &td = w.td[a.t];
    if (!td.qb) return;
    const QueryOut o{};
    bool ok;
    const RecordView rv = query_filter(w, o, td, MODE, &ok);
    const uint32_t d = td.in.d;
    const uint32_t r = blockIdx.x;
    if (r >= qb_regions(d)) return;
    const uint32_t *rowk = w.qrow + rv.k * QB_MAX_BINS;
    const uint32_t start = qb_sum<QB_TEST_THREADS>(rowk, r, scratch), end = start + rowk[r];
    const uint32_t w0 = r * QB_RW, nw = min(QB_RW, td.in.ntiles * TILE_WORDS - w0);
    for (uint32_t q = threadIdx.x; q < QB_RW; q += QB_TEST_THREADS) bm[q] = 0u;
    __syncthreads();
    const uint32_t i0 = r << QB_RL;
    for (uint32_t x0 = start + threadIdx.x; x0 < end; x0 += QB_TEST_THREADS * QB_PER) {
        uint32_t e[QB_PER];
#pragma unroll
        for (uint32_t u = 0; u < QB_PER; ++u) {
            const uint32_t x = x0 + u * QB_TEST_THREADS;
            e[u] = x < end ? w.qbkt[x] - i0 : QB_DEAD;
        }
#pragma unroll
        for (uint32_t u = 0; u < QB_PER; ++u)
            if (e[u] < (1u << QB_RL)) atomicOr(&bm[e[u] >> 5], 1u << (e[u] & 31u));
    }
    __syncthreads();
    uint32_t *out = w.pbits + (uint64_t)td.in.tile0 * TILE_WORDS + w0;
    for (uint32_t q = threadIdx.x; q < nw; q += QB_TEST_THREADS) out[q] = bm[q];
}

// The received value of a positive whose value number is vn (NO_SLOT: not
// coded, so 0): its run's polynomial at the abscissa of its sorted rank
// sigma[vn].  A rank outside the record, or run starts that do not bracket
// it, flag the tensor and read as 0.  kn: the run starts of a chord-
// segmented record (staged in LDS, or the record's own).
// GEN: records may use chord runs or the double exponential; without it
// (the usual equal runs of polynomials) the kernels stay at half the
// registers.
template <bool GEN>
__device__ __forceinline__ float positive_value(const RecordView &rv, const float *cf, const uint32_t *kn,
                                                uint32_t vn, TDesc &td, uint64_t *counts_out, uint32_t t) {
    if (vn >= rv.nv) return 0.0f;
    const uint32_t rank = sigma_get(rv.sigma, (uint64_t)vn * rv.b, rv.b);
    uint32_t s, lo, ns;
    bool good = rank < rv.nv;
    if (good) {
        if (GEN && rv.segmode == SEG_CHORD)
            good = run_of_rank_knots(kn, rank, rv.nv, rv.seff, &s, &lo, &ns);
        else
            run_of_rank(rank, rv.nv, rv.seff, &s, &lo, &ns);
    }
    if (!good) {
        atomicOr(&td.flags, FLAG_DEC_MISMATCH);
        if (counts_out) atomicOr((unsigned long long *)&counts_out[4 * t + 3], FLAG_DEC_MISMATCH);
        return 0.0f;
    }
    const double tt = abscissa(rank - lo, ns);
    const float *row = cf + s * (rv.deff + 1u);
    if (GEN && rv.model == FIT_DEXP)
        return (float)((double)row[0] * exp((double)row[1] * tt) + (double)row[2] * exp((double)row[3] * tt));
    return horner(row, rv.deff, tt);
}

// Emit pass: positives in ascending order at their tensor-wide ranks.
//  A. the tile's 128 positives words and their prefix counts (block scan);
//     each thread lists the positives among its 16 elements at their
//     tile-local ranks;
//  B. thread p takes positives p, p + 256, ...: consecutive threads handle
//     consecutive ranks, so the reorder-map reads and the list outputs are
//     coalesced; the receiver also stores each value into the dense output,
//     which the probe pass has already zeroed.
// The next tile's positives words are read before this tile's B and C run.
constexpr uint32_t EMIT_COEF = 512;   // coefficients staged in LDS (else read from the payload)
constexpr uint32_t EMIT_KNOTS = 256;  // chord run starts staged in LDS (else read from the payload)
// The emit passes run 128-thread blocks, one tile each: a tile of a top-r
// gradient holds some 40 positives, so a block's second half only waited;
// two blocks in its place keep twice the tiles in flight (the receiver's
// pass: transformer_355m_x24 0.284 -> 0.227 ms, vgg16_138m 93 -> 71 us).
constexpr uint32_t EMIT_THREADS = 128;
static_assert(EMIT_THREADS >= TILE_WORDS, "each thread of an emit block reads one word of the tile's positives bitmap");
// A tile's wait is mostly memory latency, so the passes want many blocks per
// CU: six waves per SIMD (80 VGPRs, with the record and tensor fields in
// scalar registers) give 12 blocks, as many as the LDS holds, instead of the
// 8 that the receiver's pass got at 128 VGPRs (its time on
// transformer_355m_x24 0.233 -> 0.216 ms, vgg16_138m 69 -> 59 us).  The
// general decoder (chord runs, the double exponential) takes five, which it
// fits without spilling.
#define EMIT_WAVES_PER_EU(GEN) __attribute__((amdgpu_waves_per_eu((GEN) ? 5 : 6)))

// Stage a record's coefficients and run starts in LDS when they fit (the
// caller synchronises before use); the pointers to read them from: LDS or
// the record.
__device__ __forceinline__ void stage_record(const RecordView &rv, float *cf, uint32_t *kn, const float **cf_use,
                                             const uint32_t **kn_use) {
    const uint32_t ncoef = rv.seff * (rv.deff + 1u);
    const uint32_t nkn = rv.segmode == SEG_CHORD && rv.seff > 1 ? rv.seff - 1 : 0u;
    *cf_use = rv.coef;
    *kn_use = rv.knots;
    if (ncoef <= EMIT_COEF) {
        for (uint32_t x = threadIdx.x; x < ncoef; x += blockDim.x) cf[x] = rv.coef[x];
        *cf_use = cf;
    }
    if (nkn <= EMIT_KNOTS) {
        for (uint32_t x = threadIdx.x; x < nkn; x += blockDim.x) kn[x] = rv.knots[x];
        *kn_use = kn;
    }
}

// records of another layout than the kernel's (GEN) decode as empty and are
// flagged: the receiver's configuration sizes the records, so it names the
// segmentation and the model the sender used
template <bool GEN>
__device__ __forceinline__ void match_layout(RecordView &rv, TDesc &td, uint64_t *counts_out, uint32_t t) {
    if (!GEN && (rv.segmode != SEG_EQUAL || rv.model != FIT_POLY)) {
        rv.nv = 0;
        if (threadIdx.x == 0) {
            atomicOr(&td.flags, FLAG_DEC_MISMATCH);
            if (counts_out) atomicOr((unsigned long long *)&counts_out[4 * t + 3], FLAG_DEC_MISMATCH);
        }
    }
}

template <int MODE, bool GEN = false>
__global__ __launch_bounds__(EMIT_THREADS) EMIT_WAVES_PER_EU(GEN) void k_emit(Work w, QueryOut o) {
    __shared__ uint32_t scratch[EMIT_THREADS / 64 + 1];
    __shared__ uint32_t pw[TILE_WORDS];
    __shared__ uint32_t pre[TILE_WORDS];
    __shared__ uint16_t slot[TILE];  // local index of the positive of rank p
    __shared__ float cf[MODE == Q_DECODE ? EMIT_COEF : 1];
    __shared__ uint32_t kn[MODE == Q_DECODE ? EMIT_KNOTS : 1];
    constexpr uint32_t GROUPS = TILE / (4 * EMIT_THREADS);  // 4 groups of 4 elements per thread
    const float *cfu = cf;                              // the tensor's coefficients: LDS or the record
    const uint32_t *knu = kn;                           // its run starts: LDS or the record
    // The next tile's positives words, first rank and tensor are read one
    // tile ahead, and the tensor's fields (descriptor, record header) only
    // when the tensor changes, so a tile waits on no chain of dependent
    // reads.  The barriers order LDS only: the read-ahead and the output
    // stores stay in flight across them.
    uint32_t tile = blockIdx.x;
    uint32_t word = 0, q0n = 0, tn = 0;
    // the value stage's layout over the tensors needs only the per-tensor
    // set-up the probe pass did; block 0 runs it here instead of in a kernel
    // of its own
    if (MODE == Q_ENCODE && o.setup && blockIdx.x == 0) value_layout_block<EMIT_THREADS>(w);
    if (tile < w.ntiles_total) {
        q0n = w.toff[tile];
        tn = tensor_of_tile(w, tile);
        if (threadIdx.x < TILE_WORDS) word = w.pbits[(uint64_t)tile * TILE_WORDS + threadIdx.x];
    }
    uint32_t cur_t = 0xffffffffu, tile0 = 0, d = 0;
    uint64_t toff_el = 0, tslot = 0;
    RecordView rv{};
    // the policy's view of the tensor: positives, values coded, key
    uint32_t npos = 0, ncoded = 0, policy = POLICY_P0, pseed = 0;
    bool sparse_vals = false;  // sender: values from g~ (0 off the selection)
    for (; tile < w.ntiles_total; tile += gridDim.x) {
        const uint32_t t = tn;
        TDesc &td = w.td[t];
        if (t != cur_t) {
            tile0 = uni(td.in.tile0);
            d = uni(td.in.d);
            toff_el = uni(td.in.off);
            tslot = uni(td.in.slot);
            if (MODE == Q_ENCODE) {
                npos = uni(td.npos);
                ncoded = uni(td.nv);
                policy = uni(td.in.policy);
                pseed = uni(td.in.seed);
                sparse_vals = uni(td.in.value_src) == VALUES_SPARSE;
            }
            if (MODE == Q_DECODE) {
                bool ok = true;
                rv = read_record(td.in.rec, td.in.rec_cap, d, &ok);
                match_layout<GEN>(rv, td, o.counts_out, t);
                uniform_record(rv);
                // the receiver's own positives, and the header's values count
                npos = uni(td.nv_dec);
                ncoded = rv.policy == POLICY_P0 ? npos : min(rv.nv, npos);
                policy = rv.policy;
                pseed = rv.seed;
                stage_record(rv, cf, kn, &cfu, &knu);
            }
            cur_t = t;
        }
        const uint32_t lt = tile - tile0;
        const uint32_t q0 = q0n;
        uint32_t tot;
        const uint32_t ex = block_excl_scan_n<EMIT_THREADS, true>(__popc(word), scratch, &tot);
        if (threadIdx.x < TILE_WORDS) {
            pw[threadIdx.x] = word;
            pre[threadIdx.x] = ex;
        }
        lds_barrier();
        // A: list the positives
        uint32_t nib[GROUPS], rank0[GROUPS];
#pragma unroll
        for (uint32_t u = 0; u < GROUPS; ++u) {
            const uint32_t e0 = u * 4 * EMIT_THREADS + threadIdx.x * 4;
            const uint32_t wd = pw[e0 >> 5], sh = e0 & 31u;
            nib[u] = (wd >> sh) & 0xfu;
            rank0[u] = pre[e0 >> 5] + __popc(sh ? wd << (32u - sh) : 0u);
            uint32_t r = rank0[u];
#pragma unroll
            for (uint32_t v = 0; v < 4; ++v)
                if ((nib[u] >> v) & 1u) slot[r++] = e0 + v;
        }
        // the next tile's positives words, in flight during B
        const uint32_t nt = tile + gridDim.x;
        word = 0;
        if (nt < w.ntiles_total) {
            q0n = w.toff[nt];
            tn = tensor_of_tile(w, nt);
            if (threadIdx.x < TILE_WORDS) word = w.pbits[(uint64_t)nt * TILE_WORDS + threadIdx.x];
        }
        lds_barrier();
        // B: one positive per thread
        const uint32_t base = lt * TILE;
        for (uint32_t p = threadIdx.x; p < tot; p += EMIT_THREADS) {
            const uint32_t i = base + slot[p];
            const uint32_t q = q0 + p;
            if (MODE == Q_ENCODE) {
                const uint32_t vn = policy_slot(q, npos, ncoded, policy, pseed);
                if (vn != NO_SLOT) {
                    float x = o.g[toff_el + i];
                    // g~ is 0 at a false positive: i not in the selection
                    // (tslot is a multiple of the tile, so bit i & 31)
                    if (sparse_vals && !((w.selbits[(tslot + i) >> 5] >> (i & 31u)) & 1u)) x = 0.0f;
                    const uint64_t at = tslot + vn;
                    w.V[at] = x;
                    w.keyA[at] = ~order_key(x);  // ascending order of ~key = descending values
                    w.valA[at] = vn;
                }
            } else if (MODE == Q_PLAIN) {
                if (q < o.cap) o.idx_out[q] = i;
            } else {
                const float y = positive_value<GEN>(rv, cfu, knu, policy_slot(q, npos, ncoded, policy, pseed), td,
                                                    o.counts_out, t);
                o.dense_out[toff_el + i] = y;  // zeros elsewhere come from the probe pass
                const uint64_t at = toff_el + q;
                if (o.idx_out) o.idx_out[at] = i;
                if (o.val_out) o.val_out[at] = y;
            }
        }
        lds_barrier();  // pw, pre, slot, cf and kn are rewritten by the next tile
    }
}

// Summing emit pass: one block per tile of the dense gradient.  The tile's
// sum is kept in LDS; the payloads are added in order p = 0, 1, ...: each
// payload's positives in the tile are listed (as in k_emit), decoded one per
// thread, and added to their elements, with a barrier between payloads so
// that every element sees its terms in payload order.  The tile is then
// scaled and written once, zeros included, by full-row stores.
__global__ __launch_bounds__(NTHREADS) void k_emit_sum(Work w, QueryOut o) {
    __shared__ uint32_t scratch[NWAVES + 1];
    __shared__ uint32_t pw[TILE_WORDS];
    __shared__ uint32_t pre[TILE_WORDS];
    __shared__ uint16_t slot[TILE];
    __shared__ float acc[TILE];
    __shared__ float cf[EMIT_COEF];
    __shared__ uint32_t kn[EMIT_KNOTS];
    constexpr uint32_t GROUPS = TILE / (4 * NTHREADS);
    for (uint32_t tile = blockIdx.x; tile < o.ntiles1; tile += gridDim.x) {
        const uint32_t t = uni(tensor_of_tile(w, tile));  // payload 0's descriptor of the tensor
        const uint32_t lt = tile - uni(w.td[t].in.tile0);
        const uint32_t d = uni(w.td[t].in.d);
        const uint64_t toff_el = uni(w.td[t].in.off);
        for (uint32_t e = threadIdx.x; e < TILE; e += NTHREADS) acc[e] = 0.0f;
        for (uint32_t p = 0; p < o.npay; ++p) {
            const uint32_t v = p * o.ntens + t;
            TDesc &td = w.td[v];
            const uint32_t ptile = p * o.ntiles1 + tile;
            const uint32_t word = threadIdx.x < TILE_WORDS ? w.pbits[(uint64_t)ptile * TILE_WORDS + threadIdx.x] : 0u;
            const uint32_t q0 = uni(w.toff[ptile]);
            bool ok = true;
            RecordView rv = read_record(td.in.rec, td.in.rec_cap, d, &ok);
            uniform_record(rv);
            const uint32_t npos = uni(td.nv_dec);
            const uint32_t ncoded = rv.policy == POLICY_P0 ? npos : min(rv.nv, npos);
            uint32_t tot;
            const uint32_t ex = block_excl_scan(__popc(word), scratch, &tot);
            if (threadIdx.x < TILE_WORDS) {
                pw[threadIdx.x] = word;
                pre[threadIdx.x] = ex;
            }
            const float *cfu;
            const uint32_t *knu;
            stage_record(rv, cf, kn, &cfu, &knu);
            __syncthreads();
#pragma unroll
            for (uint32_t u = 0; u < GROUPS; ++u) {
                const uint32_t e0 = u * 4 * NTHREADS + threadIdx.x * 4;
                const uint32_t wd = pw[e0 >> 5], sh = e0 & 31u;
                const uint32_t nib = (wd >> sh) & 0xfu;
                uint32_t r = pre[e0 >> 5] + __popc(sh ? wd << (32u - sh) : 0u);
#pragma unroll
                for (uint32_t c = 0; c < 4; ++c)
                    if ((nib >> c) & 1u) slot[r++] = (uint16_t)(e0 + c);
            }
            __syncthreads();
            for (uint32_t x = threadIdx.x; x < tot; x += NTHREADS) {
                const uint32_t vn = policy_slot(q0 + x, npos, ncoded, rv.policy, rv.seed);
                acc[slot[x]] += positive_value<true>(rv, cfu, knu, vn, td, o.counts_out, v);
            }
            __syncthreads();  // pw, pre, slot, cf and kn are rewritten by the next payload
        }
        // scale and store the tile
        float *dst = o.dense_out + toff_el + (uint64_t)lt * TILE;
        const uint32_t n_el = min(TILE, d - lt * TILE);
        if (n_el == TILE && ((uintptr_t)dst & 15u) == 0) {
            for (uint32_t x = threadIdx.x; x < TILE / 4; x += NTHREADS) {
                const float4 a = ((const float4 *)acc)[x];
                ((float4 *)dst)[x] = make_float4(o.scale * a.x, o.scale * a.y, o.scale * a.z, o.scale * a.w);
            }
        } else {
            for (uint32_t x = threadIdx.x; x < n_el; x += NTHREADS) dst[x] = o.scale * acc[x];
        }
        __syncthreads();  // acc is cleared for the next tile
    }
}

// One probe block per CU (its LDS holds a filter copy), each owning at
// least PB_TILES tiles so that all of its waves have work.
static int probe_grid(const Work &w) {
    const uint32_t cus = std::min((uint32_t)device_cus(), PSTAT_MAX);  // one look-back entry per block
    const uint32_t by_tiles = (w.ntiles_total + PB_TILES - 1) / PB_TILES;
    return (int)std::max(1u, std::min(cus, by_tiles));
}

hipError_t launch_query_encode(const Work &w, const float *g, int grid_persist, uint64_t *counts_out, hipStream_t s,
                               hipEvent_t after_probe) {
    QueryOut o{};
    o.g = g;
    o.setup = 1;
    o.counts_out = counts_out;
    // the pass also scans its tile counts (probe_scan) and writes the
    // records' headers
    k_probe<Q_ENCODE><<<probe_grid(w), PB_THREADS, 0, s>>>(w, o);
    trace_mark(s, "k_probe<Q_ENCODE>");
    if (after_probe) {
        hipError_t e = hipEventRecord(after_probe, s);
        if (e != hipSuccess) return e;
    }
    k_emit<Q_ENCODE><<<resident_grid(k_emit<Q_ENCODE>, EMIT_THREADS, w.ntiles_total), EMIT_THREADS, 0, s>>>(w, o);
    trace_mark(s, "k_emit<Q_ENCODE>");
    return hipGetLastError();
}

hipError_t launch_query_bucketed(const Work &w, const QbTensor &q, uint32_t k, uint32_t min_bits, hipStream_t s) {
    if (k < 1 || q.nch_cap == 0 || q.nsl_cap == 0 || q.nreg == 0 || q.ncol < q.nch_cap || q.ncol < q.nsl_cap)
        return hipSuccess;
    const QbArgs a{q.t, k, min_bits, q.nsl_cap, q.ncol};
    // round 0's counts; each later round's are its previous test's
    k_qb_count<Q_DECODE><<<q.nch_cap, QB_THREADS, 0, s>>>(w, a);
    trace_mark(s, "k_qb_count");
    for (uint32_t j = 0; j <= k; ++j) {
        k_qb_scan<Q_DECODE><<<j < k ? q.nsl_cap : q.nreg, QB_THREADS, 0, s>>>(w, a, j);
        trace_mark(s, "k_qb_scan");
        k_qb_scatter<Q_DECODE><<<q.ncol, QB_THREADS, 0, s>>>(w, a, j);
        trace_mark(s, "k_qb_scatter");
        if (j < k) {
            k_qb_test<Q_DECODE><<<q.nsl_cap, QB_TEST_THREADS, 0, s>>>(w, a, j);
            trace_mark(s, "k_qb_test");
        }
    }
    k_qb_fill<Q_DECODE><<<q.nreg, QB_TEST_THREADS, 0, s>>>(w, a);
    trace_mark(s, "k_qb_fill");
    return hipGetLastError();
}

hipError_t launch_query_plain(const Work &w, uint32_t *idx_out, uint64_t cap, uint64_t *n_out, int grid_persist,
                              hipStream_t s) {
    QueryOut o{};
    o.idx_out = idx_out;
    o.cap = cap;
    o.n_out = n_out;
    // the pass also scans its tile counts (probe_scan)
    k_probe<Q_PLAIN><<<probe_grid(w), PB_THREADS, 0, s>>>(w, o);
    trace_mark(s, "k_probe<Q_PLAIN>");
    k_emit<Q_PLAIN><<<resident_grid(k_emit<Q_PLAIN>, EMIT_THREADS, w.ntiles_total), EMIT_THREADS, 0, s>>>(w, o);
    trace_mark(s, "k_emit<Q_PLAIN>");
    return hipGetLastError();
}

hipError_t launch_probe_decode(const Work &w, float *dense_out, uint64_t *counts_out, uint32_t max_blocks,
                               hipStream_t s) {
    QueryOut o{};
    o.counts_out = counts_out;
    o.dense_out = dense_out;
    // std::min: HIP's host min() takes ints, and max_blocks may be ~0u
    const uint32_t grid = std::min<uint32_t>((uint32_t)probe_grid(w), std::max<uint32_t>(1u, max_blocks));
    // the pass also scans its tile counts (probe_scan)
    k_probe<Q_DECODE><<<grid, PB_THREADS, 0, s>>>(w, o);
    trace_mark(s, "k_probe<Q_DECODE>");
    return hipGetLastError();
}

hipError_t launch_emit_decode(const Work &w, float *dense_out, uint32_t *idx_out, float *val_out,
                              uint64_t *counts_out, bool general, hipStream_t s) {
    QueryOut o{};
    o.counts_out = counts_out;
    o.dense_out = dense_out;
    o.idx_out = idx_out;
    o.val_out = val_out;
    if (general)
        k_emit<Q_DECODE, true><<<resident_grid(k_emit<Q_DECODE, true>, EMIT_THREADS, w.ntiles_total), EMIT_THREADS, 0, s>>>(
            w, o);
    else
        k_emit<Q_DECODE><<<resident_grid(k_emit<Q_DECODE>, EMIT_THREADS, w.ntiles_total), EMIT_THREADS, 0, s>>>(w, o);
    trace_mark(s, "k_emit<Q_DECODE>");
    return hipGetLastError();
}

hipError_t launch_query_decode_sum(const Work &w, uint32_t npay, uint32_t ntens, uint32_t ntiles1, float scale,
                                   float *dense_out, uint64_t *counts_out, hipStream_t s) {
    QueryOut o{};
    o.counts_out = counts_out;
    o.dense_out = dense_out;
    o.scale = scale;
    o.npay = npay;
    o.ntens = ntens;
    o.ntiles1 = ntiles1;
    // the pass also scans its tile counts (probe_scan)
    k_probe<Q_SUM><<<probe_grid(w), PB_THREADS, 0, s>>>(w, o);
    trace_mark(s, "k_probe<Q_SUM>");
    k_emit_sum<<<resident_grid(k_emit_sum, NTHREADS, ntiles1), NTHREADS, 0, s>>>(w, o);
    trace_mark(s, "k_emit_sum");
    return hipGetLastError();
}

}  // namespace dr
