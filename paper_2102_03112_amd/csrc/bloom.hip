// bloom.hip -- Bloom-filter index compression (Sections 2 and 4).
//
// Insert: every selected index s sets bits h_j(s), j < k.  Device-wide
// atomics into a filter larger than a CU's LDS are slow on this GPU, so the
// insert buckets the k n bit positions by 2^16-bit slice of the filter
// (count, scan, scatter), and one block per slice then sets its bits in
// LDS and writes the slice out whole.  OR is commutative, so the filter
// does not depend on the order of any of this.
//
// Query (policy P0, Section 4): every i of the tensor's index range whose k
// bits are all set is a positive, reported in ascending order.  Each wave
// owns 1024 consecutive indices and tests them probe by probe: after probe
// j only the indices still alive are kept, compacted into an LDS queue in
// index order (ballot + mbcnt), so lanes do not idle while a few indices
// need many probes.  The key-dependent half of MurmurHash3 is computed once
// per index.  Tiles chain their positive counts with a decoupled look-back.
#include "launch.hpp"

namespace dr {

// ---------------------------------------------------------------------------
// Insert
// ---------------------------------------------------------------------------
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

// items of chunk c of tensor td: [c * chunk, min(n, (c+1) * chunk))
__global__ __launch_bounds__(NTHREADS) void k_bloom_count(Work w, uint32_t j0, uint32_t j1) {
    extern __shared__ uint32_t lh[];
    const uint32_t t = tensor_of_chunk(w, blockIdx.x);
    const TDesc &td = w.td[t];
    const uint32_t c = blockIdx.x - td.in.bl_chunk0;
    if (c >= td.in.bl_nchunks) return;
    const uint32_t n = td.n, chunk = td.in.bl_chunk;
    const uint32_t nact = (n + chunk - 1) / chunk;
    if (c >= nact) return;
    const uint32_t m_bits = td.m_words * 32u;
    const uint32_t nsl = (m_bits + SLICE_BITS - 1) >> SLICE_LOG2;
    for (uint32_t s = threadIdx.x; s < nsl; s += NTHREADS) lh[s] = 0;
    __syncthreads();
    const uint32_t q0 = c * chunk, q1 = min(n, q0 + chunk);
    const uint32_t *S = w.S + td.in.slot;
    const uint32_t je = min(j1, td.in.k);
    if (je <= j0) return;
    for (uint32_t q = q0 + threadIdx.x; q < q1; q += NTHREADS) {
        const uint32_t km = mm3_key(S[q]);
        for (uint32_t j = j0; j < je; ++j) atomicAdd(&lh[bloom_pos(km, j, m_bits) >> SLICE_LOG2], 1u);
    }
    __syncthreads();
    uint32_t *tab = w.btab + td.in.bl_tab0;
    for (uint32_t s = threadIdx.x; s < nsl; s += NTHREADS) tab[(uint64_t)s * td.in.bl_nchunks + c] = lh[s];
}

constexpr uint32_t SCAN_THREADS = 1024;

// per tensor: exclusive scan of the (slice, chunk) counts in slice-major order
__global__ __launch_bounds__(SCAN_THREADS) void k_bloom_scan(Work w, uint32_t j0, uint32_t j1) {
    const TDesc &td = w.td[blockIdx.x];
    __shared__ uint32_t scratch[SCAN_THREADS / 64 + 1];
    __shared__ uint32_t carry;
    if (j0 >= td.in.k) return;
    (void)j1;
    const uint32_t n = td.n, chunk = td.in.bl_chunk;
    const uint32_t nact = (n + chunk - 1) / chunk;
    const uint32_t nsl = (td.m_words * 32u + SLICE_BITS - 1) >> SLICE_LOG2;
    const uint32_t nch = td.in.bl_nchunks;
    uint32_t *tab = w.btab + td.in.bl_tab0;
    const uint64_t total = (uint64_t)nsl * nact;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (uint64_t f0 = 0; f0 < total; f0 += SCAN_THREADS) {
        const uint64_t f = f0 + threadIdx.x;
        uint64_t a = 0;
        uint32_t v = 0;
        if (f < total) {
            a = (f / nact) * nch + (f % nact);
            v = tab[a];
        }
        uint32_t tot;
        const uint32_t base = carry;
        const uint32_t ex = block_excl_scan_n<SCAN_THREADS>(v, scratch, &tot);
        if (f < total) tab[a] = base + ex;
        if (threadIdx.x == 0) carry = base + tot;
        __syncthreads();
    }
}

__global__ __launch_bounds__(NTHREADS) void k_bloom_scatter(Work w, uint32_t j0, uint32_t j1) {
    extern __shared__ uint32_t lc[];
    const uint32_t t = tensor_of_chunk(w, blockIdx.x);
    const TDesc &td = w.td[t];
    const uint32_t c = blockIdx.x - td.in.bl_chunk0;
    if (c >= td.in.bl_nchunks) return;
    const uint32_t n = td.n, chunk = td.in.bl_chunk;
    const uint32_t nact = (n + chunk - 1) / chunk;
    if (c >= nact) return;
    const uint32_t m_bits = td.m_words * 32u;
    const uint32_t nsl = (m_bits + SLICE_BITS - 1) >> SLICE_LOG2;
    const uint32_t *tab = w.btab + td.in.bl_tab0;
    for (uint32_t s = threadIdx.x; s < nsl; s += NTHREADS) lc[s] = tab[(uint64_t)s * td.in.bl_nchunks + c];
    __syncthreads();
    const uint32_t q0 = c * chunk, q1 = min(n, q0 + chunk);
    const uint32_t *S = w.S + td.in.slot;
    const uint32_t je = min(j1, td.in.k);
    uint16_t *pos = w.bpos + td.in.bl_pos0;
    for (uint32_t q = q0 + threadIdx.x; q < q1; q += NTHREADS) {
        const uint32_t km = mm3_key(S[q]);
        for (uint32_t j = j0; j < je; ++j) {
            const uint32_t p = bloom_pos(km, j, m_bits);
            const uint32_t at = atomicAdd(&lc[p >> SLICE_LOG2], 1u);
            pos[at] = (uint16_t)(p & (SLICE_BITS - 1));
        }
    }
}

__global__ __launch_bounds__(NTHREADS) void k_bloom_fill(Work w, uint32_t j0, uint32_t j1) {
    __shared__ uint32_t words[SLICE_WORDS];
    const uint32_t t = tensor_of_slice(w, blockIdx.x);
    const TDesc &td = w.td[t];
    const uint32_t s = blockIdx.x - td.in.bl_slice0;
    if (s >= td.in.bl_nslices) return;
    const uint32_t m_words = td.m_words;
    const uint32_t m_bits = m_words * 32u;
    const uint32_t nsl = (m_bits + SLICE_BITS - 1) >> SLICE_LOG2;
    if (s >= nsl) return;
    uint32_t *out = td.in.bits + (uint64_t)s * SLICE_WORDS;
    const uint32_t lim = min(SLICE_WORDS, m_words - s * SLICE_WORDS);
    // the first round starts from an empty slice, later rounds add to it
    for (uint32_t i = threadIdx.x; i < SLICE_WORDS; i += NTHREADS) words[i] = (j0 > 0 && i < lim) ? out[i] : 0u;
    __syncthreads();
    const uint32_t je = min(j1, td.in.k);
    const uint32_t n = td.n, chunk = td.in.bl_chunk;
    const uint32_t nact = (n + chunk - 1) / chunk;
    if (nact > 0 && je > j0) {
        const uint32_t *tab = w.btab + td.in.bl_tab0;
        const uint32_t start = tab[(uint64_t)s * td.in.bl_nchunks];
        const uint32_t end = (s + 1 < nsl) ? tab[(uint64_t)(s + 1) * td.in.bl_nchunks] : n * (je - j0);
        const uint16_t *pos = w.bpos + td.in.bl_pos0;
        for (uint32_t q = start + threadIdx.x; q < end; q += NTHREADS) {
            const uint32_t p = pos[q];
            atomicOr(&words[p >> 5], 1u << (p & 31u));
        }
    }
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < lim; i += NTHREADS) out[i] = words[i];
}

hipError_t launch_bloom_insert(const Work &w, uint32_t total_chunks, uint32_t total_slices, uint32_t max_slices,
                               uint32_t hash_per_round, uint32_t kmax, hipStream_t s) {
    // LDS for one counter per slice of the largest filter
    const size_t lds = (size_t)max_slices * 4u;
    uint32_t j0 = 0;
    do {
        const uint32_t j1 = j0 + hash_per_round;
        if (total_chunks) {
            k_bloom_count<<<total_chunks, NTHREADS, lds, s>>>(w, j0, j1);
            k_bloom_scan<<<w.ntensors, SCAN_THREADS, 0, s>>>(w, j0, j1);
            k_bloom_scatter<<<total_chunks, NTHREADS, lds, s>>>(w, j0, j1);
        }
        k_bloom_fill<<<total_slices, NTHREADS, 0, s>>>(w, j0, j1);
        j0 = j1;
    } while (j0 < kmax);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Full-range query
// ---------------------------------------------------------------------------
enum QueryMode { Q_ENCODE = 0, Q_PLAIN = 1, Q_DECODE = 2 };

struct QueryOut {
    const float *g;         // encode: dense gradient (values of the positives)
    uint32_t *idx_out;      // plain: output list; decode: optional positives
    uint64_t cap;           // plain: output capacity
    uint64_t *n_out;        // plain: device count
    const uint8_t *payload; // decode: payload base
    float *dense_out;       // decode: dense gradient
    float *val_out;         // decode: optional values
};

struct RecordView {
    const uint32_t *bits;
    const float *coef;
    const uint32_t *sigma;
    uint32_t m_bits, k, nv, deff, seff, b;
};

// Reads a record header and checks it against the record's capacity and
// the tensor's size; an invalid record decodes as empty (k = 0) and is
// flagged, so a damaged payload cannot send reads past its record.
__device__ __forceinline__ RecordView read_record(const uint8_t *rec, uint64_t cap, uint32_t d, bool *ok) {
    RecordView v;
    const uint32_t *h = (const uint32_t *)rec;
    const uint64_t m_bits = *(const uint64_t *)(rec + 32);
    v.m_bits = (uint32_t)m_bits;
    v.nv = (uint32_t)(*(const uint64_t *)(rec + 24));
    v.k = h[10];
    v.deff = h[12];
    v.seff = h[13];
    v.b = h[14];
    v.bits = (const uint32_t *)(rec + HDR_BYTES);
    const uint32_t coef_off = HDR_BYTES + (v.m_bits / 32u) * 4u;
    v.coef = (const float *)(rec + coef_off);
    const uint64_t need = (uint64_t)HDR_BYTES + m_bits / 8u + 4ull * v.seff * (v.deff + 1ull) +
                          4ull * (((uint64_t)v.nv * v.b + 31u) / 32u);
    const uint64_t nv64 = *(const uint64_t *)(rec + 24);
    *ok = h[0] == HDR_MAGIC && h[1] == HDR_BYTES && m_bits >= 32 && (m_bits & 31u) == 0 && m_bits < (1ull << 32) &&
          v.k >= 1 && v.k <= 32 && v.deff <= MAX_DEG && v.b >= 1 && v.b <= 32 && nv64 <= d &&
          (v.nv == 0 || (v.seff >= 1 && v.seff <= v.nv && v.b >= sigma_bits(v.nv))) && need <= cap;
    if (!*ok) {
        v.k = 0;
        v.nv = 0;
        v.m_bits = 32;
    }
    v.sigma = (const uint32_t *)(rec + coef_off + v.seff * (v.deff + 1u) * 4u);
    return v;
}

// entry q of a packed b-bit stream (b <= 32)
__device__ __forceinline__ uint32_t sigma_get(const uint32_t *sig, uint32_t q, uint32_t b) {
    const uint64_t bit = (uint64_t)q * b;
    const uint32_t w0 = sig[bit >> 5], sh = (uint32_t)(bit & 31u);
    uint64_t v = w0 >> sh;
    if (sh + b > 32u) v |= (uint64_t)sig[(bit >> 5) + 1] << (32u - sh);
    return b == 32u ? (uint32_t)v : (uint32_t)(v & ((1ull << b) - 1ull));
}

// value of sorted rank `rank` among nv values fitted in seff runs of degree deff
__device__ __forceinline__ float eval_rank(const float *coef, uint32_t rank, uint32_t nv, uint32_t seff,
                                           uint32_t deff) {
    // run s is the largest with floor(s nv / seff) <= rank
    const uint64_t s = (((uint64_t)rank + 1u) * seff - 1u) / nv;
    const uint64_t lo = s * nv / seff, hi = (s + 1) * nv / seff;
    const uint64_t ns = hi - lo, j = rank - lo;
    const double t = ns > 1 ? (double)(2 * (int64_t)j - (int64_t)(ns - 1)) / (double)(ns - 1) : 0.0;
    const float *c = coef + s * (deff + 1u);
    double y = (double)c[deff];
    for (int p = (int)deff - 1; p >= 0; --p) y = y * t + (double)c[p];
    return (float)y;
}

constexpr uint32_t QWAVE = 1024;  // indices per wave per tile

template <int MODE>
__global__ __launch_bounds__(NTHREADS) void k_query(Work w, QueryOut o) {
    __shared__ uint16_t qe[NWAVES][QWAVE];
    __shared__ uint32_t qk[NWAVES][QWAVE];
    __shared__ float stage[MODE == Q_DECODE ? TILE : 1];
    __shared__ uint32_t wcount[NWAVES];
    __shared__ uint32_t tkt, tile_excl;
    const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
    uint32_t *ticket = &w.tickets[MODE == Q_DECODE ? 3 : 2];
    unsigned long long *lb = MODE == Q_DECODE ? w.lb3 : w.lb2;
    for (;;) {
        const uint32_t tile = next_ticket(ticket, &tkt);
        if (tile >= w.ntiles_total) break;
        const uint32_t t = tensor_of_tile(w.td, w.ntensors, tile);
        TDesc &td = w.td[t];
        const uint32_t lt = tile - td.in.tile0;
        const uint32_t d = td.in.d;
        RecordView rv;
        if (MODE == Q_DECODE) {
            bool ok = true;
            rv = read_record(o.payload + td.in.rec_off, td.in.rec_cap, d, &ok);
            if (!ok && threadIdx.x == 0) atomicOr(&td.flags, FLAG_DEC_MISMATCH);
        } else {
            rv.bits = td.in.bits;
            rv.m_bits = td.m_words * 32u;
            rv.k = td.in.k;
        }
        const uint32_t m_bits = rv.m_bits, k = rv.k;
        const uint32_t *bits = rv.bits;
        const uint32_t wbase = lt * TILE + wv * QWAVE;  // first index of this wave
        uint16_t *me = qe[wv];
        uint32_t *mk = qk[wv];
        // probe 0 over the wave's 1024 indices
        uint32_t cnt = 0;
        for (uint32_t c = 0; c < QWAVE / 64; ++c) {
            const uint32_t e = c * 64 + lane;
            const uint32_t i = wbase + e;
            const bool valid = i < d && k > 0;
            const uint32_t km = mm3_key(i);
            bool hit = false;
            if (valid) hit = test_bit(bits, bloom_pos(km, 0, m_bits));
            const uint64_t mask = ballot(hit);
            if (hit) {
                const uint32_t at = cnt + lanes_below(mask);
                me[at] = (uint16_t)e;
                mk[at] = km;
            }
            cnt += popc64(mask);
        }
        // probes 1..k-1 over the survivors, compacting in place
        for (uint32_t j = 1; j < k && cnt > 0; ++j) {
            __builtin_amdgcn_wave_barrier();
            const uint32_t L = cnt;
            cnt = 0;
            for (uint32_t b0 = 0; b0 < L; b0 += 64) {
                const uint32_t x = b0 + lane;
                const bool act = x < L;
                uint32_t e = 0, km = 0;
                if (act) {
                    e = me[x];
                    km = mk[x];
                }
                const bool hit = act && test_bit(bits, bloom_pos(km, j, m_bits));
                const uint64_t mask = ballot(hit);
                __builtin_amdgcn_wave_barrier();
                if (hit) {
                    const uint32_t at = cnt + lanes_below(mask);
                    me[at] = (uint16_t)e;
                    mk[at] = km;
                }
                cnt += popc64(mask);
                __builtin_amdgcn_wave_barrier();
            }
        }
        if (lane == 0) wcount[wv] = cnt;
        if (MODE == Q_DECODE) {
            for (uint32_t e = threadIdx.x; e < TILE; e += NTHREADS) stage[e] = 0.0f;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t tot = 0;
            for (uint32_t q = 0; q < NWAVES; ++q) tot += wcount[q];
            tile_excl = (uint32_t)lookback(lb, tile, td.in.tile0, tot);
            if (lt == td.in.ntiles - 1) {
                const uint32_t nv = tile_excl + tot;
                if (MODE == Q_ENCODE) td.nv = nv;
                if (MODE == Q_PLAIN) *o.n_out = nv;
                if (MODE == Q_DECODE) {
                    td.nv_dec = nv;
                    if (nv != rv.nv) atomicOr(&td.flags, FLAG_DEC_MISMATCH);
                }
            }
        }
        __syncthreads();
        uint32_t wpre = 0;
        for (uint32_t q = 0; q < wv; ++q) wpre += wcount[q];
        const uint32_t qbase = tile_excl + wpre;
        for (uint32_t x = lane; x < cnt; x += 64) {
            const uint32_t e = me[x];
            const uint32_t i = wbase + e;
            const uint32_t q = qbase + x;
            if (MODE == Q_ENCODE) {
                const float v = o.g[td.in.off + i];
                const uint64_t at = td.in.slot + q;
                w.P[at] = i;
                w.V[at] = v;
                w.keyA[at] = ~order_key(v);  // ascending order of ~key = descending values
                w.valA[at] = q;
            } else if (MODE == Q_PLAIN) {
                if (q < o.cap) o.idx_out[q] = i;
            } else {
                float y = 0.0f;
                if (rv.nv > 0 && q < rv.nv) {
                    const uint32_t rank = sigma_get(rv.sigma, q, rv.b);
                    if (rank < rv.nv)
                        y = eval_rank(rv.coef, rank, rv.nv, rv.seff, rv.deff);
                    else
                        atomicOr(&td.flags, FLAG_DEC_MISMATCH);
                }
                stage[wv * QWAVE + e] = y;
                const uint64_t at = td.in.off + q;
                if (o.idx_out) o.idx_out[at] = i;
                if (o.val_out) o.val_out[at] = y;
            }
        }
        if (MODE == Q_DECODE) {
            __syncthreads();
            float *dst = o.dense_out + td.in.off + (uint64_t)lt * TILE;
            const uint32_t lim = min(TILE, d - lt * TILE);
            for (uint32_t e = threadIdx.x; e < lim; e += NTHREADS) dst[e] = stage[e];
        }
        __syncthreads();
    }
}

hipError_t launch_query_encode(const Work &w, const float *g, int grid_persist, hipStream_t s) {
    QueryOut o{};
    o.g = g;
    k_query<Q_ENCODE><<<grid_persist, NTHREADS, 0, s>>>(w, o);
    return hipGetLastError();
}

hipError_t launch_query_plain(const Work &w, uint32_t *idx_out, uint64_t cap, uint64_t *n_out, int grid_persist,
                              hipStream_t s) {
    QueryOut o{};
    o.idx_out = idx_out;
    o.cap = cap;
    o.n_out = n_out;
    k_query<Q_PLAIN><<<grid_persist, NTHREADS, 0, s>>>(w, o);
    return hipGetLastError();
}

hipError_t launch_query_decode(const Work &w, const uint8_t *payload, float *dense_out, uint32_t *idx_out,
                               float *val_out, int grid_persist, hipStream_t s) {
    QueryOut o{};
    o.payload = payload;
    o.dense_out = dense_out;
    o.idx_out = idx_out;
    o.val_out = val_out;
    k_query<Q_DECODE><<<grid_persist, NTHREADS, 0, s>>>(w, o);
    return hipGetLastError();
}

}  // namespace dr
