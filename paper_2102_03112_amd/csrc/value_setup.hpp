// value_setup.hpp -- the value path's set-up once |P| is known: per tensor
// (the sender's probe pass runs it where it learns a tensor's |P|) and over
// the tensors (block 0 of the sender's emit pass); both in the standalone
// value path's own kernel.
#pragma once

#include "dr_common.hpp"

namespace dr {

__device__ __forceinline__ void fit_shape(uint32_t nv, uint32_t degree, uint32_t nseg, uint32_t *seff,
                                          uint32_t *deff) {
    if (nv == 0) {
        *seff = 0;
        *deff = 0;
        return;
    }
    uint32_t cap = nv / (degree + 1u);
    if (cap < 1) cap = 1;
    *seff = nseg < cap ? nseg : cap;
    *deff = nv >= degree + 1u ? degree : nv - 1u;
}

// One tensor's value set-up once |P| is known (one thread): run shape,
// reorder-map width, sort tiles and words, and, for a payload, the record
// layout and header.  counts_out, if given, starts as zeros: the flags word
// is OR-ed, as other kernels do.
__device__ inline void value_setup_tensor(const Work &w, uint32_t t, int payload, uint64_t *counts_out) {
    TDesc &td = w.td[t];
    const uint32_t nv = td.nv;
    uint32_t seff, deff;
    fit_shape(nv, td.in.degree, td.in.nseg, &seff, &deff);
    td.seff = seff;
    td.deff = deff;
    const uint32_t b = sigma_bits(nv);
    td.b = b;
    td.model = td.in.fit_model == FIT_DEXP && nv >= 4 ? FIT_DEXP : FIT_POLY;
    const uint32_t ntl = (nv + TILE - 1) / TILE;
    const uint32_t nwd = (uint32_t)(((uint64_t)nv * b + 31u) / 32u);
    td.sntiles = ntl;
    td.swords = nwd;
    if (counts_out) {
        counts_out[4 * t + 0] = td.n;
        counts_out[4 * t + 1] = td.npos;
        if (td.flags) atomicOr((unsigned long long *)&counts_out[4 * t + 3], td.flags);
    }
    if (payload) {
        const uint32_t coef_off = HDR_BYTES + td.m_words * 4u;
        const uint32_t sigma_off = coef_off + seff * (deff + 1u) * 4u;
        const uint32_t rec_bytes = sigma_off + nwd * 4u;
        td.coef_off = coef_off;
        td.sigma_off = sigma_off;
        td.rec_bytes = rec_bytes;
        uint32_t *h = (uint32_t *)td.in.rec;
        h[H_MAGIC] = HDR_MAGIC;
        h[H_BYTES] = HDR_BYTES;
        h[H_D] = td.in.d;
        h[H_NSEL] = td.n;
        h[H_NPOS] = td.npos;
        h[H_NVAL] = nv;
        h[H_MBITS] = td.m_words * 32u;
        h[H_K] = td.in.k;
        // MurmurHash3_x86_32, seeds 0..k-1, over the whole array or per part
        h[H_HASH] = td.in.layout == LAYOUT_PARTITIONED ? HASH_ID_PARTITIONED : HASH_ID_STANDARD;
        h[H_POLICY] = td.in.policy;
        h[H_SEED] = td.in.seed;
        h[H_DEFF] = deff;
        h[H_SEFF] = seff;
        h[H_B] = b;
        h[H_RECBYTES] = rec_bytes;
        h[H_SEGMODE] = td.in.seg_mode | (td.model << 8) | (td.in.value_src << 16);
    }
}

// The value stage's layout over the tensors, after value_setup_tensor of
// each (one block of NT threads; every thread must call it): each tensor's
// first sort tile and first reorder-map word, and the totals.
template <uint32_t NT>
__device__ void value_layout_block(const Work &w) {
    __shared__ uint32_t scratch[NT / 64 + 1];
    __shared__ uint32_t carry_tiles, carry_words, carry_vals;
    if (threadIdx.x == 0) {
        carry_tiles = 0;
        carry_words = 0;
        carry_vals = 0;
    }
    __syncthreads();
    for (uint32_t t0 = 0; t0 < w.ntensors; t0 += NT) {
        const uint32_t t = t0 + threadIdx.x;
        uint32_t ntl = 0, nwd = 0, nv = 0;
        if (t < w.ntensors) {
            const TDesc &td = w.td[t];
            ntl = td.sntiles;
            nwd = td.swords;
            nv = td.nv;
        }
        uint32_t tot_t, tot_w, tot_v;
        const uint32_t bt = carry_tiles, bw = carry_words, bv = carry_vals;
        const uint32_t ex_t = block_excl_scan_n<NT>(ntl, scratch, &tot_t);
        const uint32_t ex_w = block_excl_scan_n<NT>(nwd, scratch, &tot_w);
        block_excl_scan_n<NT>(nv, scratch, &tot_v);
        if (t < w.ntensors) {
            w.td[t].stile0 = bt + ex_t;
            w.td[t].sw0 = bw + ex_w;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            carry_tiles = bt + tot_t;
            carry_words = bw + tot_w;
            carry_vals = bv + tot_v;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        w.glob->sort_tiles = carry_tiles;
        w.glob->sigma_words = carry_words;
        w.glob->values = carry_vals;
    }
}

// Both, in one block (the standalone value path).
template <uint32_t NT>
__device__ void value_setup_block(const Work &w, int payload, uint64_t *counts_out) {
    for (uint32_t t = threadIdx.x; t < w.ntensors; t += NT) value_setup_tensor(w, t, payload, counts_out);
    __syncthreads();
    value_layout_block<NT>(w);
}

}  // namespace dr
