// dr_common.hpp -- device-side building blocks shared by the codec's kernels.
//
// Layout conventions
//  * A gradient is split into tensors; tensor t covers global elements
//    [off, off + d).  Every tensor is also given a padded "slot" of
//    ntiles * TILE elements starting at tile0 * TILE in the per-element work
//    arrays, so per-tensor buffers never overlap and tiles never straddle
//    tensors.
//  * Work is split into tiles of TILE consecutive elements of one tensor.
//    A pass that must emit results in ascending index order first records,
//    per tile, a bitmap of what it keeps and a count; a per-tensor scan of
//    the counts gives each tile its output offset; an emit pass then writes
//    the results in order.  No tile ever waits on another.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dr {

constexpr uint32_t TILE = 4096;               // elements per tile
constexpr uint32_t TILE_WORDS = TILE / 32;    // bitmap words per tile
constexpr uint32_t NTHREADS = 256;            // threads per block (4 waves of 64)
constexpr uint32_t NWAVES = NTHREADS / 64;
constexpr uint32_t R_NONZERO = 0xFFFFFFFFu;   // select every nonzero
constexpr uint32_t CHUNK_TILES = 16;          // Bloom insert from the bitmap: fewest tiles per chunk
constexpr uint32_t MAX_CHUNKS = 512;           // Bloom insert: most item chunks per tensor (two scatter blocks per CU)
constexpr uint32_t DIR_SLICE_LOG2 = 20;        // direct insert: 2^20-bit (128 KiB) slices in LDS
constexpr uint32_t DIR_SLICE_WORDS = 1u << (DIR_SLICE_LOG2 - 5);
constexpr uint64_t DIR_MAX_BITS = 8ull << DIR_SLICE_LOG2;  // at most 8 slices per tensor
// Bucketed query (filters larger than an XCD's L2): rounds of one hash
// each route the live indices to filter slices of 2^QB_SL bits held in LDS;
// the positives are then bucketed by index region of 2^QB_RL indices.  Bins
// of a round are slices or regions, at most QB_MAX_BINS of either; a chunk
// is QB_CH list entries, staged QB_SUB at a time.
constexpr uint32_t QB_SL = 19;                  // filter slice: 2^19 bits (64 KiB)
constexpr uint32_t QB_SW = 1u << (QB_SL - 5);
constexpr uint32_t QB_RL = 19;                  // index region: 2^19 indices (64 KiB of bitmap)
constexpr uint32_t QB_RW = 1u << (QB_RL - 5);
constexpr uint32_t QB_MAX_BINS = 2048;
constexpr uint32_t QB_THREADS = 1024;
constexpr uint32_t QB_PER = 9;                  // entries per thread of a staged batch
constexpr uint32_t QB_SUB = QB_THREADS * QB_PER;
constexpr uint32_t QB_CH = 4 * QB_SUB;          // entries per chunk
constexpr uint32_t QB_MAX_D = 1u << 30;         // largest tensor taken this way (regions <= QB_MAX_BINS)
constexpr uint32_t QB_DEAD = 0xffffffffu;       // list entry of an index that failed a probe
constexpr int BUFFER_RSRC_WORD3 = 0x00020000;  // gfx9 buffer descriptor word 3 (32-bit dword format)
constexpr uint32_t SLICE_LOG2_MIN = 14;       // Bloom fill slices: 2^14 to 2^20 bits (2 to 128 KiB of LDS)
constexpr uint32_t SLICE_LOG2_MAX = 20;
constexpr uint32_t SLICE_WORDS_MAX = (1u << SLICE_LOG2_MAX) / 32;
constexpr uint32_t BL_MAX_SLICES = 1024;      // Bloom insert: slices per filter (filters up to 2^30 bits)
constexpr uint32_t HIST1_BITS = 11;           // first top-r digit: key bits 30..20
constexpr uint32_t HIST1_BINS = 1u << HIST1_BITS;
constexpr uint32_t HIST1_SHIFT = 20;
// Copies of each tensor's histogram of the candidates' key bits 19..10: the
// filter pass's blocks add to copy (block mod HISTA_COPIES), which spreads
// their atomics over that many times more cache lines.
constexpr uint32_t HISTA_COPIES = 8;
// Sampled top-r: a large tensor whose r is a small share of d takes the
// first digit's histogram from a sample (segment j of SAMPLE_SEG elements
// in every srate, at j srate + srate / 2) and reads the tensor once, in a
// filter pass that keeps the bins of a bracket [bL, bH] (at most NBR bins)
// around the sample's estimate of the threshold as candidates.  A bracket
// that the exact counts contradict is redone from a full histogram.
constexpr uint32_t SAMPLE_SEG = 64;
constexpr uint32_t SAMPLE_SEGS_PER_BLOCK = 64;   // 16 waves x 4 segments
constexpr uint64_t SAMPLE_MIN_D = 1ull << 22;
constexpr uint32_t SHIST_COPIES = 4;             // copies of the sample histogram (block mod 4)
constexpr uint32_t NBR = 4;                      // most first-digit bins in a bracket
constexpr uint32_t HISTA_BINS = NBR * 1024;      // candidate histogram: (bin - bL, key bits 19..10)
// The filter pass's exact counts per sampled tensor: elements above the
// bracket and candidates in each of its bins, added by block mod
// FCNT_COPIES.
constexpr uint32_t FCNT_COPIES = 16;
constexpr uint32_t FCNT_W = 1 + NBR;
constexpr uint32_t SORT_BINS = 256;           // 8-bit LSD radix digits
constexpr uint32_t FIT_CHUNKS = 8;            // partial-moment blocks per fitted run
constexpr uint32_t MAX_DEG = 7;
constexpr uint32_t MAX_SEG = 4096;            // most runs per tensor
// index policies (Section 4; Sections 10.4, 10.5)
constexpr uint32_t POLICY_P0 = 0, POLICY_RANDOM = 1, POLICY_LEFTMOST = 2, POLICY_MIDDLE = 3, POLICY_RIGHTMOST = 4;
constexpr uint32_t NO_SLOT = 0xffffffffu;
// segmentation of the sorted values (Section 5)
constexpr uint32_t SEG_EQUAL = 0, SEG_CHORD = 1;
// value models (Section 5): polynomial, double exponential a e^(bt) + c e^(dt)
constexpr uint32_t FIT_POLY = 0, FIT_DEXP = 1;
// where the sender's coded values come from (Section 4): g, or g~ (0 off S)
constexpr uint32_t VALUES_DENSE = 0, VALUES_SPARSE = 1;
// filter layouts: each hash over the whole array, or hash j over part j of k;
// a record's hash id names the layout
constexpr uint32_t LAYOUT_STANDARD = 0, LAYOUT_PARTITIONED = 1;
constexpr uint32_t HASH_ID_STANDARD = 1, HASH_ID_PARTITIONED = 2;
constexpr uint32_t NMOM = 3 * MAX_DEG + 2;    // 2D+1 power sums + D+1 right-hand sides (room for D=7)
constexpr uint32_t HDR_BYTES = 64;
// payload record header: sixteen little-endian u32 words
enum HdrWord : uint32_t {
    H_MAGIC = 0, H_BYTES, H_D, H_NSEL, H_NPOS, H_NVAL, H_MBITS, H_K, H_HASH, H_POLICY, H_SEED, H_DEFF, H_SEFF, H_B,
    H_RECBYTES, H_SEGMODE
};
constexpr uint32_t HDR_MAGIC = 0x31435244u;   // "DRC1"

// Static per-tensor set-up, written by the host (through kernel arguments).
struct TInit {
    uint64_t off;        // first element of the tensor in g / dense_out
    uint64_t rec_off;    // byte offset of the tensor's payload record
    uint64_t slot;       // first element of the tensor's padded slot (= tile0 * TILE)
    uint64_t bl_pos0;    // first entry of this tensor in the Bloom position buffer
    uint64_t bl_tab0;    // first entry of this tensor in the Bloom count table
    uint32_t *bits;      // filter words (payload record or caller buffer)
    float *coef;         // coefficient output; null: the payload record
    uint32_t *sigma;     // reorder-map output; null: the payload record
    uint8_t *rec;        // payload record, or null
    double mC;           // -ln(fpr) / (ln 2)^2: m = 32 ceil(ceil(n mC) / 32)
    uint32_t d;          // elements
    uint32_t r;          // requested count, or R_NONZERO
    uint32_t tile0;      // first tile
    uint32_t ntiles;     // ceil(d / TILE), at least 1
    uint32_t k;          // hash functions
    uint32_t degree;     // requested polynomial degree
    uint32_t nseg;       // requested runs
    uint32_t m_words_in; // filter words fixed by the caller, or 0: derive from n
    uint32_t fit_blk0;   // first block of this tensor in the fit grid
    uint32_t bl_chunk;   // Bloom insert: bitmap tiles (from the bitmap) or items (from a list) per chunk
    uint32_t bl_chunk0;  // first Bloom chunk of this tensor
    uint32_t bl_nchunks; // Bloom chunks reserved for this tensor
    uint32_t bl_slice0;  // first Bloom slice of this tensor
    uint32_t bl_nslices; // Bloom slices reserved (covers the largest possible filter)
    uint32_t hb0, hbn;   // top-r histogram blocks of this tensor
    uint32_t coef_stride;// floats per run in `coef` when it is given
    uint32_t slice_log2; // Bloom fill slice size (bits, log2)
    uint64_t rec_cap;    // payload record capacity in bytes (receiver checks the header against it)
    uint64_t bl_poscap;  // Bloom insert: positions reserved for this tensor per round
    // direct insert (filters of at most DIR_MAX_BITS bits): block (s, c) sets
    // the bits of slice s from item chunk c in LDS and writes them to its
    // own partial slice; an OR over the chunks then gives the filter
    uint64_t dir_pb;     // first partial word of this tensor
    uint32_t dir_blk0;   // first direct-insert block of this tensor
    uint32_t dir_sl0;    // first slice of this tensor (over all tensors)
    uint32_t dir_nsl;    // slices planned (covers the largest possible filter)
    uint32_t dir_g;      // item chunks
    uint32_t dir_sw;     // words per partial slice: min(DIR_SLICE_WORDS, planned filter words)
    uint32_t dir_per;    // bitmap tiles (from the bitmap) or items (from a list) per chunk
    uint32_t policy;     // index policy (POLICY_*)
    uint32_t seed;       // key of the random policy
    uint32_t seg_mode;   // SEG_EQUAL or SEG_CHORD (nseg == 0: the heuristic count)
    uint32_t fit_model;  // FIT_POLY or FIT_DEXP (then degree is 3: rows (a, b, c, d))
    uint32_t bnd0;       // chord segmentation: first segment-start entry of this tensor
    uint32_t seg_slot;   // chord segmentation over the whole grid: the tensor's state, or NO_SEG_SLOT
    uint32_t value_src;  // VALUES_DENSE or VALUES_SPARSE
    uint32_t layout;     // LAYOUT_STANDARD or LAYOUT_PARTITIONED
    // sampled top-r (srate 0: the exact histogram; hb0, hbn then count the
    // sample's blocks)
    uint32_t srate;      // one sampled segment in srate (a power of 2)
    uint32_t nsamp;      // elements in the sample
    uint32_t slo, shi;   // sample ranks that bound the bracket: rho -/+ delta
    uint32_t rb0, rbn;   // blocks of the full histogram for a redo
};

// Chord segmentation over the whole grid (at most SEG_GRID_RUNS runs per
// tensor, at most SEG_GRID_TENSORS such tensors): each step evaluates the
// runs a split has just made, in parallel over SEG_GRID_BLOCKS blocks; the
// last block to finish picks and makes the next split.
constexpr uint32_t NO_SEG_SLOT = 0xFFFFFFFFu;
constexpr uint32_t SEG_GRID_RUNS = 64;
constexpr uint32_t SEG_GRID_TENSORS = 64;
constexpr uint32_t SEG_GRID_BLOCKS = 256;
struct SegState {
    double cd[SEG_GRID_RUNS];  // each run's farthest allowed split distance (0: none)
    uint32_t ci[SEG_GRID_RUNS];  // and the rank that ends its left part
    uint32_t count;            // runs so far (their starts are in the tensor's bounds)
    uint32_t req;              // runs requested
    uint32_t done;             // no further split
    uint32_t pend;             // first of the runs to evaluate (npend of them)
    uint32_t npend;
    uint32_t arrive;           // blocks done with this step
};
struct SegPart {               // one block's farthest point of each run evaluated
    double d[2];
    uint32_t i[2];
};

// Per-tensor descriptor, in device memory.
struct TDesc {
    TInit in;
    // --- produced on the device ---
    uint32_t n;          // |S|
    uint32_t m_words;    // filter words
    uint32_t nv;         // values coded on the sender: |P| for P0, else min(|S|, |P|)
    uint32_t nv_dec;     // |P| on the receiver
    uint32_t npos;       // |P| on the sender
    uint32_t seff, deff; // runs and degree actually used
    uint32_t b;          // reorder-map bits per entry
    uint32_t flags;      // DR_FLAG_* bits (+ internal error bits)
    uint32_t b1;         // top-r: first-digit bin holding the threshold
    uint32_t need1;      // top-r: how many to take from bin b1
    uint32_t ncand;      // top-r: elements in bin b1
    uint32_t T;          // top-r: exact threshold key
    uint32_t needT;      // top-r: how many elements with key == T to take
    uint32_t ntie;       // top-r: elements with key == T
    uint32_t idx_star;   // top-r: largest index taken among key == T (when ties split)
    uint32_t bL, bH;     // top-r: the filter pass's bracket of first-digit bins
    uint32_t sfail;      // top-r: the sampled bracket missed the threshold and was redone
    uint32_t bA;         // top-r: bin of key bits 19..10 holding the threshold (~0: all of b1)
    uint32_t needA;      // top-r: how many to take from bin bA
    uint32_t nsub;       // top-r: candidates in bin bA (the short list)
    uint32_t stile0;     // value sort: first tile
    uint32_t sntiles;    // value sort: tiles
    uint32_t sw0;        // reorder map: first word in the packing grid
    uint32_t swords;     // reorder map: words
    uint32_t coef_off;   // payload record: byte offset of the coefficients
    uint32_t sigma_off;  // payload record: byte offset of the reorder map
    uint32_t rec_bytes;  // payload record: bytes in use
    uint32_t bl_end;     // Bloom insert: positions bucketed in the current round
    uint32_t model;      // value model used: FIT_DEXP needs at least 4 values, else FIT_POLY
    uint32_t qb;         // the bucketed query found this tensor's filter and wrote its positives bitmap
};

static_assert(sizeof(TInit) % 4 == 0 && sizeof(TDesc) % 4 == 0, "descriptor layout");

// device-wide totals produced on the device
struct Glob {
    uint32_t sort_tiles;      // value-sort tiles over all tensors
    uint32_t sigma_words;     // reorder-map words over all tensors
    uint32_t values;          // sum of |P|
    uint32_t redo;            // top-r: some sampled bracket missed (the redo's filter pass has work)
    uint32_t sort_ticket[4];  // value sort: next tile of each pass, in start order
};

// internal flag bits (besides DR_FLAG_NONFINITE = 1)
constexpr uint32_t FLAG_NONFINITE = 1u;
constexpr uint32_t FLAG_DEC_MISMATCH = 2u;   // receiver |P| differs from the header
constexpr uint32_t FLAG_COUNT = 4u;          // selection count differs from r
constexpr uint32_t FLAG_CAPACITY = 8u;       // a device-side capacity was exceeded
constexpr uint32_t FLAG_STALLED = 16u;       // a bounded wait gave up (internal error)
constexpr uint32_t PSTAT_MAX = 4096;         // probe pass blocks with a look-back entry (at most)

// Views of the workspace carved on the host.
struct Work {
    TDesc *td;
    Glob *glob;
    uint64_t *counts_out;     // the round trip's per-tensor counts (nullable): late flags go here too
    uint32_t *tile_tensor;    // tensor of each tile (filled by k_init)
    uint32_t ntensors;
    uint32_t ntiles_total;    // sum of ntiles
    uint64_t slots;           // padded elements = ntiles_total * TILE
    uint64_t *pstat;          // probe pass look-back: per block (flag << 62 | trailing count), zeroed at set-up
    uint32_t *tcnt;           // per-tile counts of the current ordered pass
    uint32_t *toff;           // per-tile exclusive offsets within the tensor
    uint32_t *ccnt;           // top-r candidates per tile
    uint32_t *pbits;          // positives of a full-range query, one bit per index (slots / 32 words)
    uint32_t *hist;           // top-r first-digit histogram per tensor
    uint32_t *selbits;        // selection bitmap (paper's d-bit string B), slots / 32 words
    uint32_t *cand_key;       // top-r candidates (keys), per tensor slot
    uint32_t *cand_idx;       // top-r candidates (indices)
    uint32_t *histA;          // top-r: per tensor, HISTA_COPIES histograms of the candidates' (bin - bL, key bits 19..10)
    uint32_t *shist;          // sampled top-r: per tensor, SHIST_COPIES first-digit histograms of the sample
    uint32_t *fcnt;           // sampled top-r: [tensor][FCNT_COPIES][FCNT_W] counts of the filter pass
    uint32_t *sub_key;        // top-r short list (borrows P, which is written later)
    uint32_t *sub_idx;        // top-r short list (borrows V)
    uint32_t *S;              // selected indices, per tensor slot
    uint32_t *P;              // sender's positives, per tensor slot
    float *V;                 // g[P]
    uint32_t *keyA, *keyB;    // sort keys
    uint32_t *valA, *valB;    // sort payloads
    uint64_t *sstat;          // sort look-back: (flag << 32 | count) per pass, tile and digit
    uint32_t *sdig;           // sort: per-tensor totals of each pass's digits (4 x SORT_BINS)
    uint32_t *srow;           // sort: per tensor digit totals
    uint32_t *sig;            // unpacked reorder map, per tensor slot
    float *vsorted;           // values in sorted order, per tensor slot
    double *fit_part;         // fit: partial moments
    uint32_t fit_runs;
    uint32_t *bpos;           // Bloom insert: bucketed in-slice positions
    uint32_t *btab;           // Bloom insert: per (slice, chunk) counts, then offsets within the slice
    uint32_t *brow;           // Bloom insert: per reserved slice, its count; brow + bslices: its start
    uint32_t bslices;         // Bloom insert: reserved slices over all tensors
    uint32_t *bounds;         // chord segmentation: segment starts (S_eff + 1 per tensor)
    SegState *segst;          // chord segmentation over the grid: per state slot
    SegPart *segpart;         // and SEG_GRID_BLOCKS partial results per slot
    // bucketed query (one tensor at a time): the live indices of a round
    // (qlist, with QB_DEAD for the ones that failed), the same bucketed by
    // bin (qbkt), per (bin, chunk) counts then offsets (qtab, bins x
    // qb_nch words) and each round's bin totals (qrow, QB_MAX_BINS per round)
    uint32_t *qlist, *qbkt, *qtab, *qrow;
    uint64_t qcap;            // entries of qlist and qbkt
};

// ---------------------------------------------------------------------------
// MurmurHash3_x86_32 of the 4-byte little-endian encoding of an index.
// The key-dependent part is computed once per index and reused for every
// seed, since it does not depend on the seed.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t rotl32(uint32_t x, uint32_t r) { return (x << r) | (x >> (32u - r)); }

__device__ __forceinline__ uint32_t mm3_key(uint32_t i) {
    uint32_t k = i * 0xcc9e2d51u;
    k = rotl32(k, 15);
    return k * 0x1b873593u;
}

__device__ __forceinline__ uint32_t mm3_seed(uint32_t kmix, uint32_t seed) {
    uint32_t h = seed ^ kmix;
    h = rotl32(h, 13);
    h = h * 5u + 0xe6546b64u;
    h ^= 4u;  // input length in bytes
    h ^= h >> 16;
    h *= 0x85ebca6bu;
    h ^= h >> 13;
    h *= 0xc2b2ae35u;
    h ^= h >> 16;
    return h;
}

// Bit position of hash j for a key mix in an m-bit filter: floor(h m / 2^32).
__device__ __forceinline__ uint32_t bloom_pos(uint32_t kmix, uint32_t j, uint32_t m_bits) {
    return __umulhi(mm3_seed(kmix, j), m_bits);
}

__device__ __forceinline__ uint32_t test_bit(const uint32_t *w, uint32_t p) { return (w[p >> 5] >> (p & 31u)) & 1u; }

// Bit positions of a filter in its layout.  Standard: hash j over the whole
// m-bit array.  Partitioned: part j covers [ps[j], ps[j+1]), ps[j] =
// floor(j m / k), and hash j maps into it by the same multiply-shift.
struct PosMap {
    uint32_t m_bits;
    const uint32_t *ps;  // the k + 1 part starts (LDS) of a partitioned filter, else null
    __device__ __forceinline__ uint32_t operator()(uint32_t kmix, uint32_t j) const {
        const uint32_t h = mm3_seed(kmix, j);
        if (ps) {
            const uint32_t a = ps[j];
            return a + __umulhi(h, ps[j + 1] - a);
        }
        return __umulhi(h, m_bits);
    }
};

// Part starts floor(j m / k), j = 0..k, written by threads 0..k of the
// block (the caller synchronises before use).
__device__ __forceinline__ void fill_part_starts(uint32_t *ps, uint32_t m_bits, uint32_t k) {
    if (threadIdx.x <= k && k > 0) ps[threadIdx.x] = (uint32_t)(((uint64_t)threadIdx.x * m_bits) / k);
}

// ---------------------------------------------------------------------------
// Block barrier for LDS traffic only: waits for this wave's LDS operations,
// not for its global loads, stores or atomics, which stay in flight across it
// (__syncthreads also drains those).  For barriers that order LDS accesses
// alone; not where one thread reads global memory that another thread of
// the block wrote before the barrier.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Wave (64-lane) primitives.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)); }

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

// number of set bits of `mask` in lanes below this one
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint32_t popc64(uint64_t m) { return (uint32_t)__popcll(m); }

// inclusive prefix sum across the wave
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
    const uint32_t lane = lane_id();
#pragma unroll
    for (uint32_t o = 1; o < 64; o <<= 1) {
        uint32_t t = __shfl_up(v, o, 64);
        if (lane >= o) v += t;
    }
    return v;
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
    for (uint32_t o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
    for (uint32_t o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Exclusive scan of one value per thread over a block of NT threads.
// `scratch` holds NT/64+1 words of LDS; returns the block total in *total.
// Contains barriers: every thread of the block must call it.  LDS_ONLY: its
// barriers leave the caller's global memory operations in flight.
template <uint32_t NT, bool LDS_ONLY = false>
__device__ __forceinline__ uint32_t block_excl_scan_n(uint32_t v, uint32_t *scratch, uint32_t *total) {
    constexpr uint32_t NW = NT / 64;
    const uint32_t lane = threadIdx.x & 63u, w = threadIdx.x >> 6;
    uint32_t inc = wave_incl_scan(v);
    if (lane == 63) scratch[w] = inc;
    if (LDS_ONLY)
        lds_barrier();
    else
        __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t s = 0;
        for (uint32_t i = 0; i < NW; ++i) {
            uint32_t t = scratch[i];
            scratch[i] = s;
            s += t;
        }
        scratch[NW] = s;
    }
    if (LDS_ONLY)
        lds_barrier();
    else
        __syncthreads();
    uint32_t r = scratch[w] + inc - v;
    *total = scratch[NW];
    if (LDS_ONLY)
        lds_barrier();
    else
        __syncthreads();
    return r;
}

__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t *scratch, uint32_t *total) {
    return block_excl_scan_n<NTHREADS>(v, scratch, total);
}

// ---------------------------------------------------------------------------
// Tiles.
// ---------------------------------------------------------------------------
// ---------------------------------------------------------------------------
// Equal-count runs of the value fit (rank -> run, abscissa, polynomial).
// ---------------------------------------------------------------------------
// floor(a / b) for a < 2^53, b >= 1: a double-precision estimate, then one
// integer correction step (the estimate is off by at most one).
__device__ __forceinline__ uint64_t udiv53(uint64_t a, uint32_t b) {
    uint64_t q = (uint64_t)((double)a / (double)b);
    if (q * b > a)
        --q;
    else if ((q + 1) * b <= a)
        ++q;
    return q;
}

// Run s holds sorted ranks [floor(s n / S), floor((s+1) n / S)); the run of
// `rank` is the largest s with floor(s n / S) <= rank, i.e.
// floor(((rank + 1) S - 1) / n).  n < 2^32 and S <= 4096 keep every
// product below 2^53.
__device__ __forceinline__ void run_of_rank(uint32_t rank, uint32_t n, uint32_t seff, uint32_t *s, uint32_t *lo,
                                            uint32_t *ns) {
    const uint32_t r = (uint32_t)udiv53(((uint64_t)rank + 1u) * seff - 1u, n);
    const uint32_t a = (uint32_t)udiv53((uint64_t)r * n, seff);
    const uint32_t b = (uint32_t)udiv53(((uint64_t)r + 1u) * n, seff);
    *s = r;
    *lo = a;
    *ns = b - a;
}

// Run of a sorted rank under chord segmentation: the runs start at 0 and at
// the seff - 1 interior starts knots[0..seff-2] (ascending), and the last
// ends at n.  Binary search for the last start <= rank; false if the starts
// do not bracket the rank (a damaged record).
__device__ __forceinline__ bool run_of_rank_knots(const uint32_t *knots, uint32_t rank, uint32_t n, uint32_t seff,
                                                  uint32_t *s, uint32_t *lo, uint32_t *ns) {
    uint32_t a = 0, b = seff;  // the run is in [a, b)
    while (b - a > 1) {
        const uint32_t mid = (a + b) >> 1;
        if (knots[mid - 1] <= rank)
            a = mid;
        else
            b = mid;
    }
    const uint32_t st = a ? knots[a - 1] : 0u;
    const uint32_t en = a + 1 < seff ? knots[a] : n;
    *s = a;
    *lo = st;
    *ns = en - st;
    return st <= rank && rank < en;
}

// abscissa of local rank j in a run of ns points: (2j - (ns-1)) / (ns-1)
__device__ __forceinline__ double abscissa(uint64_t j, uint64_t ns) {
    return ns > 1 ? (double)(2 * (int64_t)j - (int64_t)(ns - 1)) / (double)(ns - 1) : 0.0;
}

// Horner's rule in double on fp32 coefficients c[0..deg], rounded to fp32
__device__ __forceinline__ float horner(const float *c, uint32_t deg, double t) {
    double y = (double)c[deg];
    for (int p = (int)deg - 1; p >= 0; --p) y = y * t + (double)c[p];
    return (float)y;
}

// ---------------------------------------------------------------------------
// Index policies: which positives are coded, and as which value.
// ---------------------------------------------------------------------------
// P1 keeps positive q iff pi(q) < ncoded, as value pi(q): pi is a keyed
// pseudo-random permutation of [0, npos), a 4-round Feistel network on 2h-bit
// words (h = ceil(ceil(log2 npos) / 2), at least 1; round j is MurmurHash3 of
// the 4-byte half with seed (seed + j), cut to h bits) restricted to
// [0, npos) by cycle walking (Black and Rogaway, CT-RSA 2002).  The walk
// ends: pi's cycle through q returns to q, which is in the domain.
__device__ __forceinline__ uint32_t feistel_perm(uint32_t q, uint32_t npos, uint32_t seed) {
    uint32_t bits = 0;
    while (bits < 32 && (1ull << bits) < npos) ++bits;
    const uint32_t h = max(1u, (bits + 1) / 2);
    const uint32_t mask = h >= 32 ? 0xffffffffu : ((1u << h) - 1u);
    uint32_t y = q;
    do {
        uint32_t L = (y >> h) & mask, R = y & mask;
#pragma unroll
        for (uint32_t j = 0; j < 4; ++j) {
            const uint32_t t = L ^ (mm3_seed(mm3_key(R), seed + j) & mask);
            L = R;
            R = t;
        }
        y = (L << h) | R;
    } while (y >= npos);
    return y;
}

// value number of positive rank q under `policy`, or NO_SLOT if dropped
__device__ __forceinline__ uint32_t policy_slot(uint32_t q, uint32_t npos, uint32_t ncoded, uint32_t policy,
                                                uint32_t seed) {
    switch (policy) {
        case POLICY_P0: return q;
        case POLICY_RANDOM: {
            const uint32_t p = feistel_perm(q, npos, seed);
            return p < ncoded ? p : NO_SLOT;
        }
        case POLICY_LEFTMOST: return q < ncoded ? q : NO_SLOT;
        case POLICY_MIDDLE: {
            const uint32_t s0 = (npos - ncoded) / 2;
            return (q >= s0 && q - s0 < ncoded) ? q - s0 : NO_SLOT;
        }
        default: return q >= npos - ncoded ? q - (npos - ncoded) : NO_SLOT;
    }
}

// Raw buffer view of `bytes` bytes at p (both the same on every lane of the
// wave; readfirstlane states it, so the descriptor sits in scalar
// registers).  A load at an offset past the view returns 0 and touches no
// memory, so bounds checks need neither branches nor clamps.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_view(const void *p, uint32_t bytes) {
    const uint64_t a = (uint64_t)(uintptr_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    void *q = (void *)(uintptr_t)(((uint64_t)hi << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(q, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes),
                                             BUFFER_RSRC_WORD3);
}

__device__ __forceinline__ uint32_t buffer_u32(__amdgpu_buffer_rsrc_t v, uint32_t byte_off) {
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(v, byte_off, 0, 0);
}

// tensor holding global tile `tile` (one read of the table k_init fills)
__device__ __forceinline__ uint32_t tensor_of_tile(const Work &w, uint32_t tile) { return w.tile_tensor[tile]; }

// Magnitude key: IEEE bits with the sign cleared (orders like |x|).
__device__ __forceinline__ uint32_t mag_key(float x) { return __float_as_uint(x) & 0x7fffffffu; }

// Order-preserving u32 image of a float (unsigned order == float order).
__device__ __forceinline__ uint32_t order_key(float x) {
    uint32_t u = __float_as_uint(x);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float order_key_inv(uint32_t k) {
    uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    return __uint_as_float(u);
}

// Filter words for |S| = n (Remark 2 of Section 10.2): m = 32 ceil(ceil(n mC)
// / 32), at least 32 bits, at most the words reserved for the tensor.
__device__ __forceinline__ uint32_t filter_words(TDesc &td) {
    if (td.in.m_words_in) return td.in.m_words_in;
    const double raw = ceil((double)td.n * td.in.mC);
    uint64_t words = ((uint64_t)raw + 31u) / 32u;
    if (words < 1) words = 1;
    const uint64_t cap = ((uint64_t)td.in.bl_nslices << td.in.slice_log2) / 32u;
    if (words > cap) {
        atomicOr(&td.flags, FLAG_CAPACITY);
        words = cap;
    }
    return (uint32_t)words;
}

// Width of one reorder-map entry: smallest b >= 1 with 2^b >= n.
__device__ __forceinline__ uint32_t sigma_bits(uint32_t n) {
    if (n <= 2) return 1;
    return 32u - __clz(n - 1u);
}

}  // namespace dr
