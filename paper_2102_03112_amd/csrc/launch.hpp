// launch.hpp -- host-side launchers of the codec's kernels (one per .hip file
// that defines them), called by the C ABI in api.hip.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <stdint.h>

#include "dr_common.hpp"
#include "ranges.hpp"

namespace dr {

int device_cus();  // compute units of the current device

// Resident blocks per CU of `kernel` at `threads` threads on the current
// device (hipOccupancyMaxActiveBlocksPerMultiprocessor), cached per kernel
// address, block size and device.
int blocks_per_cu(const void *kernel, int threads);

// A grid of persistent blocks: as many as can be resident at once on the
// current device (so every block starts at once and none waits for another
// to finish), but no more than `work` units.
template <typename K>
int resident_grid(K kernel, int threads, uint32_t work) {
    const uint32_t g = (uint32_t)(blocks_per_cu((const void *)kernel, threads) * device_cus());
    return (int)(work < g ? (work ? work : 1u) : g);
}

// Opt-in per-kernel timing (dr_trace_begin / dr_trace_end): when tracing is
// on for the calling host thread, an event is recorded on the stream after
// each kernel launch; the time between consecutive events is that kernel's.
void trace_mark(hipStream_t s, const char *kernel);

constexpr int INIT_CHUNK = 14;  // tensors per set-up launch (kernel argument size)

struct InitArgs {
    uint32_t first, count;
    TInit t[INIT_CHUNK];
};

struct ZeroRange {
    void *p;
    uint64_t words;  // 32-bit words to clear
};
struct ZeroArgs {
    ZeroRange z[8];
    uint32_t n;
};
// k_init's arguments stay within 4 KiB
static_assert(sizeof(Work) + sizeof(InitArgs) + sizeof(ZeroArgs) <= 4096, "set-up kernel arguments");

// select.hip
// descriptors of one chunk of tensors, plus clearing the zero ranges
hipError_t launch_init(const Work &w, const InitArgs &a, const ZeroArgs &z, hipStream_t s);
// hist_blocks: the first-digit histograms (exact, or of the samples);
// redo_blocks: the full histograms of sampled tensors whose bracket missed
// (0: no tensor is sampled, and the redo passes are not launched)
hipError_t launch_topr(const Work &w, const float *g, uint32_t hist_blocks, uint32_t redo_blocks, bool any_topr,
                       hipStream_t s);
hipError_t launch_nonzero(const Work &w, const float *g, int grid_persist, hipStream_t s);
hipError_t launch_compact_selection(const Work &w, const float *g, float *val_out, int grid_persist, hipStream_t s);
hipError_t launch_tile_popc(const Work &w, const uint32_t *bits, int grid_persist, hipStream_t s);

// bloom.hip
// Insert in rounds of `hash_per_round` hash functions (the position buffer
// holds that many positions per reserved item); items come from the
// selection bitmap or from the list w.S.
hipError_t launch_bloom_direct(const Work &w, bool from_bitmap, uint32_t blocks, uint32_t slices, hipStream_t s);
hipError_t launch_bloom_insert(const Work &w, bool from_bitmap, uint32_t total_chunks, uint32_t total_slices,
                               uint32_t max_slices, uint32_t hash_per_round, uint32_t kmax, hipStream_t s);
// the sender's query: probe (with the per-tensor value set-up and headers),
// then emit (with the layout over the tensors); after_probe, if given, is
// recorded between the two
hipError_t launch_query_encode(const Work &w, const float *g, int grid_persist, uint64_t *counts_out, hipStream_t s,
                               hipEvent_t after_probe = nullptr);
// The receiver's bucketed query of one tensor (a filter larger than an
// XCD's L2): rounds of one hash each, then the positives bitmap; the probe
// pass that follows counts it.  Caps of the work it was planned for:
// nsl_cap filter slices, nch_cap round-0 list chunks, nreg index regions.
struct QbTensor {
    uint32_t t, nsl_cap, nch_cap, nreg;
    uint32_t ncol;  // columns of the count table: max(nch_cap, nsl_cap)
};
hipError_t launch_query_bucketed(const Work &w, const QbTensor &q, uint32_t k, uint32_t min_bits, hipStream_t s);
hipError_t launch_query_plain(const Work &w, uint32_t *idx_out, uint64_t cap, uint64_t *n_out, int grid_persist,
                              hipStream_t s);
// the receiver's query in two halves: the probe pass (at most max_blocks
// blocks) with the tile scan, then the emit pass
hipError_t launch_probe_decode(const Work &w, float *dense_out, uint64_t *counts_out, uint32_t max_blocks,
                               hipStream_t s);
hipError_t launch_emit_decode(const Work &w, float *dense_out, uint32_t *idx_out, float *val_out,
                              uint64_t *counts_out, bool general, hipStream_t s);
// Several payloads of one tensor layout into one dense sum: the work's
// tensors are payload-major (tensor t of payload p is p * ntens + t).
hipError_t launch_query_decode_sum(const Work &w, uint32_t npay, uint32_t ntens, uint32_t ntiles1, float scale,
                                   float *dense_out, uint64_t *counts_out, hipStream_t s);

// valuefit.hip
// the standalone calls' device counts: at most n_cap items are used, and
// flags_out (nullable) receives FLAG_CAPACITY if the count exceeds n_cap
hipError_t launch_keygen(const Work &w, const float *vals, const uint64_t *n, uint64_t n_cap, uint64_t *flags_out,
                         int grid_persist, hipStream_t s);
hipError_t launch_value_setup(const Work &w, bool payload, uint64_t *counts_out, hipStream_t s);
hipError_t launch_sort(const Work &w, uint32_t cap_tiles, hipStream_t s);
hipError_t launch_segment(const Work &w, uint32_t grid_req, bool block_pass, hipStream_t s);
// the fit's moments with the packing of the reorder maps (one launch), the
// solve, then the double-exponential passes if any tensor asks for them
hipError_t launch_fit(const Work &w, uint32_t fit_blocks, uint64_t vals_est, bool dexp, hipStream_t s);
hipError_t launch_curvefit_decode(const Work &w, const float *coef, const uint32_t *sigma, const uint64_t *n,
                                  uint64_t n_cap, float *vals_out, uint64_t *flags_out, int grid_persist,
                                  hipStream_t s);
// device count <-> tensor 0's descriptor (standalone calls)
hipError_t launch_import_n(const Work &w, const uint64_t *n, uint64_t n_cap, uint64_t *flags_out, hipStream_t s);
hipError_t launch_export_n(const Work &w, uint64_t *n_out, int field, hipStream_t s);

}  // namespace dr
