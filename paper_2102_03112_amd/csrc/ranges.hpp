// ranges.hpp -- the index ranges that kernels derive from a tensor's plan
// (which bitmap words, list entries or sorted values a block touches).
// They are __host__ __device__ so that the library's host-side range check
// (dr_check_ranges) replays exactly the arithmetic the kernels run, on every
// chunk and tile of a configuration, without a GPU.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dr {

struct Range32 {
    uint32_t lo, hi;  // [lo, hi); lo <= hi always
};

__host__ __device__ __forceinline__ uint32_t umin32(uint32_t a, uint32_t b) { return a < b ? a : b; }

// Direct Bloom insert from the selection bitmap: chunk c of a tensor of
// `ntiles` tiles covers tiles [c per, (c+1) per), in bitmap words of the
// tensor's slot.  Chunks past the tensor's last tile (a small tensor gets
// more chunks than it has tiles) are empty: both ends are clamped, so the
// length hi - lo never wraps.
__host__ __device__ __forceinline__ Range32 dir_bitmap_chunk(uint32_t ntiles, uint32_t per, uint32_t c,
                                                             uint32_t tile_words) {
    const uint64_t t1 = (uint64_t)(c + 1u) * per;
    const uint32_t hi = (uint32_t)((t1 < ntiles ? t1 : ntiles) * tile_words);
    const uint64_t lo64 = (uint64_t)c * per * tile_words;
    return Range32{lo64 < hi ? (uint32_t)lo64 : hi, hi};
}

// Direct Bloom insert from an index list of n items: chunk c covers items
// [c per, (c+1) per) clamped to n.
__host__ __device__ __forceinline__ Range32 dir_list_chunk(uint32_t n, uint32_t per, uint32_t c) {
    const uint64_t a = (uint64_t)c * per, b = a + per;
    const uint32_t hi = (uint32_t)(b < n ? b : n);
    return Range32{a < hi ? (uint32_t)a : hi, hi};
}

// Value sort: tile lt of a tensor holding nv values covers values
// [lt tile, lt tile + tile) clamped to nv.
__host__ __device__ __forceinline__ Range32 sort_tile_values(uint32_t nv, uint32_t lt, uint32_t tile) {
    const uint64_t a = (uint64_t)lt * tile, b = a + tile;
    const uint32_t hi = (uint32_t)(b < nv ? b : nv);
    return Range32{a < hi ? (uint32_t)a : hi, hi};
}

// Probe pass: block b of `grid` owns tiles [b per, b per + per) of all
// ntiles_total, per = ceil(ntiles_total / grid), clamped to the end.
__host__ __device__ __forceinline__ Range32 probe_block_tiles(uint32_t ntiles_total, uint32_t grid, uint32_t b) {
    const uint32_t per = (ntiles_total + grid - 1u) / grid;
    const uint64_t a = (uint64_t)b * per;
    const uint32_t lo = (uint32_t)(a < ntiles_total ? a : ntiles_total);
    const uint64_t e = (uint64_t)lo + per;
    return Range32{lo, (uint32_t)(e < ntiles_total ? e : ntiles_total)};
}

}  // namespace dr
