// Host emulation of the few HIP device facilities the bucketed-query kernels
// use: every thread of a block is a std::thread, __syncthreads a block
// barrier, wave intrinsics exchanges through a per-wave buffer.
#pragma once
#include <stdint.h>
#include <stddef.h>
#include <algorithm>
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <thread>
#include <cstring>
#include <cmath>
using std::ceil;
using std::max;
using std::min;
struct dim3 {
    uint32_t x = 0, y = 0, z = 0;
};
extern thread_local dim3 threadIdx, blockIdx;
extern dim3 blockDim, gridDim;
#define __global__
#define __device__
#define __host__
#define __forceinline__ inline
#define __launch_bounds__(...)
#define __shared__ static
#define __restrict__
#define __HIP_MEMORY_SCOPE_AGENT 0
void emu_block_barrier();
uint64_t emu_wave_xchg(uint64_t v, uint32_t src_lane);  // every lane of the wave calls it
inline uint32_t emu_lane() { return threadIdx.x & 63u; }
inline void __syncthreads() { emu_block_barrier(); }
#define __builtin_amdgcn_s_barrier() emu_block_barrier()
#define __builtin_amdgcn_fence(...) std::atomic_thread_fence(std::memory_order_seq_cst)
#define __builtin_amdgcn_wave_barrier() ((void)0)
#define __builtin_amdgcn_s_sleep(n) std::this_thread::yield()
#define __builtin_amdgcn_readfirstlane(x) (x)
inline uint32_t __builtin_amdgcn_mbcnt_lo(uint32_t m, uint32_t x) {
    const uint32_t l = emu_lane();
    return x + (uint32_t)__builtin_popcount(l < 32 ? (m & ((1u << l) - 1u)) : m);
}
inline uint32_t __builtin_amdgcn_mbcnt_hi(uint32_t m, uint32_t x) {
    const uint32_t l = emu_lane();
    return x + (l < 32 ? 0u : (uint32_t)__builtin_popcount(m & ((1u << (l - 32)) - 1u)));
}
inline uint64_t __ballot(bool p) {
    uint64_t m = 0;
    for (uint32_t s = 0; s < 64; ++s) m |= (emu_wave_xchg(p ? 1u : 0u, s) & 1ull) << s;
    return m;
}
template <typename T>
inline T emu_shfl(T v, uint32_t src) {
    uint64_t raw = 0;
    memcpy(&raw, &v, sizeof(T));
    raw = emu_wave_xchg(raw, src & 63u);
    T r;
    memcpy(&r, &raw, sizeof(T));
    return r;
}
#include <cstring>
template <typename T> inline T __shfl_xor(T v, int o, int = 64) { return emu_shfl(v, emu_lane() ^ (uint32_t)o); }
template <typename T> inline T __shfl_up(T v, unsigned d, int = 64) {
    const uint32_t l = emu_lane();
    return emu_shfl(v, l >= d ? l - d : l);
}
template <typename T> inline T __shfl_down(T v, unsigned d, int = 64) {
    const uint32_t l = emu_lane();
    return emu_shfl(v, l + d < 64 ? l + d : l);
}
template <typename T> inline T __shfl(T v, int s, int = 64) { return emu_shfl(v, (uint32_t)s); }
inline int __popc(uint32_t x) { return __builtin_popcount(x); }
inline int __popcll(uint64_t x) { return __builtin_popcountll(x); }
inline int __ffs(uint32_t x) { return __builtin_ffs((int)x); }
inline int __ffsll(unsigned long long x) { return __builtin_ffsll((long long)x); }
inline uint32_t __float_as_uint(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
inline float __uint_as_float(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
inline int __clz(uint32_t x) { return x ? __builtin_clz(x) : 32; }
inline uint32_t __umulhi(uint32_t a, uint32_t b) { return (uint32_t)(((uint64_t)a * b) >> 32); }
inline uint32_t atomicAdd(uint32_t *p, uint32_t v) { return __atomic_fetch_add(p, v, __ATOMIC_SEQ_CST); }
inline uint32_t atomicOr(uint32_t *p, uint32_t v) { return __atomic_fetch_or(p, v, __ATOMIC_SEQ_CST); }
inline unsigned long long atomicAdd(unsigned long long *p, unsigned long long v) { return __atomic_fetch_add(p, v, __ATOMIC_SEQ_CST); }
inline unsigned long long atomicOr(unsigned long long *p, unsigned long long v) { return __atomic_fetch_or(p, v, __ATOMIC_SEQ_CST); }
#define __hip_atomic_load(p, o, s) __atomic_load_n((p), __ATOMIC_SEQ_CST)
#define __hip_atomic_store(p, v, o, s) __atomic_store_n((p), (v), __ATOMIC_SEQ_CST)
struct __amdgpu_buffer_rsrc_t {
    const uint8_t *base;
    uint32_t bytes;
};
inline __amdgpu_buffer_rsrc_t __builtin_amdgcn_make_buffer_rsrc(void *p, short, int bytes, int) {
    return {(const uint8_t *)p, (uint32_t)bytes};
}
inline uint32_t __builtin_amdgcn_raw_buffer_load_b32(__amdgpu_buffer_rsrc_t v, uint32_t off, int, int) {
    if ((uint64_t)off + 4 > v.bytes) return 0;
    uint32_t r;
    memcpy(&r, v.base + off, 4);
    return r;
}
typedef int hipError_t;
typedef void *hipStream_t;
