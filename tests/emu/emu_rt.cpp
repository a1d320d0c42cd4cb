// Emulated block execution: NT std::threads per block, one block at a time.
#include "hip/hip_runtime.h"
#include <chrono>
#include <condition_variable>
#include <functional>
#include <mutex>
#include <vector>

thread_local dim3 threadIdx, blockIdx;
dim3 blockDim, gridDim;

struct Bar {
    std::mutex m;
    std::condition_variable cv;
    int expected = 0, arrived = 0;
    uint64_t gen = 0;
    void reset(int n) { expected = n; arrived = 0; }
    void wait(const char *what) {
        std::unique_lock<std::mutex> l(m);
        const uint64_t g = gen;
        if (++arrived == expected) {
            arrived = 0;
            ++gen;
            cv.notify_all();
            return;
        }
        if (!cv.wait_for(l, std::chrono::seconds(30), [&] { return gen != g; })) {
            fprintf(stderr, "DEADLOCK at %s: block %u thread %u (arrived %d of %d)\n", what, blockIdx.x, threadIdx.x,
                    arrived, expected);
            fflush(stderr);
            std::_Exit(3);
        }
    }
    void drop() {
        std::lock_guard<std::mutex> l(m);
        --expected;
        if (expected > 0 && arrived == expected) {
            arrived = 0;
            ++gen;
            cv.notify_all();
        }
    }
};

static Bar g_block;
static Bar g_wave[16];
static uint64_t g_xbuf[16][64];

void emu_block_barrier() { g_block.wait("block barrier"); }
uint64_t emu_wave_xchg(uint64_t v, uint32_t src) {
    const uint32_t w = threadIdx.x >> 6, l = threadIdx.x & 63u;
    g_xbuf[w][l] = v;
    g_wave[w].wait("wave exchange (write)");
    const uint64_t r = g_xbuf[w][src];
    g_wave[w].wait("wave exchange (read)");
    return r;
}

void emu_launch(uint32_t grid, uint32_t nt, const std::function<void()> &body) {
    gridDim.x = grid;
    blockDim.x = nt;
    for (uint32_t b = 0; b < grid; ++b) {
        g_block.reset((int)nt);
        for (uint32_t w = 0; w < (nt + 63) / 64; ++w) g_wave[w].reset((int)std::min<uint32_t>(64, nt - 64 * w));
        std::vector<std::thread> th;
        th.reserve(nt);
        for (uint32_t t = 0; t < nt; ++t)
            th.emplace_back([=, &body] {
                threadIdx.x = t;
                blockIdx.x = b;
                body();
                g_wave[t >> 6].drop();
                g_block.drop();
            });
        for (auto &x : th) x.join();
    }
}
