// Host->device transfer of small blobs through kernel arguments, so that no
// pageable host copy (and no implicit host synchronization) is involved.
#include "internal.h"

#include <string.h>

#include <algorithm>
#include <utility>
#include <vector>

namespace sparcml {
namespace {

__global__ void k_upload(uint32_t* dst, Blob b)
{
    for (uint32_t i = threadIdx.x; i < b.nwords; i += blockDim.x) dst[i] = b.words[i];
}

}  // namespace

hipError_t upload(void* dst, const void* src, size_t bytes, hipStream_t s)
{
    // bytes is a multiple of 4 for every caller (descriptor tables).
    const uint8_t* p = static_cast<const uint8_t*>(src);
    uint32_t* d = static_cast<uint32_t*>(dst);
    size_t words = (bytes + 3) / 4, done = 0;
    while (done < words) {
        Blob b;
        b.nwords = (uint32_t)std::min<size_t>(words - done, kBlobWords);
        memset(b.words, 0, sizeof(b.words));
        const size_t nb = std::min<size_t>((size_t)b.nwords * 4, bytes - done * 4);
        memcpy(b.words, p + done * 4, nb);
        hipLaunchKernelGGL(k_upload, dim3(1), dim3(256), 0, s, d + done, b);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        done += b.nwords;
    }
    return hipSuccess;
}

namespace {

// Every launch of a group between enabling and reading gets its own event
// pair, so that reading once after many calls averages all of them without
// synchronizing in between.  Pairs are kept for reuse; past kMaxPairs a
// group's finished pairs are folded into a running sum.
constexpr size_t kMaxPairs = 4096;

struct Group {
    std::vector<std::pair<hipEvent_t, hipEvent_t>> pool;  // created events, reused
    size_t used = 0;                                      // pairs recorded since enabling
    double folded_ms = 0.0;                               // folded pairs' total
    uint64_t folded_n = 0;
};

struct Timers {
    bool enabled = false;
    Group g[kTSlots];
};
thread_local Timers g_timers;

// Total ms and count of the first `used` pairs of a group (waits for them).
bool sum_pairs(Group& g, double* ms, uint64_t* n)
{
    for (size_t i = 0; i < g.used; ++i) {
        float t = 0.0f;
        if (hipEventSynchronize(g.pool[i].second) != hipSuccess ||
            hipEventElapsedTime(&t, g.pool[i].first, g.pool[i].second) != hipSuccess)
            return false;
        *ms += t;
        ++*n;
    }
    return true;
}

}  // namespace

void timer_begin(int slot, hipStream_t s)
{
    Timers& t = g_timers;
    if (!t.enabled) return;
    Group& g = t.g[slot];
    if (g.used == kMaxPairs) {
        if (!sum_pairs(g, &g.folded_ms, &g.folded_n)) return;
        g.used = 0;
    }
    if (g.used == g.pool.size()) {
        hipEvent_t a, b;
        if (hipEventCreate(&a) != hipSuccess) return;
        if (hipEventCreate(&b) != hipSuccess) {
            hipEventDestroy(a);
            return;
        }
        g.pool.emplace_back(a, b);
    }
    hipEventRecord(g.pool[g.used].first, s);
}

void timer_end(int slot, hipStream_t s)
{
    Timers& t = g_timers;
    if (!t.enabled) return;
    Group& g = t.g[slot];
    if (g.used == g.pool.size()) return;  // begin failed
    hipEventRecord(g.pool[g.used].second, s);
    ++g.used;
}

int timer_enable(int on)
{
    g_timers.enabled = on != 0;
    for (Group& g : g_timers.g) {
        g.used = 0;
        g.folded_ms = 0.0;
        g.folded_n = 0;
    }
    return 0;
}

int timer_read(int slot, float* ms)
{
    if (slot < 0 || slot >= kTSlots || !ms) return -1;
    Group& g = g_timers.g[slot];
    double sum = g.folded_ms;
    uint64_t n = g.folded_n;
    if (!sum_pairs(g, &sum, &n)) return -5;
    if (n == 0) return -1;
    *ms = (float)(sum / (double)n);
    return 0;
}

}  // namespace sparcml
