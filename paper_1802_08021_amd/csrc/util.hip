// Host->device transfer of small blobs through kernel arguments, so that no
// pageable host copy (and no implicit host synchronization) is involved.
#include "internal.h"

#include <string.h>

#include <algorithm>

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

struct Timers {
    bool enabled = false;
    bool created = false;
    hipEvent_t ev[kTSlots][2];
    bool recorded[kTSlots] = {};
};
thread_local Timers g_timers;

}  // namespace

void timer_begin(int slot, hipStream_t s)
{
    Timers& t = g_timers;
    if (!t.enabled) return;
    if (!t.created) {
        for (int i = 0; i < kTSlots; ++i)
            for (int j = 0; j < 2; ++j)
                if (hipEventCreate(&t.ev[i][j]) != hipSuccess) return;
        t.created = true;
    }
    hipEventRecord(t.ev[slot][0], s);
}

void timer_end(int slot, hipStream_t s)
{
    Timers& t = g_timers;
    if (!t.enabled || !t.created) return;
    hipEventRecord(t.ev[slot][1], s);
    t.recorded[slot] = true;
}

int timer_enable(int on)
{
    g_timers.enabled = on != 0;
    for (bool& r : g_timers.recorded) r = false;
    return 0;
}

int timer_read(int slot, float* ms)
{
    Timers& t = g_timers;
    if (slot < 0 || slot >= kTSlots || !ms || !t.created || !t.recorded[slot]) return -1;
    if (hipEventSynchronize(t.ev[slot][1]) != hipSuccess) return -5;
    return hipEventElapsedTime(ms, t.ev[slot][0], t.ev[slot][1]) == hipSuccess ? 0 : -5;
}

}  // namespace sparcml
