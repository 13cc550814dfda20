// Top-k sparsification by magnitude on gfx950 (§2.2 "Structured
// Sparsification"; Alg. 1: TopK and the error update eps = acc - TopK(acc)).
//
// Exact radix select on the 31-bit magnitude key (IEEE bits, sign cleared),
// normally in one pass over the data.  A histogram of the top 11 key bits
// over a sample of the row (1024 segments of 256 elements) gives a gather
// bin safely below the k-th largest key; the gather pass collects, per
// 4096-element wave unit, every entry in that bin or above it as {element,
// value bits} in index order (a few per unit).  If the row then holds at
// least k gathered keys, the k-th largest key K* and how many entries equal
// to it are still needed follow from the gathered keys alone (11-, 10- and
// 10-bit histograms), which also give every unit its counts; a scan over
// the units gives output offsets, and the selection is written from the
// gathered entries (equal keys: lowest index first), zeroing the residual
// at the selected positions.  Otherwise the row takes the exact gather bin
// from a histogram of all its keys and gathers again; a row with a unit
// holding more than kSlots entries even then takes two more histogram
// passes, a count pass and a write pass over its data.  Every path is
// exact: the sample only decides how much data is read.
#include "internal.h"

#include <algorithm>

namespace sparcml {
namespace {

constexpr uint32_t kUnit = 4096;  // elements per wave unit (64 iterations of 64 lanes)
constexpr uint32_t kSlots = 32;   // gathered entries per unit
constexpr int kHistBlocksPerRank = 64;
constexpr uint32_t kExactGatherBlocks = 64;  // workgroups per row of the exact path's gather (grid-stride)
constexpr uint64_t kSampleSegs = 1024;  // 256-element segments sampled per row
// Gathered keys are also listed per row in kSub sub-lists (unit u appends to
// sub-list u mod kSub, reserving its place with one atomic on that
// sub-list's counter, each counter on a cache line of its own, so that no
// counter takes more than a few hundred atomics); a full sub-list counts as
// an overflow.
constexpr uint32_t kSub = 64;
constexpr uint32_t kSubCap = 1024;                     // keys per sub-list
constexpr uint32_t kList = kSub * kSubCap;             // keys listed per row
constexpr uint32_t kCntStride = 32;                    // counter words apart (128 B)

__device__ __forceinline__ uint32_t mag_key(float v) { return __float_as_uint(v) & 0x7FFFFFFFu; }

struct RankState {
    uint32_t prefix;  // key bits fixed so far (gather: the lowest 11-bit bin gathered)
    uint32_t full;    // 0: K* from the gathered keys; 1: refined by passes over the data
    uint64_t krem;    // entries still to take from keys matching the prefix
    uint32_t exact;   // 0: gather bin estimated from a sample; 1: from the full histogram
    uint32_t pad;
};

// Keys of row r from element lo to hi (lo a multiple of 4), in float4 loads
// where the row is 16-byte aligned; f(element, key) in any order.
template <typename F>
__device__ __forceinline__ void for_keys(const float* row, uint64_t lo, uint64_t hi, uint32_t t,
                                         uint32_t nt, F&& f)
{
    if ((reinterpret_cast<uintptr_t>(row) & 15u) == 0u) {
        // batches of four float4 loads per thread, all issued before use
        const uint64_t step = 16ull * nt, hb = lo + ((hi - lo) / step) * step;
        for (uint64_t e = lo + 4ull * t; e < hb; e += step) {
            float4 v[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] = *reinterpret_cast<const float4*>(row + e + 4ull * nt * q);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint64_t b = e + 4ull * nt * q;
                f(b, mag_key(v[q].x));
                f(b + 1, mag_key(v[q].y));
                f(b + 2, mag_key(v[q].z));
                f(b + 3, mag_key(v[q].w));
            }
        }
        const uint64_t hv = hb + ((hi - hb) & ~3ull);
        for (uint64_t e = hb + 4ull * t; e < hv; e += 4ull * nt) {
            const float4 v = *reinterpret_cast<const float4*>(row + e);
            f(e, mag_key(v.x));
            f(e + 1, mag_key(v.y));
            f(e + 2, mag_key(v.z));
            f(e + 3, mag_key(v.w));
        }
        for (uint64_t e = hv + t; e < hi; e += nt) f(e, mag_key(row[e]));
    } else {
        for (uint64_t e = lo + t; e < hi; e += nt) f(e, mag_key(row[e]));
    }
}

// PASS 0: bins = key >> 20 (2048); PASS 1: (key >> 10) & 1023 among keys
// whose top 11 bits match; PASS 2: key & 1023 among keys whose top 21 bits
// match.
template <int PASS>
__global__ void __launch_bounds__(256) k_hist(const float* x, uint64_t N, const RankState* st,
                                              uint32_t* hist)
{
    constexpr uint32_t NB = PASS == 0 ? 2048u : 1024u;
    constexpr int SHIFT = PASS == 0 ? 20 : (PASS == 1 ? 10 : 0);
    constexpr int PSHIFT = PASS == 1 ? 20 : 10;
    __shared__ uint32_t s_h[NB];
    const uint32_t r = blockIdx.y;
    if (PASS == 0 ? st[r].exact == 0u : st[r].full == 0u) return;  // row not on this path
    for (uint32_t i = threadIdx.x; i < NB; i += 256) s_h[i] = 0;
    __syncthreads();
    const uint32_t prefix = PASS == 0 ? 0u : st[r].prefix;
    const float* row = x + (uint64_t)r * N;
    const uint64_t per = ((N + gridDim.x - 1) / gridDim.x + 3) & ~3ull;
    const uint64_t lo = min((uint64_t)blockIdx.x * per, N), hi = min(lo + per, N);
    for_keys(row, lo, hi, threadIdx.x, 256u, [&](uint64_t, uint32_t key) {
        if (PASS == 0 || (key >> PSHIFT) == prefix) atomicAdd(&s_h[(key >> SHIFT) & (NB - 1)], 1u);
    });
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < NB; i += 256)
        if (s_h[i]) atomicAdd(&hist[(uint64_t)r * 2048 + i], s_h[i]);
}

// Find the bin holding the krem-th largest remaining key; refine the state
// and clear the histogram for the next pass.
template <int PASS>
__global__ void __launch_bounds__(256) k_select(RankState* st, uint32_t* hist)
{
    constexpr uint32_t NB = PASS == 0 ? 2048u : 1024u, PER = NB / 256;
    constexpr int BITS = PASS == 0 ? 11 : 10;
    __shared__ uint64_t s_w[4];
    const uint32_t r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    if (PASS == 0 ? st[r].exact == 0u : st[r].full == 0u) return;
    // read the state before the barrier below; one thread rewrites it after
    const uint64_t krem = st[r].krem;
    const uint32_t prefix = st[r].prefix;
    uint32_t* h = hist + (uint64_t)r * 2048;
    // thread tid owns bins [lo, lo+PER); threads are ordered from the top
    const uint32_t lo = NB - (tid + 1) * PER;
    uint32_t cnt[PER];
    uint64_t mine = 0;
#pragma unroll
    for (uint32_t i = 0; i < PER; ++i) {
        cnt[i] = h[lo + i];
        mine += cnt[i];
    }
    uint64_t incl = mine;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint64_t y = __shfl_up(incl, o);
        if (lane >= (uint32_t)o) incl += y;
    }
    if (lane == 63) s_w[wv] = incl;
    __syncthreads();
    uint64_t above = incl - mine;  // entries in bins above this thread's bins
    for (uint32_t w = 0; w < wv; ++w) above += s_w[w];
    uint64_t run = above;
    for (int i = (int)PER - 1; i >= 0; --i) {
        if (run < krem && run + cnt[i] >= krem) {
            st[r].prefix = (prefix << BITS) | (lo + (uint32_t)i);
            st[r].krem = krem - run;
        }
        run += cnt[i];
    }
#pragma unroll
    for (uint32_t i = 0; i < PER; ++i) h[lo + i] = 0;
}

// mode 0: start from a sampled gather bin; 1: from the exact one; 2: more
// keys per unit than a unit gathers are selected -- straight to the passes
// over the data (marked as overflowed, so that no gather runs).
__global__ void k_init(RankState* st, uint32_t P, uint64_t k, uint32_t* hist, uint32_t* overflow, uint32_t mode,
                       uint32_t* kcnt)
{
    const uint64_t gid = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid < (uint64_t)P * kSub) kcnt[gid * kCntStride] = 0;
    if (gid < P) {
        st[gid].prefix = 0;
        st[gid].full = 0;
        st[gid].krem = k;
        st[gid].exact = mode >= 1u ? 1u : 0u;
        st[gid].pad = 0;
        overflow[gid] = mode == 2u ? 1u : 0u;
    }
    if (gid < (uint64_t)P * 2048) hist[gid] = 0;
}

__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* s_w, uint32_t* total)
{
    const uint32_t lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
    uint32_t incl = v;
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o);
        if (lane >= (uint32_t)o) incl += y;
    }
    __syncthreads();
    if (lane == 63) s_w[wv] = incl;
    __syncthreads();
    uint32_t ex = incl - v, t = 0;
    for (uint32_t w = 0; w < nw; ++w) {
        if (w < wv) ex += s_w[w];
        t += s_w[w];
    }
    *total = t;
    return ex;
}

// Sample histogram of the top 11 key bits: kSampleSegs segments of 256
// consecutive elements spread evenly over the row (all of a short row).
__global__ void __launch_bounds__(256) k_sample(const float* x, uint64_t N, uint32_t stride, uint32_t* hist)
{
    __shared__ uint32_t s_h[2048];
    const uint32_t r = blockIdx.y;
    for (uint32_t i = threadIdx.x; i < 2048; i += 256) s_h[i] = 0;
    __syncthreads();
    const float* row = x + (uint64_t)r * N;
    const uint64_t nseg = (N + 255) / 256, step = (uint64_t)gridDim.x * stride;
    for (uint64_t g = (uint64_t)blockIdx.x * stride; g < nseg; g += 4 * step) {
        float v[4];
        bool ok[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {  // four segments' loads in flight
            const uint64_t e = (g + q * step) * 256 + threadIdx.x;
            ok[q] = g + q * step < nseg && e < N;
            v[q] = ok[q] ? row[e] : 0.0f;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (ok[q]) atomicAdd(&s_h[mag_key(v[q]) >> 20], 1u);
    }
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < 2048; i += 256)
        if (s_h[i]) atomicAdd(&hist[(uint64_t)r * 2048 + i], s_h[i]);
}

// The gather bin of a row from its sample: the 11-bit bin of the t-th
// largest sampled key, t = k f + 4 sqrt(k f) + 16 for sample fraction f --
// low enough that the row holds at least k keys at or above it, barring a
// sample off by more than four standard deviations (checked after the
// gather).  Clears the histogram.
__global__ void __launch_bounds__(256) k_estimate(RankState* st, uint32_t* hist, uint64_t k, double f)
{
    __shared__ uint32_t s_w[4];
    __shared__ uint32_t s_bin;
    const uint32_t r = blockIdx.x, tid = threadIdx.x;
    if (st[r].exact != 0u) return;  // the row starts from the exact bin
    uint32_t* h = hist + (uint64_t)r * 2048;
    const double kf = (double)k * f;
    const uint64_t t = (uint64_t)ceil(kf + 4.0 * sqrt(kf) + 16.0);
    // thread tid owns bins [lo, lo + 8), threads ordered from the top
    const uint32_t lo = 2048u - (tid + 1u) * 8u;
    uint32_t cnt[8], mine = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        cnt[i] = h[lo + i];
        mine += cnt[i];
    }
    if (tid == 0) s_bin = 0u;  // the whole row when the sample holds fewer than t keys
    uint32_t total;
    uint64_t run = block_excl_scan(mine, s_w, &total);
    for (int i = 7; i >= 0; --i) {
        if (run < t && run + cnt[i] >= t) s_bin = lo + (uint32_t)i;
        run += cnt[i];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 8; ++i) h[lo + i] = 0;
    if (tid == 0) st[r].prefix = s_bin;
}

// Per wave unit: every entry whose top 11 key bits are at or above the
// gather bin goes as {element, value bits} into the unit's kSlots slots in
// index order, and its key into the row's key list (a unit with more, or a
// full list, flags its row for the next path).  A separate residual
// receives a copy of the row here.
__global__ void __launch_bounds__(256) k_gather(const float* x, uint64_t N, uint32_t U, const RankState* st,
                                                uint2* cand, uint32_t* ccnt, uint32_t* overflow, float* residual,
                                                uint32_t exact, uint32_t* klist, uint32_t* kcnt)
{
    const uint32_t r = blockIdx.y, lane = threadIdx.x & 63;
    if (st[r].exact != exact) return;  // not this path
    // units one a wave, grid-stride: the fallback launch takes a grid
    // smaller than the row's units (most rows skip it at once)
    for (uint32_t u = blockIdx.x * 4 + (threadIdx.x >> 6); u < U; u += gridDim.x * 4) {
        if (overflow[r] != 0u) return;  // gathered too many
        const uint32_t bin = st[r].prefix;
        const float* row = x + (uint64_t)r * N;
        float* res = residual && residual != x ? residual + (uint64_t)r * N : nullptr;
        const uint64_t lo = (uint64_t)u * kUnit, hi = min(lo + kUnit, N);
        uint2* cu = cand + ((uint64_t)r * U + u) * kSlots;
        const uint32_t sub = u % kSub;
        uint32_t* kl = klist + ((uint64_t)r * kSub + sub) * kSubCap;
        uint32_t* kc = kcnt + ((uint64_t)r * kSub + sub) * kCntStride;
        // The unit's count first, then its entries: into the unit's slots in
        // index order and, at a place reserved with one atomic, into the row's
        // key list.  Returns whether the unit's entries are to be written.
        auto reserve = [&](uint32_t nc, uint32_t* base) {
            uint32_t b = kSubCap;
            if (lane == 0) {
                ccnt[(uint64_t)r * U + u] = nc;
                if (nc > kSlots) {
                    atomicOr(&overflow[r], 1u);
                } else if (nc) {
                    b = atomicAdd(kc, nc);
                    if (b + nc > kSubCap) atomicOr(&overflow[r], 1u);
                }
            }
            *base = (uint32_t)__builtin_amdgcn_readfirstlane((int)b);
            return nc != 0u && nc <= kSlots && *base + nc <= kSubCap;
        };
        auto put = [&](uint32_t at, uint32_t base, uint64_t e, float v) {
            cu[at] = make_uint2((uint32_t)e, __float_as_uint(v));
            kl[base + at] = mag_key(v);
        };
        const bool rvec = res == nullptr || (reinterpret_cast<uintptr_t>(res) & 15u) == 0u;
        if ((reinterpret_cast<uintptr_t>(row) & 15u) == 0u && rvec && hi - lo == kUnit) {
            // the unit's 16 float4 per lane, all requested before use (loads
            // marked nontemporal: the row is streamed once); lane i holds
            // elements 4i..4i+3 of every 256, so entries are placed in index
            // order by a wave scan per 256 elements that hold any
            float4 vs[kUnit / 256];
    #pragma unroll
            for (uint32_t q = 0; q < kUnit / 256; ++q)
                vs[q] = load_nt(row + lo + 256u * q + 4u * lane);
            // in-bin flags of the lane's elements, bit k of nibble q for element
            // 256q + 4 lane + k (two words of eight nibbles: a handful of
            // registers instead of 64 lane masks)
            auto in4 = [&](const float4& v) {
                return (uint32_t)((mag_key(v.x) >> 20) >= bin) | (uint32_t)((mag_key(v.y) >> 20) >= bin) << 1 |
                       (uint32_t)((mag_key(v.z) >> 20) >= bin) << 2 | (uint32_t)((mag_key(v.w) >> 20) >= bin) << 3;
            };
            uint32_t fl[2] = {0u, 0u};
    #pragma unroll
            for (uint32_t q = 0; q < kUnit / 256; ++q) {
                fl[q / 8] |= in4(vs[q]) << (4 * (q % 8));
                if (res) store_nt(res + lo + 256u * q + 4u * lane, vs[q]);
            }
            const uint32_t mine = (uint32_t)__popc(fl[0]) + (uint32_t)__popc(fl[1]);
            const uint32_t nc = (uint32_t)__builtin_amdgcn_readlane((int)wave_scan(mine), 63);
            uint32_t base;
            if (reserve(nc, &base)) {
                uint32_t run = 0;
    #pragma unroll
                for (uint32_t q = 0; q < kUnit / 256; ++q) {
                    const uint32_t f = (fl[q / 8] >> (4 * (q % 8))) & 15u;
                    const uint32_t n4 = (uint32_t)__popc(f);
                    if (__ballot(n4 != 0u) == 0ull) continue;  // no entry in these 256 elements
                    const uint64_t e = lo + 256u * q + 4u * lane;
                    const uint32_t incl = wave_scan(n4);
                    uint32_t at = run + incl - n4;
                    if (f & 1u) put(at++, base, e, vs[q].x);
                    if (f & 2u) put(at++, base, e + 1, vs[q].y);
                    if (f & 4u) put(at++, base, e + 2, vs[q].z);
                    if (f & 8u) put(at, base, e + 3, vs[q].w);
                    run += (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
                }
            }
        } else {
            // short or unaligned unit: count (and copy), then read again to place
            uint32_t nc = 0;
            for (uint64_t e0 = lo; e0 < hi; e0 += 64) {
                const uint64_t e = e0 + lane;
                const float v = e < hi ? row[e] : 0.0f;
                nc += (uint32_t)__popcll(__ballot(e < hi && (mag_key(v) >> 20) >= bin));
                if (res && e < hi) res[e] = v;
            }
            uint32_t base;
            if (reserve(nc, &base)) {
                uint32_t run = 0;
                for (uint64_t e0 = lo; e0 < hi; e0 += 64) {
                    const uint64_t e = e0 + lane;
                    const float v = e < hi ? row[e] : 0.0f;
                    const bool in = e < hi && (mag_key(v) >> 20) >= bin;
                    const uint64_t m = __ballot(in);
                    if (in) put(run + (uint32_t)__popcll(m & ((1ull << lane) - 1ull)), base, e, v);
                    run += (uint32_t)__popcll(m);
                }
            }
        }
    }
}

// Bin (of NB, ordered from the top) holding the krem-th largest key of a
// histogram held one bin per thread (thread t: bin NB-1-t); returns the bin
// and, through *rem, krem less the keys in the bins above it.
__device__ uint32_t block_find(uint32_t cnt, uint64_t krem, uint32_t NB, uint64_t* rem, uint32_t* s_w,
                               uint32_t* s_res)
{
    uint32_t total;
    const uint32_t above = block_excl_scan(cnt, s_w, &total);
    if (above < krem && above + cnt >= krem) {
        s_res[0] = NB - 1u - threadIdx.x;
        s_res[1] = (uint32_t)(krem - above);
    }
    __syncthreads();
    *rem = s_res[1];
    return s_res[0];
}

// K* and the ties still needed, from the key list of row r (every key at or
// above its gather bin), for the rows on the path `exact` names.  After the
// sampled gather (exact = 0) a row that gathered fewer than k keys, or
// overflowed, is sent to the exact path instead; after the exact gather a row
// that overflowed is sent to the passes over its data.
__global__ void __launch_bounds__(1024) k_cand_select(uint64_t k, RankState* st, const uint32_t* klist,
                                                      uint32_t* kcnt, uint32_t* overflow, uint32_t exact)
{
    __shared__ uint32_t s_h[2048];
    __shared__ uint32_t s_w[16];
    __shared__ uint32_t s_res[2];
    const uint32_t r = blockIdx.x, t = threadIdx.x;
    if (st[r].exact != exact || st[r].full != 0u) return;  // row not on this path (whole workgroup)
    // keys gathered for the row (the sub-list counters) and the overflow flag
    uint32_t total;
    block_excl_scan(t < kSub ? kcnt[((uint64_t)r * kSub + t) * kCntStride] : 0u, s_w, &total);
    const bool ov = overflow[r] != 0u;
    if (exact == 0u && (ov || total < k)) {
        // the sampled bin failed: the exact one from a histogram of the row,
        // then a second gather
        if (t == 0) {
            st[r].exact = 1u;
            st[r].prefix = 0u;
            st[r].krem = k;
            overflow[r] = 0u;
        }
        if (t < kSub) kcnt[((uint64_t)r * kSub + t) * kCntStride] = 0u;
        return;
    }
    if (ov) {  // too many to gather even from the exact bin: passes over the data
        if (t == 0) st[r].full = 1u;
        return;
    }
    // every listed key: 16 threads per sub-list, four loads per thread in
    // flight: f(key)
    const uint32_t sub = t / 16u, j = t % 16u;
    const uint32_t* kl = klist + ((uint64_t)r * kSub + sub) * kSubCap;
    const uint32_t n = kcnt[((uint64_t)r * kSub + sub) * kCntStride];
    auto for_keys = [&](auto&& f) {
        for (uint32_t i0 = j; i0 < n; i0 += 64u) {
            uint32_t key[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) key[q] = i0 + 16u * q < n ? kl[i0 + 16u * q] : 0u;
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (i0 + 16u * q < n) f(key[q]);
        }
    };
    // The listed keys are every key at or above the gather bin, so the k-th
    // largest of them is the row's: its top 11 bits (2048 bins, two per
    // thread), then bits 19..10, then bits 9..0.
    uint64_t krem = k;
    s_h[t] = 0;
    s_h[t + 1024] = 0;
    __syncthreads();
    for_keys([&](uint32_t key) { atomicAdd(&s_h[key >> 20], 1u); });
    __syncthreads();
    uint32_t bin;
    {
        // thread t: bins 2047-2t and 2046-2t
        const uint32_t hb = s_h[2047u - 2u * t], lb = s_h[2046u - 2u * t];
        uint32_t total;
        const uint32_t above = block_excl_scan(hb + lb, s_w, &total);
        if (above < krem && above + hb >= krem) {
            s_res[0] = 2047u - 2u * t;
            s_res[1] = (uint32_t)(krem - above);
        } else if (above + hb < krem && above + hb + lb >= krem) {
            s_res[0] = 2046u - 2u * t;
            s_res[1] = (uint32_t)(krem - above - hb);
        }
        __syncthreads();
        bin = s_res[0];
        krem = s_res[1];
    }
    __syncthreads();
    s_h[t] = 0;
    __syncthreads();
    for_keys([&](uint32_t key) {
        if ((key >> 20) == bin) atomicAdd(&s_h[(key >> 10) & 1023u], 1u);
    });
    __syncthreads();
    const uint32_t b2 = block_find(s_h[1023u - t], krem, 1024u, &krem, s_w, s_res);
    const uint32_t p21 = bin << 10 | b2;
    __syncthreads();
    s_h[t] = 0;
    __syncthreads();
    for_keys([&](uint32_t key) {
        if ((key >> 10) == p21) atomicAdd(&s_h[key & 1023u], 1u);
    });
    __syncthreads();
    const uint32_t b3 = block_find(s_h[1023u - t], krem, 1024u, &krem, s_w, s_res);
    if (t == 0) {
        st[r].prefix = p21 << 10 | b3;
        st[r].krem = krem;
    }
}


// Per unit: entries with key > K* and key == K*.  A wave takes kUPW
// consecutive units: from the gathered entries on a settled row (all loads
// in flight together), from the data on a row refined over it.
constexpr uint32_t kUPW = 8;  // units per wave in the count and write kernels

__global__ void __launch_bounds__(256) k_count(const float* x, uint64_t N, uint32_t U, const RankState* st,
                                               const uint2* cand, const uint32_t* ccnt, uint32_t* cgt,
                                               uint32_t* ceq)
{
    const uint32_t r = blockIdx.y, lane = threadIdx.x & 63;
    const uint32_t u0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * kUPW;
    if (u0 >= U) return;
    const uint32_t K = st[r].prefix;
    if (st[r].full == 0u) {
        uint32_t n[kUPW], key[kUPW];
#pragma unroll
        for (uint32_t j = 0; j < kUPW; ++j) n[j] = u0 + j < U ? ccnt[(uint64_t)r * U + u0 + j] : 0u;
#pragma unroll
        for (uint32_t j = 0; j < kUPW; ++j)
            key[j] = lane < n[j] ? cand[((uint64_t)r * U + u0 + j) * kSlots + lane].y & 0x7FFFFFFFu : 0u;
#pragma unroll
        for (uint32_t j = 0; j < kUPW; ++j) {
            const uint32_t g = (uint32_t)__popcll(__ballot(lane < n[j] && key[j] > K));
            const uint32_t q = (uint32_t)__popcll(__ballot(lane < n[j] && key[j] == K));
            if (lane == 0 && u0 + j < U) {
                cgt[(uint64_t)r * U + u0 + j] = g;
                ceq[(uint64_t)r * U + u0 + j] = q;
            }
        }
        return;
    }
    const float* row = x + (uint64_t)r * N;
    for (uint32_t u = u0; u < min(u0 + kUPW, U); ++u) {
        const uint64_t lo = (uint64_t)u * kUnit, hi = min(lo + kUnit, N);
        uint32_t gt = 0, eq = 0;
        for (uint64_t e = lo + lane; e < hi; e += 64) {
            const uint32_t key = mag_key(row[e]);
            gt += key > K;
            eq += key == K;
        }
        for (int o = 32; o > 0; o >>= 1) {
            gt += __shfl_xor(gt, o);
            eq += __shfl_xor(eq, o);
        }
        if (lane == 0) {
            cgt[(uint64_t)r * U + u] = gt;
            ceq[(uint64_t)r * U + u] = eq;
        }
    }
}


// Unit offsets: equal keys are taken in index order until `need` of them.
__global__ void __launch_bounds__(1024) k_unit_scan(uint32_t U, const RankState* st, const uint32_t* cgt,
                                                    const uint32_t* ceq, uint32_t* beq, uint32_t* bout)
{
    __shared__ uint32_t s_w[16];
    const uint32_t r = blockIdx.x;
    const uint64_t need = st[r].krem;
    const uint32_t per = (U + 1023) / 1024;
    const uint32_t lo = min(threadIdx.x * per, U), hi = min(lo + per, U);
    const uint32_t* g = cgt + (uint64_t)r * U;
    const uint32_t* q = ceq + (uint64_t)r * U;
    // the first kScanPer of a thread's units read at once (all of them at the
    // common sizes), the rest in turn
    constexpr uint32_t kScanPer = 8;
    const uint32_t h8 = min(hi, lo + kScanPer);
    uint32_t gv[kScanPer], qv[kScanPer];
#pragma unroll
    for (uint32_t j = 0; j < kScanPer; ++j) {
        gv[j] = lo + j < h8 ? g[lo + j] : 0u;
        qv[j] = lo + j < h8 ? q[lo + j] : 0u;
    }
    uint32_t seq = 0;
#pragma unroll
    for (uint32_t j = 0; j < kScanPer; ++j) seq += qv[j];
    for (uint32_t i = h8; i < hi; ++i) seq += q[i];
    uint32_t tot;
    uint32_t run_eq = block_excl_scan(seq, s_w, &tot);
    // selections of a unit: its keys above K*, and its ties while needed
    auto take = [&](uint32_t re, uint32_t gi, uint32_t qi) {
        return gi + (re >= need ? 0u : (uint32_t)min<uint64_t>(need - re, qi));
    };
    uint32_t ssel = 0;
    {
        uint32_t re = run_eq;
#pragma unroll
        for (uint32_t j = 0; j < kScanPer; ++j) {
            ssel += take(re, gv[j], qv[j]);
            re += qv[j];
        }
        for (uint32_t i = h8; i < hi; ++i) {
            ssel += take(re, g[i], q[i]);
            re += q[i];
        }
    }
    uint32_t run_out = block_excl_scan(ssel, s_w, &tot);
#pragma unroll
    for (uint32_t j = 0; j < kScanPer; ++j) {
        if (lo + j < h8) {
            beq[(uint64_t)r * U + lo + j] = run_eq;
            bout[(uint64_t)r * U + lo + j] = run_out;
        }
        run_out += take(run_eq, gv[j], qv[j]);
        run_eq += qv[j];
    }
    for (uint32_t i = h8; i < hi; ++i) {
        beq[(uint64_t)r * U + i] = run_eq;
        bout[(uint64_t)r * U + i] = run_out;
        run_out += take(run_eq, g[i], q[i]);
        run_eq += q[i];
    }
}

// One unit of a row refined over its data: the selection compacted in index
// order from the data itself.
__device__ void write_unit(const float* x, uint64_t N, uint64_t k, uint32_t U, uint32_t r, uint32_t u,
                           const RankState* st, const uint32_t* beq, const uint32_t* bout, uint32_t* out_idx,
                           float* out_val, float* residual)
{
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t K = st[r].prefix;
    const uint64_t need = st[r].krem;
    const float* row = x + (uint64_t)r * N;
    float* res = residual ? residual + (uint64_t)r * N : nullptr;
    const bool inplace = res == row;
    uint32_t* oi = out_idx + (uint64_t)r * k;
    float* ov = out_val + (uint64_t)r * k;
    uint64_t eq_run = beq[(uint64_t)r * U + u];
    uint32_t out_run = bout[(uint64_t)r * U + u];
    const uint64_t lo = (uint64_t)u * kUnit, hi = min(lo + kUnit, N);
    const uint64_t lt = (1ull << lane) - 1ull;
    const bool res_vec = res == nullptr || inplace || (reinterpret_cast<uintptr_t>(res) & 15u) == 0u;
    if ((reinterpret_cast<uintptr_t>(row) & 15u) == 0u && res_vec && hi - lo == kUnit) {
        // The unit's 16 float4 per lane, all requested before use; per 256
        // elements (lane i: elements 4i..4i+3) ties and selections are placed
        // in index order by wave scans of the per-lane counts.
        float4 vs[kUnit / 256];
#pragma unroll
        for (uint32_t q = 0; q < kUnit / 256; ++q)
            vs[q] = *reinterpret_cast<const float4*>(row + lo + 256u * q + 4u * lane);
#pragma unroll
        for (uint32_t q = 0; q < kUnit / 256; ++q) {
            const uint64_t e = lo + 256u * q + 4u * lane;
            const float v4[4] = {vs[q].x, vs[q].y, vs[q].z, vs[q].w};
            uint32_t neq = 0;
            bool isq[4], gt[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t key = mag_key(v4[i]);
                isq[i] = key == K;
                gt[i] = key > K;
                neq += isq[i] ? 1u : 0u;
            }
            const uint32_t eincl = wave_scan(neq);
            uint64_t eb = eq_run + (eincl - neq);  // ties before this lane's first
            bool sel[4];
            uint32_t nsel = 0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                sel[i] = gt[i] || (isq[i] && eb < need);
                eb += isq[i] ? 1u : 0u;
                nsel += sel[i] ? 1u : 0u;
            }
            const uint32_t sincl = wave_scan(nsel);
            uint32_t o = out_run + (sincl - nsel);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (sel[i]) {
                    oi[o] = (uint32_t)(e + i);
                    ov[o] = v4[i];
                    ++o;
                }
            }
            if (res) {
                if (inplace) {
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        if (sel[i]) res[e + i] = 0.0f;
                } else {
                    *reinterpret_cast<float4*>(res + e) =
                        make_float4(sel[0] ? 0.0f : v4[0], sel[1] ? 0.0f : v4[1], sel[2] ? 0.0f : v4[2],
                                    sel[3] ? 0.0f : v4[3]);
                }
            }
            eq_run += (uint32_t)__builtin_amdgcn_readlane((int)eincl, 63);
            out_run += (uint32_t)__builtin_amdgcn_readlane((int)sincl, 63);
        }
        return;
    }
    for (uint64_t e0 = lo; e0 < hi; e0 += 64) {
        const uint64_t e = e0 + lane;
        const bool valid = e < hi;
        const float v = valid ? row[e] : 0.0f;
        const uint32_t key = mag_key(v);
        const bool eq = valid && key == K;
        const uint64_t beq_w = __ballot(eq);
        const bool take_eq = eq && (eq_run + (uint64_t)__popcll(beq_w & lt)) < need;
        const bool sel = (valid && key > K) || take_eq;
        const uint64_t bsel = __ballot(sel);
        if (sel) {
            const uint32_t o = out_run + (uint32_t)__popcll(bsel & lt);
            oi[o] = (uint32_t)e;
            ov[o] = v;
        }
        if (res && valid) {
            if (inplace) {
                if (sel) res[e] = 0.0f;
            } else {
                res[e] = sel ? 0.0f : v;
            }
        }
        eq_run += (uint64_t)__popcll(beq_w);
        out_run += (uint32_t)__popcll(bsel);
    }
}

// Per kUPW units of a wave: a row settled by its gathered entries writes
// its selection from them (a unit's entries in index order, one per lane):
// key > K*, or key == K* while ties are still needed, at the unit's offset,
// zeroing the residual there; a row refined over its data compacts it.
__global__ void __launch_bounds__(256) k_write(const float* x, uint64_t N, uint64_t k, uint32_t U,
                                               const RankState* st, const uint2* cand, const uint32_t* ccnt,
                                               const uint32_t* beq, const uint32_t* bout, uint32_t* out_idx,
                                               float* out_val, float* residual)
{
    const uint32_t r = blockIdx.y, lane = threadIdx.x & 63;
    const uint32_t u0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * kUPW;
    if (u0 >= U) return;
    if (st[r].full != 0u) {
        for (uint32_t u = u0; u < min(u0 + kUPW, U); ++u)
            write_unit(x, N, k, U, r, u, st, beq, bout, out_idx, out_val, residual);
        return;
    }
    const uint32_t K = st[r].prefix;
    const uint64_t need = st[r].krem;
    const uint64_t lt = (1ull << lane) - 1ull;
    uint32_t n[kUPW], eqb[kUPW], ob[kUPW];
    uint2 c[kUPW];
#pragma unroll
    for (uint32_t j = 0; j < kUPW; ++j) {
        const bool in = u0 + j < U;
        n[j] = in ? ccnt[(uint64_t)r * U + u0 + j] : 0u;  // <= kSlots on a settled row
        eqb[j] = in ? beq[(uint64_t)r * U + u0 + j] : 0u;
        ob[j] = in ? bout[(uint64_t)r * U + u0 + j] : 0u;
    }
#pragma unroll
    for (uint32_t j = 0; j < kUPW; ++j)
        c[j] = lane < n[j] ? cand[((uint64_t)r * U + u0 + j) * kSlots + lane] : make_uint2(0u, 0u);
#pragma unroll
    for (uint32_t j = 0; j < kUPW; ++j) {
        const uint32_t key = c[j].y & 0x7FFFFFFFu;
        const bool eq = lane < n[j] && key == K;
        const uint64_t beq_w = __ballot(eq);
        const bool sel = (lane < n[j] && key > K) || (eq && (uint64_t)eqb[j] + (uint64_t)__popcll(beq_w & lt) < need);
        const uint64_t bsel = __ballot(sel);
        if (sel) {
            const uint64_t o = (uint64_t)r * k + ob[j] + (uint32_t)__popcll(bsel & lt);
            out_idx[o] = c[j].x;
            out_val[o] = __uint_as_float(c[j].y);
            if (residual) residual[(uint64_t)r * N + c[j].x] = 0.0f;
        }
    }
}

struct TLayout {
    RankState* st;
    uint32_t *hist, *cgt, *ceq, *beq, *bout, *ccnt, *overflow, *klist, *kcnt;
    uint2* cand;
    uint32_t U;
    size_t bytes;
};

TLayout tlayout(int P, uint64_t N, void* ws)
{
    Carve c(ws);
    TLayout l{};
    l.U = (uint32_t)((N + kUnit - 1) / kUnit);
    l.st = c.take<RankState>(P);
    l.overflow = c.take<uint32_t>(P);
    l.kcnt = c.take<uint32_t>((size_t)P * kSub * kCntStride);
    l.klist = c.take<uint32_t>((size_t)P * kList);
    l.ccnt = c.take<uint32_t>((size_t)P * l.U);
    l.cand = c.take<uint2>((size_t)P * l.U * kSlots);
    l.hist = c.take<uint32_t>((size_t)P * 2048);
    l.cgt = c.take<uint32_t>((size_t)P * l.U);
    l.ceq = c.take<uint32_t>((size_t)P * l.U);
    l.beq = c.take<uint32_t>((size_t)P * l.U);
    l.bout = c.take<uint32_t>((size_t)P * l.U);
    l.bytes = align_up(c.used, 256);
    return l;
}

}  // namespace

size_t topk_workspace(int P, uint64_t N, uint64_t /*k*/) { return tlayout(P, N, nullptr).bytes; }

hipError_t topk_run(int P, const float* x, uint64_t N, uint64_t k, uint32_t* out_idx,
                    float* out_val, float* residual, void* ws, hipStream_t s)
{
    if (k == 0) {
        if (residual && residual != x)
            return hipMemcpyAsync(residual, x, (size_t)P * N * sizeof(float), hipMemcpyDeviceToDevice, s);
        return hipSuccess;
    }
    const TLayout l = tlayout(P, N, ws);
    // expected selections per unit decide where a row starts
    const double per_unit = (double)k * kUnit / (double)N;
    const uint32_t mode = per_unit > kSlots ? 2u : (per_unit > kSlots / 4 ? 1u : 0u);
    const uint64_t ninit = (uint64_t)P * 2048;  // covers P * kSub counters too
    hipLaunchKernelGGL(k_init, dim3((uint32_t)((ninit + 255) / 256)), dim3(256), 0, s, l.st,
                       (uint32_t)P, k, l.hist, l.overflow, mode, l.kcnt);
    const uint32_t hb = (uint32_t)std::min<uint64_t>(kHistBlocksPerRank, (N + 4095) / 4096);
    const dim3 hgrid(hb, P), ugrid((l.U + 3) / 4, P);
    // sample: every stride-th 256-element segment, about kSampleSegs of them
    const uint64_t nseg = (N + 255) / 256;
    const uint64_t stride = std::max<uint64_t>(1, nseg / kSampleSegs);
    uint64_t sampled = 0;
    for (uint64_t g = 0; g < nseg; g += stride) sampled += std::min<uint64_t>(256, N - g * 256);
    const double frac = (double)sampled / (double)N;
    const uint32_t sb = (uint32_t)std::min<uint64_t>(64, (nseg + stride - 1) / stride);
    timer_begin(kTTopkSelect, s);
    if (mode == 0) {
        hipLaunchKernelGGL(k_sample, dim3(sb, P), dim3(256), 0, s, x, N, (uint32_t)stride, l.hist);
        hipLaunchKernelGGL(k_estimate, dim3(P), dim3(256), 0, s, l.st, l.hist, k, frac);
        hipLaunchKernelGGL(k_gather, ugrid, dim3(256), 0, s, x, N, l.U, l.st, l.cand, l.ccnt, l.overflow,
                           residual, 0u, l.klist, l.kcnt);
        // settles the rows whose sampled bin held; the others go exact
        hipLaunchKernelGGL(k_cand_select, dim3(P), dim3(1024), 0, s, k, l.st, l.klist, l.kcnt, l.overflow, 0u);
    }
    // rows on the exact path: the exact boundary bin, a gather from it
    hipLaunchKernelGGL(k_hist<0>, hgrid, dim3(256), 0, s, x, N, l.st, l.hist);
    hipLaunchKernelGGL(k_select<0>, dim3(P), dim3(256), 0, s, l.st, l.hist);
    const dim3 xgrid(std::min<uint32_t>((l.U + 3) / 4, kExactGatherBlocks), P);
    hipLaunchKernelGGL(k_gather, xgrid, dim3(256), 0, s, x, N, l.U, l.st, l.cand, l.ccnt, l.overflow,
                       residual, 1u, l.klist, l.kcnt);
    hipLaunchKernelGGL(k_cand_select, dim3(P), dim3(1024), 0, s, k, l.st, l.klist, l.kcnt, l.overflow, 1u);
    // rows whose boundary bin overflowed the gather buffer (the others return at once)
    hipLaunchKernelGGL(k_hist<1>, hgrid, dim3(256), 0, s, x, N, l.st, l.hist);
    hipLaunchKernelGGL(k_select<1>, dim3(P), dim3(256), 0, s, l.st, l.hist);
    hipLaunchKernelGGL(k_hist<2>, hgrid, dim3(256), 0, s, x, N, l.st, l.hist);
    hipLaunchKernelGGL(k_select<2>, dim3(P), dim3(256), 0, s, l.st, l.hist);
    timer_end(kTTopkSelect, s);
    timer_begin(kTTopkWrite, s);
    const dim3 wgrid((l.U + 4 * kUPW - 1) / (4 * kUPW), P);
    hipLaunchKernelGGL(k_count, wgrid, dim3(256), 0, s, x, N, l.U, l.st, l.cand, l.ccnt, l.cgt, l.ceq);
    hipLaunchKernelGGL(k_unit_scan, dim3(P), dim3(1024), 0, s, l.U, l.st, l.cgt, l.ceq, l.beq, l.bout);
    hipLaunchKernelGGL(k_write, wgrid, dim3(256), 0, s, x, N, k, l.U, l.st, l.cand, l.ccnt, l.beq, l.bout,
                       out_idx, out_val, residual);
    timer_end(kTTopkWrite, s);
    return hipGetLastError();
}

}  // namespace sparcml
