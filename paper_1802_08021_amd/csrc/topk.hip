// Top-k sparsification by magnitude on gfx950 (§2.2 "Structured
// Sparsification"; Alg. 1: TopK and the error update eps = acc - TopK(acc)).
//
// Exact radix select on the 31-bit magnitude key (IEEE bits, sign cleared):
// three histogram passes (11 + 10 + 10 bits) narrow the k-th largest key K*
// and how many entries equal to K* are still needed; a count pass and a scan
// over 4096-element wave units then give every unit its output offset, and a
// write pass compacts the selection in index order (equal keys: lowest index
// first) with wave ballots, optionally zeroing the residual.
#include "internal.h"

#include <algorithm>

namespace sparcml {
namespace {

constexpr uint32_t kUnit = 4096;  // elements per wave unit (64 iterations of 64 lanes)
constexpr int kHistBlocksPerRank = 64;

struct RankState {
    uint32_t prefix;  // key bits fixed so far
    uint32_t pad;
    uint64_t krem;    // entries still to take from keys matching the prefix
};

__device__ __forceinline__ uint32_t mag_key(float v) { return __float_as_uint(v) & 0x7FFFFFFFu; }

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
    for (uint32_t i = threadIdx.x; i < NB; i += 256) s_h[i] = 0;
    __syncthreads();
    const uint32_t prefix = PASS == 0 ? 0u : st[r].prefix;
    const float* row = x + (uint64_t)r * N;
    const uint64_t per = (N + gridDim.x - 1) / gridDim.x;
    const uint64_t lo = (uint64_t)blockIdx.x * per, hi = min(lo + per, N);
    for (uint64_t e = lo + threadIdx.x; e < hi; e += 256) {
        const uint32_t key = mag_key(row[e]);
        if (PASS == 0 || (key >> PSHIFT) == prefix) atomicAdd(&s_h[(key >> SHIFT) & (NB - 1)], 1u);
    }
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

__global__ void k_init(RankState* st, uint32_t P, uint64_t k, uint32_t* hist)
{
    const uint64_t gid = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid < P) {
        st[gid].prefix = 0;
        st[gid].krem = k;
    }
    if (gid < (uint64_t)P * 2048) hist[gid] = 0;
}

// Per wave unit: entries with key > K* and key == K*.
__global__ void __launch_bounds__(256) k_count(const float* x, uint64_t N, uint32_t U,
                                               const RankState* st, uint32_t* cgt, uint32_t* ceq)
{
    const uint32_t r = blockIdx.y, lane = threadIdx.x & 63;
    const uint32_t u = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (u >= U) return;
    const uint32_t K = st[r].prefix;
    const float* row = x + (uint64_t)r * N;
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
    uint32_t seq = 0;
    for (uint32_t i = lo; i < hi; ++i) seq += q[i];
    uint32_t tot;
    uint32_t run_eq = block_excl_scan(seq, s_w, &tot);
    uint32_t ssel = 0;
    {
        uint32_t re = run_eq;
        for (uint32_t i = lo; i < hi; ++i) {
            const uint64_t take = re >= need ? 0 : min<uint64_t>(need - re, q[i]);
            ssel += g[i] + (uint32_t)take;
            re += q[i];
        }
    }
    uint32_t run_out = block_excl_scan(ssel, s_w, &tot);
    for (uint32_t i = lo; i < hi; ++i) {
        beq[(uint64_t)r * U + i] = run_eq;
        bout[(uint64_t)r * U + i] = run_out;
        const uint64_t take = run_eq >= need ? 0 : min<uint64_t>(need - run_eq, q[i]);
        run_out += g[i] + (uint32_t)take;
        run_eq += q[i];
    }
}

__global__ void __launch_bounds__(256) k_write(const float* x, uint64_t N, uint64_t k, uint32_t U,
                                               const RankState* st, const uint32_t* beq,
                                               const uint32_t* bout, uint32_t* out_idx, float* out_val,
                                               float* residual)
{
    const uint32_t r = blockIdx.y, lane = threadIdx.x & 63;
    const uint32_t u = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (u >= U) return;
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

struct TLayout {
    RankState* st;
    uint32_t *hist, *cgt, *ceq, *beq, *bout;
    uint32_t U;
    size_t bytes;
};

TLayout tlayout(int P, uint64_t N, void* ws)
{
    Carve c(ws);
    TLayout l{};
    l.U = (uint32_t)((N + kUnit - 1) / kUnit);
    l.st = c.take<RankState>(P);
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
    const uint64_t ninit = (uint64_t)P * 2048;
    hipLaunchKernelGGL(k_init, dim3((uint32_t)((ninit + 255) / 256)), dim3(256), 0, s, l.st,
                       (uint32_t)P, k, l.hist);
    const uint32_t hb = (uint32_t)std::min<uint64_t>(kHistBlocksPerRank, (N + 4095) / 4096);
    const dim3 hgrid(hb, P);
    timer_begin(kTTopkSelect, s);
    hipLaunchKernelGGL(k_hist<0>, hgrid, dim3(256), 0, s, x, N, l.st, l.hist);
    hipLaunchKernelGGL(k_select<0>, dim3(P), dim3(256), 0, s, l.st, l.hist);
    hipLaunchKernelGGL(k_hist<1>, hgrid, dim3(256), 0, s, x, N, l.st, l.hist);
    hipLaunchKernelGGL(k_select<1>, dim3(P), dim3(256), 0, s, l.st, l.hist);
    hipLaunchKernelGGL(k_hist<2>, hgrid, dim3(256), 0, s, x, N, l.st, l.hist);
    hipLaunchKernelGGL(k_select<2>, dim3(P), dim3(256), 0, s, l.st, l.hist);
    timer_end(kTTopkSelect, s);
    timer_begin(kTTopkWrite, s);
    const dim3 ugrid((l.U + 3) / 4, P);
    hipLaunchKernelGGL(k_count, ugrid, dim3(256), 0, s, x, N, l.U, l.st, l.cgt, l.ceq);
    hipLaunchKernelGGL(k_unit_scan, dim3(P), dim3(1024), 0, s, l.U, l.st, l.cgt, l.ceq, l.beq, l.bout);
    hipLaunchKernelGGL(k_write, ugrid, dim3(256), 0, s, x, N, k, l.U, l.st, l.beq, l.bout, out_idx,
                       out_val, residual);
    timer_end(kTTopkWrite, s);
    return hipGetLastError();
}

}  // namespace sparcml
