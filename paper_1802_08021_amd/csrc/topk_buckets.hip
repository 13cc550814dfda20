// Bucketed top-k with error feedback on gfx950 (§8.4: every group of B
// consecutive coordinates sends its kb largest entries and keeps the rest;
// Alg. 1: acc = eps + alpha * grad, eps = acc - TopK(acc)).
//
// One wave per bucket, B = 64 * EPT: lane l holds the EPT consecutive
// coordinates at l * EPT, so a wave reads and writes its bucket with
// coalesced 16-byte accesses.  Selection is kb rounds of a wave-wide maximum
// over 64-bit keys (|acc| bits above the complemented index: the largest
// magnitude wins, the lowest index on ties); each lane then writes its
// selected entries at its prefix count, which lists the bucket's entries in
// ascending index order.  The kernel is HBM-bound: acc is formed, selected
// and written back in registers (grad and eps read once, eps written once).
#include "internal.h"

#include <algorithm>

namespace sparcml {
namespace {

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v)
{
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint64_t w = __shfl_xor(v, o);
        v = w > v ? w : v;
    }
    return v;
}

template <int EPT>
__global__ void __launch_bounds__(256) k_topk_buckets(const float* grad, float* eps, uint32_t N, float alpha,
                                                      uint32_t nb, uint32_t kb, uint64_t K, uint32_t* out_idx,
                                                      float* out_val)
{
    constexpr uint32_t B = 64u * EPT;
    const uint32_t lane = threadIdx.x & 63u;
    const uint32_t q = blockIdx.x * 4u + (threadIdx.x >> 6);  // bucket
    if (q >= nb) return;                                    // whole wave
    const uint32_t r = blockIdx.y;
    const uint32_t j0 = q * B;
    const uint32_t len = min(B, N - j0);
    float* e = eps + (uint64_t)r * N + j0;
    const float* g = grad ? grad + (uint64_t)r * N + j0 : nullptr;
    const uint32_t c0 = lane * EPT;  // this lane's first coordinate in the bucket
    const bool vec = EPT >= 4 && len == B &&
                     ((reinterpret_cast<uintptr_t>(e) | (g ? reinterpret_cast<uintptr_t>(g) : 0u)) & 15u) == 0;

    float acc[EPT];
    if (vec) {
#pragma unroll
        for (int i = 0; i < EPT; i += 4) {
            float4 a = *reinterpret_cast<const float4*>(e + c0 + i);
            if (g) {
                const float4 b = *reinterpret_cast<const float4*>(g + c0 + i);
                a.x = __fadd_rn(a.x, __fmul_rn(alpha, b.x));
                a.y = __fadd_rn(a.y, __fmul_rn(alpha, b.y));
                a.z = __fadd_rn(a.z, __fmul_rn(alpha, b.z));
                a.w = __fadd_rn(a.w, __fmul_rn(alpha, b.w));
            }
            acc[i] = a.x;
            acc[i + 1] = a.y;
            acc[i + 2] = a.z;
            acc[i + 3] = a.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            const uint32_t c = c0 + i;
            float a = 0.0f;
            if (c < len) {
                a = e[c];
                if (g) a = __fadd_rn(a, __fmul_rn(alpha, g[c]));
            }
            acc[i] = a;
        }
    }

    // key: |acc| bits (sign cleared) above the complemented row index;
    // 0 marks a coordinate past the row's end or one already taken
    uint64_t key[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const uint32_t c = c0 + i;
        key[i] = c < len ? ((uint64_t)(__float_as_uint(acc[i]) & 0x7FFFFFFFu) << 32) | (0xFFFFFFFFu - (j0 + c))
                         : 0ull;
    }
    uint64_t taken = 0;  // bit i: coordinate c0 + i selected
    const uint32_t take = min(kb, len);
    for (uint32_t t = 0; t < take; ++t) {
        uint64_t best = 0;
#pragma unroll
        for (int i = 0; i < EPT; ++i) best = key[i] > best ? key[i] : best;
        const uint64_t top = wave_max_u64(best);
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            if (key[i] == top) {
                key[i] = 0;
                taken |= 1ull << i;
            }
        }
    }

    // selected entries in ascending index order at the bucket's output
    // offset (every bucket before the last one contributes kb)
    const uint32_t cnt = (uint32_t)__popcll(taken);
    const uint32_t excl = wave_scan(cnt) - cnt;
    uint64_t o = (uint64_t)r * K + (uint64_t)q * kb + excl;
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        if ((taken >> i) & 1ull) {
            out_idx[o] = j0 + c0 + i;
            out_val[o] = acc[i];
            ++o;
            acc[i] = 0.0f;  // eps = acc - TopK(acc)
        }
    }
    if (vec) {
#pragma unroll
        for (int i = 0; i < EPT; i += 4) store_nt(e + c0 + i, make_float4(acc[i], acc[i + 1], acc[i + 2], acc[i + 3]));
    } else {
#pragma unroll
        for (int i = 0; i < EPT; ++i)
            if (c0 + i < len) e[c0 + i] = acc[i];
    }
}

}  // namespace

uint64_t topk_buckets_count(uint64_t N, uint64_t bucket, uint64_t kb)
{
    const uint64_t nb = (N + bucket - 1) / bucket;
    const uint64_t last = N - (nb - 1) * bucket;
    return (nb - 1) * kb + std::min(last, kb);
}

hipError_t topk_buckets_run(int P, const float* grad, float* eps, uint64_t N, float alpha, uint32_t bucket,
                            uint32_t kb, uint32_t* out_idx, float* out_val, hipStream_t s)
{
    const uint32_t nb = (uint32_t)((N + bucket - 1) / bucket);
    const uint64_t K = topk_buckets_count(N, bucket, kb);
    const dim3 grid((nb + 3) / 4, P);
    timer_begin(kTTopkBuckets, s);
    switch (bucket) {
#define SPARCML_TB(E)                                                                                    \
    case 64u * E:                                                                                        \
        hipLaunchKernelGGL(k_topk_buckets<E>, grid, dim3(256), 0, s, grad, eps, (uint32_t)N, alpha, nb, kb, K, \
                           out_idx, out_val);                                                            \
        break;
        SPARCML_TB(1)
        SPARCML_TB(2)
        SPARCML_TB(4)
        SPARCML_TB(8)
        SPARCML_TB(16)
        SPARCML_TB(32)
        SPARCML_TB(64)
#undef SPARCML_TB
    default: return hipErrorInvalidValue;
    }
    timer_end(kTTopkBuckets, s);
    return hipGetLastError();
}

}  // namespace sparcml
