// Bucketed top-k with error feedback on gfx950 (§8.4: every group of B
// consecutive coordinates sends its kb largest entries and keeps the rest;
// Alg. 1: acc = eps + alpha * grad, eps = acc - TopK(acc)).
//
// One wave per bucket, B = 64 * EPT: each lane holds EPT coordinates, 4
// consecutive ones in each 256-coordinate group, so that every wave-wide
// load or store is one contiguous kilobyte.  Selection is kb rounds of a wave-wide maximum
// over 64-bit keys (|acc| bits above the complemented index: the largest
// magnitude wins, the lowest index on ties); each lane then writes its
// selected entries at its prefix count in LDS, which lists the bucket's
// entries in ascending index order, and kb lanes store them at once.  The
// kernel is HBM-bound: acc is formed, selected and written back in
// registers (grad and eps read once, eps written once; the loads and the
// store of eps are marked nontemporal, which measured markedly faster).
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
    // Lane l holds G = min(EPT, 4) consecutive coordinates in each of NG
    // groups: coordinate u * 64G + l * G + k, so every wave-wide access of a
    // group is one contiguous run of 64G floats (whole cache lines).
    constexpr int G = EPT < 4 ? EPT : 4;
    constexpr int NG = EPT / G;
    constexpr uint32_t B = 64u * EPT;
    const uint32_t lane = threadIdx.x & 63u;
    const uint32_t wv = threadIdx.x >> 6;
    const uint32_t q = blockIdx.x * 4u + wv;  // bucket
    if (q >= nb) return;                      // whole wave
    const uint32_t r = blockIdx.y;
    const uint32_t j0 = q * B;
    const uint32_t len = min(B, N - j0);
    float* e = eps + (uint64_t)r * N + j0;
    const float* g = grad ? grad + (uint64_t)r * N + j0 : nullptr;
    const bool vec = G == 4 && len == B &&
                     ((reinterpret_cast<uintptr_t>(e) | (g ? reinterpret_cast<uintptr_t>(g) : 0u)) & 15u) == 0;

    float acc[EPT];  // acc[u * G + k]: coordinate u * 64G + lane * G + k
    if (vec) {
#pragma unroll
        for (int u = 0; u < NG; ++u) {
            const uint32_t c = u * 256u + lane * 4u;
            float4 v = load_nt(e + c);
            if (g) {
                const float4 w = load_nt(g + c);
                v.x = __fadd_rn(v.x, __fmul_rn(alpha, w.x));
                v.y = __fadd_rn(v.y, __fmul_rn(alpha, w.y));
                v.z = __fadd_rn(v.z, __fmul_rn(alpha, w.z));
                v.w = __fadd_rn(v.w, __fmul_rn(alpha, w.w));
            }
            acc[u * 4] = v.x;
            acc[u * 4 + 1] = v.y;
            acc[u * 4 + 2] = v.z;
            acc[u * 4 + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            const uint32_t c = (i / G) * 64u * G + lane * G + (i % G);
            float v = 0.0f;
            if (c < len) {
                v = e[c];
                if (g) v = __fadd_rn(v, __fmul_rn(alpha, g[c]));
            }
            acc[i] = v;
        }
    }

    // key: |acc| bits (sign cleared) above the complemented row index;
    // 0 marks a coordinate past the row's end or one already taken
    uint64_t key[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const uint32_t c = (i / G) * 64u * G + lane * G + (i % G);
        key[i] = c < len ? ((uint64_t)(__float_as_uint(acc[i]) & 0x7FFFFFFFu) << 32) | (0xFFFFFFFFu - (j0 + c))
                         : 0ull;
    }
    uint64_t taken = 0;  // bit i: acc[i] selected
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

    // Selected entries in ascending index order (group, then lane, then k):
    // each lane stages its own in the wave's LDS row at the count of
    // selected entries before them, then lanes 0..take-1 write the bucket's
    // output (offset q * kb: every bucket before the last contributes kb)
    // with one coalesced store per array.
    __shared__ uint32_t s_i[4][64];
    __shared__ float s_v[4][64];
    uint32_t before = 0;  // selected entries of earlier groups
#pragma unroll
    for (int u = 0; u < NG; ++u) {
        const uint32_t bits = (uint32_t)((taken >> (u * G)) & ((1u << G) - 1u));
        const uint32_t cnt = (uint32_t)__popc(bits);
        const uint32_t incl = wave_scan(cnt);
        uint32_t pos = before + incl - cnt;
#pragma unroll
        for (int k = 0; k < G; ++k) {
            if ((bits >> k) & 1u) {
                s_i[wv][pos] = j0 + u * 64u * G + lane * G + k;
                s_v[wv][pos] = acc[u * G + k];
                ++pos;
                acc[u * G + k] = 0.0f;  // eps = acc - TopK(acc)
            }
        }
        before += (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane < take) {
        const uint64_t o = (uint64_t)r * K + (uint64_t)q * kb + lane;
        out_idx[o] = s_i[wv][lane];
        out_val[o] = s_v[wv][lane];
    }
    if (vec) {
#pragma unroll
        for (int u = 0; u < NG; ++u)
            store_nt(e + u * 256u + lane * 4u, make_float4(acc[u * 4], acc[u * 4 + 1], acc[u * 4 + 2], acc[u * 4 + 3]));
    } else {
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            const uint32_t c = (i / G) * 64u * G + lane * G + (i % G);
            if (c < len) e[c] = acc[i];
        }
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
