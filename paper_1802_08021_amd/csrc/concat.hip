// Sum of P vectors whose index ranges are disjoint -- the gathered shares
// of the split-allgather allreduce (§5.3.2) -- which is their concatenation
// (§5.1, case (2)).  Part s covers [lo_s, lo_s + len_s); it is sparse
// (absolute indices) or dense (len_s values), with fp32 values or QSGD codes
// (one scale, or one per bucket of B entries, §6) dequantized on the fly.
//
// Sparse result: every part's entries are copied to its offset in the
// output (prefix of the parts' counts): a (chunk, part) grid of 4096-entry
// chunks, coalesced grid-stride copies.  Dense result: a (tile, part) grid over 4096-index
// tiles of each part's range; a dense part's tile is copied (or decoded)
// straight through, a sparse part's tile is scattered into LDS (zeros
// elsewhere) and written with coalesced stores.  Both are HBM-bound: every
// input byte is read once and every output byte written once.
#include "internal.h"
#include "qsgd_device.h"

#include <algorithm>
#include <vector>

namespace sparcml {
namespace {

constexpr uint32_t kTile = 4096;
constexpr uint32_t kChunk = 4096;  // sparse entries per workgroup (256 threads x 16)

struct CDesc {
    const uint32_t* idx;
    const float* val;
    const uint8_t* qval;
    const float* qscale;
    uint64_t nnz;  // stored entries (len for a dense part)
    uint64_t lo;   // first index of the part's range
    uint64_t len;  // range length
    uint64_t off;  // sparse result: first output position
    uint32_t dense;
    uint32_t pad;
};

// Value of stored entry i of a part.
__device__ __forceinline__ float entry(const CDesc& d, uint64_t i, uint32_t qbits, uint32_t bshift)
{
    if (!qbits) return d.val[i];
    const float unit = level_unit(d.qscale[bshift < 64u ? (i >> bshift) : 0], qbits);
    return dequant(load_code(d.qval, i, qbits), qbits, unit);
}

__device__ __forceinline__ uint64_t lower_bound_idx(const uint32_t* a, uint64_t lo, uint64_t hi, uint64_t x)
{
    while (lo < hi) {
        const uint64_t mid = lo + ((hi - lo) >> 1);
        if ((uint64_t)a[mid] < x) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

__global__ void __launch_bounds__(256) k_concat_sparse(const CDesc* tab, uint32_t qbits, uint32_t bshift,
                                                       uint32_t* out_idx, float* out_val)
{
    const CDesc d = tab[blockIdx.y];
    const uint64_t c0 = (uint64_t)blockIdx.x * kChunk;
    if (c0 >= d.nnz) return;
    const uint64_t c1 = min(c0 + kChunk, d.nnz);
    for (uint64_t i = c0 + threadIdx.x; i < c1; i += 256) {
        out_idx[d.off + i] = d.idx[i];
        out_val[d.off + i] = entry(d, i, qbits, bshift);
    }
}

__global__ void __launch_bounds__(256) k_concat_dense(const CDesc* tab, uint32_t qbits, uint32_t bshift,
                                                      float* out)
{
    __shared__ float s_tile[kTile];
    __shared__ uint64_t s_rng[2];
    const CDesc d = tab[blockIdx.y];
    const uint64_t t0 = (uint64_t)blockIdx.x * kTile;  // tile start within the part
    if (t0 >= d.len) return;                           // uniform over the block
    const uint32_t w = (uint32_t)min((uint64_t)kTile, d.len - t0);
    float* o = out + d.lo + t0;
    if (d.dense) {
        // 4 consecutive values per thread and step
        const bool vec = !qbits && ((reinterpret_cast<uintptr_t>(o) | reinterpret_cast<uintptr_t>(d.val + t0)) & 15u) == 0;
        for (uint32_t j = threadIdx.x * 4; j < w; j += 1024) {
            if (vec && j + 4 <= w) {
                *reinterpret_cast<float4*>(o + j) = *reinterpret_cast<const float4*>(d.val + t0 + j);
            } else {
                for (uint32_t q = 0; q < 4 && j + q < w; ++q) o[j + q] = entry(d, t0 + j + q, qbits, bshift);
            }
        }
        return;
    }
    for (uint32_t j = threadIdx.x; j < kTile; j += 256) s_tile[j] = 0.0f;
    if (threadIdx.x < 2)
        s_rng[threadIdx.x] = lower_bound_idx(d.idx, 0, d.nnz, d.lo + t0 + (threadIdx.x ? w : 0u));
    __syncthreads();
    for (uint64_t i = s_rng[0] + threadIdx.x; i < s_rng[1]; i += 256) {
        const uint64_t j = (uint64_t)d.idx[i] - (d.lo + t0);
        if (j < kTile) s_tile[j] = entry(d, i, qbits, bshift);
    }
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < w; j += 256) o[j] = s_tile[j];
}

}  // namespace

size_t concat_workspace(int P) { return align_up(sizeof(CDesc) * (size_t)P, 256); }

hipError_t concat_run(int P, const ConcatPart* parts, uint32_t qbits, uint64_t bucket, int dense,
                      uint32_t* out_idx, float* out_val, void* ws, hipStream_t s)
{
    std::vector<CDesc> host(P);
    uint64_t off = 0, max_nnz = 0, max_len = 0;
    for (int p = 0; p < P; ++p) {
        const ConcatPart& c = parts[p];
        host[p] = CDesc{c.idx, c.val, c.qval, c.qscale, c.nnz, c.lo, c.len, off, c.dense ? 1u : 0u, 0u};
        off += c.nnz;
        max_nnz = std::max(max_nnz, c.nnz);
        max_len = std::max(max_len, c.len);
    }
    CDesc* tab = static_cast<CDesc*>(ws);
    hipError_t e = upload(tab, host.data(), sizeof(CDesc) * P, s);
    if (e != hipSuccess) return e;
    // bucket (a power of two) as a shift; 64 = one scale per part
    const uint32_t bshift = bucket ? (uint32_t)__builtin_ctzll(bucket) : 64u;
    timer_begin(kTConcat, s);
    if (dense) {
        if (max_len)
            hipLaunchKernelGGL(k_concat_dense, dim3((uint32_t)((max_len + kTile - 1) / kTile), P), dim3(256), 0,
                               s, tab, qbits, bshift, out_val);
    } else if (max_nnz) {
        hipLaunchKernelGGL(k_concat_sparse, dim3((uint32_t)((max_nnz + kChunk - 1) / kChunk), P), dim3(256), 0,
                           s, tab, qbits, bshift, out_idx, out_val);
    }
    timer_end(kTConcat, s);
    return hipGetLastError();
}

}  // namespace sparcml
