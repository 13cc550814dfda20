// Sum of P vectors whose index ranges are disjoint -- the gathered shares
// of the split-allgather allreduce (§5.3.2) -- which is their concatenation
// (§5.1, case (2)).  Part s covers [lo_s, lo_s + len_s); it is sparse
// (absolute indices) or dense (len_s values), with fp32 values or QSGD codes
// (one scale, or one per bucket of B entries, §6) dequantized on the fly.
//
// Sparse result: every part's entries are copied to its offset in the
// output (prefix of the parts' counts): a (chunk, part) grid of 4096-entry
// chunks, coalesced grid-stride copies.  Dense result: a (tile, part) grid
// over 16384-index tiles of each part's range; a dense part's tile is
// copied (or decoded) straight through, 16-byte stores with all loads in
// flight first; a sparse part's tile is scattered into LDS 4096 indices at
// a time (zeros elsewhere) and written with coalesced stores.  Both are HBM-bound: every
// input byte is read once and every output byte written once.
#include "internal.h"
#include "qsgd_device.h"

#include <algorithm>
#include <vector>

namespace sparcml {
namespace {

constexpr uint32_t kTile = 4096;    // LDS tile of a sparse part in a dense result
constexpr uint32_t kDTile = 16384;  // dense-result indices per workgroup
constexpr uint32_t kChunk = 4096;   // sparse-result entries per workgroup (256 threads x 16)

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

// Four consecutive values of a dense part from stored entry i (a multiple
// of 4; a bucket holds a multiple of 4 entries): one 16-byte load (fp32) or
// one 1/2/4-byte load of their codes and one scale.
__device__ __forceinline__ float4 dense4(const CDesc& d, uint64_t i, uint32_t qbits, uint32_t bshift)
{
    if (!qbits) return *reinterpret_cast<const float4*>(d.val + i);
    uint32_t c;  // the 4 codes, element q at bit q * qbits
    if (qbits == 8u) c = *reinterpret_cast<const uint32_t*>(d.qval + i);
    else if (qbits == 4u) c = *reinterpret_cast<const uint16_t*>(d.qval + (i >> 1));
    else c = d.qval[i >> 2];
    const float unit = level_unit(d.qscale[bshift < 64u ? (i >> bshift) : 0], qbits);
    const uint32_t m = (1u << qbits) - 1u;
    return make_float4(dequant(c & m, qbits, unit), dequant((c >> qbits) & m, qbits, unit),
                       dequant((c >> (2 * qbits)) & m, qbits, unit), dequant((c >> (3 * qbits)) & m, qbits, unit));
}

// A (tile, part) grid over kDTile-index tiles of every part's range.
__global__ void __launch_bounds__(256) k_concat_dense(const CDesc* tab, uint32_t qbits, uint32_t bshift,
                                                      float* out)
{
    __shared__ float s_tile[kTile];
    __shared__ uint64_t s_rng[2];
    const CDesc d = tab[blockIdx.y];
    const uint64_t t0 = (uint64_t)blockIdx.x * kDTile;  // tile start within the part
    if (t0 >= d.len) return;                            // uniform over the block
    const uint32_t w = (uint32_t)min((uint64_t)kDTile, d.len - t0);
    float* o = out + d.lo + t0;
    if (d.dense) {
        const bool ovec = (reinterpret_cast<uintptr_t>(o) & 15u) == 0;
        const bool ivec = qbits ? ((reinterpret_cast<uintptr_t>(d.qval) & 3u) == 0)
                                : ((reinterpret_cast<uintptr_t>(d.val) & 15u) == 0);
        if (w == kDTile && ivec && ovec) {
            // whole aligned tile: every load issued before the first store
            constexpr int U = kDTile / 1024;
            float4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = dense4(d, t0 + u * 1024 + threadIdx.x * 4, qbits, bshift);
#pragma unroll
            for (int u = 0; u < U; ++u) store_nt(o + u * 1024 + threadIdx.x * 4, v[u]);
            return;
        }
        for (uint32_t j = threadIdx.x * 4; j < w; j += 1024) {
            if (j + 4 <= w && ivec) {
                const float4 v = dense4(d, t0 + j, qbits, bshift);
                if (ovec) {
                    store_nt(o + j, v);
                } else {
                    o[j] = v.x;
                    o[j + 1] = v.y;
                    o[j + 2] = v.z;
                    o[j + 3] = v.w;
                }
            } else {
                for (uint32_t q = 0; q < 4 && j + q < w; ++q) o[j + q] = entry(d, t0 + j + q, qbits, bshift);
            }
        }
        return;
    }
    // sparse part: kTile-index sub-tiles, each scattered into LDS and
    // written out whole
    for (uint32_t sub = 0; sub < w; sub += kTile) {
        const uint32_t sw = min(kTile, w - sub);
        const uint64_t base = d.lo + t0 + sub;  // absolute index of the sub-tile
        __syncthreads();  // the previous sub-tile's reads of s_tile / s_rng are done
        for (uint32_t j = threadIdx.x; j < kTile; j += 256) s_tile[j] = 0.0f;
        if (threadIdx.x < 2) s_rng[threadIdx.x] = lower_bound_idx(d.idx, 0, d.nnz, base + (threadIdx.x ? sw : 0u));
        __syncthreads();
        for (uint64_t i = s_rng[0] + threadIdx.x; i < s_rng[1]; i += 256) {
            const uint64_t j = (uint64_t)d.idx[i] - base;
            if (j < kTile) s_tile[j] = entry(d, i, qbits, bshift);
        }
        __syncthreads();
        for (uint32_t j = threadIdx.x; j < sw; j += 256) o[sub + j] = s_tile[j];
    }
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
            hipLaunchKernelGGL(k_concat_dense, dim3((uint32_t)((max_len + kDTile - 1) / kDTile), P), dim3(256), 0,
                               s, tab, qbits, bshift, out_val);
    } else if (max_nnz) {
        hipLaunchKernelGGL(k_concat_sparse, dim3((uint32_t)((max_nnz + kChunk - 1) / kChunk), P), dim3(256), 0,
                           s, tab, qbits, bshift, out_idx, out_val);
    }
    timer_end(kTConcat, s);
    return hipGetLastError();
}

}  // namespace sparcml
