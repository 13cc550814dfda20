// Dense representation of one sparse stream (§5.1 "Switching to a Dense
// Format"): every index of [0, N) written once, +0.0 where the stream has no
// pair.  Each workgroup owns a 4096-index tile: it finds the tile's slice of
// the sorted stream by binary search, scatters into an LDS copy of the tile
// and writes the tile out with coalesced stores.
#include "internal.h"
#include "qsgd_device.h"

#include <algorithm>

namespace sparcml {
namespace {

constexpr uint32_t kTile = 4096;

__device__ __forceinline__ uint32_t lower_bound_u32(const uint32_t* a, uint32_t lo, uint32_t hi,
                                                    uint64_t x)
{
    while (lo < hi) {
        const uint32_t mid = lo + ((hi - lo) >> 1);
        if ((uint64_t)a[mid] < x) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

__global__ void __launch_bounds__(256) k_densify(const uint32_t* idx, const float* val,
                                                 const uint8_t* qval, const float* qscale,
                                                 uint32_t qbits, uint32_t nnz, uint64_t lo, uint64_t N,
                                                 float* out)
{
    __shared__ float s_tile[kTile];
    __shared__ uint32_t s_rng[2];
    const uint64_t tlo = lo + (uint64_t)blockIdx.x * kTile;  // absolute index of the tile
    const uint64_t thi = min(tlo + kTile, lo + N);
    for (uint32_t j = threadIdx.x; j < kTile; j += 256) s_tile[j] = 0.0f;
    if (threadIdx.x < 2) s_rng[threadIdx.x] = lower_bound_u32(idx, 0u, nnz, threadIdx.x ? thi : tlo);
    __syncthreads();
    const float unit = qbits ? level_unit(*qscale, qbits) : 0.0f;
    for (uint32_t i = s_rng[0] + threadIdx.x; i < s_rng[1]; i += 256) {
        const uint64_t j = (uint64_t)idx[i] - tlo;
        if (j < kTile) s_tile[j] = qbits ? dequant(load_code(qval, i, qbits), qbits, unit) : val[i];
    }
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < kTile; j += 256)
        if (tlo + j < thi) out[tlo - lo + j] = s_tile[j];
}

__global__ void k_dequant(const uint8_t* qval, const float* qscale, uint32_t qbits, uint64_t n,
                          float* out)
{
    const float unit = level_unit(*qscale, qbits);
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        out[i] = dequant(load_code(qval, i, qbits), qbits, unit);
}

}  // namespace

hipError_t dequant_run(const uint8_t* qval, const float* qscale, uint32_t qbits, uint64_t n,
                       float* out, hipStream_t s)
{
    if (n == 0) return hipSuccess;
    const uint64_t blocks = std::min<uint64_t>((n + 255) / 256, 65536);
    hipLaunchKernelGGL(k_dequant, dim3((uint32_t)blocks), dim3(256), 0, s, qval, qscale, qbits, n, out);
    return hipGetLastError();
}

hipError_t densify_run(const uint32_t* idx, const float* val, const uint8_t* qval,
                       const float* qscale, uint32_t qbits, uint64_t nnz, uint64_t N,
                       int is_dense, float* dense, hipStream_t s, uint64_t lo)
{
    if (is_dense) {
        if (qbits) return dequant_run(qval, qscale, qbits, N, dense, s);
        return hipMemcpyAsync(dense, val, N * sizeof(float), hipMemcpyDeviceToDevice, s);
    }
    const uint64_t tiles = (N + kTile - 1) / kTile;
    timer_begin(kTDensify, s);
    hipLaunchKernelGGL(k_densify, dim3((uint32_t)tiles), dim3(256), 0, s, idx, val, qval, qscale,
                       qbits, (uint32_t)nnz, lo, N, dense);
    timer_end(kTDensify, s);
    return hipGetLastError();
}

}  // namespace sparcml
