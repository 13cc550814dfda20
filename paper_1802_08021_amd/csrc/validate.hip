// Validation of sparse streams (§5.1 "Vector Representations": a sparse
// vector is a list of index/value pairs; the reduction's merges assume the
// indices of a stream strictly ascending and inside the vector's range).
// One read-only pass over every stream's indices; the first offending
// position (lowest stream, then lowest position) is kept with an atomic
// minimum in the workspace and read back by the host.
#include "internal.h"

#include <algorithm>
#include <vector>

namespace sparcml {
namespace {

struct IdxDesc {
    const uint32_t* idx;
    uint64_t nnz;
};

// Grid: (blocks over positions, P).  bad = stream << 40 | position.
__global__ void __launch_bounds__(256) k_validate(const IdxDesc* tab, uint64_t lo, uint64_t hi,
                                                  unsigned long long* bad)
{
    const uint32_t r = blockIdx.y;
    const IdxDesc d = tab[r];
    const uint64_t step = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < d.nnz; i += step) {
        const uint64_t x = d.idx[i];
        const bool ok = x >= lo && x < hi && (i == 0 || (uint64_t)d.idx[i - 1] < x);
        if (!ok) atomicMin(bad, (unsigned long long)r << 40 | i);
    }
}

__global__ void k_validate_init(unsigned long long* bad) { *bad = ~0ull; }

}  // namespace

size_t validate_workspace(int P) { return align_up(sizeof(IdxDesc) * (size_t)P, 256) + 256; }

hipError_t validate_run(int P, const uint32_t* const* idx, const uint64_t* nnz, uint64_t lo, uint64_t hi,
                        void* ws, hipStream_t s, int* bad_stream, uint64_t* bad_pos)
{
    Carve c(ws);
    IdxDesc* tab = c.take<IdxDesc>((size_t)P);
    unsigned long long* bad = c.take<unsigned long long>(1);
    std::vector<IdxDesc> host(P);
    uint64_t maxn = 0;
    for (int r = 0; r < P; ++r) {
        host[r] = IdxDesc{idx[r], nnz[r]};
        maxn = std::max(maxn, nnz[r]);
    }
    hipError_t e = upload(tab, host.data(), sizeof(IdxDesc) * P, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_validate_init, dim3(1), dim3(1), 0, s, bad);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (maxn) {
        const uint64_t blocks = std::min<uint64_t>((maxn + 255) / 256, 1024);
        hipLaunchKernelGGL(k_validate, dim3((uint32_t)blocks, (uint32_t)P), dim3(256), 0, s, tab, lo, hi, bad);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    unsigned long long res = 0;
    if ((e = hipMemcpyAsync(&res, bad, sizeof(res), hipMemcpyDeviceToHost, s)) != hipSuccess) return e;
    if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
    *bad_stream = res == ~0ull ? -1 : (int)(res >> 40);
    *bad_pos = res & ((1ull << 40) - 1);
    return hipSuccess;
}

}  // namespace sparcml
