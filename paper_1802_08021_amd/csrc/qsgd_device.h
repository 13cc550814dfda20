// Device helpers for QSGD codes (§6: buckets of packed low-precision items
// plus a full-precision scale).  A code is (sign << (bits-1)) | level.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sparcml {

// Code of element i from a packed array (8/qbits codes per byte, element i
// at bit (i % (8/qbits)) * qbits of byte i / (8/qbits)).
// (q: any pointer to bytes -- generic, or marked global)
template <class BytePtr>
__device__ __forceinline__ uint32_t load_code(BytePtr q, uint64_t i, uint32_t qbits)
{
    const uint32_t plog = qbits == 8u ? 0u : (qbits == 4u ? 1u : 2u);  // log2(codes per byte)
    const uint32_t byte = q[i >> plog];
    const uint32_t sh = (uint32_t)(i & ((1u << plog) - 1u)) * qbits;
    return (byte >> sh) & ((1u << qbits) - 1u);
}

// Value of one level: scale / s, s = 2^(qbits-1) - 1, correctly rounded.
__device__ __forceinline__ float level_unit(float scale, uint32_t qbits)
{
    return __fdiv_rn(scale, (float)((1u << (qbits - 1u)) - 1u));
}

// +-level * unit; level 0 gives +0.0.
__device__ __forceinline__ float dequant(uint32_t code, uint32_t qbits, float unit)
{
    const uint32_t l = code & ((1u << (qbits - 1u)) - 1u);
    const float mag = __fmul_rn((float)l, unit);
    return l == 0u ? 0.0f : (((code >> (qbits - 1u)) & 1u) ? -mag : mag);
}

}  // namespace sparcml
