// The exact-sum bf16 pair of an fp32 value (hi = bf16(x), lo = bf16(x - hi), both rounded to nearest
// even) in the interleaved layout the prefill GEMMs read (pair_at, stage_kernels.h).  Shared by the
// kernels that produce GEMM operands: RMSNorm, SwiGLU, and the prefill attention output.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace stg {

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t pair_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ void split_pair(float v, uint16_t &hi, uint16_t &lo) {
    hi = pair_bf16(v);
    lo = pair_bf16(v - __uint_as_float((uint32_t)hi << 16));
}

// The hi and lo of four consecutive elements of a 32-wide block (p: the first one's hi, 8-byte
// aligned): two 8-byte stores, the lo 32 elements further.
__device__ __forceinline__ void store_pair4(uint16_t *p, float4 v) {
    uint16_t h[4], l[4];
    split_pair(v.x, h[0], l[0]);
    split_pair(v.y, h[1], l[1]);
    split_pair(v.z, h[2], l[2]);
    split_pair(v.w, h[3], l[3]);
    *reinterpret_cast<uint2 *>(p) = make_uint2(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16));
    *reinterpret_cast<uint2 *>(p + 32) = make_uint2(l[0] | ((uint32_t)l[1] << 16), l[2] | ((uint32_t)l[3] << 16));
}

}  // namespace stg
