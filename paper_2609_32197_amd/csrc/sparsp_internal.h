// Internal declarations shared by the HIP translation units of libsparsp:
// the host interface (sparsp_launch.h) plus device helpers. Kernels are
// launched only through the launchers declared there; argument checking has
// already happened in api.cpp when they are called.
#pragma once

#include <hip/hip_runtime.h>

#include "sparsp_launch.h"

namespace sparsp {

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// float32 -> bfloat16 bits, round to nearest even (finite inputs; NaN kept quiet).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float x) {
    uint32_t u = __float_as_uint(x);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

// 16-byte global load and store with the non-temporal hint, for data that
// streams through once (the caches keep less of it).
__device__ __forceinline__ uint4 load_nt(const char* p) {
    typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
    return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p)));
}
__device__ __forceinline__ void store_nt(char* p, uint4 v) {
    typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(__builtin_bit_cast(u32x4_t, v), reinterpret_cast<u32x4_t*>(p));
}

}  // namespace sparsp
