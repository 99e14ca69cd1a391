// Device-side helpers shared by the MPM kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mpm {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// Storage types: bfloat16 is handled as raw 16-bit patterns.
struct Bf16 {
    static constexpr int kBytes = 2;
};
struct F32 {
    static constexpr int kBytes = 4;
};

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// float32 -> bfloat16 bits, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ u32x4 load16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

__device__ __forceinline__ void store16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// Streaming store for rows written once and not read back by this kernel.
__device__ __forceinline__ void store16_stream(void* p, u32x4 v)
{
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

// Mean of two 16-byte groups of storage values: float32 arithmetic, one
// rounding to the storage type.
__device__ __forceinline__ u32x4 mean16(u32x4 a, u32x4 b, Bf16)
{
    u32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        float lo = (bf16_lo(a[e]) + bf16_lo(b[e])) * 0.5f;
        float hi = (bf16_hi(a[e]) + bf16_hi(b[e])) * 0.5f;
        r[e] = f32_to_bf16_rne(lo) | (f32_to_bf16_rne(hi) << 16);
    }
    return r;
}

__device__ __forceinline__ u32x4 mean16(u32x4 a, u32x4 b, F32)
{
    u32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e)
        r[e] = __float_as_uint((__uint_as_float(a[e]) + __uint_as_float(b[e])) * 0.5f);
    return r;
}

__device__ __forceinline__ int wave_sum(int v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

}  // namespace mpm
