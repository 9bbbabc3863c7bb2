// Device helpers shared by the DPB kernels (gfx950, wave64).
#pragma once

#include "dpb_internal.hpp"

namespace dpb {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// Orders LDS traffic among the lanes of one wave (no workgroup barrier).
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// float -> bf16 bits, round to nearest even.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ uint32_t parity(uint32_t v) { return __popc(v) & 1u; }

// +-a where the sign flips when popcount(m) is odd: the entry of a hashed
// direction times a coefficient (App. A.4, packed-parity equation).
__device__ __forceinline__ float signed_by_parity(float a, uint32_t m)
{
    return __uint_as_float(__float_as_uint(a) ^ (__popc(m) << 31));
}

// AbsTopK key: |s| (fp32 bits) first, then the smaller index; the sign of s
// rides in bit 0 so that the signed coefficient can be rebuilt.
__device__ __forceinline__ uint64_t make_key(float s, uint32_t idx)
{
    const uint32_t u = __float_as_uint(s);
    return ((uint64_t)(u & 0x7FFFFFFFu) << 32) | (uint64_t)(((0x7FFFFFFFu - idx) << 1) | (u >> 31));
}
__device__ __forceinline__ uint32_t key_index(uint64_t key) { return 0x7FFFFFFFu - ((uint32_t)key >> 1); }
__device__ __forceinline__ float key_value(uint64_t key)
{
    return __uint_as_float((uint32_t)(key >> 32) | (((uint32_t)key & 1u) << 31));
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

template <bool BF16>
__device__ __forceinline__ float load_act(const void* p, int64_t i)
{
    if constexpr (BF16) return bf16_bits_to_f32(((const uint16_t*)p)[i]);
    else return ((const float*)p)[i];
}

template <bool BF16>
__device__ __forceinline__ void store_act(void* p, int64_t i, float v)
{
    if constexpr (BF16) ((uint16_t*)p)[i] = (uint16_t)f32_to_bf16_rne(v);
    else ((float*)p)[i] = v;
}

// Lane exchanges without address arithmetic: XOR of the lane index by
// 1..16 inside 32-lane halves (ds_swizzle bit mode), and by 32.
template <int J>
__device__ __forceinline__ uint32_t swz_xor(uint32_t v)
{
    static_assert(J >= 1 && J <= 16, "swizzle xor within 32 lanes");
    return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, (J << 10) | 0x1F);
}
__device__ __forceinline__ float swz_xorf16(float v) { return __uint_as_float(swz_xor<16>(__float_as_uint(v))); }

// Rotates left by r (0..31).
__device__ __forceinline__ uint32_t rotl32(uint32_t v, uint32_t r) { return __builtin_amdgcn_alignbit(v, v, (32u - r) & 31u); }

// Exact split of an fp32 value into three bf16 terms (v = hi + mid + lo).
__device__ __forceinline__ void split3(float v, uint32_t& hi, uint32_t& mid, uint32_t& lo)
{
    hi = f32_to_bf16_rne(v);
    const float r1 = v - bf16_bits_to_f32(hi);
    mid = f32_to_bf16_rne(r1);
    lo = f32_to_bf16_rne(r1 - bf16_bits_to_f32(mid));
}

}  // namespace dpb
