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

// Two fp32 values rounded to nearest even as one word of bf16 (lo in bits
// 0-15): a single hardware conversion on gfx950, equal to f32_to_bf16_rne of
// each half for every non-NaN input.
typedef float dpb_f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 dpb_bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((dpb_f32x2){lo, hi}, dpb_bf16x2));
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
// Exchange with the lane whose index differs by J (1, 2, 4, 8, 16, 32) on the
// vector ALU, without the LDS path of swizzles and permutes: quad
// permutations for 1 and 2, rotations of 16-lane rows for 4 (two of them,
// selected by lane bit 2) and 8, and the row-swap permutes of gfx950 for 16
// and 32 (each returns both halves of the swap; lane bit 4 or 5 selects).
template <int J>
__device__ __forceinline__ uint32_t lane_xor(uint32_t v)
{
    static_assert(J == 1 || J == 2 || J == 4 || J == 8 || J == 16 || J == 32, "power of two up to 32");
    if constexpr (J == 1) {
        return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
    } else if constexpr (J == 2) {
        return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
    } else if constexpr (J == 4) {
        const uint32_t r4 = (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x124, 0xF, 0xF, false);    // row_ror 4
        const uint32_t r12 = (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x12C, 0xF, 0xF, false);   // row_ror 12
        return (__lane_id() & 4) ? r4 : r12;
    } else if constexpr (J == 8) {
        return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, false);   // row_ror 8
    } else if constexpr (J == 16) {
        const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        return (__lane_id() & 16) ? p[0] : p[1];
    } else {
        const auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        return (__lane_id() & 32) ? p[0] : p[1];
    }
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
