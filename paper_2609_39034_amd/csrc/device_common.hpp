// Device helpers shared by the SwiLA kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace swila {

constexpr float kLog2e = 1.4426950408889634f;

// bf16 <-> fp32.  Widening is exact; narrowing rounds to nearest-even and
// keeps NaN a (quiet) NaN.
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
    return __builtin_bit_cast(uint16_t, (__bf16)f);   // v_cvt_pk_bf16_f32 (RNE)
}

// e^x through the hardware base-2 exponential.
__device__ __forceinline__ float exp_fast(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }

// 1/x through the hardware reciprocal (about 1 ulp).
__device__ __forceinline__ float rcp_fast(float x) { return __builtin_amdgcn_rcpf(x); }

__device__ __forceinline__ float sigmoid(float x) { return rcp_fast(1.0f + exp_fast(-x)); }

// Four consecutive input elements (fp32, or bf16 when bf16 is set) as fp32.
// p must be 8-byte (bf16) or 16-byte (fp32) aligned.
__device__ __forceinline__ float4 load4(const void *base, size_t idx, bool bf16) {
    if (bf16) {
        const uint2 u = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(base) + idx);
        return make_float4(bf16_bits_to_f32(u.x & 0xffffu), bf16_bits_to_f32(u.x >> 16),
                           bf16_bits_to_f32(u.y & 0xffffu), bf16_bits_to_f32(u.y >> 16));
    }
    return *reinterpret_cast<const float4 *>(static_cast<const float *>(base) + idx);
}

__device__ __forceinline__ float load1(const void *base, size_t idx, bool bf16) {
    if (bf16) return bf16_bits_to_f32(static_cast<const uint16_t *>(base)[idx]);
    return static_cast<const float *>(base)[idx];
}

// Raw loads: the bits of one element (a bf16 in the low half, or an fp32), or
// of four, converted to fp32 only where they are used.  Loading and converting
// in one step makes each load wait for its data before the next is issued;
// these let a staging loop issue all of its loads first.
__device__ __forceinline__ uint32_t raw1(const void *base, size_t idx, bool bf16) {
    return bf16 ? (uint32_t) static_cast<const uint16_t *>(base)[idx]
                : static_cast<const uint32_t *>(base)[idx];
}
__device__ __forceinline__ float cvt1(uint32_t r, bool bf16) {
    return __uint_as_float(bf16 ? r << 16 : r);
}
__device__ __forceinline__ uint4 raw4(const void *base, size_t idx, bool bf16) {
    if (bf16) {
        const uint2 x = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(base) + idx);
        return make_uint4(x.x, x.y, 0u, 0u);
    }
    return *reinterpret_cast<const uint4 *>(static_cast<const float *>(base) + idx);
}
__device__ __forceinline__ float4 cvt4(uint4 r, bool bf16) {
    if (bf16)
        return make_float4(__uint_as_float(r.x << 16), __uint_as_float(r.x & 0xffff0000u),
                           __uint_as_float(r.y << 16), __uint_as_float(r.y & 0xffff0000u));
    return make_float4(__uint_as_float(r.x), __uint_as_float(r.y), __uint_as_float(r.z),
                       __uint_as_float(r.w));
}

__device__ __forceinline__ void store1(void *base, size_t idx, float x, bool bf16) {
    if (bf16)
        static_cast<uint16_t *>(base)[idx] = f32_to_bf16_bits(x);
    else
        static_cast<float *>(base)[idx] = x;
}

// Block barrier that orders LDS traffic only: waits for this wave's LDS
// operations, then for every wave of the block.  Global loads still in flight
// (prefetches) are not waited for; the compiler inserts those waits where the
// loaded registers are used.  The "memory" clobber keeps the compiler from
// moving memory accesses across it.
__device__ __forceinline__ void block_sync_lds() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// DPP lane moves within a row of 16 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xf, 0xf, true));
}

// Sum over each aligned group of L consecutive lanes; every lane of the group
// receives the total.  L is a power of two, at most 64.
template <int L>
__device__ __forceinline__ float group_sum(float x) {
    if constexpr (L >= 2) x += dpp_mov<0xb1>(x);   // quad_perm [1,0,3,2]: lane ^ 1
    if constexpr (L >= 4) x += dpp_mov<0x4e>(x);   // quad_perm [2,3,0,1]: lane ^ 2
    if constexpr (L >= 8) x += dpp_mov<0x141>(x);  // row_half_mirror: other quad of 8
    if constexpr (L >= 16) x += dpp_mov<0x140>(x); // row_mirror: other half of 16
    if constexpr (L >= 32) x += __shfl_xor(x, 16);
    if constexpr (L >= 64) x += __shfl_xor(x, 32);
    return x;
}

// Maximum over each aligned group of L consecutive lanes (L a power of two,
// at most 16); every lane of the group receives it.
template <int L>
__device__ __forceinline__ float group_max(float x) {
    if constexpr (L >= 2) x = fmaxf(x, dpp_mov<0xb1>(x));
    if constexpr (L >= 4) x = fmaxf(x, dpp_mov<0x4e>(x));
    if constexpr (L >= 8) x = fmaxf(x, dpp_mov<0x141>(x));
    if constexpr (L >= 16) x = fmaxf(x, dpp_mov<0x140>(x));
    return x;
}

}  // namespace swila
