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
