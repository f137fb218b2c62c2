// Device helpers shared by the gfx950 kernels: bf16 conversion, cross-lane
// sums over small lane groups (DPP), fast exp, and MFMA operand types.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gdn {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// bf16 bit pattern -> fp32 (exact).
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// fp32 -> bf16, round to nearest even (the conversion instruction of gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float x) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(x));
}

// exp(x) as 2^(x * log2 e) on the hardware exp2 unit.
__device__ __forceinline__ float fast_exp(float x) {
    return __builtin_amdgcn_exp2f(x * 1.4426950408889634f);
}

// DPP lane moves inside a row of 16 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
constexpr int DPP_QUAD_XOR1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int DPP_QUAD_XOR2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141;  // lane i <- lane 7-i within each group of 8
constexpr int DPP_ROW_MIRROR = 0x140;   // lane i <- lane 15-i within each row of 16

// Sum over aligned groups of G lanes (G in {1, 2, 4, 8, 16}); every lane of a
// group receives the group's sum.
template <int G>
__device__ __forceinline__ float group_sum(float x) {
    if constexpr (G >= 2) x += dpp<DPP_QUAD_XOR1>(x);
    if constexpr (G >= 4) x += dpp<DPP_QUAD_XOR2>(x);
    if constexpr (G >= 8) x += dpp<DPP_HALF_MIRROR>(x);
    if constexpr (G >= 16) x += dpp<DPP_ROW_MIRROR>(x);
    return x;
}

}  // namespace gdn
