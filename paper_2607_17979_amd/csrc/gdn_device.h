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

// ---- optional input prologue (the flags of the _ex entry points) ------------
enum : int {
    kFlagQkL2Norm = 1,      // q and k rows are L2-normalised in the kernel
    kFlagGateLogits = 2,    // g and beta hold logits: g = -softplus(a), beta = sigmoid(b)
    kFlagShortOnly = 4,     // prefill: every sequence has at most 8 tokens (multi-token decode)
};

// 1 / sqrt(sum of squares + 1e-6) of a row of D bf16 values in global memory,
// summed in index order with one rounding per term (the square of a bf16
// value is exact in fp32) and correctly rounded square root and division, so
// that every kernel, and a host computation in the same order, gets the same
// bits for the same row.
template <int D>
__device__ __forceinline__ float row_inv_norm(const uint16_t* row) {
    float acc = 0.f;
#pragma unroll
    for (int s = 0; s < D / 8; ++s) {
        const uint4 u = *reinterpret_cast<const uint4*>(row + 8 * s);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float lo = __uint_as_float(w[e] << 16), hi = __uint_as_float(w[e] & 0xFFFF0000u);
            acc = fmaf(lo, lo, acc);
            acc = fmaf(hi, hi, acc);
        }
    }
    return 1.0f / sqrtf(acc + 1e-6f);
}

// Two packed bf16 values times r, rounded to bf16 again (nearest even).
__device__ __forceinline__ uint32_t scale_bf16x2(uint32_t w, float r) {
    const uint32_t lo = f32_to_bf16(__uint_as_float(w << 16) * r);
    const uint32_t hi = f32_to_bf16(__uint_as_float(w & 0xFFFF0000u) * r);
    return lo | (hi << 16);
}
__device__ __forceinline__ uint4 scale_bf16x8(const uint4& u, float r) {
    return uint4{scale_bf16x2(u.x, r), scale_bf16x2(u.y, r), scale_bf16x2(u.z, r), scale_bf16x2(u.w, r)};
}

// g = log alpha = -softplus(a) for a gate logit a, in fp32.
__device__ __forceinline__ float gate_from_logit(float a) {
    return -(fmaxf(a, 0.f) + log1pf(expf(-fabsf(a))));
}
// beta = sigmoid(b) for a logit b, in fp32.
__device__ __forceinline__ float beta_from_logit(float b) { return 1.f / (1.f + expf(-b)); }

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
