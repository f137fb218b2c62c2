// MFMA operand helpers and scheduling shared by the gfx950 prefill kernels.
//
// MFMA lane layouts (v_mfma_f32_16x16x32_bf16, v_mfma_f32_16x16x16_bf16 and
// v_mfma_f32_16x16x4_f32): lane l = m + 16 g (m = l % 16, g = l / 16) holds
// row m of A and column m of B, its operand slots covering contraction
// indices of lane group g; the 16 x 16 fp32 result D[4 g + i][m] sits in
// element i of lane l.  Only the pairing of A and B slots matters for a
// contraction, so both operands may use any common contraction order.
#pragma once

#include "gdn_device.h"
#include "gdn_index.h"

namespace gdn {

typedef short s16x4_t __attribute__((ext_vector_type(4)));

// --- MFMA wrappers -----------------------------------------------------------
// K = 32: v_mfma_f32_16x16x32_bf16 (gfx950); K = 16: v_mfma_f32_16x16x16_bf16.
// Layout (both): A[m][k] on lane m + 16 g, B[k][n] on lane n + 16 g, slot j of
// the lane's operand vector is contraction index (K/4) g + j in hardware order;
// D[4 g + i][n] on lane n + 16 g, element i.  Only the pairing of A and B
// slots matters for a contraction, so operands may use any common order.
template <int K> struct Frag;
template <> struct Frag<32> { typedef bf16x8_t type; };
template <> struct Frag<16> { typedef s16x4_t type; };

__device__ __forceinline__ f32x4_t mma(const bf16x8_t& a, const bf16x8_t& b, const f32x4_t& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mma(const s16x4_t& a, const s16x4_t& b, const f32x4_t& c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

// fp32 MFMA 16x16x4: A[m][k] on lane m + 16 k, B[k][n] on lane n + 16 k.
__device__ __forceinline__ f32x4_t mma_f32(float a, float b, const f32x4_t& c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// A/B operand from a row-major bf16 LDS matrix, "permuted" contraction order:
// slot j < 4 -> column k0 + 4g + j, slot j >= 4 -> k0 + 16 + 4g + (j - 4).
// This is the order in which accumulator tiles supply B operands.
template <int K>
__device__ __forceinline__ typename Frag<K>::type lds_frag_perm(const uint16_t* row, int k0, int g) {
    if constexpr (K == 32) {
        const uint2 lo = *reinterpret_cast<const uint2*>(row + k0 + 4 * g);
        const uint2 hi = *reinterpret_cast<const uint2*>(row + k0 + 16 + 4 * g);
        uint4 u = {lo.x, lo.y, hi.x, hi.y};
        return __builtin_bit_cast(bf16x8_t, u);
    } else {
        const uint2 u = *reinterpret_cast<const uint2*>(row + k0 + 4 * g);
        return __builtin_bit_cast(s16x4_t, u);
    }
}

// Operand in "natural" order (slot j -> column k0 + (K/4) g + j); used where
// both operands come from LDS.
template <int K>
__device__ __forceinline__ typename Frag<K>::type lds_frag_nat(const uint16_t* row, int k0, int g) {
    if constexpr (K == 32) {
        const uint4 u = *reinterpret_cast<const uint4*>(row + k0 + 8 * g);
        return __builtin_bit_cast(bf16x8_t, u);
    } else {
        const uint2 u = *reinterpret_cast<const uint2*>(row + k0 + 4 * g);
        return __builtin_bit_cast(s16x4_t, u);
    }
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> packed bf16 pair (round to nearest even; one conversion instruction).
__device__ __forceinline__ uint32_t cvt_pk(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// hi = bf16(x), lo = bf16(x - hi) for a pair, each packed: x = hi + lo to ~2^-17.
__device__ __forceinline__ void split_pair(float a, float b, uint32_t& hi, uint32_t& lo) {
    hi = cvt_pk(a, b);
    lo = cvt_pk(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xFFFF0000u));
}

// hi / lo split with the residual from the dot-product unit: lo of element e
// is bf16(x_e + hi . m_e) with m_0 = (-1, 0), m_1 = (0, -1) as packed bf16, one
// v_dot2_f32_bf16 each (exact: x - hi is representable).  The two masks are
// kept in registers (opaque to the compiler): folding them into the
// instruction's inline-constant form placed -1 in the wrong half.
struct SplitMasks {
    uint32_t m0, m1;
};
__device__ __forceinline__ SplitMasks split_masks() {
    uint32_t a = 0x0000BF80u, b = 0xBF800000u;
    asm volatile("" : "+v"(a), "+v"(b));
    return SplitMasks{a, b};
}
__device__ __forceinline__ void split_pair(float a, float b, uint32_t& hi, uint32_t& lo, const SplitMasks& sm) {
    hi = cvt_pk(a, b);
    const bf16x2_t h = __builtin_bit_cast(bf16x2_t, hi);
    const float la = __builtin_amdgcn_fdot2_f32_bf16(h, __builtin_bit_cast(bf16x2_t, sm.m0), a, false);
    const float lb = __builtin_amdgcn_fdot2_f32_bf16(h, __builtin_bit_cast(bf16x2_t, sm.m1), b, false);
    lo = cvt_pk(la, lb);
}

// B operand (hi and lo parts) from accumulator tiles t0 (contraction rows
// k0..k0+15) and t1 (rows k0+16..k0+31), in the permuted order.
template <int K>
__device__ __forceinline__ void acc_frag(const f32x4_t& t0, const f32x4_t& t1,
                                         typename Frag<K>::type& hi, typename Frag<K>::type& lo) {
    if constexpr (K == 32) {
        uint4 uh, ul;
        split_pair(t0[0], t0[1], uh.x, ul.x);
        split_pair(t0[2], t0[3], uh.y, ul.y);
        split_pair(t1[0], t1[1], uh.z, ul.z);
        split_pair(t1[2], t1[3], uh.w, ul.w);
        hi = __builtin_bit_cast(bf16x8_t, uh);
        lo = __builtin_bit_cast(bf16x8_t, ul);
    } else {
        uint2 uh, ul;
        split_pair(t0[0], t0[1], uh.x, ul.x);
        split_pair(t0[2], t0[3], uh.y, ul.y);
        hi = __builtin_bit_cast(s16x4_t, uh);
        lo = __builtin_bit_cast(s16x4_t, ul);
    }
}

// The same with the dot-product residual.
__device__ __forceinline__ void acc_frag(const f32x4_t& t0, const f32x4_t& t1, bf16x8_t& hi, bf16x8_t& lo,
                                         const SplitMasks& sm) {
    uint4 uh, ul;
    split_pair(t0[0], t0[1], uh.x, ul.x, sm);
    split_pair(t0[2], t0[3], uh.y, ul.y, sm);
    split_pair(t1[0], t1[1], uh.z, ul.z, sm);
    split_pair(t1[2], t1[3], uh.w, ul.w, sm);
    hi = __builtin_bit_cast(bf16x8_t, uh);
    lo = __builtin_bit_cast(bf16x8_t, ul);
}

// B operand, hi part only.
template <int K>
__device__ __forceinline__ typename Frag<K>::type acc_frag_hi(const f32x4_t& t0, const f32x4_t& t1) {
    if constexpr (K == 32) {
        uint4 u = {cvt_pk(t0[0], t0[1]), cvt_pk(t0[2], t0[3]), cvt_pk(t1[0], t1[1]), cvt_pk(t1[2], t1[3])};
        return __builtin_bit_cast(bf16x8_t, u);
    } else {
        uint2 u = {cvt_pk(t0[0], t0[1]), cvt_pk(t0[2], t0[3])};
        return __builtin_bit_cast(s16x4_t, u);
    }
}

// B operand, lo part, given the hi part from acc_frag_hi<32>: the same
// residuals as acc_frag<32> (bf16 of x - hi for each element).
__device__ __forceinline__ bf16x8_t acc_frag_lo32(const f32x4_t& t0, const f32x4_t& t1, const bf16x8_t& hi) {
    const uint4 h = __builtin_bit_cast(uint4, hi);
    const uint4 l = {cvt_pk(t0[0] - __uint_as_float(h.x << 16), t0[1] - __uint_as_float(h.x & 0xFFFF0000u)),
                     cvt_pk(t0[2] - __uint_as_float(h.y << 16), t0[3] - __uint_as_float(h.y & 0xFFFF0000u)),
                     cvt_pk(t1[0] - __uint_as_float(h.z << 16), t1[1] - __uint_as_float(h.z & 0xFFFF0000u)),
                     cvt_pk(t1[2] - __uint_as_float(h.w << 16), t1[3] - __uint_as_float(h.w & 0xFFFF0000u))};
    return __builtin_bit_cast(bf16x8_t, l);
}

// Round x to bf16 hi and the residual to lo (scalar form, for LDS stores).
__device__ __forceinline__ void split_bf16(float x, uint16_t& hi, uint16_t& lo) {
    hi = f32_to_bf16(x);
    lo = f32_to_bf16(x - bf16_to_f32(hi));
}

}  // namespace gdn
