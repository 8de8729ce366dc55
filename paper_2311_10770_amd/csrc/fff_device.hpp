// fff_device.hpp -- gfx950 device helpers for the FFF kernels: bf16 packing,
// sub-wave all-reduce over DPP and permlane swaps, and the activations.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace fff {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float tile_v4f __attribute__((ext_vector_type(4)));  // a 16x16 MFMA result per lane

// bf16 -> fp32 is exact: the bf16 bits are the top half of the fp32 bits.
__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return uint32_t(f32_to_bf16(lo)) | (uint32_t(f32_to_bf16(hi)) << 16);
}

// c + a.lo*b.lo + a.hi*b.hi with bf16 pairs; the bf16 products are exact in fp32.
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c,
                                           false);
}

__device__ __forceinline__ uint32_t word(const uint4& v, int j) {
    return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
}
__device__ __forceinline__ float fword(const float4& v, int j) {
    return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
}

// Sum of v over each aligned group of LANES lanes (16, 32 or 64); every lane of
// the group receives the same bits.  Within a 16-lane row the butterfly uses
// DPP row rotations; across rows it uses the gfx950 permlane swaps, which hand
// each lane its partner row's value.  Every step adds two values that are
// bitwise equal across the pair, so all lanes end with identical sums and take
// the same branch.
template <int LANES>
__device__ __forceinline__ float group_sum(float v) {
    static_assert(LANES == 16 || LANES == 32 || LANES == 64, "group of 16, 32 or 64 lanes");
    v += __builtin_amdgcn_update_dpp(0.0f, v, 0x128, 0xf, 0xf, false);  // row_ror:8
    v += __builtin_amdgcn_update_dpp(0.0f, v, 0x124, 0xf, 0xf, false);  // row_ror:4
    v += __builtin_amdgcn_update_dpp(0.0f, v, 0x122, 0xf, 0xf, false);  // row_ror:2
    v += __builtin_amdgcn_update_dpp(0.0f, v, 0x121, 0xf, 0xf, false);  // row_ror:1
    if constexpr (LANES >= 32) {
        const uint32_t u = __float_as_uint(v);
        const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
        v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    if constexpr (LANES == 64) {
        const uint32_t u = __float_as_uint(v);
        const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
        v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    return v;
}

enum { ACT_GELU_ERF = 0, ACT_GELU_TANH = 1, ACT_IDENTITY = 2 };

// GELU(z) = z * Phi(z) = z/2 * erfc(-z/sqrt 2); erfc keeps full relative
// accuracy for negative z, where 1 + erf(z/sqrt 2) would cancel.  The tanh
// approximation z/2 (1 + tanh u), u = sqrt(2/pi)(z + 0.044715 z^3), is
// evaluated as z / (1 + exp(-2u)) (the same function, since
// (1 + tanh u)/2 = 1/(1 + exp(-2u))), which does not cancel for negative z.
__device__ __forceinline__ float gelu_tanh_u(float z) { return 0.79788456080286535588f * (z + 0.044715f * z * z * z); }

__device__ __forceinline__ float activation(float z, int act) {
    if (act == ACT_GELU_ERF) return 0.5f * z * erfcf(-0.70710678118654752440f * z);
    if (act == ACT_GELU_TANH) return z / (1.0f + expf(-2.0f * gelu_tanh_u(z)));
    return z;
}

// d act / dz.  GELU: Phi(z) + z phi(z) with phi the standard normal density.
// Tanh form: with s = 1/(1 + exp(-2u)) and 1 - s = 1/(1 + exp(2u)),
// d/dz [z s] = s + 2 z s (1 - s) du/dz.  Identity: 1.
__device__ __forceinline__ float activation_grad(float z, int act) {
    if (act == ACT_GELU_ERF)
        return 0.5f * erfcf(-0.70710678118654752440f * z) + z * 0.39894228040143267794f * expf(-0.5f * z * z);
    if (act == ACT_GELU_TANH) {
        const float u = gelu_tanh_u(z);
        const float s = 1.0f / (1.0f + expf(-2.0f * u));
        const float sm = 1.0f / (1.0f + expf(2.0f * u));
        return s + 2.0f * z * s * sm * 0.79788456080286535588f * (1.0f + 0.134145f * z * z);
    }
    return 1.0f;
}

}  // namespace fff
