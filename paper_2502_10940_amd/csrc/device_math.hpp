// device_math.hpp -- pointwise helpers for the gfx950 kernels: bf16 rounding
// and the CoLA nonlinearity sigma with its derivative.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cola {

// bf16 bits -> float (exact).
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two floats -> packed bf16 pair (lo in bits 15:0), round to nearest even,
// in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// float -> bf16 bits, round to nearest even (a NaN stays a NaN).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    return pack_bf16x2(f, 0.0f) & 0xffffu;
}

// x rounded to bf16 (nearest even) and back: the value a bf16 store keeps.
__device__ __forceinline__ float round_bf16(float x) {
    return __uint_as_float(pack_bf16x2(x, 0.0f) << 16);
}

// logistic sigmoid s(z) = 1 / (1 + e^{-z}); e^{-z} = inf for very negative z
// gives s = 0 exactly, never NaN.
// bf16 path: hardware exp and reciprocal (about 1 ulp each in fp32, far below
// the bf16 rounding that follows).
__device__ __forceinline__ float logistic_fast(float z) {
    return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}
__device__ __forceinline__ float logistic_exact(float z) {
    return 1.0f / (1.0f + expf(-z));
}

// Standard normal CDF Phi(z) = erfc(-z / sqrt 2) / 2 and density phi(z).
template <bool FAST>
__device__ __forceinline__ float normal_cdf(float z) {
    return 0.5f * erfcf(-z * 0.70710678118654752f);
}
template <bool FAST>
__device__ __forceinline__ float normal_pdf(float z) {
    return 0.39894228040143268f * (FAST ? __expf(-0.5f * z * z) : expf(-0.5f * z * z));
}

// sigma(z) and sigma'(z) for act 0 (identity), 1 (SiLU = z s(z),
// SiLU' = s (1 + z (1 - s))) and 2 (GeLU = z Phi(z), GeLU' = Phi + z phi).
// FAST selects the hardware exp and reciprocal (bf16 path).
template <bool FAST>
__device__ __forceinline__ float act_sigma(int act, float z) {
    if (act == 0) return z;
    if (act == 2) return z * normal_cdf<FAST>(z);
    float s = FAST ? logistic_fast(z) : logistic_exact(z);
    return z * s;
}

template <bool FAST>
__device__ __forceinline__ float act_sigma_prime(int act, float z) {
    if (act == 0) return 1.0f;
    if (act == 2) return normal_cdf<FAST>(z) + z * normal_pdf<FAST>(z);
    float s = FAST ? logistic_fast(z) : logistic_exact(z);
    return s * (1.0f + z * (1.0f - s));
}

// Both at once (the dZ epilogue needs sigma' and, for CoLA-M, H = sigma(z)),
// sharing the transcendental work.
template <bool FAST>
__device__ __forceinline__ void act_sigma_both(int act, float z, float& sig, float& sigp) {
    if (act == 0) {
        sig = z;
        sigp = 1.0f;
    } else if (act == 2) {
        const float cdf = normal_cdf<FAST>(z);
        sig = z * cdf;
        sigp = cdf + z * normal_pdf<FAST>(z);
    } else {
        const float s = FAST ? logistic_fast(z) : logistic_exact(z);
        sig = z * s;
        sigp = s * (1.0f + z * (1.0f - s));
    }
}

// The same with the activation fixed at compile time (ACT = 0 identity,
// 1 SiLU, 2 GeLU): the GEMM epilogues choose ACT once per block, so the
// unrolled per-element code has no branches.
template <int ACT, bool FAST>
__device__ __forceinline__ float act_sigma_c(float z) {
    if constexpr (ACT == 0) return z;
    else if constexpr (ACT == 2) return z * normal_cdf<FAST>(z);
    else return z * (FAST ? logistic_fast(z) : logistic_exact(z));
}

template <int ACT, bool FAST>
__device__ __forceinline__ void act_sigma_both_c(float z, float& sig, float& sigp) {
    if constexpr (ACT == 0) {
        sig = z;
        sigp = 1.0f;
    } else if constexpr (ACT == 2) {
        const float cdf = normal_cdf<FAST>(z);
        sig = z * cdf;
        sigp = cdf + z * normal_pdf<FAST>(z);
    } else {
        const float s = FAST ? logistic_fast(z) : logistic_exact(z);
        sig = z * s;
        sigp = s * (1.0f + z * (1.0f - s));
    }
}

}  // namespace cola
