// Internal device helpers shared by the MoE layer kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

typedef uint16_t bf16_t;  // raw bfloat16 bits
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float -> bfloat16, round to nearest even (gfx950 converts in hardware: v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f)); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const bf16x2_t v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

// Lanes of this wave whose expert equals this lane's (valid lanes only), from nbits ballots
// over the id bits (E <= 2^nbits).
__device__ __forceinline__ uint64_t same_expert_lanes(int e, bool valid, int nbits) {
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < nbits; ++b) {
        const bool bit = valid && ((e >> b) & 1);
        const uint64_t m = __ballot(bit);
        peers &= bit ? m : ~m;
    }
    return peers;
}

// Activations of the expert FFN (fp32).
__device__ __forceinline__ float act_gelu(float u) { return 0.5f * u * (1.0f + erff(u * 0.70710678118654752f)); }

__device__ __forceinline__ float act_gelu_tanh(float u) {
    const float c = 0.79788456080286536f;  // sqrt(2/pi)
    return 0.5f * u * (1.0f + tanhf(c * (u + 0.044715f * u * u * u)));
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

// Fast activations for the bf16 epilogues (their error is far below bf16 rounding).
//
// erf from Abramowitz & Stegun, Handbook of Mathematical Functions, formula 7.1.26
// (Hastings' rational approximation): for a >= 0,
//     erf(a) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-a^2) + eps,
//     t = 1 / (1 + p a),  |eps| <= 1.5e-7.
// GELU(u) = u Phi(u) = u (1 + erf(u / sqrt 2)) / 2; with Q = (poly) exp(-a^2), a = |u|/sqrt 2:
//     u >= 0:  u (1 - Q / 2)        u < 0:  u Q / 2
// The constants are folded for the vector unit: t = 1 / (1 + (p / sqrt 2) |u|), the
// coefficients carry the 1/2, and exp(-a^2) = 2^(-u^2 log2(e) / 2).
__device__ __forceinline__ float act_gelu_fast(float u) {
    const float t = __builtin_amdgcn_rcpf(fmaf(fabsf(u), 0.3275911f * 0.70710678118654752f, 1.0f));
    float poly = 0.5f * 1.061405429f;
    poly = fmaf(poly, t, 0.5f * -1.453152027f);
    poly = fmaf(poly, t, 0.5f * 1.421413741f);
    poly = fmaf(poly, t, 0.5f * -0.284496736f);
    poly = fmaf(poly, t, 0.5f * 0.254829592f);
    const float q = poly * t * __builtin_amdgcn_exp2f((u * -0.72134752044448170f) * u);
    return u >= 0.f ? u - u * q : u * q;
}

// silu(z) = z / (1 + e^-z) with the hardware exponential and reciprocal (about 1 ulp each).
__device__ __forceinline__ float silu_fast(float z) { return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }

__host__ __device__ constexpr int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ constexpr int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

}  // namespace moe
