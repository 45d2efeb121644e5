// Bottleneck activations of the branch nonlinearity.
//
// The CosNet of Sec. 3.2 Eq. 2 applies cos twice, with the rank-space mixing
// M between the two applications.  The activation ablation (Sec. 4.4, Table 5)
// swaps cos for tanh, LeakyReLU or GELU and also runs each one as a single
// application without M.  Every application keeps the per-rank affine map
// w (.) h + p in front of f, so w = 1, p = 0 is the bare activation.
// LeakyReLU has negative slope 0.01 and GELU is the exact a Phi(a), with Phi
// the standard normal distribution function.
#pragma once

#include <hip/hip_runtime.h>

namespace noble {

enum class Act : int { Cos = 0, Tanh = 1, Leaky = 2, Gelu = 3 };

constexpr float kLeakySlope = 0.01f;

// sin and cos of x: reduction to one period in turns (x / 2 pi minus the
// nearest integer), then the hardware v_sin_f32 / v_cos_f32, which take their
// argument in turns.  Absolute error about 1e-6 for |x| in the range the
// layer produces, far below the bf16 operand rounding that follows.
__device__ __forceinline__ float turns(float x) {
    const float t = x * 0.15915494309189535f;
    return t - __builtin_rintf(t);
}
__device__ __forceinline__ float fast_cos(float x) { return __builtin_amdgcn_cosf(turns(x)); }
__device__ __forceinline__ void fast_sincos(float x, float& s, float& c) {
    const float t = turns(x);
    s = __builtin_amdgcn_sinf(t);
    c = __builtin_amdgcn_cosf(t);
}

// Standard normal distribution function as erfc(-a / sqrt 2) / 2: the form
// 1 + erf(a / sqrt 2) loses every digit to cancellation once a is a few units
// below zero, erfc keeps the relative accuracy of the tail.
__device__ __forceinline__ float std_normal_cdf(float a) { return 0.5f * erfcf(-a * 0.70710678118654752f); }

// f(a).  FAST selects the turn-reduced hardware cosine (bf16 path); the
// float32 path uses the device math library throughout.
template <Act F, bool FAST>
__device__ __forceinline__ float act_value(float a) {
    if constexpr (F == Act::Cos) {
        if constexpr (FAST) return fast_cos(a);
        else return cosf(a);
    } else if constexpr (F == Act::Tanh) {
        return tanhf(a);
    } else if constexpr (F == Act::Leaky) {
        return a > 0.f ? a : kLeakySlope * a;
    } else {
        return a * std_normal_cdf(a);
    }
}

// f(a) and f'(a): d cos = -sin; d tanh = 1 - tanh^2; LeakyReLU's slope is 1
// above zero and kLeakySlope otherwise; d (a Phi(a)) = Phi(a) + a phi(a), phi
// the standard normal density.  1 - tanh^2 is evaluated as sech^2 =
// 4 e / (1 + e)^2 with e = exp(-2 |a|): taken as 1 - t t from a rounded t it
// cancels where tanh saturates (about 10% relative error at |a| = 8 in
// float32), and the gradient of a saturated unit would carry that error.
template <Act F, bool FAST>
__device__ __forceinline__ void act_value_slope(float a, float& f, float& d) {
    if constexpr (F == Act::Cos) {
        float s, c;
        if constexpr (FAST) fast_sincos(a, s, c);
        else sincosf(a, &s, &c);
        f = c;
        d = -s;
    } else if constexpr (F == Act::Tanh) {
        const float e = expf(-2.f * fabsf(a));
        const float q = 1.f + e;
        f = tanhf(a);
        d = 4.f * e / (q * q);
    } else if constexpr (F == Act::Leaky) {
        f = a > 0.f ? a : kLeakySlope * a;
        d = a > 0.f ? 1.f : kLeakySlope;
    } else {
        const float cdf = std_normal_cdf(a);
        f = a * cdf;
        d = cdf + a * 0.39894228040143268f * expf(-0.5f * a * a);
    }
}

}  // namespace noble
