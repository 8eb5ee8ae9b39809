// Internal helpers shared by the HIP kernels and the host launcher (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace sgd {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf2f(bf16 x) {
    return __uint_as_float(((uint32_t)__builtin_bit_cast(uint16_t, x)) << 16);
}
// float -> bf16, round to nearest even (gfx950 v_cvt_pk_bf16_f32)
__device__ __forceinline__ bf16 f2bf(float x) { return (bf16)x; }

template <typename T> struct ElemIO;
template <> struct ElemIO<float> {
    __device__ static __forceinline__ float load(const float* p) { return *p; }
    __device__ static __forceinline__ void store(float* p, float v) { *p = v; }
};
template <> struct ElemIO<bf16> {
    __device__ static __forceinline__ float load(const bf16* p) { return bf2f(*p); }
    __device__ static __forceinline__ void store(bf16* p, float v) { *p = f2bf(v); }
};

// Activations of the MLP epilogues, built on the hardware exponential (v_exp_f32) and
// reciprocal (v_rcp_f32); errors are a few 1e-7 absolute, far below the bf16 outputs'
// resolution and the fp32 workload's tolerance.
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }
// erf by Abramowitz & Stegun, Handbook of Mathematical Functions, 7.1.26 (|error| <= 1.5e-7):
// erf(x) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) exp(-x^2), t = 1 / (1 + p x), x >= 0
__device__ __forceinline__ float erf_as(float x) {
    const float ax = fabsf(x);
    const float t = fast_rcp(1.0f + 0.3275911f * ax);
    const float poly = t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
    const float y = 1.0f - poly * __expf(-ax * ax);
    return copysignf(y, x);
}
__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.0f + erf_as(x * 0.70710678118654752f)); }
// 0.5 x (1 + tanh(u)) = x / (1 + exp(-2u)), u = sqrt(2/pi) (x + 0.044715 x^3); the exponent
// -2u log2(e) = x (c0 + c1 x^2) goes straight to v_exp_f32 (exp2): five VALU operations plus
// the exponential and the reciprocal.  Limits: exp2 -> inf gives x * 0, exp2 -> 0 gives x.
__device__ __forceinline__ float gelu_tanh(float x) {
    const float c0 = -2.302208198144325f;    // -2 sqrt(2/pi) log2(e)
    const float c1 = -0.1029432395800235f;   // -2 sqrt(2/pi) 0.044715 log2(e)
    return x * fast_rcp(1.0f + __builtin_amdgcn_exp2f(x * fmaf(c1, x * x, c0)));
}
__device__ __forceinline__ float silu(float x) { return x * fast_rcp(1.0f + __expf(-x)); }

__device__ __forceinline__ float warp_sum(float v) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
__device__ __forceinline__ double warp_sum(double v) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
__device__ __forceinline__ float warp_max(float v) {
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

inline int cdiv(long a, long b) { return (int)((a + b - 1) / b); }

__device__ __forceinline__ float apply_act(int act, float x) {
    switch (act) {
        case ACT_GELU_ERF: return gelu_erf(x);
        case ACT_GELU_TANH: return gelu_tanh(x);
        case ACT_SILU: return silu(x);
        default: return x;
    }
}

}  // namespace sgd
