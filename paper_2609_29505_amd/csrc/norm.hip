// Pre-norms of the residual branches: RMSNorm, LayerNorm, and LayerNorm with AdaLN
// modulation fused (y = LN(x) (1 + scale_b) + shift_b).
#include "common.h"
#include "kernels.h"

namespace sgd {

// One wave per row (four rows per workgroup): the row's float4 groups stay in registers
// between the statistics (wave reductions, no workgroup barrier) and the output pass; gains,
// shifts and modulation vectors are read as float4, bf16 outputs stored four at a time.
template <typename OutT>
__device__ __forceinline__ void store4(OutT* p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store4<float>(float* p, float a, float b, float c, float d) {
    *(float4*)p = make_float4(a, b, c, d);
}
template <>
__device__ __forceinline__ void store4<bf16>(bf16* p, float a, float b, float c, float d) {
    bf16x4 s;
    s[0] = f2bf(a); s[1] = f2bf(b); s[2] = f2bf(c); s[3] = f2bf(d);
    *(bf16x4*)p = s;
}

template <typename OutT, int VPL>
__global__ __launch_bounds__(256) void norm_kernel(NormArgs a) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= a.M) return;  // whole waves: no barrier below
    const float* x = a.x + (long)row * a.d;
    const int nvec = a.d / 4;
    float4 v[VPL];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
        const int c = lane + i * 64;
        v[i] = c < nvec ? ((const float4*)x)[c] : make_float4(0.f, 0.f, 0.f, 0.f);
        s += (a.kind == 0) ? (v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w)
                           : (v[i].x + v[i].y + v[i].z + v[i].w);
    }
    s = warp_sum(s);
    const float invd = 1.0f / (float)a.d;
    float mean = 0.f, rstd;
    if (a.kind == 0) {
        rstd = 1.0f / sqrtf(s * invd + a.eps);
    } else {
        mean = s * invd;
        float q = 0.f;
#pragma unroll
        for (int i = 0; i < VPL; ++i) {
            const int c = lane + i * 64;
            if (c < nvec) {
                const float dx = v[i].x - mean, dy = v[i].y - mean, dz = v[i].z - mean, dw = v[i].w - mean;
                q += dx * dx + dy * dy + dz * dz + dw * dw;
            }
        }
        q = warp_sum(q);
        rstd = 1.0f / sqrtf(q * invd + a.eps);
    }
    OutT* y = (OutT*)a.y + (long)row * a.d;
    const long mrow = a.kind == 2 ? (long)(row / a.ntok) * a.mod_ld : 0;
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
        const int c = lane + i * 64;
        if (c >= nvec) continue;
        float t[4] = {(v[i].x - mean) * rstd, (v[i].y - mean) * rstd, (v[i].z - mean) * rstd, (v[i].w - mean) * rstd};
        if (a.kind == 0) {
            const float4 w = ((const float4*)a.w)[c];
            t[0] *= w.x; t[1] *= w.y; t[2] *= w.z; t[3] *= w.w;
        } else if (a.kind == 1) {
            const float4 w = ((const float4*)a.w)[c], b = ((const float4*)a.b)[c];
            t[0] = t[0] * w.x + b.x; t[1] = t[1] * w.y + b.y; t[2] = t[2] * w.z + b.z; t[3] = t[3] * w.w + b.w;
        } else {
            const float4 sc = *(const float4*)(a.scale + mrow + c * 4), sh = *(const float4*)(a.shift + mrow + c * 4);
            t[0] = t[0] * (1.0f + sc.x) + sh.x; t[1] = t[1] * (1.0f + sc.y) + sh.y;
            t[2] = t[2] * (1.0f + sc.z) + sh.z; t[3] = t[3] * (1.0f + sc.w) + sh.w;
        }
        store4<OutT>(y + c * 4, t[0], t[1], t[2], t[3]);
    }
}

hipError_t launch_norm(int dtype, const NormArgs& a, hipStream_t st) {
    const int nvec = a.d / 4;
    const int vpl = (nvec + 63) / 64;
    dim3 grid((a.M + 3) / 4), block(256);
#define NORM_CASE(V)                                                                              \
    if (vpl <= V) {                                                                               \
        if (dtype == 1) hipLaunchKernelGGL((norm_kernel<bf16, V>), grid, block, 0, st, a);       \
        else hipLaunchKernelGGL((norm_kernel<float, V>), grid, block, 0, st, a);                 \
        return hipGetLastError();                                                                 \
    }
    NORM_CASE(2)
    NORM_CASE(4)
    NORM_CASE(5)
    NORM_CASE(8)
    NORM_CASE(16)
    NORM_CASE(32)
#undef NORM_CASE
    return hipErrorInvalidValue;
}

}  // namespace sgd
