// Pre-norms of the residual branches: RMSNorm, LayerNorm, and LayerNorm with AdaLN
// modulation fused (y = LN(x) (1 + scale_b) + shift_b).
#include "common.h"
#include "kernels.h"

namespace sgd {

// WPR waves per row (one for many rows, four for few long rows), 256-thread workgroups: the
// row's float4 groups stay in registers between the statistics (wave reductions, combined
// across the row's waves through LDS) and the output pass; gains, shifts and modulation
// vectors are read as float4, bf16 outputs stored four at a time.
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

// sum over the WPR waves of one row (every wave of the workgroup reaches the barrier)
template <int WPR>
__device__ __forceinline__ float row_sum(float v, float* red) {
    v = warp_sum(v);
    if (WPR == 1) return v;
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < WPR; ++i) t += red[(w / WPR) * WPR + i];
    return t;
}

template <typename OutT, int VPL, int WPR>
__global__ __launch_bounds__(256) void norm_kernel(NormArgs a) {
    constexpr int TPR = 64 * WPR;  // threads per row
    __shared__ float red[4];
    const int t = threadIdx.x % TPR;
    const int row = blockIdx.x * (256 / TPR) + threadIdx.x / TPR;
    const bool live = row < a.M;  // dead rows still join the row_sum barriers
    const float* x = a.x + (long)(live ? row : 0) * a.d;
    const int nvec = a.d / 4;
    float4 v[VPL];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
        const int c = t + i * TPR;
        v[i] = (live && c < nvec) ? ((const float4*)x)[c] : make_float4(0.f, 0.f, 0.f, 0.f);
        s += (a.kind == 0) ? (v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w)
                           : (v[i].x + v[i].y + v[i].z + v[i].w);
    }
    s = row_sum<WPR>(s, red);
    const float invd = 1.0f / (float)a.d;
    float mean = 0.f, rstd;
    if (a.kind == 0) {
        rstd = 1.0f / sqrtf(s * invd + a.eps);
    } else {
        mean = s * invd;
        float q = 0.f;
#pragma unroll
        for (int i = 0; i < VPL; ++i) {
            const int c = t + i * TPR;
            if (c < nvec) {
                const float dx = v[i].x - mean, dy = v[i].y - mean, dz = v[i].z - mean, dw = v[i].w - mean;
                q += dx * dx + dy * dy + dz * dz + dw * dw;
            }
        }
        q = row_sum<WPR>(q, red);
        rstd = 1.0f / sqrtf(q * invd + a.eps);
    }
    if (!live) return;
    OutT* y = (OutT*)a.y + (long)row * a.d;
    const long mrow = a.kind == 2 ? (long)(row / a.ntok) * a.mod_ld : 0;
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
        const int c = t + i * TPR;
        if (c >= nvec) continue;
        float o[4] = {(v[i].x - mean) * rstd, (v[i].y - mean) * rstd, (v[i].z - mean) * rstd, (v[i].w - mean) * rstd};
        if (a.kind == 0) {
            const float4 w = ((const float4*)a.w)[c];
            o[0] *= w.x; o[1] *= w.y; o[2] *= w.z; o[3] *= w.w;
        } else if (a.kind == 1) {
            const float4 w = ((const float4*)a.w)[c], b = ((const float4*)a.b)[c];
            o[0] = o[0] * w.x + b.x; o[1] = o[1] * w.y + b.y; o[2] = o[2] * w.z + b.z; o[3] = o[3] * w.w + b.w;
        } else {
            const float4 sc = *(const float4*)(a.scale + mrow + c * 4), sh = *(const float4*)(a.shift + mrow + c * 4);
            o[0] = o[0] * (1.0f + sc.x) + sh.x; o[1] = o[1] * (1.0f + sc.y) + sh.y;
            o[2] = o[2] * (1.0f + sc.z) + sh.z; o[3] = o[3] * (1.0f + sc.w) + sh.w;
        }
        store4<OutT>(y + c * 4, o[0], o[1], o[2], o[3]);
    }
}

template <int WPR>
static hipError_t launch_norm_wpr(int dtype, const NormArgs& a, hipStream_t st) {
    const int vpl = (a.d / 4 + 64 * WPR - 1) / (64 * WPR);
    dim3 grid((a.M + (4 / WPR) - 1) / (4 / WPR)), block(256);
#define NORM_CASE(V)                                                                              \
    if (vpl <= V) {                                                                               \
        if (dtype == 1) hipLaunchKernelGGL((norm_kernel<bf16, V, WPR>), grid, block, 0, st, a);  \
        else hipLaunchKernelGGL((norm_kernel<float, V, WPR>), grid, block, 0, st, a);            \
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

hipError_t launch_norm(int dtype, const NormArgs& a, hipStream_t st) {
    // few rows (LLaDA: 1024): four waves per row.  Many rows: two waves per row when the row's
    // float4 groups split evenly over 128 lanes (U-ViT, d = 1024: 13.9 -> 12.5 us), else one
    // (DiT d = 1152 and SDXL d = 1280 measured slower with two: uneven lanes)
    if (a.M < 4096) return launch_norm_wpr<4>(dtype, a, st);
    return (a.d / 4) % 128 == 0 ? launch_norm_wpr<2>(dtype, a, st) : launch_norm_wpr<1>(dtype, a, st);
}

}  // namespace sgd
