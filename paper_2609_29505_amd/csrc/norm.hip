// Pre-norms of the residual branches: RMSNorm, LayerNorm, and LayerNorm with AdaLN
// modulation fused (y = LN(x) (1 + scale_b) + shift_b).  One 256-thread workgroup per row;
// the row stays in registers between the statistics and the output pass.
#include "common.h"
#include "kernels.h"

namespace sgd {

__device__ __forceinline__ float block_sum(float v, float* red) {
    v = warp_sum(v);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) t += red[i];
    return t;
}

template <typename OutT, int VPT>
__global__ __launch_bounds__(256) void norm_kernel(NormArgs a) {
    __shared__ float red[4];
    const int row = blockIdx.x;
    const float* x = a.x + (long)row * a.d;
    const int nvec = a.d / 4;
    float4 v[VPT];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int c = threadIdx.x + i * 256;
        v[i] = c < nvec ? ((const float4*)x)[c] : make_float4(0.f, 0.f, 0.f, 0.f);
        s += (a.kind == 0) ? (v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w)
                           : (v[i].x + v[i].y + v[i].z + v[i].w);
    }
    s = block_sum(s, red);
    const float invd = 1.0f / (float)a.d;
    float mean = 0.f, rstd;
    if (a.kind == 0) {
        rstd = 1.0f / sqrtf(s * invd + a.eps);
    } else {
        mean = s * invd;
        float q = 0.f;
#pragma unroll
        for (int i = 0; i < VPT; ++i) {
            const int c = threadIdx.x + i * 256;
            if (c < nvec) {
                const float dx = v[i].x - mean, dy = v[i].y - mean, dz = v[i].z - mean, dw = v[i].w - mean;
                q += dx * dx + dy * dy + dz * dz + dw * dw;
            }
        }
        q = block_sum(q, red);
        rstd = 1.0f / sqrtf(q * invd + a.eps);
    }
    OutT* y = (OutT*)a.y + (long)row * a.d;
    const long mrow = a.kind == 2 ? (long)(row / a.ntok) * a.mod_ld : 0;
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int c = threadIdx.x + i * 256;
        if (c >= nvec) continue;
        float r[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int col = c * 4 + e;
            float t = (r[e] - mean) * rstd;
            if (a.kind == 0) t = t * a.w[col];
            else if (a.kind == 1) t = t * a.w[col] + a.b[col];
            else t = t * (1.0f + a.scale[mrow + col]) + a.shift[mrow + col];
            ElemIO<OutT>::store(y + col, t);
        }
    }
}

hipError_t launch_norm(int dtype, const NormArgs& a, hipStream_t st) {
    const int nvec = a.d / 4;
    const int vpt = (nvec + 255) / 256;
    dim3 grid(a.M), block(256);
#define NORM_CASE(V)                                                                              \
    if (vpt <= V) {                                                                               \
        if (dtype == 1) hipLaunchKernelGGL((norm_kernel<bf16, V>), grid, block, 0, st, a);       \
        else hipLaunchKernelGGL((norm_kernel<float, V>), grid, block, 0, st, a);                 \
        return hipGetLastError();                                                                 \
    }
    NORM_CASE(1)
    NORM_CASE(2)
    NORM_CASE(4)
    NORM_CASE(8)
#undef NORM_CASE
    return hipErrorInvalidValue;
}

}  // namespace sgd
