// Bandwidth-bound kernels of the step: the frozen-run residual update, stream set-up,
// the sampler update and the DiT conditioning path.
#include "common.h"
#include "kernels.h"

namespace sgd {

// h <- (((h + D_1) + D_2) + ... + D_r), one coalesced float4 pass for a maximal run of
// consecutive frozen units; optional bf16 snapshots of h after individual units (U-ViT
// in-blocks feed their output to a long skip connection).  The cached updates are read four
// at a time, so every wave keeps four loads in flight per element group instead of one; the
// additions stay in stack order (bitwise the same result).
__device__ __forceinline__ void frozen_snap(const FrozenRun& f, int u, long i, const float4& v) {
    if (!f.snap[u]) return;
    if (f.snap_bf16) {
        bf16x4 s;
        s[0] = f2bf(v.x); s[1] = f2bf(v.y); s[2] = f2bf(v.z); s[3] = f2bf(v.w);
        ((bf16x4*)f.snap[u])[i] = s;
    } else {
        ((float4*)f.snap[u])[i] = v;
    }
}

__global__ __launch_bounds__(256) void frozen_run_kernel(FrozenRun f) {
    const long n4 = f.n / 4;
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n4; i += (long)gridDim.x * 256) {
        float4 v = ((const float4*)f.h)[i];
        int u = 0;
        for (; u + 4 <= f.r; u += 4) {
            float4 d[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) d[k] = ((const float4*)f.delta[u + k])[i];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                v.x = v.x + d[k].x;
                v.y = v.y + d[k].y;
                v.z = v.z + d[k].z;
                v.w = v.w + d[k].w;
                frozen_snap(f, u + k, i, v);
            }
        }
        for (; u < f.r; ++u) {
            const float4 d = ((const float4*)f.delta[u])[i];
            v.x = v.x + d.x;
            v.y = v.y + d.y;
            v.z = v.z + d.z;
            v.w = v.w + d.w;
            frozen_snap(f, u, i, v);
        }
        ((float4*)f.h)[i] = v;
    }
}

hipError_t launch_frozen_run(const FrozenRun& f, hipStream_t st) {
    const long n4 = f.n / 4;
    long blocks = (n4 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(frozen_run_kernel, dim3((unsigned)blocks), dim3(256), 0, st, f);
    return hipGetLastError();
}

// sinusoidal timestep embedding [cos(t f_i), sin(t f_i)], f_i = 10000^(-i/half); evaluated
// in double precision (a few thousand values per step)
__device__ __forceinline__ float temb(float t, int k, int dim) {
    const int half = dim / 2;
    const int i = k < half ? k : k - half;
    const double f = exp(-9.210340371976184 * (double)i / (double)half);
    const double arg = (double)t * f;
    return (float)(k < half ? cos(arg) : sin(arg));
}

__global__ __launch_bounds__(256) void stream_init_kernel(const float* z, float* h, int B, int N, int d,
                                                          int time_token, float t) {
    const long n4 = (long)B * N * d / 4;
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n4; i += (long)gridDim.x * 256) {
        float4 v = ((const float4*)z)[i];
        if (time_token) {
            const long e = i * 4;
            const long tok = (e / d) % N;
            if (tok == 0) {
                const int c = (int)(e % d);
                v.x = temb(t, c, d);
                v.y = temb(t, c + 1, d);
                v.z = temb(t, c + 2, d);
                v.w = temb(t, c + 3, d);
            }
        }
        ((float4*)h)[i] = v;
    }
}

hipError_t launch_stream_init(const float* z, float* h, int B, int N, int d, int time_token, float t,
                              hipStream_t st) {
    const long n4 = (long)B * N * d / 4;
    long blocks = (n4 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(stream_init_kernel, dim3((unsigned)blocks), dim3(256), 0, st, z, h, B, N, d,
                       time_token, t);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void state_update_kernel(float* z, const float* h, int B, int N, int d,
                                                           int r0, int r1, float alpha, float beta) {
    const int rows = r1 - r0;
    const long per_sample = (long)rows * d / 4;
    const long n4 = (long)B * per_sample;
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n4; i += (long)gridDim.x * 256) {
        const long b = i / per_sample;
        const long off = ((long)b * N + r0) * d / 4 + (i - b * per_sample);
        float4 zv = ((const float4*)z)[off];
        const float4 hv = ((const float4*)h)[off];
        zv.x = alpha * zv.x - beta * hv.x;
        zv.y = alpha * zv.y - beta * hv.y;
        zv.z = alpha * zv.z - beta * hv.z;
        zv.w = alpha * zv.w - beta * hv.w;
        ((float4*)z)[off] = zv;
    }
}

hipError_t launch_state_update(float* z, const float* h, int B, int N, int d, int r0, int r1, float alpha,
                               float beta, hipStream_t st) {
    const long n4 = (long)B * (r1 - r0) * d / 4;
    if (n4 <= 0) return hipSuccess;
    long blocks = (n4 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(state_update_kernel, dim3((unsigned)blocks), dim3(256), 0, st, z, h, B, N, d, r0, r1,
                       alpha, beta);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void cond_silu_kernel(const float* y, float* x, int B, int d, float t) {
    const long n = (long)B * d;
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const int k = (int)(i % d);
        x[i] = silu(temb(t, k, d) + y[i]);
    }
}

hipError_t launch_cond_silu(const float* y, float* x, int B, int d, float t, hipStream_t st) {
    const long n = (long)B * d;
    hipLaunchKernelGGL(cond_silu_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, y, x, B, d, t);
    return hipGetLastError();
}

// AdaLN modulation: mod[b, j] = sum_k x[b, k] W[j, k] + bias[j] for j < n_out.
// A workgroup owns 64 output features for every sample; the weight rows stream through
// LDS once in 64-wide k chunks.
template <typename WT>
__global__ __launch_bounds__(256) void adaln_mod_kernel(const float* x, const WT* W, const float* bias,
                                                        float* mod, int B, int d, int n_out) {
    constexpr int FJ = 64, KC = 64, SB = 32;  // features, k chunk, samples per pass
    __shared__ float sw[FJ][KC + 1];
    __shared__ float sx[SB][KC + 1];
    const int tid = threadIdx.x;
    const int j0 = blockIdx.x * FJ;
    const int f = tid & 63, sg = tid >> 6;  // feature, sample group (4 groups)
    for (int b0 = 0; b0 < B; b0 += SB) {
        float acc[SB / 4];
#pragma unroll
        for (int i = 0; i < SB / 4; ++i) acc[i] = 0.f;
        for (int k0 = 0; k0 < d; k0 += KC) {
            __syncthreads();
            for (int i = tid; i < FJ * KC; i += 256) {
                const int r = i / KC, c = i % KC;
                const int jj = j0 + r, kk = k0 + c;
                sw[r][c] = (jj < n_out && kk < d) ? ElemIO<WT>::load(W + (long)jj * d + kk) : 0.f;
            }
            for (int i = tid; i < SB * KC; i += 256) {
                const int r = i / KC, c = i % KC;
                const int bb = b0 + r, kk = k0 + c;
                sx[r][c] = (bb < B && kk < d) ? x[(long)bb * d + kk] : 0.f;
            }
            __syncthreads();
#pragma unroll 4
            for (int c = 0; c < KC; ++c) {
                const float w = sw[f][c];
#pragma unroll
                for (int i = 0; i < SB / 4; ++i) acc[i] = fmaf(sx[sg + 4 * i][c], w, acc[i]);
            }
        }
        const int j = j0 + f;
        if (j < n_out) {
#pragma unroll
            for (int i = 0; i < SB / 4; ++i) {
                const int bb = b0 + sg + 4 * i;
                if (bb < B) mod[(long)bb * n_out + j] = acc[i] + (bias ? bias[j] : 0.f);
            }
        }
    }
}

hipError_t launch_adaln_mod(int dtype, const float* x, const void* W, const float* bias, float* mod, int B,
                            int d, int n_out, hipStream_t st) {
    dim3 grid((n_out + 63) / 64), block(256);
    if (dtype == 1)
        hipLaunchKernelGGL(adaln_mod_kernel<bf16>, grid, block, 0, st, x, (const bf16*)W, bias, mod, B, d, n_out);
    else
        hipLaunchKernelGGL(adaln_mod_kernel<float>, grid, block, 0, st, x, (const float*)W, bias, mod, B, d,
                           n_out);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void to_bf16_kernel(const float* x, bf16* y, long n) {
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long)gridDim.x * 256) y[i] = f2bf(x[i]);
}

hipError_t launch_to_bf16(const float* x, void* y, long n, hipStream_t st) {
    long blocks = (n + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(to_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, st, x, (bf16*)y, n);
    return hipGetLastError();
}

}  // namespace sgd
