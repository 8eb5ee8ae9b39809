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

// Squared norms for the input-aware baselines (drift of a unit's input, deviation of an
// output): per block, sum (x - y)^2 and sum x^2 over the selected rows, float4 loads, fp64
// accumulation, wave then workgroup reduction in a fixed order, so repeated runs give the
// same bits.  A thread's copy store follows its own loads of the same element (copy may be y).
__global__ __launch_bounds__(256) void sumsq_kernel(const float* x, const float* y, float* copy, int B, int N,
                                                    int d, int r0, int r1, int have_y, double* partial) {
    const long per_sample = (long)(r1 - r0) * d / 4;
    const long n4 = (long)B * per_sample;
    double a = 0.0, b = 0.0;
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n4; i += (long)gridDim.x * 256) {
        const long s = i / per_sample;
        const long off = ((long)s * N + r0) * d / 4 + (i - s * per_sample);
        const float4 v = ((const float4*)x)[off];
        if (have_y) {
            const float4 p = ((const float4*)y)[off];
            // differences of fp32 values are exact in fp64
            const double dx = (double)v.x - p.x, dy = (double)v.y - p.y, dz = (double)v.z - p.z,
                         dw = (double)v.w - p.w;
            a += dx * dx + dy * dy + dz * dz + dw * dw;
        }
        b += (double)v.x * v.x + (double)v.y * v.y + (double)v.z * v.z + (double)v.w * v.w;
        if (copy) ((float4*)copy)[off] = v;
    }
    __shared__ double red[2][4];
    a = warp_sum(a);
    b = warp_sum(b);
    const int wv = threadIdx.x / 64;
    if ((threadIdx.x & 63) == 0) {
        red[0][wv] = a;
        red[1][wv] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        partial[2 * blockIdx.x] = ((red[0][0] + red[0][1]) + red[0][2]) + red[0][3];
        partial[2 * blockIdx.x + 1] = ((red[1][0] + red[1][1]) + red[1][2]) + red[1][3];
    }
}

hipError_t launch_sumsq(const float* x, const float* y, float* copy, int B, int N, int d, int r0, int r1,
                        int have_y, double* partial, hipStream_t st) {
    hipLaunchKernelGGL(sumsq_kernel, dim3(kSumBlocks), dim3(256), 0, st, x, y, copy, B, N, d, r0, r1, have_y,
                       partial);
    return hipGetLastError();
}

// one workgroup per tensor: kSumBlocks partial pairs -> one pair, fixed order
__global__ __launch_bounds__(256) void sumsq_finish_kernel(const double* partial, double* out) {
    const double* p = partial + (size_t)blockIdx.x * 2 * kSumBlocks;
    double a = 0.0, b = 0.0;
    for (int i = threadIdx.x; i < kSumBlocks; i += 256) {
        a += p[2 * i];
        b += p[2 * i + 1];
    }
    __shared__ double red[2][4];
    a = warp_sum(a);
    b = warp_sum(b);
    const int wv = threadIdx.x / 64;
    if ((threadIdx.x & 63) == 0) {
        red[0][wv] = a;
        red[1][wv] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        out[2 * blockIdx.x] = ((red[0][0] + red[0][1]) + red[0][2]) + red[0][3];
        out[2 * blockIdx.x + 1] = ((red[1][0] + red[1][1]) + red[1][2]) + red[1][3];
    }
}

hipError_t launch_sumsq_finish(const double* partial, int count, double* out, hipStream_t st) {
    hipLaunchKernelGGL(sumsq_finish_kernel, dim3(count), dim3(256), 0, st, partial, out);
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
// mod[b, j] = sum_k x[b, k] W[j, k] + bias[j]: the DiT AdaLN modulation (6 d outputs per
// sample) in fp32 from the fp32 SiLU(c) rows and the stored weights.  A workgroup computes a
// 64-feature x 32-sample tile; thread (f, s) holds features 4f..4f+3 of samples s, s + 16, so
// each 4-deep k step is six 16-byte LDS reads for 32 FMAs.  LDS rows are padded to 68 floats
// (16-byte aligned, conflict-free 16-byte reads); the next k chunk is prefetched into
// registers (weights 16 bytes per thread, activations two float4 per thread).
template <typename WT> struct Wvec;
template <> struct Wvec<bf16> {
    typedef u32x4 raw;  // 8 weights
    static constexpr int PER = 8;
    __device__ static void expand(const raw& r, float* o) {
        for (int e = 0; e < 4; ++e) {
            o[2 * e] = __uint_as_float(r[e] << 16);
            o[2 * e + 1] = __uint_as_float(r[e] & 0xffff0000u);
        }
    }
};
template <> struct Wvec<float> {
    typedef f32x4 raw;  // 4 weights
    static constexpr int PER = 4;
    __device__ static void expand(const raw& r, float* o) {
        for (int e = 0; e < 4; ++e) o[e] = r[e];
    }
};

template <typename WT>
__global__ __launch_bounds__(256) void adaln_mod_kernel(const float* x, ModBatch mb, int B, int d, int n_out) {
    const WT* W = (const WT*)mb.W[blockIdx.z];
    const float* bias = mb.bias[blockIdx.z];
    float* mod = mb.mod[blockIdx.z];
    constexpr int FJ = 64, SB = 32, KC = 64, LD = KC + 4;
    constexpr int WV = Wvec<WT>::PER;                     // weights per vector load
    constexpr int WLOADS = FJ * KC / WV / 256;            // weight vectors per thread per chunk
    __shared__ __attribute__((aligned(16))) float sw[FJ * LD];
    __shared__ __attribute__((aligned(16))) float sx[SB * LD];
    const int tid = threadIdx.x;
    const int j0 = blockIdx.x * FJ, b0 = blockIdx.y * SB;
    const int f4 = (tid & 15) * 4, s0 = tid >> 4;  // features f4..f4+3, samples s0, s0 + 16

    typename Wvec<WT>::raw rw[WLOADS];
    f32x4 rx[2];
    auto gload = [&](int k0) {
#pragma unroll
        for (int t = 0; t < WLOADS; ++t) {
            const int i = tid + t * 256;
            const int r = i / (KC / WV), c = (i % (KC / WV)) * WV;
            const int jj = min(j0 + r, n_out - 1);  // clamped rows are never stored
            rw[t] = *(const typename Wvec<WT>::raw*)(W + (long)jj * d + k0 + c);
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int i = tid + t * 256;
            const int r = i / (KC / 4), c = (i % (KC / 4)) * 4;
            const int bb = min(b0 + r, B - 1);
            rx[t] = *(const f32x4*)(x + (long)bb * d + k0 + c);
        }
    };
    auto lstore = [&]() {
#pragma unroll
        for (int t = 0; t < WLOADS; ++t) {
            const int i = tid + t * 256;
            const int r = i / (KC / WV), c = (i % (KC / WV)) * WV;
            float w[WV];
            Wvec<WT>::expand(rw[t], w);
#pragma unroll
            for (int e = 0; e < WV; e += 4) *(f32x4*)(sw + r * LD + c + e) = f32x4{w[e], w[e + 1], w[e + 2], w[e + 3]};
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int i = tid + t * 256;
            const int r = i / (KC / 4), c = (i % (KC / 4)) * 4;
            *(f32x4*)(sx + r * LD + c) = rx[t];
        }
    };

    float acc[4][2] = {};
    gload(0);
    for (int k0 = 0; k0 < d; k0 += KC) {
        __syncthreads();  // the previous chunk has been consumed
        lstore();
        __syncthreads();
        if (k0 + KC < d) gload(k0 + KC);
#pragma unroll 4
        for (int c = 0; c < KC; c += 4) {
            f32x4 w[4], xv[2];
#pragma unroll
            for (int q = 0; q < 4; ++q) w[q] = *(const f32x4*)(sw + (f4 + q) * LD + c);
            xv[0] = *(const f32x4*)(sx + s0 * LD + c);
            xv[1] = *(const f32x4*)(sx + (s0 + 16) * LD + c);
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int s = 0; s < 2; ++s)
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[q][s] = fmaf(xv[s][e], w[q][e], acc[q][s]);
        }
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int bb = b0 + s0 + 16 * s;
        if (bb >= B) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int j = j0 + f4 + q;
            if (j < n_out) mod[(long)bb * n_out + j] = acc[q][s] + (bias ? bias[j] : 0.f);
        }
    }
}

// bf16 weights: the same product on the matrix cores.  SiLU(c) is fp32; it is split into
// three bf16 parts, x = hi + mid + lo (each part the round-to-nearest-even bf16 of what the
// previous parts leave: x - hi has at most 16 significant bits and x - hi - mid at most 8, so
// hi + mid + lo == x exactly), and bf16 x bf16 products are exact in fp32: the MFMAs sum the
// fp32 products of the FMA kernel above, in another order.  A workgroup owns 32 features x 32
// samples (v_mfma_f32_32x32x16_bf16: A = the x parts, one sample per lane row; B = the weight
// rows, one feature per lane column) and walks k in chunks of 256: the chunk's 32 weight rows
// and 32 x rows are read with 16-byte loads in which every wave covers whole 128-byte lines
// (reading the MFMA layout straight from memory touches 32 lines per load instruction, and the
// kernel was bound by that request rate), stored to LDS, and wave w takes the chunk's k step w.
// A thread issues the loads of up to kModG chunks before storing the first (one memory round
// trip for d <= 1536).  The partial tiles of the sixteen waves are summed in LDS in wave order
// (deterministic).
constexpr int kModWaves = 16, kModKC = 16 * kModWaves, kModG = 6;
constexpr int kModWS = kModKC * 2 + 16, kModXS = kModKC * 4 + 16;  // padded LDS row bytes
__global__ __launch_bounds__(kModWaves * 64) void adaln_mod_mfma_kernel(const float* x, ModBatch mb, int B, int d,
                                                                        int n_out) {
    const bf16* W = (const bf16*)mb.W[blockIdx.z];
    const float* bias = mb.bias[blockIdx.z];
    float* mod = mb.mod[blockIdx.z];
    __shared__ __attribute__((aligned(16))) char sw[32 * kModWS];
    __shared__ __attribute__((aligned(16))) char sx[32 * kModXS];
    __shared__ float red[kModWaves][32 * 32];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int j0 = blockIdx.x * 32, b0 = blockIdx.y * 32;
    // loads of a chunk: weight row tid / 32, bytes 16 (tid % 32) of its 512; x rows tid / 64
    // and tid / 64 + 16, bytes 16 (tid % 64) of their 1024
    const int wr = tid >> 5, wc = (tid & 31) * 16, xr = tid >> 6, xc = (tid & 63) * 16;
    const bool win = j0 + wr < n_out, xin0 = b0 + xr < B, xin1 = b0 + xr + 16 < B;
    const char* wsrc = (const char*)(W + (long)(win ? j0 + wr : 0) * d) + wc;
    const char* xsrc0 = (const char*)(x + (long)(xin0 ? b0 + xr : 0) * d) + xc;
    const char* xsrc1 = (const char*)(x + (long)(xin1 ? b0 + xr + 16 : 0) * d) + xc;
    // fragments: lane l reads row l % 32 at k offset 8 (l / 32) of the wave's k step
    const int col = lane & 31, fk = wave * 16 + (lane >> 5) * 8;
    const char* fw = sw + col * kModWS + fk * 2;
    const char* fx = sx + col * kModXS + fk * 4;
    const int nch = (d + kModKC - 1) / kModKC;
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    for (int c0 = 0; c0 < nch; c0 += kModG) {
        u32x4 rw[kModG], rx0[kModG], rx1[kModG];
        const u32x4 z{0u, 0u, 0u, 0u};
#pragma unroll
        for (int g = 0; g < kModG; ++g) {
            const int kb = (c0 + g) * kModKC;  // (d is a multiple of 16: a load lies wholly inside or past d)
            const bool kw = c0 + g < nch && kb + wc / 2 < d, kx = c0 + g < nch && kb + xc / 4 < d;
            rw[g] = win && kw ? *(const u32x4*)(wsrc + (long)kb * 2) : z;
            rx0[g] = xin0 && kx ? *(const u32x4*)(xsrc0 + (long)kb * 4) : z;
            rx1[g] = xin1 && kx ? *(const u32x4*)(xsrc1 + (long)kb * 4) : z;
        }
#pragma unroll
        for (int g = 0; g < kModG; ++g) {
            if (c0 + g >= nch) break;
            __syncthreads();  // every wave has read the previous chunk's fragments
            *(u32x4*)(sw + wr * kModWS + wc) = rw[g];
            *(u32x4*)(sx + xr * kModXS + xc) = rx0[g];
            *(u32x4*)(sx + (xr + 16) * kModXS + xc) = rx1[g];
            __syncthreads();
            if ((c0 + g) * kModKC + wave * 16 < d) {
                const bf16x8 wf = *(const bf16x8*)fw;
                const f32x4 xa = *(const f32x4*)fx, xb = *(const f32x4*)(fx + 16);
                bf16x8 hi, mid, lo;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float v = e < 4 ? xa[e] : xb[e - 4];
                    hi[e] = f2bf(v);
                    const float r1 = v - bf2f(hi[e]);
                    mid[e] = f2bf(r1);
                    lo[e] = f2bf(r1 - bf2f(mid[e]));
                }
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lo, wf, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(mid, wf, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(hi, wf, acc, 0, 0, 0);
            }
        }
    }
    // lane l holds feature column l % 32 and, for register r, sample row
    // (r / 4) * 8 + (l / 32) * 4 + r % 4 of the tile
#pragma unroll
    for (int r = 0; r < 16; ++r) red[wave][((r >> 2) * 8 + (lane >> 5) * 4 + (r & 3)) * 32 + col] = acc[r];
    __syncthreads();
    const int i = tid >> 5, j = tid & 31;  // one output per thread: sample i, feature j
    float v = red[0][tid];
#pragma unroll
    for (int w = 1; w < kModWaves; ++w) v += red[w][tid];
    if (b0 + i < B && j0 + j < n_out) mod[(long)(b0 + i) * n_out + j0 + j] = v + (bias ? bias[j0 + j] : 0.f);
}

// Wide variant for many output features (the DiT modulation, 6 d outputs per block): a
// workgroup owns 32 samples x 32 WV features and each of its WV waves owns 32 features over
// the whole k range, so no partial tiles are exchanged and SiLU(c) is read once per 32 WV
// features.  k goes in 64-deep chunks through LDS: x split once into its three bf16 parts by
// the thread that loads it, the weight rows with 16-byte loads covering whole 128-byte lines;
// every thread keeps the loads of kWideG chunks in flight.  Per output the products go into
// one accumulator, k step by k step (lo, mid, hi each), whatever WV is: the launcher picks WV
// for the grid size and the results do not depend on it.
constexpr int kWideKC = 64, kWideG = 3;
constexpr int kWideRS = kWideKC * 2 + 16;  // padded LDS row bytes (bf16 weights and x parts)
template <int WV>
__global__ __launch_bounds__(WV * 64) void adaln_mod_wide_kernel(const float* x, ModBatch mb, int B, int d,
                                                                 int n_out) {
    constexpr int NT = WV * 64, FW = WV * 32, XP = 512 / NT;  // x passes per chunk
    __shared__ __attribute__((aligned(16))) char sw[FW * kWideRS];
    __shared__ __attribute__((aligned(16))) char sx[3 * 32 * kWideRS];
    const bf16* W = (const bf16*)mb.W[blockIdx.z];
    const float* bias = mb.bias[blockIdx.z];
    float* mod = mb.mod[blockIdx.z];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int j0 = blockIdx.x * FW, b0 = blockIdx.y * 32;
    // loads of a chunk: x rows tid / 16 + (NT / 16) p, floats 4 (tid % 16) .. + 3 of their 64;
    // weight rows tid / 8 + (NT / 8) i, bf16 8 (tid % 8) .. + 7 of their 64
    const int xr = tid >> 4, xe = (tid & 15) * 4, wr = tid >> 3, we = (tid & 7) * 8;
    bool xin[XP], win[4];
    const float* xsrc[XP];
    const bf16* wsrc[4];
#pragma unroll
    for (int p = 0; p < XP; ++p) {
        const int b = b0 + xr + (NT / 16) * p;
        xin[p] = b < B;
        xsrc[p] = x + (long)(xin[p] ? b : 0) * d + xe;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int j = j0 + wr + (NT / 8) * i;
        win[i] = j < n_out;
        wsrc[i] = W + (long)(win[i] ? j : 0) * d + we;
    }
    // fragments: lane l takes x parts of sample l % 32 and weight row 32 wave + l % 32, at k
    // offset 8 (l / 32) of each 16-deep step
    const int col = lane & 31, kh = (lane >> 5) * 8;
    const char* fw = sw + (wave * 32 + col) * kWideRS + kh * 2;
    const char* fx = sx + col * kWideRS + kh * 2;
    const int nch = d / kWideKC;
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    for (int c0 = 0; c0 < nch; c0 += kWideG) {
        f32x4 rx[kWideG][XP];
        u32x4 rw[kWideG][4];
#pragma unroll
        for (int g = 0; g < kWideG; ++g) {
            const bool ok = c0 + g < nch;
            const int k = (c0 + g) * kWideKC;
#pragma unroll
            for (int p = 0; p < XP; ++p)
                rx[g][p] = ok && xin[p] ? *(const f32x4*)(xsrc[p] + k) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int i = 0; i < 4; ++i)
                rw[g][i] = ok && win[i] ? *(const u32x4*)(wsrc[i] + k) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int g = 0; g < kWideG; ++g) {
            if (c0 + g >= nch) break;
            __syncthreads();  // every wave has read the previous chunk's fragments
#pragma unroll
            for (int p = 0; p < XP; ++p) {
                bf16x4 hi, mid, lo;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float v = rx[g][p][e];
                    hi[e] = f2bf(v);
                    const float r1 = v - bf2f(hi[e]);
                    mid[e] = f2bf(r1);
                    lo[e] = f2bf(r1 - bf2f(mid[e]));
                }
                char* xd = sx + (xr + (NT / 16) * p) * kWideRS + xe * 2;
                *(bf16x4*)xd = hi;
                *(bf16x4*)(xd + 32 * kWideRS) = mid;
                *(bf16x4*)(xd + 64 * kWideRS) = lo;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) *(u32x4*)(sw + (wr + (NT / 8) * i) * kWideRS + we * 2) = rw[g][i];
            __syncthreads();
#pragma unroll
            for (int q = 0; q < kWideKC / 16; ++q) {
                const bf16x8 wf = *(const bf16x8*)(fw + q * 32);
                const bf16x8 xh = *(const bf16x8*)(fx + q * 32);
                const bf16x8 xm = *(const bf16x8*)(fx + 32 * kWideRS + q * 32);
                const bf16x8 xl = *(const bf16x8*)(fx + 64 * kWideRS + q * 32);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xl, wf, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xm, wf, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xh, wf, acc, 0, 0, 0);
            }
        }
    }
    // lane l holds feature 32 wave + l % 32 and, for register r, sample row
    // (r / 4) * 8 + (l / 32) * 4 + r % 4 of the tile
    const int j = j0 + wave * 32 + col;
    if (j >= n_out) return;
    const float bj = bias ? bias[j] : 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int i = (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        if (b0 + i < B) mod[(long)(b0 + i) * n_out + j] = acc[r] + bj;
    }
}

hipError_t launch_adaln_mod_batch(int dtype, const float* x, const ModBatch& mb, int B, int d, int n_out,
                                  hipStream_t st) {
    if (d % 64) return hipErrorInvalidValue;  // whole 64-deep k chunks (the model requires d % 128 == 0)
    if (mb.n < 1 || mb.n > kMaxModUnits) return hipErrorInvalidValue;
    if (dtype == 1 && n_out >= 2048) {
        // many features (DiT: 6 d per block): the widest workgroups that still give two per CU
        const long tiles = (long)((B + 31) / 32) * mb.n;
        const auto groups = [&](int wv) { return (long)((n_out + 32 * wv - 1) / (32 * wv)) * tiles; };
        if (groups(8) >= 512) {
            dim3 grid((n_out + 255) / 256, (B + 31) / 32, mb.n);
            hipLaunchKernelGGL(adaln_mod_wide_kernel<8>, grid, dim3(512), 0, st, x, mb, B, d, n_out);
        } else if (groups(4) >= 512) {
            dim3 grid((n_out + 127) / 128, (B + 31) / 32, mb.n);
            hipLaunchKernelGGL(adaln_mod_wide_kernel<4>, grid, dim3(256), 0, st, x, mb, B, d, n_out);
        } else {
            dim3 grid((n_out + 63) / 64, (B + 31) / 32, mb.n);
            hipLaunchKernelGGL(adaln_mod_wide_kernel<2>, grid, dim3(128), 0, st, x, mb, B, d, n_out);
        }
    } else if (dtype == 1) {
        dim3 grid((n_out + 31) / 32, (B + 31) / 32, mb.n), block(kModWaves * 64);
        hipLaunchKernelGGL(adaln_mod_mfma_kernel, grid, block, 0, st, x, mb, B, d, n_out);
    } else {
        dim3 grid((n_out + 63) / 64, (B + 31) / 32, mb.n), block(256);
        hipLaunchKernelGGL(adaln_mod_kernel<float>, grid, block, 0, st, x, mb, B, d, n_out);
    }
    return hipGetLastError();
}

hipError_t launch_adaln_mod(int dtype, const float* x, const void* W, const float* bias, float* mod, int B,
                            int d, int n_out, hipStream_t st) {
    ModBatch mb;
    mb.n = 1;
    mb.W[0] = W;
    mb.bias[0] = bias;
    mb.mod[0] = mod;
    return launch_adaln_mod_batch(dtype, x, mb, B, d, n_out, st);
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
