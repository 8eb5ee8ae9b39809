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

template <typename OutT, int VPL, int WPR, bool FOLD>
__device__ __forceinline__ void norm_body(const NormArgs& a) {
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
    }
    if (FOLD && live) {
        // the frozen run ending at this unit: its cached updates in stack order, written back.
        // G updates are loaded together before they are added (still one at a time, in stack
        // order), so a run costs one memory round trip per group of G, not per update; G keeps
        // at most 16 float4 of updates in registers.
        const long roff = (long)row * nvec;
        constexpr int G = VPL >= 16 ? 1 : (16 / VPL < 4 ? 16 / VPL : 4);
        for (int k0 = 0; k0 < a.nfold; k0 += G) {
            float4 dv[G][VPL];
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int i = 0; i < VPL; ++i) {
                    const int c = t + i * TPR;
                    dv[g][i] = (k0 + g < a.nfold && c < nvec) ? ((const float4*)a.fold[k0 + g] + roff)[c]
                                                              : make_float4(0.f, 0.f, 0.f, 0.f);
                }
#pragma unroll
            for (int g = 0; g < G; ++g) {
                if (k0 + g >= a.nfold) break;
#pragma unroll
                for (int i = 0; i < VPL; ++i) {
                    v[i].x = v[i].x + dv[g][i].x;
                    v[i].y = v[i].y + dv[g][i].y;
                    v[i].z = v[i].z + dv[g][i].z;
                    v[i].w = v[i].w + dv[g][i].w;
                }
            }
        }
#pragma unroll
        for (int i = 0; i < VPL; ++i) {
            const int c = t + i * TPR;
            if (c < nvec) ((float4*)x)[c] = v[i];
        }
    }
    // every multiply-add below is an explicit fmaf (or an explicit plain product): the compiler
    // may contract a*b + c differently in different instantiations, and a pre-norm that absorbed
    // a frozen run must give bitwise the rows of the plain one
#pragma unroll
    for (int i = 0; i < VPL; ++i)
        s += (a.kind == 0) ? fmaf(v[i].w, v[i].w, fmaf(v[i].z, v[i].z, fmaf(v[i].y, v[i].y, v[i].x * v[i].x)))
                           : (v[i].x + v[i].y + v[i].z + v[i].w);
    s = row_sum<WPR>(s, red);
    const float invd = 1.0f / (float)a.d;
    float mean = 0.f, rstd;
    if (a.kind == 0) {
        rstd = 1.0f / sqrtf(fmaf(s, invd, a.eps));
    } else {
        mean = s * invd;
        float q = 0.f;
#pragma unroll
        for (int i = 0; i < VPL; ++i) {
            const int c = t + i * TPR;
            if (c < nvec) {
                const float dx = v[i].x - mean, dy = v[i].y - mean, dz = v[i].z - mean, dw = v[i].w - mean;
                q += fmaf(dw, dw, fmaf(dz, dz, fmaf(dy, dy, dx * dx)));
            }
        }
        q = row_sum<WPR>(q, red);
        rstd = 1.0f / sqrtf(fmaf(q, invd, a.eps));
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
            o[0] = fmaf(o[0], w.x, b.x); o[1] = fmaf(o[1], w.y, b.y);
            o[2] = fmaf(o[2], w.z, b.z); o[3] = fmaf(o[3], w.w, b.w);
        } else {
            const float4 sc = *(const float4*)(a.scale + mrow + c * 4), sh = *(const float4*)(a.shift + mrow + c * 4);
            o[0] = fmaf(o[0], 1.0f + sc.x, sh.x); o[1] = fmaf(o[1], 1.0f + sc.y, sh.y);
            o[2] = fmaf(o[2], 1.0f + sc.z, sh.z); o[3] = fmaf(o[3], 1.0f + sc.w, sh.w);
        }
        store4<OutT>(y + c * 4, o[0], o[1], o[2], o[3]);
    }
}

template <typename OutT, int VPL, int WPR, bool FOLD>
__global__ __launch_bounds__(256) void norm_kernel(NormArgs a) {
    norm_body<OutT, VPL, WPR, FOLD>(a);
}

// A pre-norm that first adds the partial products of a split residual GEMM to its rows, in
// K-range order: the body of a folding pre-norm under a name of its own, so that launch
// counts and traces keep it apart from the folds of frozen runs.
template <typename OutT, int VPL, int WPR>
__global__ __launch_bounds__(256) void norm_parts_kernel(NormArgs a) {
    norm_body<OutT, VPL, WPR, true>(a);
}

template <int WPR>
static hipError_t launch_norm_wpr(int dtype, const NormArgs& a, bool parts, hipStream_t st) {
    const int vpl = (a.d / 4 + 64 * WPR - 1) / (64 * WPR);
    dim3 grid((a.M + (4 / WPR) - 1) / (4 / WPR)), block(256);
#define NORM_CASE(V)                                                                                       \
    if (vpl <= V) {                                                                                        \
        if (parts) {                                                                                       \
            if (dtype == 1) hipLaunchKernelGGL((norm_parts_kernel<bf16, V, WPR>), grid, block, 0, st, a);  \
            else hipLaunchKernelGGL((norm_parts_kernel<float, V, WPR>), grid, block, 0, st, a);            \
        } else if (a.nfold > 0) {                                                                          \
            if (dtype == 1) hipLaunchKernelGGL((norm_kernel<bf16, V, WPR, true>), grid, block, 0, st, a);  \
            else hipLaunchKernelGGL((norm_kernel<float, V, WPR, true>), grid, block, 0, st, a);            \
        } else {                                                                                           \
            if (dtype == 1) hipLaunchKernelGGL((norm_kernel<bf16, V, WPR, false>), grid, block, 0, st, a); \
            else hipLaunchKernelGGL((norm_kernel<float, V, WPR, false>), grid, block, 0, st, a);           \
        }                                                                                                  \
        return hipGetLastError();                                                                          \
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

hipError_t launch_norm(int dtype, const NormArgs& a, hipStream_t st, bool parts) {
    // few rows (LLaDA: 1024): four waves per row.  Many rows: two waves per row when the row's
    // float4 groups split evenly over 128 lanes (U-ViT, d = 1024: 13.9 -> 12.5 us), else one
    // (DiT d = 1152 and SDXL d = 1280 measured slower with two: uneven lanes)
    if (parts && a.nfold < 1) return hipErrorInvalidValue;
    if (a.M < 4096) return launch_norm_wpr<4>(dtype, a, parts, st);
    return (a.d / 4) % 128 == 0 ? launch_norm_wpr<2>(dtype, a, parts, st) : launch_norm_wpr<1>(dtype, a, parts, st);
}

// GroupNorm + SiLU of the SDXL UNet ResNet blocks, y = SiLU(GN(x) w + b) in bf16 for x
// [B, N, C] (the fp32 stream or a bf16 convolution output), in three launches with coalesced
// rows: (1) per block of kGnRows positions, a workgroup of C / 4 threads (thread t owns
// channels 4t .. 4t+3, all in one group) sums x and x^2 over its rows and combines the
// threads of each group in a fixed order into fp64 partials; (2) one wave per (sample, group)
// adds the partials (lane j takes blocks j, j + 64, ... in order, then a fixed butterfly over
// the lanes) and forms the mean and 1 / sqrt(biased variance + eps); (3) the same row blocks
// normalise, apply the gain and shift, SiLU, and store bf16.  Full row blocks unroll their
// row loop, so every row's load is in flight at once.
template <typename TI>
__device__ __forceinline__ float4 ld4_any(const TI* p);
template <>
__device__ __forceinline__ float4 ld4_any<float>(const float* p) { return *(const float4*)p; }
template <>
__device__ __forceinline__ float4 ld4_any<bf16>(const bf16* p) {
    const bf16x4 v = *(const bf16x4*)p;
    return make_float4(bf2f(v[0]), bf2f(v[1]), bf2f(v[2]), bf2f(v[3]));
}

constexpr int kGnRows = 16;

template <typename TI>
__global__ __launch_bounds__(1024) void gn_partial_kernel(GroupNormArgs a, double* partial) {
    const int nblk = (a.N + kGnRows - 1) / kGnRows;
    const int b = blockIdx.x / nblk, blk = blockIdx.x - b * nblk;
    const int t = threadIdx.x, q4 = (a.C / a.groups) / 4;  // channel quads per group
    const TI* x = (const TI*)a.x + ((long)b * a.N + (long)blk * kGnRows) * a.C + 4 * t;
    const int rows = min(kGnRows, a.N - blk * kGnRows);
    float s = 0.f, ss = 0.f;
    auto add = [&](int r) {
        const float4 v = ld4_any<TI>(x + (long)r * a.C);
        s += (v.x + v.y) + (v.z + v.w);
        ss += (v.x * v.x + v.y * v.y) + (v.z * v.z + v.w * v.w);
    };
    if (rows == kGnRows) {
#pragma unroll
        for (int r = 0; r < kGnRows; ++r) add(r);
    } else {
        for (int r = 0; r < rows; ++r) add(r);
    }
    extern __shared__ double red[];  // [C / 4][2]
    red[2 * t] = s;
    red[2 * t + 1] = ss;
    __syncthreads();
    if (t < a.groups) {
        double gs = 0.0, gss = 0.0;
        for (int i = 0; i < q4; ++i) {
            gs += red[2 * (t * q4 + i)];
            gss += red[2 * (t * q4 + i) + 1];
        }
        double* o = partial + (((long)b * nblk + blk) * a.groups + t) * 2;
        o[0] = gs;
        o[1] = gss;
    }
}

__global__ __launch_bounds__(256) void gn_stats_kernel(GroupNormArgs a, const double* partial, float* stats) {
    const int i = blockIdx.x * 4 + (threadIdx.x >> 6);  // sample * groups + group: one wave each
    const int lane = threadIdx.x & 63;
    if (i >= a.B * a.groups) return;  // whole waves
    const int b = i / a.groups, g = i - b * a.groups;
    const int nblk = (a.N + kGnRows - 1) / kGnRows;
    double s = 0.0, ss = 0.0;
    for (int blk = lane; blk < nblk; blk += 64) {
        const double* p = partial + (((long)b * nblk + blk) * a.groups + g) * 2;
        s += p[0];
        ss += p[1];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        s += __shfl_xor(s, off);
        ss += __shfl_xor(ss, off);
    }
    if (lane != 0) return;
    const double cnt = (double)a.N * (a.C / a.groups);
    const double mean = s / cnt;
    const double var = fmax(ss / cnt - mean * mean, 0.0);
    stats[2 * i] = (float)mean;
    stats[2 * i + 1] = (float)(1.0 / sqrt(var + (double)a.eps));
}

template <typename TI>
__global__ __launch_bounds__(1024) void gn_apply_kernel(GroupNormArgs a, const float* stats) {
    const int nblk = (a.N + kGnRows - 1) / kGnRows;
    const int b = blockIdx.x / nblk, blk = blockIdx.x - b * nblk;
    const int t = threadIdx.x, cg = a.C / a.groups, c = 4 * t, g = c / cg;
    const float mean = stats[2 * (b * a.groups + g)], rstd = stats[2 * (b * a.groups + g) + 1];
    const float4 ww = *(const float4*)(a.w + c), bv = *(const float4*)(a.b + c);
    const long off = ((long)b * a.N + (long)blk * kGnRows) * a.C + c;
    const TI* x = (const TI*)a.x + off;
    bf16* y = (bf16*)a.y + off;
    const int rows = min(kGnRows, a.N - blk * kGnRows);
    auto apply = [&](int r) {
        const float4 v = ld4_any<TI>(x + (long)r * a.C);
        bf16x4 o;
        o[0] = f2bf(silu((v.x - mean) * rstd * ww.x + bv.x));
        o[1] = f2bf(silu((v.y - mean) * rstd * ww.y + bv.y));
        o[2] = f2bf(silu((v.z - mean) * rstd * ww.z + bv.z));
        o[3] = f2bf(silu((v.w - mean) * rstd * ww.w + bv.w));
        *(bf16x4*)(y + (long)r * a.C) = o;
    };
    if (rows == kGnRows) {
#pragma unroll
        for (int r = 0; r < kGnRows; ++r) apply(r);
    } else {
        for (int r = 0; r < rows; ++r) apply(r);
    }
}

size_t group_norm_scratch_bytes(int B, int N, int groups) {
    const int nblk = (N + kGnRows - 1) / kGnRows;
    return (size_t)B * nblk * groups * 2 * sizeof(double) + (size_t)B * groups * 2 * sizeof(float);
}

hipError_t launch_group_norm_silu(int in_bf16, const GroupNormArgs& a, void* scratch, hipStream_t st) {
    const int nblk = (a.N + kGnRows - 1) / kGnRows;
    double* partial = (double*)scratch;
    float* stats = (float*)(partial + (size_t)a.B * nblk * a.groups * 2);
    const dim3 rows(a.B * nblk), threads(a.C / 4);
    const size_t lds = (size_t)(a.C / 4) * 2 * sizeof(double);
    if (in_bf16) hipLaunchKernelGGL(gn_partial_kernel<bf16>, rows, threads, lds, st, a, partial);
    else hipLaunchKernelGGL(gn_partial_kernel<float>, rows, threads, lds, st, a, partial);
    hipLaunchKernelGGL(gn_stats_kernel, dim3((a.B * a.groups + 3) / 4), dim3(256), 0, st, a,
                       (const double*)partial, stats);
    if (in_bf16) hipLaunchKernelGGL(gn_apply_kernel<bf16>, rows, threads, 0, st, a, (const float*)stats);
    else hipLaunchKernelGGL(gn_apply_kernel<float>, rows, threads, 0, st, a, (const float*)stats);
    return hipGetLastError();
}

}  // namespace sgd
