// Branch GEMMs of the active units in fp32: C = A . B^T with fused epilogues, and the
// dtype dispatch (the bf16 path is in gemm_bf16.hip).
//
// fp32 path: LDS-tiled FMA kernel (the fp32 workload is small and latency-bound).  Each
// thread holds columns c and c + 32 of its rows, so paired epilogues (gated MLPs: gate and
// up projections of one output column) read both halves from registers.
#include "common.h"
#include "kernels.h"

namespace sgd {

// ---------------------------------------------------------------------------- epilogue

template <typename OutT>
struct Epi {
    EpiParams p;

    int tw = 0;  // EP_HEADS: projection of this tile (0 q, 1 k, 2 v^T); tiles never straddle two

    __device__ __forceinline__ void store_qk(int row, int nn, float v) const {
        const int b = row / p.ntok, tok = row - b * p.ntok;
        const int hh = nn / p.dh, j = nn - hh * p.dh;
        OutT* base = (OutT*)(tw == 0 ? p.q : p.k);
        ElemIO<OutT>::store(base + (((long)b * p.H + hh) * p.np + tok) * p.dh + j, v);
    }
    __device__ __forceinline__ void store_vt(int row, int nn, float v) const {
        const int b = row / p.ntok, tok = row - b * p.ntok;
        const int hh = nn / p.dh, j = nn - hh * p.dh;
        ElemIO<OutT>::store((OutT*)p.vt + (((long)b * p.H + hh) * p.dh + j) * p.np + tok, v);
    }
    // V^T columns of a tile (tw == 2): their own store loop
    __device__ __forceinline__ void single_vt(int row, int n, float v) const {
        if (p.bias) v += p.bias[n];
        store_vt(row, n - (tw - p.which0) * p.d, v);
    }

    // one element at product column n
    __device__ __forceinline__ void single(int row, int n, float v) const {
        switch (p.kind) {
            case EP_HEADS: {
                if (p.bias) v += p.bias[n];
                store_qk(row, n - (tw - p.which0) * p.d, v);
                break;
            }
            case EP_ACT: {
                if (p.bias) v += p.bias[n];
                ElemIO<OutT>::store((OutT*)p.out + (long)row * p.ldo + n, apply_act(p.act, v));
                break;
            }
            case EP_RESID: {
                if (p.bias) v += p.bias[n];
                if (p.gate) v *= p.gate[(long)(row / p.ntok) * p.gate_ld + n];
                const long idx = (long)row * p.d + n;
                const float hn = p.h[idx] + v;
                p.h[idx] = hn;
                if (p.delta_mode == 1) p.delta[idx] = v;
                else if (p.delta_mode == 2) p.delta[idx] = p.delta[idx] + v;
                if (p.hcopy) ElemIO<OutT>::store((OutT*)p.hcopy + idx, hn);
                break;
            }
            case EP_SKIP: {
                if (p.bias) v += p.bias[n];
                const long idx = (long)row * p.d + n;
                if (p.delta_mode == 1) v = v + p.delta[idx];
                p.h[idx] = v;
                if (p.hcopy) ElemIO<OutT>::store((OutT*)p.hcopy + idx, v);
                break;
            }
            default: break;
        }
    }

    // two elements of one row: product columns n and n + half (half = BN / 2).
    // For EP_GATED, `on` is the output column of the pair.
    __device__ __forceinline__ void pair(int row, int n, int half, int on, float lo, float hi) const {
        if (p.kind == EP_GATED) {
            float g = lo, u = hi;
            if (p.bias) { g += p.bias[on]; u += p.bias[p.F + on]; }
            ElemIO<OutT>::store((OutT*)p.out + (long)row * p.ldo + on, apply_act(p.act, g) * u);
            return;
        }
        if (p.kind == EP_HEADS && p.rope) {
            const int nn = n - (tw - p.which0) * p.d;
            const int j = nn % p.dh;  // < dh/2 by construction (BN == dh)
            if (p.bias) { lo += p.bias[n]; hi += p.bias[n + half]; }
            if (tw == 2) {
                store_vt(row, nn, lo);
                store_vt(row, nn + half, hi);
                return;
            }
            {
                const int tok = row % p.ntok;
                const float inv = exp2f(-(2.0f * (float)j / (float)p.dh) * p.rope_log2_theta);
                float s, c;
                sincosf((float)tok * inv, &s, &c);
                const float a = lo * c - hi * s;
                const float b = hi * c + lo * s;
                lo = a;
                hi = b;
            }
            store_qk(row, nn, lo);
            store_qk(row, nn + half, hi);
            return;
        }
        single(row, n, lo);
        single(row, n + half, hi);
    }
};

__device__ __forceinline__ bool kind_paired(const EpiParams& p) {
    return p.kind == EP_GATED || (p.kind == EP_HEADS && p.rope);
}

// ---------------------------------------------------------------------------- fp32 FMA

// 64 x 64 tile, BK = 16, 256 threads, 4 x 4 outputs per thread.  Thread (ty, tx) owns rows
// ty + 16 i and columns tx + 16 j (j = 0..3): columns tx and tx + 32 form pairs.
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs g, EpiParams ep) {
    constexpr int BM = 64, BN = 64, BK = 16;
    __shared__ float sa[BK][BM + 4];
    __shared__ float sb[BK][BN + 4];
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int nt_m = (g.M + BM - 1) / BM;
    const bool gated = ep.kind == EP_GATED;
    const int t = blockIdx.x;
    const int tm = t % nt_m, tn = t / nt_m;
    const int m0 = tm * BM;
    const int F = g.N / 2;
    float acc[4][4] = {};
    // loader: 64 rows x 16 k = 1024 elements, 4 per thread (one float4 along k)
    const int lr = tid >> 2, lk = (tid & 3) * 4;
    const int ar = min(m0 + lr, g.M - 1);
    long br;
    if (gated) br = lr < 32 ? (long)tn * 32 + lr : (long)F + tn * 32 + (lr - 32);
    else br = (long)tn * BN + lr;
    for (int k0 = 0; k0 < g.K; k0 += BK) {
        const bool second = g.A1 && k0 >= g.K0;
        const float* ap = second ? (const float*)g.A1 + (long)ar * g.lda1 + (k0 - g.K0) + lk
                                 : (const float*)g.A0 + (long)ar * g.lda0 + k0 + lk;
        float4 av = *(const float4*)ap;
        float4 bv = *(const float4*)((const float*)g.B + br * g.ldb + k0 + lk);
        sa[lk + 0][lr] = av.x; sa[lk + 1][lr] = av.y; sa[lk + 2][lr] = av.z; sa[lk + 3][lr] = av.w;
        sb[lk + 0][lr] = bv.x; sb[lk + 1][lr] = bv.y; sb[lk + 2][lr] = bv.z; sb[lk + 3][lr] = bv.w;
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < BK; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = sa[kk][ty + 16 * i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = sb[kk][tx + 16 * j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
    Epi<float> e{ep};
    const bool paired = kind_paired(ep);
    if (ep.kind == EP_HEADS) e.tw = ep.which0 + (tn * BN) / ep.d;
    if (ep.kind == EP_HEADS && e.tw == 2 && !paired) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = m0 + ty + 16 * i;
            if (row >= g.M) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) e.single_vt(row, tn * BN + tx + 16 * j, acc[i][j]);
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = m0 + ty + 16 * i;
        if (row >= g.M) continue;
        if (paired) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int lc = tx + 16 * j;
                e.pair(row, tn * BN + lc, 32, tn * 32 + lc, acc[i][j], acc[i][j + 2]);
            }
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) e.single(row, tn * BN + tx + 16 * j, acc[i][j]);
        }
    }
}

// ---------------------------------------------------------------------------- dispatch

bool gemm_shape_ok(int dtype, const GemmArgs& g, const EpiParams& e, int tile) {
    if (g.M <= 0 || g.N <= 0 || g.K <= 0) return false;
    if (dtype == 1) return gemm_bf16_shape_ok(g, e, tile);
    if (g.K % 16 || g.N % 64) return false;
    if (g.A1 && (g.K0 % 16)) return false;
    if (e.kind == EP_HEADS && (e.rope || e.d % 64)) return false;
    return true;
}

hipError_t launch_gemm(int dtype, const GemmArgs& g, const EpiParams& e, hipStream_t st, int tile) {
    if (dtype == 1) return launch_gemm_bf16(g, e, st, tile);
    const int nt_m = (g.M + 63) / 64, nt_n = g.N / 64;
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(nt_m * nt_n), dim3(256), 0, st, g, e);
    return hipGetLastError();
}

}  // namespace sgd
