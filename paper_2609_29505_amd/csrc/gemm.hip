// Branch GEMMs of the active units in fp32: C = A . B^T with fused epilogues, and the
// dtype dispatch (the bf16 path is in gemm_bf16.hip).
//
// fp32 path: matrix-core kernel (v_mfma_f32_32x32x2_f32) with small tiles and K split across
// the waves of a workgroup (the fp32 workload is small and latency-bound); paired epilogues
// (gated MLPs: gate and up projections of one output column) read both halves from LDS.
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

// ---------------------------------------------------------------------------- fp32 MFMA

// 32 x 32 output tile per workgroup on v_mfma_f32_32x32x2_f32 (fp32 products, fp32
// accumulation).  The four waves split K: k unit u (8 values) goes to wave u % 4, and in a unit
// lanes 0-31 contract k = 8u .. 8u+3 and lanes 32-63 k = 8u+4 .. 8u+7 (four MFMA steps), so each
// lane reads one float4 of its A row and one of its B row per unit, straight from global
// memory.  The partial tiles meet in LDS and are summed in wave order (deterministic); every
// thread then applies the epilogue to its elements.  Gated tiles hold 16 gate and the matching
// 16 up columns (pairs c, c + 16).
constexpr int kF32Waves = 4, kF32Chunk = 4;  // k units per wave per pass (loads issued together)
__global__ __launch_bounds__(kF32Waves * 64) void gemm_f32_kernel(GemmArgs g, EpiParams ep) {
    __shared__ float red[kF32Waves][32 * 33];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 31, half = lane >> 5;
    const int nt_m = (g.M + 31) / 32;
    const int tm = blockIdx.x % nt_m, tn = blockIdx.x / nt_m;
    const int m0 = tm * 32;
    const bool gated = ep.kind == EP_GATED;
    const int F = g.N / 2;
    // operand rows of this lane: A row m0 + col (clamped; rows past M are never stored), B row
    // of product column col of the tile
    const int ar = min(m0 + col, g.M - 1);
    const long br = gated ? (col < 16 ? (long)tn * 16 + col : (long)F + tn * 16 + (col - 16)) : (long)tn * 32 + col;
    const float* bp = (const float*)g.B + br * g.ldb + half * 4;
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    const int units = g.K / 8;
    for (int u0 = wave; u0 < units; u0 += kF32Waves * kF32Chunk) {
        f32x4 av[kF32Chunk], bv[kF32Chunk];
#pragma unroll
        for (int c = 0; c < kF32Chunk; ++c) {
            const int u = u0 + c * kF32Waves;
            const int k = u * 8 + half * 4;
            if (u < units) {
                const bool second = g.A1 && k >= g.K0;
                const float* ap = second ? (const float*)g.A1 + (long)ar * g.lda1 + (k - g.K0)
                                         : (const float*)g.A0 + (long)ar * g.lda0 + k;
                av[c] = *(const f32x4*)ap;
                bv[c] = *(const f32x4*)(bp + u * 8);
            } else {
                av[c] = f32x4{0.f, 0.f, 0.f, 0.f};
                bv[c] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
        }
#pragma unroll
        for (int c = 0; c < kF32Chunk; ++c)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av[c][e], bv[c][e], acc, 0, 0, 0);
    }
    // lane l holds tile column l % 32 and, for register r, row (r / 4) * 8 + (l / 32) * 4 + r % 4
#pragma unroll
    for (int r = 0; r < 16; ++r) red[wave][((r >> 2) * 8 + half * 4 + (r & 3)) * 33 + col] = acc[r];
    __syncthreads();
    auto tile_at = [&](int row, int c) {
        float v = red[0][row * 33 + c];
#pragma unroll
        for (int w = 1; w < kF32Waves; ++w) v += red[w][row * 33 + c];
        return v;
    };
    Epi<float> e{ep};
    if (ep.kind == EP_HEADS) e.tw = ep.which0 + (tn * 32) / ep.d;
    if (gated) {
        // 32 rows x 16 (gate, up) pairs, two per thread
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int pidx = tid + i * kF32Waves * 64, row = pidx >> 4, c = pidx & 15;
            if (m0 + row < g.M) e.pair(m0 + row, tn * 32 + c, 16, tn * 16 + c, tile_at(row, c), tile_at(row, c + 16));
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int idx = tid + i * kF32Waves * 64, row = idx >> 5, c = idx & 31;
        if (m0 + row >= g.M) continue;
        const float v = tile_at(row, c);
        if (ep.kind == EP_HEADS && e.tw == 2) e.single_vt(m0 + row, tn * 32 + c, v);
        else e.single(m0 + row, tn * 32 + c, v);
    }
}

// ---------------------------------------------------------------------------- dispatch

bool gemm_shape_ok(int dtype, const GemmArgs& g, const EpiParams& e, int tile) {
    if (g.M <= 0 || g.N <= 0 || g.K <= 0) return false;
    if (dtype == 1) return gemm_bf16_shape_ok(g, e, tile);
    if (g.ksplit != 1 || e.kind == EP_PARTIAL) return false;  // split products: bf16 only
    if (g.K % 16 || g.N % 64) return false;
    if (g.A1 && (g.K0 % 16)) return false;
    if (e.kind == EP_HEADS && (e.rope || e.d % 64)) return false;
    return true;
}

hipError_t launch_gemm(int dtype, const GemmArgs& g, const EpiParams& e, hipStream_t st, int tile) {
    if (dtype == 1) return launch_gemm_bf16(g, e, st, tile);
    if (g.ksplit != 1 || e.kind == EP_PARTIAL) return hipErrorInvalidValue;
    const int nt_m = (g.M + 31) / 32, nt_n = g.N / 32;
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(nt_m * nt_n), dim3(kF32Waves * 64), 0, st, g, e);
    return hipGetLastError();
}

}  // namespace sgd
