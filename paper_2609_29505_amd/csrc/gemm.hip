// Branch GEMMs of the active units: C = A . B^T with fused epilogues.
//
// bf16 path: CDNA4 matrix cores (v_mfma_f32_32x32x16_bf16), LDS-staged tiles with a
// register prefetch of the next K tile and a double-buffered LDS, XCD-aware tile order.
// fp32 path: LDS-tiled FMA kernel (used by the fp32 workload, which is latency-bound).
//
// Column layout inside a wave: every wave owns the same column offsets in both halves
// of the block tile, so each lane holds column c and c + BN/2 of a row.  Paired
// epilogues use this for rotary embeddings (pairs i, i + d_h/2 inside one head) and for
// gated MLPs (gate and up projections of the same output column).
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

// XCD-aware tile order: the hardware hands workgroup g to XCD g % 8.  Give each XCD a
// contiguous range of logical tiles, row tiles fastest, so the row tiles that share a B
// (weight) tile run together on one XCD and share its L2.
__device__ __forceinline__ int xcd_tile(int g, int total) {
    if (total % 8 != 0) return g;
    return (g % 8) * (total / 8) + g / 8;
}

// ---------------------------------------------------------------------------- bf16 MFMA

template <int BM, int BN, int WAVES_M, int WAVES_N>
struct BfCfg {
    static constexpr int BK = 64;
    static constexpr int LDS = BK + 8;  // padded row (elements): 144 B rows, conflict-free b128 reads
    static constexpr int NT = WAVES_M * WAVES_N * 64;
    static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    static constexpr int TM = WM / 32, TN = WN / 32;
    static constexpr int A_CHUNKS = BM * BK / 8 / NT;  // 16-byte chunks per thread
    static constexpr int B_CHUNKS = BN * BK / 8 / NT;
    static constexpr int STAGE = (BM + BN) * LDS;      // elements per LDS stage
    static_assert(TN % 2 == 0, "wave tile must cover both halves");
    static_assert(BM * BK / 8 % NT == 0 && BN * BK / 8 % NT == 0, "chunk split");
};

template <int BM, int BN, int WAVES_M, int WAVES_N, bool GATED>
__global__ __launch_bounds__(WAVES_M* WAVES_N * 64) void gemm_bf16_kernel(GemmArgs g, EpiParams ep) {
    using C = BfCfg<BM, BN, WAVES_M, WAVES_N>;
    __shared__ __attribute__((aligned(16))) bf16 lds[2 * C::STAGE];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nt_m = (g.M + BM - 1) / BM;
    const int nt_n = GATED ? g.N / BN : g.N / BN;
    const int t = xcd_tile(blockIdx.x, nt_m * nt_n);
    const int tm = t % nt_m, tn = t / nt_m;
    const int m0 = tm * BM;
    const int half_out = BN / 2;
    const int F = g.N / 2;

    // global source rows of this thread's chunks
    const bf16* a_src0[C::A_CHUNKS];
    const bf16* a_src1[C::A_CHUNKS];
    const bf16* b_src[C::B_CHUNKS];
    const int cchunk = tid & 7;
#pragma unroll
    for (int i = 0; i < C::A_CHUNKS; ++i) {
        int r = (tid >> 3) + i * (C::NT / 8);
        int gr = min(m0 + r, g.M - 1);
        a_src0[i] = (const bf16*)g.A0 + (long)gr * g.lda0 + cchunk * 8;
        a_src1[i] = g.A1 ? (const bf16*)g.A1 + (long)gr * g.lda1 + cchunk * 8 : a_src0[i];
    }
#pragma unroll
    for (int i = 0; i < C::B_CHUNKS; ++i) {
        int r = (tid >> 3) + i * (C::NT / 8);
        long gr;
        if (GATED) gr = r < half_out ? (long)tn * half_out + r : (long)F + tn * half_out + (r - half_out);
        else gr = (long)tn * BN + r;
        b_src[i] = (const bf16*)g.B + gr * g.ldb + cchunk * 8;
    }

    u32x4 ra[C::A_CHUNKS], rb[C::B_CHUNKS];
    auto gload = [&](int kt) {
        const int k0 = kt * C::BK;
        const bool second = g.A1 && k0 >= g.K0;
#pragma unroll
        for (int i = 0; i < C::A_CHUNKS; ++i)
            ra[i] = *(const u32x4*)(second ? a_src1[i] + (k0 - g.K0) : a_src0[i] + k0);
#pragma unroll
        for (int i = 0; i < C::B_CHUNKS; ++i) rb[i] = *(const u32x4*)(b_src[i] + k0);
    };
    auto lstore = [&](int buf) {
        bf16* sa = lds + buf * C::STAGE;
        bf16* sb = sa + BM * C::LDS;
#pragma unroll
        for (int i = 0; i < C::A_CHUNKS; ++i) {
            int r = (tid >> 3) + i * (C::NT / 8);
            *(u32x4*)(sa + r * C::LDS + cchunk * 8) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < C::B_CHUNKS; ++i) {
            int r = (tid >> 3) + i * (C::NT / 8);
            *(u32x4*)(sb + r * C::LDS + cchunk * 8) = rb[i];
        }
    };

    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int wm0 = wm * C::WM;
    int colbase[C::TN];
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
        colbase[j] = j < C::TN / 2 ? wn * (C::WN / 2) + j * 32 : BN / 2 + wn * (C::WN / 2) + (j - C::TN / 2) * 32;

    f32x16 acc[C::TM][C::TN];
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    const int KT = g.K / C::BK;
    gload(0);
    lstore(0);
    __syncthreads();
    const int lrow = lane & 31, lk = (lane >> 5) * 8;
    for (int kt = 0; kt < KT; ++kt) {
        if (kt + 1 < KT) gload(kt + 1);
        const bf16* sa = lds + (kt & 1) * C::STAGE;
        const bf16* sb = sa + BM * C::LDS;
#pragma unroll
        for (int ks = 0; ks < C::BK / 16; ++ks) {
            bf16x8 af[C::TM], bfr[C::TN];
#pragma unroll
            for (int i = 0; i < C::TM; ++i)
                af[i] = *(const bf16x8*)(sa + (wm0 + i * 32 + lrow) * C::LDS + ks * 16 + lk);
#pragma unroll
            for (int j = 0; j < C::TN; ++j)
                bfr[j] = *(const bf16x8*)(sb + (colbase[j] + lrow) * C::LDS + ks * 16 + lk);
#pragma unroll
            for (int i = 0; i < C::TM; ++i)
#pragma unroll
                for (int j = 0; j < C::TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < KT) lstore((kt + 1) & 1);
        __syncthreads();
    }

    // epilogue
    Epi<bf16> e{ep};
    const bool paired = kind_paired(ep);
    if (ep.kind == EP_HEADS) e.tw = ep.which0 + (tn * BN) / ep.d;
    if (ep.kind == EP_HEADS && e.tw == 2 && !paired) {
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm0 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                if (row >= g.M) continue;
#pragma unroll
                for (int j = 0; j < C::TN; ++j) e.single_vt(row, tn * BN + colbase[j] + lrow, acc[i][j][r]);
            }
        return;
    }
#pragma unroll
    for (int i = 0; i < C::TM; ++i) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = m0 + wm0 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
            if (row >= g.M) continue;
            if (paired) {
#pragma unroll
                for (int j = 0; j < C::TN / 2; ++j) {
                    const int lc = colbase[j] + lrow;  // < BN/2
                    const int n = tn * BN + lc;
                    e.pair(row, n, BN / 2, tn * half_out + lc, acc[i][j][r], acc[i][j + C::TN / 2][r]);
                }
            } else {
#pragma unroll
                for (int j = 0; j < C::TN; ++j) e.single(row, tn * BN + colbase[j] + lrow, acc[i][j][r]);
            }
        }
    }
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

namespace {
struct TileShape { int bm, bn; };
TileShape bf16_tile(const GemmArgs& g, const EpiParams& e, int tile) {
    if (tile == 1) return {256, 256};
    if (tile == 2) return {256, 128};
    if (tile == 3) return {128, 128};
    // rotary pairs must sit in one head: the tile is one 128-wide head
    // a head-major tile must lie inside one projection (d % 128 == 0)
    if (e.kind == EP_HEADS) return {g.M >= 2048 ? 256 : 128, 128};
    const long tiles256 = (long)((g.M + 255) / 256) * (g.N / 256);
    if (g.N % 256 == 0 && tiles256 >= 256) return {256, 256};
    const long tiles_256x128 = (long)((g.M + 255) / 256) * (g.N / 128);
    if (tiles_256x128 >= 256) return {256, 128};
    return {128, 128};
}
}  // namespace

bool gemm_shape_ok(int dtype, const GemmArgs& g, const EpiParams& e, int tile) {
    if (g.M <= 0 || g.N <= 0 || g.K <= 0) return false;
    if (dtype == 1) {
        TileShape ts = bf16_tile(g, e, tile);
        if (g.K % 64 || g.N % ts.bn) return false;
        if (g.A1 && (g.K0 % 64)) return false;
        if (e.kind == EP_HEADS && (e.d % ts.bn || (e.rope && (e.dh != 128 || ts.bn != 128)))) return false;
        return true;
    }
    if (g.K % 16 || g.N % 64) return false;
    if (g.A1 && (g.K0 % 16)) return false;
    if (e.kind == EP_HEADS && (e.rope || e.d % 64)) return false;
    return true;
}

template <int BM, int BN, int WM_, int WN_>
static hipError_t run_bf16(const GemmArgs& g, const EpiParams& e, hipStream_t st) {
    const int nt_m = (g.M + BM - 1) / BM, nt_n = g.N / BN;
    dim3 grid(nt_m * nt_n), block(WM_ * WN_ * 64);
    if (e.kind == EP_GATED)
        hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM_, WN_, true>), grid, block, 0, st, g, e);
    else
        hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM_, WN_, false>), grid, block, 0, st, g, e);
    return hipGetLastError();
}

hipError_t launch_gemm(int dtype, const GemmArgs& g, const EpiParams& e, hipStream_t st, int tile) {
    if (dtype == 1) {
        TileShape ts = bf16_tile(g, e, tile);
        if (ts.bm == 256 && ts.bn == 256) return run_bf16<256, 256, 2, 2>(g, e, st);
        if (ts.bm == 256 && ts.bn == 128) return run_bf16<256, 128, 2, 2>(g, e, st);
        return run_bf16<128, 128, 2, 2>(g, e, st);
    }
    const int nt_m = (g.M + 63) / 64, nt_n = g.N / 64;
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(nt_m * nt_n), dim3(256), 0, st, g, e);
    return hipGetLastError();
}

}  // namespace sgd
