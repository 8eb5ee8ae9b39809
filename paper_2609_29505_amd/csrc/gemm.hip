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

// ---------------------------------------------------------------------------- bf16 MFMA, v2
//
// Global -> LDS with buffer_load_dwordx4 ... lds: the loads land in LDS without passing
// through VGPRs, and the buffer descriptor's range check turns rows beyond the matrix into
// zeros, so no address clamping is needed.  One load instruction moves 8 rows x 64 bf16
// (1 KB) into LDS at consecutive lane positions; the lane -> source-chunk mapping applies an
// XOR swizzle: chunk c of row r sits at position c ^ ((r >> 1) & 7).  With 64 four-byte
// banks (256 B), two 128-byte rows share a bank line, so the 16-byte fragment reads of 16
// consecutive rows (one LDS cycle) then cover all 64 banks exactly once.
//
// KSPLIT > 1 splits each 64-wide K tile across waves (each wave covers the whole block tile
// on its share of the 16-wide k steps) and sums the partial tiles through LDS in a fixed
// order at the end; this halves the LDS read traffic per FLOP for small block tiles.

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, unsigned bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

template <int N>
__device__ __forceinline__ void wait_vm() {
    // s_waitcnt vmcnt(N) (gfx9 encoding: vmcnt[3:0] | vmcnt[5:4] << 14; other counters at max)
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int KSPLIT, int STAGES, int BK_ = 64>
struct Cfg2 {
    static constexpr int BK = BK_;
    static constexpr int NW = WAVES_M * WAVES_N * KSPLIT;
    static constexpr int NT = NW * 64;
    static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    static constexpr int TM = WM / 32, TN = WN / 32;
    static constexpr int ROWB = BK * 2;                 // bytes per tile row
    static constexpr int CH = BK / 8;                   // 16-byte chunks per row
    static constexpr int RPL = 64 / CH;                 // rows per load instruction (1 KB)
    static constexpr int RPB = 256 / ROWB;              // rows per 256-byte bank line
    static constexpr int A_BYTES = BM * ROWB, B_BYTES = BN * ROWB;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static constexpr int A_LOADS = BM / RPL / NW, B_LOADS = BN / RPL / NW;  // per wave per stage
    static constexpr int KS_PER_WAVE = (BK / 16) / KSPLIT;
    static constexpr int RED_BYTES = KSPLIT > 1 ? BM * BN * 4 : NW * TN * 16 * 64 * 4;
    static constexpr int LDS_BYTES = STAGE_BYTES * STAGES > RED_BYTES ? STAGE_BYTES * STAGES : RED_BYTES;
    static_assert(TN % 2 == 0, "paired column layout");
    static_assert(BM % (RPL * NW) == 0 && BN % (RPL * NW) == 0, "load split");
    static_assert(BK == 32 || BK == 64, "tile depth");
    static_assert((BK / 16) % KSPLIT == 0, "k split");
};

template <int BM, int BN, int WAVES_M, int WAVES_N, int KSPLIT, int STAGES, bool GATED, int BK_ = 64>
__global__ __launch_bounds__(WAVES_M* WAVES_N* KSPLIT * 64) void gemm2_kernel(GemmArgs g, EpiParams ep) {
    using C = Cfg2<BM, BN, WAVES_M, WAVES_N, KSPLIT, STAGES, BK_>;
    __shared__ __attribute__((aligned(1024))) char lds[C::LDS_BYTES];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int nt_m = (g.M + BM - 1) / BM;
    const int nt_n = g.N / BN;
    const int t = xcd_tile(blockIdx.x, nt_m * nt_n);
    const int tm = t % nt_m, tn = t / nt_m;
    const int m0 = tm * BM;
    const int half_out = BN / 2;
    const int F = g.N / 2;

    // descriptors: A may come from two sources split along K
    const __amdgpu_buffer_rsrc_t ra0 = make_rsrc(g.A0, (unsigned)((long)g.M * g.lda0 * 2));
    const __amdgpu_buffer_rsrc_t ra1 = g.A1 ? make_rsrc(g.A1, (unsigned)((long)g.M * g.lda1 * 2)) : ra0;
    const long b_rows = GATED ? 2L * F : (long)g.N;
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(g.B, (unsigned)(b_rows * g.ldb * 2));

    // Swizzle: chunk c of tile row r sits at position c ^ key(r), key(r) = (r / RPB) % CH.
    // Lane L of a load writes row g * RPL + L / CH at position L % CH, g = wave + i * NW; its
    // key is (g * RPL / RPB + L / 16) % CH, which does not depend on i because NW is even.
    static_assert(C::NW % 2 == 0, "swizzle key needs an even wave count");
    const int lr = lane / C::CH;
    const int lkey = ((wave * (C::RPL / C::RPB)) + (lane >> 4)) % C::CH;
    const int lc = (lane % C::CH) ^ lkey;
    const unsigned a0_base = (unsigned)((long)(m0 + wave * C::RPL + lr) * g.lda0 * 2 + lc * 16);
    const unsigned a1_base = (unsigned)((long)(m0 + wave * C::RPL + lr) * g.lda1 * 2 + lc * 16);
    const unsigned a0_step = (unsigned)(C::NW * C::RPL * g.lda0 * 2), a1_step = (unsigned)(C::NW * C::RPL * g.lda1 * 2);
    const unsigned b_lane = (unsigned)(lr * g.ldb * 2 + lc * 16);

    auto issue = [&](int kt, int stage) {
        const int k0 = kt * C::BK;
        char* sa = lds + stage * C::STAGE_BYTES;
        char* sb = sa + C::A_BYTES;
        const bool second = g.A1 && k0 >= g.K0;
        const int ka = second ? (k0 - g.K0) * 2 : k0 * 2;
        const __amdgpu_buffer_rsrc_t ra = second ? ra1 : ra0;
        const unsigned abase = second ? a1_base : a0_base, astep = second ? a1_step : a0_step;
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < C::A_LOADS; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(sa + ((wave + i * C::NW) * C::RPL) * C::ROWB),
                                                     16, abase + i * astep, ka, 0, 0);
#pragma unroll
        for (int i = 0; i < C::B_LOADS; ++i) {
            const int r0 = (wave + i * C::NW) * C::RPL;  // first tile row of this load group (uniform)
            long gr;
            if (GATED) gr = r0 < half_out ? (long)tn * half_out + r0 : (long)F + tn * half_out + (r0 - half_out);
            else gr = (long)tn * BN + r0;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(sb + r0 * C::ROWB), 16, b_lane,
                                                     (int)(gr * g.ldb * 2) + k0 * 2, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    };

    const int kw = wave % KSPLIT;  // k-step share
    const int tw = wave / KSPLIT;  // wave tile position
    const int wm = tw / WAVES_N, wn = tw % WAVES_N;
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
    constexpr int LOADS = C::A_LOADS + C::B_LOADS;
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        if (s < KT) issue(s, s);
    const int lrow = lane & 31, lhalf = lane >> 5;
    for (int kt = 0; kt < KT; ++kt) {
        // wait until tile kt has landed: at most (STAGES - 2) younger tiles may be in flight
        if (kt + STAGES - 2 < KT) wait_vm<LOADS * (STAGES - 2)>();
        else wait_vm<0>();
        __syncthreads();
        if (kt + STAGES - 1 < KT) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
        const char* sa = lds + (kt % STAGES) * C::STAGE_BYTES;
        const char* sb = sa + C::A_BYTES;
        // fragments of k-step q + 1 are read while the MFMAs of k-step q run
        bf16x8 af[2][C::TM], bfr[2][C::TN];
        auto frags = [&](int q, int buf) {
            const int c = (q * KSPLIT + kw) * 2 + lhalf;
#pragma unroll
            for (int i = 0; i < C::TM; ++i) {
                const int r = wm0 + i * 32 + lrow;
                af[buf][i] = *(const bf16x8*)(sa + r * C::ROWB + ((c ^ ((r / C::RPB) % C::CH)) << 4));
            }
#pragma unroll
            for (int j = 0; j < C::TN; ++j) {
                const int r = colbase[j] + lrow;
                bfr[buf][j] = *(const bf16x8*)(sb + r * C::ROWB + ((c ^ ((r / C::RPB) % C::CH)) << 4));
            }
        };
        frags(0, 0);
#pragma unroll
        for (int q = 0; q < C::KS_PER_WAVE; ++q) {
            // pin the order: the next k-step's LDS reads are issued before this k-step's MFMAs
            __builtin_amdgcn_sched_barrier(0);
            if (q + 1 < C::KS_PER_WAVE) frags(q + 1, (q + 1) & 1);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < C::TM; ++i)
#pragma unroll
                for (int j = 0; j < C::TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[q & 1][i], bfr[q & 1][j], acc[i][j], 0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    }

    // ---- epilogue.  The accumulators go to LDS with fully unrolled stores (static register
    // indices), and the epilogue proper runs as a runtime loop over LDS, so the register
    // tile is never indexed dynamically.
    __syncthreads();  // every wave is done reading the stage buffers
    float* red = (float*)lds;
    Epi<bf16> e{ep};
    const bool paired = kind_paired(ep);
    if (ep.kind == EP_HEADS) e.tw = ep.which0 + (tn * BN) / ep.d;
    const bool vt_tile = ep.kind == EP_HEADS && e.tw == 2 && !paired;
    // one (row tile i, column pair jp) unit: 16 rows per lane, columns c and c + BN/2
    auto unit = [&](int i, int jp, const float* lo_src, const float* hi_src) {
        const int lc0 = colbase[jp] + lrow;  // < BN/2
        const int n = tn * BN + lc0;
        for (int r = 0; r < 16; ++r) {
            const int row = m0 + wm0 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
            if (row >= g.M) continue;
            const float lo = lo_src[r << 6], hi = hi_src[r << 6];
            if (paired) e.pair(row, n, BN / 2, tn * half_out + lc0, lo, hi);
            else if (vt_tile) { e.single_vt(row, n, lo); e.single_vt(row, n + BN / 2, hi); }
            else { e.single(row, n, lo); e.single(row, n + BN / 2, hi); }
        }
    };
    if (KSPLIT > 1) {
        // fixed-order sum of the partial tiles of each wave tile: its k-share 0 stores,
        // shares 1.. add in turn
        float* part = red + tw * (C::TM * C::TN * 16 * 64);
        for (int w = 0; w < KSPLIT; ++w) {
            if (kw == w) {
#pragma unroll
                for (int i = 0; i < C::TM; ++i)
#pragma unroll
                    for (int j = 0; j < C::TN; ++j)
#pragma unroll
                        for (int r = 0; r < 16; ++r) {
                            float* p = part + (((i * C::TN + j) * 16 + r) << 6) + lane;
                            *p = w == 0 ? acc[i][j][r] : *p + acc[i][j][r];
                        }
            }
            __syncthreads();
        }
        for (int u = kw; u < C::TM * (C::TN / 2); u += KSPLIT) {
            const int i = u / (C::TN / 2), jp = u % (C::TN / 2);
            unit(i, jp, part + ((i * C::TN + jp) * 16 << 6) + lane,
                 part + ((i * C::TN + jp + C::TN / 2) * 16 << 6) + lane);
        }
        return;
    }
    float* slot = red + wave * (C::TN * 16 * 64);  // this wave's private staging area
#pragma unroll
    for (int i = 0; i < C::TM; ++i) {
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) slot[((j * 16 + r) << 6) + lane] = acc[i][j][r];
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's LDS stores are done
        __builtin_amdgcn_wave_barrier();
        for (int jp = 0; jp < C::TN / 2; ++jp)
            unit(i, jp, slot + ((jp * 16) << 6) + lane, slot + (((jp + C::TN / 2) * 16) << 6) + lane);
        __builtin_amdgcn_s_waitcnt(0xC07F);
        __builtin_amdgcn_wave_barrier();
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
// kind: 0 v1; 1 v2 2x2 waves; 2 v2 one wave tile, k split 4; 3 v2 2x1 waves, k split 2;
//       4 v2 1x2 waves, k split 2
struct TileShape { int bm, bn, kind; };
TileShape bf16_tile(const GemmArgs& g, const EpiParams& e, int tile) {
    switch (tile) {
        case 1: return {256, 256, 1};
        case 2: return {256, 128, 1};
        case 3: return {128, 128, 0};
        case 4: return {128, 128, 2};
        case 5: return {128, 128, 1};
        case 6: return {128, 128, 3};
        case 7: return {128, 256, 4};
        case 8: return {256, 256, 5};   // BK 32, 4 stages
        case 9: return {128, 128, 6};   // 2 stages: two workgroups per CU
        case 10: return {256, 128, 7};  // 3 stages
        case 11: return {256, 128, 8};  // BK 32, 4 stages
        case 12: return {256, 128, 9};  // BK 32, 2 stages: two workgroups per CU
        case 13: return {128, 128, 10}; // BK 32, 3 stages: two workgroups per CU
        default: break;
    }
    // 128 x 128 tiles with shallow pipelines so that two workgroups share a CU (measured best
    // on the 1024-row and 8192-row shapes); head-major tiles must lie inside one projection
    // (d % 128 == 0) and rotary pairs need BN == dh, which 128-wide tiles satisfy
    if (g.M >= 4096) return {128, 128, 10};
    return {128, 128, 6};
}
}  // namespace

bool gemm_shape_ok(int dtype, const GemmArgs& g, const EpiParams& e, int tile) {
    if (g.M <= 0 || g.N <= 0 || g.K <= 0) return false;
    if (dtype == 1) {
        TileShape ts = bf16_tile(g, e, tile);
        if (g.K % 64 || g.N % ts.bn) return false;
        if (g.A1 && (g.K0 % 64)) return false;  // (BK 32 tiles divide this too)
        if (e.kind == EP_HEADS && (e.d % ts.bn || (e.rope && (e.dh != 128 || ts.bn != 128)))) return false;
        if (ts.kind && ((long)g.M * g.lda0 * 2 >= (1L << 32) || (g.A1 && (long)g.M * g.lda1 * 2 >= (1L << 32)) ||
                        (long)g.N * g.ldb * 2 >= (1L << 32)))
            return false;  // 32-bit buffer ranges
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

template <int BM, int BN, int WM_, int WN_, int KS, int ST, int BK = 64>
static hipError_t run_v2(const GemmArgs& g, const EpiParams& e, hipStream_t st) {
    const int nt_m = (g.M + BM - 1) / BM, nt_n = g.N / BN;
    dim3 grid(nt_m * nt_n), block(WM_ * WN_ * KS * 64);
    if (e.kind == EP_GATED)
        hipLaunchKernelGGL((gemm2_kernel<BM, BN, WM_, WN_, KS, ST, true, BK>), grid, block, 0, st, g, e);
    else
        hipLaunchKernelGGL((gemm2_kernel<BM, BN, WM_, WN_, KS, ST, false, BK>), grid, block, 0, st, g, e);
    return hipGetLastError();
}

hipError_t launch_gemm(int dtype, const GemmArgs& g, const EpiParams& e, hipStream_t st, int tile) {
    if (dtype == 1) {
        TileShape ts = bf16_tile(g, e, tile);
        if (ts.kind == 0) return run_bf16<128, 128, 2, 2>(g, e, st);
        if (ts.kind == 1) {
            if (ts.bm == 256 && ts.bn == 256) return run_v2<256, 256, 2, 2, 1, 2>(g, e, st);
            if (ts.bm == 256 && ts.bn == 128) return run_v2<256, 128, 2, 2, 1, 2>(g, e, st);
            return run_v2<128, 128, 2, 2, 1, 3>(g, e, st);
        }
        if (ts.kind == 3) return run_v2<128, 128, 2, 1, 2, 3>(g, e, st);
        if (ts.kind == 5) return run_v2<256, 256, 2, 2, 1, 4, 32>(g, e, st);
        if (ts.kind == 6) return run_v2<128, 128, 2, 2, 1, 2>(g, e, st);
        if (ts.kind == 7) return run_v2<256, 128, 2, 2, 1, 3>(g, e, st);
        if (ts.kind == 8) return run_v2<256, 128, 2, 2, 1, 4, 32>(g, e, st);
        if (ts.kind == 9) return run_v2<256, 128, 2, 2, 1, 2, 32>(g, e, st);
        if (ts.kind == 10) return run_v2<128, 128, 2, 2, 1, 3, 32>(g, e, st);
        if (ts.kind == 4) return run_v2<128, 256, 1, 2, 2, 2>(g, e, st);
        return run_v2<128, 128, 1, 1, 4, 3>(g, e, st);
    }
    const int nt_m = (g.M + 63) / 64, nt_n = g.N / 64;
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(nt_m * nt_n), dim3(256), 0, st, g, e);
    return hipGetLastError();
}

}  // namespace sgd
