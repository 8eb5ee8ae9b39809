// Branch GEMMs of the active units in bf16: C = A . B^T on the CDNA4 matrix cores
// (v_mfma_f32_32x32x16_bf16, fp32 accumulation) with the unit's epilogue fused.
//
// Main loop.  Block tiles up to 256 x 256 with eight waves, two per SIMD, 64-deep k tiles
// (128-byte operand rows, one L2 line each).  Global -> LDS goes through registers:
// buffer_load_dwordx4 into VGPRs (the buffer descriptor's range check returns zeros for
// rows past the matrix, so ragged M and N need no clamping), then ds_write_b128 to an
// XOR-swizzled position so that the 16-byte fragment reads of 16 consecutive rows cover
// the 64 banks once.  The registers are a third pipeline stage next to the two LDS stages,
// and the register -> LDS writes and the next loads are spread one part at a time between
// the MFMAs, so neither the texture unit nor the LDS sees a burst while the MFMA pipes
// run.  Measured on gfx950: issuing a whole tile of loads at once (directly to LDS or to
// registers) left the load and MFMA phases serialised at ~35 % of peak.
//
// Epilogue.  The fp32 accumulator tile goes through LDS in row chunks (one wave row at a
// time); every thread then handles four consecutive columns of a row, so stores are
// vectorised and coalesced and paired columns (gate/up of a gated MLP, the rotary pairs
// (i, i + dh/2) of a head) are read from LDS whatever the wave layout.  V^T columns of a
// head projection are written by a column-major pass (consecutive tokens per thread).
#include "common.h"
#include "kernels.h"

namespace sgd {

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, unsigned bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

template <bool B> struct BoolC { static constexpr bool value = B; };

template <int BM_, int BN_, int WGM_, int WGN_, int BK_, int STAGES_>
struct TileCfg {
    static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_, BK = BK_, STAGES = STAGES_;
    static constexpr int NW = WGM * WGN;
    static constexpr int NT = NW * 64;
    static constexpr int WM = BM / WGM, WN = BN / WGN;   // wave tile
    static constexpr int TM = WM / 32, TN = WN / 32;     // 32 x 32 MFMA blocks per wave
    static constexpr int ROWB = BK * 2;                  // bytes per LDS tile row
    static constexpr int CH = BK / 8;                    // 16-byte chunks per row
    static constexpr int RPB = 256 / ROWB;               // rows per 256-byte bank line
    static constexpr int A_BYTES = BM * ROWB, B_BYTES = BN * ROWB;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static constexpr int KSTEPS = BK / 16;
    static constexpr int EPR = WM;                       // epilogue chunk: one wave row
    static constexpr int EPS = BN + 8;                   // fp32 row stride of the staged chunk
    static constexpr int EPI_BYTES = EPR * EPS * 4;
    static constexpr int LDS_BYTES = STAGE_BYTES * STAGES > EPI_BYTES ? STAGE_BYTES * STAGES : EPI_BYTES;
    static_assert(TM >= 1 && TN >= 1 && WM % 32 == 0 && WN % 32 == 0, "wave tile");
    static_assert(BK == 64, "128-byte operand rows: one L2 line per row and chunk-swizzled LDS rows");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS");
    static_assert((4 * EPS) % 64 == 32, "conflict-free accumulator staging");
};

// --------------------------------------------------------------------------- epilogue

struct Epi4 {
    EpiParams p;
    int N;  // product columns

    __device__ __forceinline__ static void store4(bf16* dst, const float v[4]) {
        bf16x4 s;
        s[0] = f2bf(v[0]); s[1] = f2bf(v[1]); s[2] = f2bf(v[2]); s[3] = f2bf(v[3]);
        *(bf16x4*)dst = s;
    }
    __device__ __forceinline__ void add_bias(int n, float v[4]) const {
        if (p.bias) {
            const f32x4 b = *(const f32x4*)(p.bias + n);
            v[0] += b[0]; v[1] += b[1]; v[2] += b[2]; v[3] += b[3];
        }
    }

    // EP_ACT: out[row, n..n+3] = act(v + bias)
    __device__ __forceinline__ void act(int row, int n, float v[4]) const {
        add_bias(n, v);
#pragma unroll
        for (int c = 0; c < 4; ++c) v[c] = apply_act(p.act, v[c]);
        store4((bf16*)p.out + (long)row * p.ldo + n, v);
    }
    // EP_GATED: out[row, on..on+3] = act(g + b_g) * (u + b_u)
    __device__ __forceinline__ void gated(int row, int on, float g[4], float u[4]) const {
        if (p.bias) {
            const f32x4 bg = *(const f32x4*)(p.bias + on);
            const f32x4 bu = *(const f32x4*)(p.bias + p.F + on);
#pragma unroll
            for (int c = 0; c < 4; ++c) { g[c] += bg[c]; u[c] += bu[c]; }
        }
        float o[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) o[c] = apply_act(p.act, g[c]) * u[c];
        store4((bf16*)p.out + (long)row * p.ldo + on, o);
    }
    // EP_RESID: v = (acc + bias) [* gate]; h += v; delta = v | delta += v; hcopy = bf16(h)
    __device__ __forceinline__ void resid(int row, int n, float v[4]) const {
        add_bias(n, v);
        if (p.gate) {
            const f32x4 gt = *(const f32x4*)(p.gate + (long)(row / p.ntok) * p.gate_ld + n);
#pragma unroll
            for (int c = 0; c < 4; ++c) v[c] *= gt[c];
        }
        const long idx = (long)row * p.d + n;
        f32x4 hv = *(const f32x4*)(p.h + idx);
        float hn[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) { hn[c] = hv[c] + v[c]; hv[c] = hn[c]; }
        *(f32x4*)(p.h + idx) = hv;
        if (p.delta_mode == 1) {
            *(f32x4*)(p.delta + idx) = f32x4{v[0], v[1], v[2], v[3]};
        } else if (p.delta_mode == 2) {
            f32x4 dv = *(const f32x4*)(p.delta + idx);
#pragma unroll
            for (int c = 0; c < 4; ++c) dv[c] = dv[c] + v[c];
            *(f32x4*)(p.delta + idx) = dv;
        }
        if (p.hcopy) store4((bf16*)p.hcopy + idx, hn);
    }
    // EP_SKIP: h = acc + bias [+ cached delta]; hcopy = bf16(h)
    __device__ __forceinline__ void skip(int row, int n, float v[4]) const {
        add_bias(n, v);
        const long idx = (long)row * p.d + n;
        if (p.delta_mode == 1) {
            const f32x4 dv = *(const f32x4*)(p.delta + idx);
#pragma unroll
            for (int c = 0; c < 4; ++c) v[c] = v[c] + dv[c];
        }
        *(f32x4*)(p.h + idx) = f32x4{v[0], v[1], v[2], v[3]};
        if (p.hcopy) store4((bf16*)p.hcopy + idx, v);
    }
};

// --------------------------------------------------------------------------- epilogue stage

// Stage one wave row of the accumulator tile at a time in LDS, then store it with the
// epilogue of ep.kind (every thread handles four consecutive columns of a row).
template <class C>
__device__ __forceinline__ void epilogue(f32x16 (&acc)[C::TM][C::TN], char* lds, const GemmArgs& g,
                                         const EpiParams& ep, int m0, int tn, int wm, int wn0) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int lrow = lane & 31, lhalf = lane >> 5;
    __syncthreads();  // every wave is done with the stage buffers
    float* st = (float*)lds;
    Epi4 e{ep, g.N};
    const int n0 = tn * C::BN;
    for (int ch = 0; ch < C::WGM; ++ch) {
        if (wm == ch) {
#pragma unroll
            for (int i = 0; i < C::TM; ++i)
#pragma unroll
                for (int j = 0; j < C::TN; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int row = i * 32 + (r >> 2) * 8 + lhalf * 4 + (r & 3);
                        st[row * C::EPS + wn0 + j * 32 + lrow] = acc[i][j][r];
                    }
        }
        __syncthreads();
        const int r0 = m0 + ch * C::EPR;  // first output row of the chunk
        if (ep.kind == EP_GATED) {
            constexpr int IT = C::EPR * (C::BN / 8);
            for (int it = tid; it < IT; it += C::NT) {
                const int rr = it / (C::BN / 8), c = (it % (C::BN / 8)) * 4;
                const int row = r0 + rr;
                if (row >= g.M) continue;
                const f32x4 gv = *(const f32x4*)(st + rr * C::EPS + c);
                const f32x4 uv = *(const f32x4*)(st + rr * C::EPS + C::BN / 2 + c);
                float gg[4] = {gv[0], gv[1], gv[2], gv[3]}, uu[4] = {uv[0], uv[1], uv[2], uv[3]};
                e.gated(row, tn * (C::BN / 2) + c, gg, uu);
            }
        } else if (ep.kind == EP_HEADS) {
            // q/k columns row-major (a thread stores four dims of one token), with the rotary
            // pair read from LDS; V^T columns column-major (four tokens of one dim)
            const int vstart = (2 - ep.which0) * ep.d;  // first product column of V
            const int hd = ep.dh / 2;
            constexpr int IT = C::EPR * (C::BN / 4);
            for (int it = tid; it < IT; it += C::NT) {
                const int rr = it / (C::BN / 4), c = (it % (C::BN / 4)) * 4;
                const int row = r0 + rr, n = n0 + c;
                if (row >= g.M || n >= g.N || n >= vstart) continue;
                const int proj = ep.which0 + n / ep.d;
                const int nn = n - (proj - ep.which0) * ep.d;
                const int hh = nn / ep.dh, j = nn - hh * ep.dh;
                const int b = row / ep.ntok, tok = row - b * ep.ntok;
                const f32x4 x = *(const f32x4*)(st + rr * C::EPS + c);
                float v[4] = {x[0], x[1], x[2], x[3]};
                e.add_bias(n, v);
                if (ep.rope) {
                    const bool lo = j < hd;
                    const int pc = lo ? c + hd : c - hd;  // partner columns in this tile
                    const f32x4 y = *(const f32x4*)(st + rr * C::EPS + pc);
                    float pv[4] = {y[0], y[1], y[2], y[3]};
                    e.add_bias(lo ? n + hd : n - hd, pv);
                    const int jb = lo ? j : j - hd;
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const float inv = exp2f(-(2.0f * (float)(jb + u) / (float)ep.dh) * ep.rope_log2_theta);
                        float s, co;
                        sincosf((float)tok * inv, &s, &co);
                        v[u] = lo ? v[u] * co - pv[u] * s : v[u] * co + pv[u] * s;
                    }
                }
                bf16* base = (bf16*)(proj == 0 ? ep.q : ep.k);
                Epi4::store4(base + (((long)b * ep.H + hh) * ep.np + tok) * ep.dh + j, v);
            }
            const int vc0 = vstart > n0 ? vstart - n0 : 0;  // first V column of the tile
            const int vcols = min(C::BN, g.N - n0) - vc0;
            if (vcols > 0) {
                const int ITV = vcols * (C::EPR / 4);
                for (int it = tid; it < ITV; it += C::NT) {
                    const int c = vc0 + it / (C::EPR / 4), rg = (it % (C::EPR / 4)) * 4;
                    const int n = n0 + c;
                    const int nn = n - vstart;
                    const int hh = nn / ep.dh, j = nn - hh * ep.dh;
                    const float bv = ep.bias ? ep.bias[n] : 0.f;
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int row = r0 + rg + u;
                        if (row >= g.M) break;
                        const int b = row / ep.ntok, tok = row - b * ep.ntok;
                        ((bf16*)ep.vt)[(((long)b * ep.H + hh) * ep.dh + j) * ep.np + tok] =
                            f2bf(st[(rg + u) * C::EPS + c] + bv);
                    }
                }
            }
        } else {
            constexpr int IT = C::EPR * (C::BN / 4);
            for (int it = tid; it < IT; it += C::NT) {
                const int rr = it / (C::BN / 4), c = (it % (C::BN / 4)) * 4;
                const int row = r0 + rr, n = n0 + c;
                if (row >= g.M || n >= g.N) continue;
                const f32x4 x = *(const f32x4*)(st + rr * C::EPS + c);
                float v[4] = {x[0], x[1], x[2], x[3]};
                if (ep.kind == EP_ACT) e.act(row, n, v);
                else if (ep.kind == EP_RESID) e.resid(row, n, v);
                else e.skip(row, n, v);
            }
        }
        __syncthreads();
    }
}

// --------------------------------------------------------------------------- kernel
//
// Three-stage pipeline with two LDS stages: in the period between the barriers before the
// last k-steps of tiles kt - 1 and kt, the MFMAs consume tile kt (one stage), tile kt + 1
// moves from registers into the other stage, and tile kt + 2 is loaded into the freed
// registers.  The register -> LDS writes and the loads are interleaved one part at a time
// with the period's MFMAs (part p after MFMA slot p * SLOTS / PARTS), so neither the
// texture unit nor the LDS sees a burst and both SIMD waves keep issuing MFMAs.

template <class C>
__global__ __launch_bounds__(C::NT, 2) void gemm_bf16_kernel(GemmArgs g, EpiParams ep) {
    static_assert(C::STAGES == 2, "two LDS stages plus the register stage");
    __shared__ __attribute__((aligned(1024))) char lds[C::LDS_BYTES];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool gated = ep.kind == EP_GATED;
    const int nt_m = (g.M + C::BM - 1) / C::BM;
    const int nt_n = (g.N + C::BN - 1) / C::BN;
    const int total = nt_m * nt_n;
    const int bid = blockIdx.x;
    const int t = total % 8 == 0 ? (bid % 8) * (total / 8) + bid / 8 : bid;
    const int tm = t % nt_m, tn = t / nt_m;
    const int m0 = tm * C::BM;
    const int F = g.N / 2;

    const __amdgpu_buffer_rsrc_t ra0 = buf_rsrc(g.A0, (unsigned)((long)g.M * g.lda0 * 2));
    const __amdgpu_buffer_rsrc_t ra1 = g.A1 ? buf_rsrc(g.A1, (unsigned)((long)g.M * g.lda1 * 2)) : ra0;
    const __amdgpu_buffer_rsrc_t rb = buf_rsrc(g.B, (unsigned)((long)g.N * g.ldb * 2));

    // thread -> (row, chunk) of a stage: chunk tid % CH of rows tid / CH + p * RPP; parts
    // 0 .. AP-1 are A rows, AP .. AP+BP-1 are B rows
    constexpr int RPP = C::NT / C::CH;
    constexpr int AP = C::BM / RPP, BP = C::BN / RPP, PARTS = AP + BP;
    static_assert(C::BM % RPP == 0 && C::BN % RPP == 0 && (C::BN / 2) % RPP == 0, "pass split");
    const int vc = tid % C::CH, vr = tid / C::CH;
    unsigned goff0[PARTS], goff1[AP];
    int loff[PARTS];
#pragma unroll
    for (int p = 0; p < AP; ++p) {
        const int r = vr + p * RPP;
        goff0[p] = (unsigned)((long)(m0 + r) * g.lda0 * 2 + vc * 16);
        goff1[p] = (unsigned)((long)(m0 + r) * g.lda1 * 2 + vc * 16);
        loff[p] = r * C::ROWB + ((vc ^ ((r / C::RPB) % C::CH)) << 4);
    }
#pragma unroll
    for (int p = 0; p < BP; ++p) {
        const int r = vr + p * RPP;
        long gr;
        if (gated) gr = r < C::BN / 2 ? (long)tn * (C::BN / 2) + r : (long)F + tn * (C::BN / 2) + (r - C::BN / 2);
        else gr = (long)tn * C::BN + r;
        goff0[AP + p] = (unsigned)(gr * g.ldb * 2 + vc * 16);
        loff[AP + p] = C::A_BYTES + r * C::ROWB + ((vc ^ ((r / C::RPB) % C::CH)) << 4);
    }
    u32x4 vreg[PARTS];
    auto gload = [&](int kt, int p) {
        const int k0 = kt * C::BK;
        if (p < AP) {
            const bool second = g.A1 && k0 >= g.K0;
            vreg[p] = __builtin_amdgcn_raw_buffer_load_b128(second ? ra1 : ra0, second ? goff1[p] : goff0[p],
                                                            second ? (k0 - g.K0) * 2 : k0 * 2, 0);
        } else {
            vreg[p] = __builtin_amdgcn_raw_buffer_load_b128(rb, goff0[p], k0 * 2, 0);
        }
    };
    auto lwrite = [&](int stage, int p) { *(u32x4*)(lds + stage * C::STAGE_BYTES + loff[p]) = vreg[p]; };

    const int wm = wave / C::WGN, wn = wave % C::WGN;
    const int wm0 = wm * C::WM, wn0 = wn * C::WN;
    const int lrow = lane & 31, lhalf = lane >> 5;

    f32x16 acc[C::TM][C::TN];
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    bf16x8 af[2][C::TM], bfr[2][C::TN];
    auto frags = [&](int stage, int q, int buf) {
        const char* sa = lds + stage * C::STAGE_BYTES;
        const char* sb = sa + C::A_BYTES;
        const int c = q * 2 + lhalf;
#pragma unroll
        for (int i = 0; i < C::TM; ++i) {
            const int r = wm0 + i * 32 + lrow;
            af[buf][i] = *(const bf16x8*)(sa + r * C::ROWB + ((c ^ ((r / C::RPB) % C::CH)) << 4));
        }
#pragma unroll
        for (int j = 0; j < C::TN; ++j) {
            const int r = wn0 + j * 32 + lrow;
            bfr[buf][j] = *(const bf16x8*)(sb + r * C::ROWB + ((c ^ ((r / C::RPB) % C::CH)) << 4));
        }
    };
    const int KT = g.K / C::BK;
    constexpr int MPK = C::TM * C::TN, SLOTS = C::KSTEPS * MPK;
    static_assert(PARTS <= SLOTS, "part spreading");
    // MFMAs of one k-step; `part` is the k-step's position in its period.  The period moves
    // tile wt (registers -> stage ws) and loads tile lt into the registers.  The compiler
    // inserts the vmcnt waits from the register dependences; in the branch-free steady state
    // (STEADY) that is vmcnt(PARTS - 1) before every write.
    auto mfmas = [&](int buf, int part, int wt, int ws, int lt, auto steady) {
        constexpr bool STEADY = decltype(steady)::value;
        const bool wr = STEADY || wt < KT, ld = STEADY || lt < KT;
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
#pragma unroll
            for (int j = 0; j < C::TN; ++j) {
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[buf][i], bfr[buf][j], acc[i][j], 0, 0, 0);
                const int slot = part * MPK + i * C::TN + j;
                const int p = (slot * PARTS + SLOTS - 1) / SLOTS;
                if (p < PARTS && (p * SLOTS) / PARTS == slot && wr) {
                    __builtin_amdgcn_sched_barrier(0);
                    lwrite(ws, p);
                    if (ld) gload(lt, p);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
    };

    // prologue: tile 0 into stage 0, tile 1 into the registers.  The first period has no
    // "last k-step of tile -1", so the parts of its first slot group (write tile 1, load
    // tile 2) are done here.
#pragma unroll
    for (int p = 0; p < PARTS; ++p) gload(0, p);
#pragma unroll
    for (int p = 0; p < PARTS; ++p) lwrite(0, p);
    if (KT > 1) {
#pragma unroll
        for (int p = 0; p < PARTS; ++p) gload(1, p);
#pragma unroll
        for (int p = 0; p < PARTS; ++p) {
            if ((p * SLOTS) / PARTS < MPK) {
                lwrite(1, p);
                if (KT > 2) gload(2, p);
            }
        }
    }
    __syncthreads();
    frags(0, 0, 0);
    // one k tile; the period of tile kt (from the barrier before tile kt-1's last k-step)
    // moves tile kt + 1 into stage st ^ 1 and loads tile kt + 2, and the period of tile
    // kt + 1 starts with the last k-step
    auto iter = [&](int kt, auto steady) {
        constexpr bool STEADY = decltype(steady)::value;
        const int st = kt & 1;
#pragma unroll
        for (int q = 0; q < C::KSTEPS; ++q) {
            const int cur = q & 1, nxt = cur ^ 1;
            __builtin_amdgcn_sched_barrier(0);
            if (q + 1 < C::KSTEPS) {
                frags(st, q + 1, nxt);
            } else if (STEADY || kt + 1 < KT) {
                __syncthreads();  // tile kt + 1 is in stage st ^ 1; stage st is free
                frags(st ^ 1, 0, nxt);
            }
            __builtin_amdgcn_sched_barrier(0);
            if (q + 1 < C::KSTEPS) mfmas(cur, q + 1, kt + 1, st ^ 1, kt + 2, steady);
            else mfmas(cur, 0, kt + 2, st, kt + 3, steady);
        }
    };
    static_assert(C::KSTEPS % 2 == 0, "fragment ring");
    int kt = 0;
    for (; kt + 3 < KT; ++kt) iter(kt, BoolC<true>{});
    for (; kt < KT; ++kt) iter(kt, BoolC<false>{});
    epilogue<C>(acc, lds, g, ep, m0, tn, wm, wn0);
}

// --------------------------------------------------------------------------- dispatch

namespace {
// block tiles (BM, BN); eight waves, 64-deep k tiles, two LDS stages plus the register stage
using T256x256 = TileCfg<256, 256, 4, 2, 64, 2>;  // 64 x 128 wave tiles
using T256x128 = TileCfg<256, 128, 4, 2, 64, 2>;  // 64 x 64
using T128x256 = TileCfg<128, 256, 2, 4, 64, 2>;  // 64 x 64
using T128x128 = TileCfg<128, 128, 2, 4, 64, 2>;  // 64 x 32

struct Shape { int bm, bn; double rate; };
// tile id -> block shape and its per-CU throughput relative to 256 x 256 (measured on the
// branch GEMM shapes: smaller tiles move more operand bytes per FLOP through L2 and LDS)
Shape tile_shape(int tile) {
    switch (tile) {
        case 1: return {256, 256, 1.0};
        case 2: return {256, 128, 0.78};
        case 3: return {128, 256, 0.80};
        case 4: return {128, 128, 0.51};
        default: return {0, 0, 0.0};
    }
}
}  // namespace

// Automatic choice: one workgroup per CU, so a launch of n tiles takes ceil(n / 256) rounds;
// pick the tile with the least rounds x tile area / per-CU rate (e.g. at 1024 rows the
// 4096-column GEMMs run 128 x 128 tiles, one full round, rather than 64 large tiles).
int gemm_bf16_auto_tile(const GemmArgs& g, const EpiParams& e) {
    int best = 1;
    double best_t = 1e300;
    for (int tile = 1; tile <= kGemmTiles; ++tile) {
        const Shape s = tile_shape(tile);
        if (e.kind == EP_GATED && g.N % s.bn) continue;
        if (e.kind == EP_HEADS && e.rope && (s.bn % e.dh || e.d % s.bn)) continue;
        const long tiles = (long)((g.M + s.bm - 1) / s.bm) * ((g.N + s.bn - 1) / s.bn);
        const double t = (double)((tiles + 255) / 256) * s.bm * s.bn / s.rate;
        if (t < best_t * 0.999) { best_t = t; best = tile; }
    }
    return best;
}

static bool aligned(const void* p, unsigned a) { return ((uintptr_t)p % a) == 0; }

bool gemm_bf16_shape_ok(const GemmArgs& g, const EpiParams& e, int tile) {
    if (tile == 0) tile = gemm_bf16_auto_tile(g, e);
    // vector accesses of the loader and the epilogue: 16-byte operand rows and fp32 vectors,
    // 8-byte bf16 output groups
    if (!aligned(g.A0, 16) || !aligned(g.A1, 16) || !aligned(g.B, 16) || !aligned(e.bias, 16) ||
        !aligned(e.gate, 16) || e.gate_ld % 4 || !aligned(e.h, 16) || !aligned(e.delta, 16) ||
        !aligned(e.out, 8) || !aligned(e.hcopy, 8) || !aligned(e.q, 8) || !aligned(e.k, 8) || !aligned(e.vt, 2))
        return false;
    const Shape s = tile_shape(tile);
    if (!s.bm) return false;
    if (g.K % 64 || (g.A1 && g.K0 % 64)) return false;
    if (g.N % 4 || g.lda0 % 8 || (g.A1 && g.lda1 % 8) || g.ldb % 8) return false;  // 16-byte rows
    if (e.kind == EP_GATED && (g.N % s.bn || e.ldo % 4)) return false;
    if (e.kind == EP_ACT && e.ldo % 4) return false;
    if ((e.kind == EP_RESID || e.kind == EP_SKIP) && (g.N != e.d)) return false;
    if (e.kind == EP_HEADS) {
        if (e.d % 4 || e.dh % 4) return false;
        if (e.rope && (e.dh % 8 || s.bn % e.dh || e.d % s.bn)) return false;  // whole heads per tile
    }
    if ((long)g.M * g.lda0 * 2 >= (1L << 32) || (g.A1 && (long)g.M * g.lda1 * 2 >= (1L << 32)) ||
        (long)g.N * g.ldb * 2 >= (1L << 32))
        return false;  // 32-bit buffer ranges
    return true;
}

template <class C>
static hipError_t run_tile(const GemmArgs& g, const EpiParams& e, hipStream_t st) {
    const int nt_m = (g.M + C::BM - 1) / C::BM, nt_n = (g.N + C::BN - 1) / C::BN;
    hipLaunchKernelGGL((gemm_bf16_kernel<C>), dim3(nt_m * nt_n), dim3(C::NT), 0, st, g, e);
    return hipGetLastError();
}

hipError_t launch_gemm_bf16(const GemmArgs& g, const EpiParams& e, hipStream_t st, int tile) {
    if (tile == 0) tile = gemm_bf16_auto_tile(g, e);
    switch (tile) {
        case 1: return run_tile<T256x256>(g, e, st);
        case 2: return run_tile<T256x128>(g, e, st);
        case 3: return run_tile<T128x256>(g, e, st);
        case 4: return run_tile<T128x128>(g, e, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace sgd
