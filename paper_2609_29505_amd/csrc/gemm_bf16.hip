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
#include <type_traits>
#include <utility>

#include "common.h"
#include "kernels.h"
#include "tile_order.h"

namespace sgd {

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, unsigned bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Rotary head projections: the q and k product columns of each head are taken in the order
// (0, dh/2, 1, dh/2 + 1, ...), so the two dims of every rotary pair are adjacent columns and a
// block tile of any even width holds whole pairs.  Column n of the product is weight row (and
// bias entry) rope_row(n); v columns (n >= vstart) keep their order.
__device__ __forceinline__ long rope_row(long n, int dh, long vstart) {
    if (n >= vstart) return n;
    const int hl = (int)(n % dh);
    return n - hl + ((hl & 1) ? dh / 2 + hl / 2 : hl / 2);
}

template <int I> using IntC = std::integral_constant<int, I>;

// f(IntC<0>{}), ..., f(IntC<N - 1>{})
template <class Fn, int... I>
__device__ __forceinline__ void static_for_impl(Fn& f, std::integer_sequence<int, I...>) {
    (f(IntC<I>{}), ...);
}
template <int N, class Fn>
__device__ __forceinline__ void static_for(Fn&& f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

template <int BM_, int BN_, int WGM_, int WGN_, int BK_, int STAGES_, int OCC_ = 2, int RD_ = 1>
struct TileCfg {
    static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_, BK = BK_, STAGES = STAGES_;
    static constexpr int OCC = OCC_;                     // waves per SIMD the registers allow
    static constexpr int RD = RD_;                       // k tiles in flight in registers
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
    static constexpr int EPR = WGM * 32;                 // epilogue chunk: one MFMA row block per wave row
    static constexpr int EPS = BN + 8;                   // fp32 row stride of the staged chunk
    static constexpr int EPI_BYTES = (EPR * EPS + BN) * 4;  // + one row of bias columns
    static constexpr int LDS_BYTES = STAGE_BYTES * STAGES > EPI_BYTES ? STAGE_BYTES * STAGES : EPI_BYTES;
    static_assert(TM >= 1 && TN >= 1 && WM % 32 == 0 && WN % 32 == 0, "wave tile");
    static_assert(BK == 64, "128-byte operand rows: one L2 line per row and chunk-swizzled LDS rows");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS");
    static_assert((4 * EPS) % 64 == 32, "conflict-free accumulator staging");
};

// --------------------------------------------------------------------------- epilogue
//
// Every item loop below has a compile-time trip count and runs in two phases, all loads
// (LDS values, bias, gate, h, delta) first and all stores after: a loop that alternated a
// global store with the next load made the compiler wait for each store's completion
// before reusing its registers, one memory round trip per item.

__device__ __forceinline__ void store_bf16x4(bf16* dst, const float v[4]) {
    bf16x4 s;
    s[0] = f2bf(v[0]); s[1] = f2bf(v[1]); s[2] = f2bf(v[2]); s[3] = f2bf(v[3]);
    *(bf16x4*)dst = s;
}
__device__ __forceinline__ f32x4 ld4(const float* p) { return *(const f32x4*)p; }

template <int ACT>
__device__ __forceinline__ float act_fn(float x) {
    if (ACT == ACT_GELU_ERF) return gelu_erf(x);
    if (ACT == ACT_GELU_TANH) return gelu_tanh(x);
    if (ACT == ACT_SILU) return silu(x);
    return x;
}

// calls f(tag) with the activation as a compile-time constant
template <class Fn>
__device__ __forceinline__ void with_act(int act, Fn&& f) {
    switch (act) {
        case ACT_GELU_ERF: f(std::integral_constant<int, ACT_GELU_ERF>{}); break;
        case ACT_GELU_TANH: f(std::integral_constant<int, ACT_GELU_TANH>{}); break;
        case ACT_SILU: f(std::integral_constant<int, ACT_SILU>{}); break;
        default: f(std::integral_constant<int, ACT_NONE>{}); break;
    }
}

// Stage the accumulator tile in LDS one MFMA row block per wave row at a time, then store
// it with the epilogue of ep.kind.  Every thread keeps the same four columns for all its
// items (NT is a multiple of the items per row), and the tile's bias columns sit in an LDS
// row of their own, so the q/k/v, activation and gated epilogues issue no global loads.
template <class C>
__device__ __forceinline__ void epilogue(f32x16 (&acc)[C::TM][C::TN], char* lds, const GemmArgs& g,
                                         const EpiParams& ep, int m0, int tn, int wm, int wn0, int split) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int lrow = lane & 31, lhalf = lane >> 5;
    // Thread t handles rows r0(t) + u * RPT of its columns.  When the items of a row do not
    // divide the block (192-column tiles), the threads past the last whole pass have no items
    // (r0 = EPR) and a thread's last items may fall past the chunk (EX* false: checked).
    constexpr int RI = C::BN / 4;                        // four-column items per row
    constexpr int RPT = C::NT / RI;                      // chunk rows per pass of the block
    constexpr int PER = (C::EPR + RPT - 1) / RPT;        // items per thread per chunk
    constexpr bool EXA = C::NT % RI == 0 && C::EPR % RPT == 0;
    constexpr int RIG = RI / 2, RPTG = C::NT / RIG, PERG = (C::EPR + RPTG - 1) / RPTG;  // gated: gate half
    constexpr bool EXG = C::NT % RIG == 0 && C::EPR % RPTG == 0;
    constexpr int EB = PER < 4 ? PER : 4;                // residual items per load group
    float* st = (float*)lds;
    float* sbias = st + C::EPR * C::EPS;                 // the tile's bias columns
    const int n0 = tn * C::BN;
    const bool gated = ep.kind == EP_GATED;
    const bool rope = ep.kind == EP_HEADS && ep.rope;
    const int vstart = ep.kind == EP_HEADS ? (2 - ep.which0) * ep.d : 0;  // first v^T product column
    __syncthreads();  // every wave is done with the stage buffers
    for (int c = tid; c < C::BN; c += C::NT) {
        float b = 0.f;
        if (ep.bias && split == 0) {
            if (gated) b = ep.bias[c < C::BN / 2 ? tn * (C::BN / 2) + c : ep.F + tn * (C::BN / 2) + c - C::BN / 2];
            else if (n0 + c < g.N) b = ep.bias[rope ? rope_row(n0 + c, ep.dh, vstart) : n0 + c];
        }
        sbias[c] = b;
    }
    // operand pointers and the token split held in registers before any store (a pointer
    // picked from the argument block later would be a memory load, and waiting for it
    // would wait for every store issued before)
    bf16* const qptr = (bf16*)ep.q;
    bf16* const kptr = (bf16*)ep.k;
    // sample of a row: floor((row + 0.5) / ntok) in fp32 is exact while row < 2^21
    const float rntok = 1.0f / (float)ep.ntok;
    auto sample_of = [&](int row) { return (int)(((float)row + 0.5f) * rntok); };
    const int c = (tid % RI) * 4, rr0 = tid < RI * RPT ? tid / RI : C::EPR;  // columns, first row
    const int cg = (tid % RIG) * 4, rrg0 = tid < RIG * RPTG ? tid / RIG : C::EPR;  // gated
    const int n = n0 + c;
    // q/k columns without rotation: projection, head and dims of this thread's columns
    int proj = 0, hh = 0, j = 0;
    if (ep.kind == EP_HEADS && n < g.N && n < vstart) {
        proj = ep.which0 + n / ep.d;
        const int nn = n - (proj - ep.which0) * ep.d;
        hh = nn / ep.dh;
        j = nn - hh * ep.dh;
    }
    // rotary q/k columns (pairs adjacent, see rope_row): a thread owns eight consecutive
    // columns, i.e. the four rotary pairs of dims pj .. pj+3 and pj+dh/2 .. pj+dh/2+3 of head
    // ph (one head: dh % 8 == 0), so one sine/cosine serves both dims of a pair; invt holds
    // the pairs' inverse frequencies in turns per token.  Tiles may hold columns of q and k,
    // or of k and v (v columns go through the V^T path below).
    constexpr int RIP = C::BN / 8, RPTP = C::NT / RIP, PERP = (C::EPR + RPTP - 1) / RPTP;
    constexpr bool EXP = C::NT % RIP == 0 && C::EPR % RPTP == 0;
    const int pc = (tid % RIP) * 8;  // first tile column of the thread's pairs
    const bool rope_thread = rope && n0 + pc < vstart && n0 + pc < g.N;
    const bool rope_tile = rope && n0 < vstart;
    const int rrp0 = tid < RIP * RPTP ? tid / RIP : C::EPR;
    int ph = 0, pj = 0;
    float invt[4] = {0.f, 0.f, 0.f, 0.f};
    bf16* pbase = qptr;
    if (rope_thread) {
        const int pn = n0 + pc;
        const int pproj = ep.which0 + pn / ep.d;
        const int nn = pn - (pproj - ep.which0) * ep.d;
        ph = nn / ep.dh;
        pj = (nn - ph * ep.dh) / 2;
        pbase = pproj == 0 ? qptr : kptr;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            invt[q] = exp2f(-(2.0f * (float)(pj + q) / (float)ep.dh) * ep.rope_log2_theta) * 0.159154943091895336f;
    }
    // V^T columns straight from the accumulators: in the MFMA output layout lane l holds
    // column l % 32 of a 32 x 32 block and, for register group q, rows q * 8 + (l / 32) * 4
    // + 0..3, i.e. four consecutive tokens of one V^T row (d % 32 == 0: a block is all V or
    // none)
    if (ep.kind == EP_HEADS) {
        bf16* vt = (bf16*)ep.vt;
#pragma unroll
        for (int jj = 0; jj < C::TN; ++jj) {
            const int nb = n0 + wn0 + jj * 32;  // first product column of the block
            if (nb < vstart || nb >= g.N) continue;
            const int nv = nb + lrow - vstart;
            const int vh = nv / ep.dh, vj = nv - vh * ep.dh;
            const float bv = ep.bias ? ep.bias[nb + lrow] : 0.f;
#pragma unroll
            for (int i = 0; i < C::TM; ++i)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int row0 = m0 + wm * C::WM + i * 32 + q * 8 + lhalf * 4;
                    if (row0 >= g.M) continue;
                    const int bs0 = sample_of(row0), tok0 = row0 - bs0 * ep.ntok;
                    float o[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) o[u] = acc[i][jj][q * 4 + u] + bv;
                    if (tok0 % 4 == 0 && tok0 + 3 < ep.ntok && row0 + 3 < g.M) {
                        store_bf16x4(vt + (((long)bs0 * ep.H + vh) * ep.dh + vj) * ep.np + tok0, o);
                    } else {
                        for (int u = 0; u < 4; ++u) {
                            const int row = row0 + u;
                            if (row >= g.M) break;
                            const int bs = sample_of(row), tok = row - bs * ep.ntok;
                            vt[(((long)bs * ep.H + vh) * ep.dh + vj) * ep.np + tok] = f2bf(o[u]);
                        }
                    }
                }
        }
    }
    // chunk ch holds MFMA row block ch of every wave row, so each wave's accumulators die
    // chunk by chunk; chunk row rr is tile row (rr / 32) * WM + ch * 32 + rr % 32
#pragma unroll 1
    for (int ch = 0; ch < C::TM; ++ch) {
        // static register indices: the chunk loop itself is not unrolled
#pragma unroll
        for (int i = 0; i < C::TM; ++i) {
            if (i != ch) continue;
#pragma unroll
            for (int jj = 0; jj < C::TN; ++jj)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = wm * 32 + (r >> 2) * 8 + lhalf * 4 + (r & 3);
                    st[row * C::EPS + wn0 + jj * 32 + lrow] = acc[i][jj][r];
                }
        }
        __syncthreads();
        auto grow = [&](int rr) { return m0 + (rr >> 5) * C::WM + ch * 32 + (rr & 31); };
        if (ep.kind == EP_GATED) {
            const f32x4 bg = ld4(sbias + cg), bu = ld4(sbias + C::BN / 2 + cg);
            with_act(ep.act, [&](auto actc) {
                constexpr int ACT = decltype(actc)::value;
#pragma unroll 2
                for (int u = 0; u < PERG; ++u) {
                    const int rr = rrg0 + u * RPTG, row = grow(rr);
                    if (!EXG && rr >= C::EPR) continue;
                    const f32x4 gv = ld4(st + rr * C::EPS + cg), uv = ld4(st + rr * C::EPS + C::BN / 2 + cg);
                    if (row >= g.M) continue;
                    float o[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) o[q] = act_fn<ACT>(gv[q] + bg[q]) * (uv[q] + bu[q]);
                    store_bf16x4((bf16*)ep.out + (long)row * ep.ldo + tn * (C::BN / 2) + cg, o);
                }
            });
        } else if (ep.kind == EP_ACT) {
            const f32x4 bb = ld4(sbias + c);
            with_act(ep.act, [&](auto actc) {
                constexpr int ACT = decltype(actc)::value;
#pragma unroll 2
                for (int u = 0; u < PER; ++u) {
                    const int rr = rr0 + u * RPT, row = grow(rr);
                    if (!EXA && rr >= C::EPR) continue;
                    const f32x4 v = ld4(st + rr * C::EPS + c);
                    if (row >= g.M || n >= g.N) continue;
                    const f32x4 rb = ep.rowbias ? ld4(ep.rowbias + (long)sample_of(row) * ep.rowbias_ld + n)
                                                : f32x4{0.f, 0.f, 0.f, 0.f};
                    float o[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) o[q] = act_fn<ACT>((v[q] + bb[q]) + rb[q]);
                    store_bf16x4((bf16*)ep.out + (long)row * ep.ldo + n, o);
                }
            });
        } else if (ep.kind == EP_RESID || ep.kind == EP_SKIP || ep.kind == EP_PARTIAL) {
            // EP_RESID: v = (acc + bias) [* gate]; h += v; delta = v | delta += v; hcopy = bf16(h)
            // EP_SKIP:  h = acc + bias [+ cached delta]; hcopy = bf16(h)
            // EP_PARTIAL: part s = acc (+ bias in range 0), as EP_SKIP into h + s * part_stride
            // The global operands of a group of EB items are loaded before any of its stores.
            const bool resid = ep.kind == EP_RESID;
            const bool rd_delta = resid ? ep.delta_mode == 2 : ep.kind == EP_SKIP && ep.delta_mode == 1;
            float* const hdst = ep.kind == EP_PARTIAL ? ep.h + (long)split * ep.part_stride : ep.h;
            const f32x4 bb = ld4(sbias + c);
            const int nl = min(n, g.N - 4);  // load column (N % 4 == 0)
#pragma unroll 1
            for (int u0 = 0; u0 < PER; u0 += EB) {
                f32x4 hv[EB], dv[EB], gt[EB];
#pragma unroll
                for (int w = 0; w < EB; ++w) {
                    // clamped row and column: every load stays inside the operands
                    const int row = min(grow(rr0 + (u0 + w) * RPT), g.M - 1);
                    const long idx = (long)row * ep.d + nl;
                    hv[w] = resid ? ld4(ep.h + idx) : f32x4{0.f, 0.f, 0.f, 0.f};
                    dv[w] = rd_delta ? ld4(ep.delta + idx) : f32x4{0.f, 0.f, 0.f, 0.f};
                    gt[w] = ep.gate ? ld4(ep.gate + (long)sample_of(row) * ep.gate_ld + nl) : f32x4{1.f, 1.f, 1.f, 1.f};
                }
#pragma unroll
                for (int w = 0; w < EB; ++w) {
                    const int rr = rr0 + (u0 + w) * RPT, row = grow(rr);
                    if (!EXA && rr >= C::EPR) continue;  // also items u0 + w >= PER
                    const f32x4 v = ld4(st + rr * C::EPS + c);
                    if (row >= g.M || n >= g.N) continue;
                    const long idx = (long)row * ep.d + n;
                    float x[4], hn[4];
                    if (resid) {
                        float dn[4];
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            x[q] = v[q] + bb[q];
                            if (ep.gate) x[q] *= gt[w][q];
                            hn[q] = hv[w][q] + x[q];
                            dn[q] = dv[w][q] + x[q];
                        }
                        *(f32x4*)(ep.h + idx) = f32x4{hn[0], hn[1], hn[2], hn[3]};
                        if (ep.delta_mode == 1) *(f32x4*)(ep.delta + idx) = f32x4{x[0], x[1], x[2], x[3]};
                        else if (ep.delta_mode == 2) *(f32x4*)(ep.delta + idx) = f32x4{dn[0], dn[1], dn[2], dn[3]};
                    } else {
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            hn[q] = v[q] + bb[q];
                            if (rd_delta) hn[q] = hn[q] + dv[w][q];
                        }
                        *(f32x4*)(hdst + idx) = f32x4{hn[0], hn[1], hn[2], hn[3]};
                    }
                    if (ep.hcopy) store_bf16x4((bf16*)ep.hcopy + idx, hn);
                }
            }
        } else if (rope_tile) {
            // rotation of each pair by the token's angle: hardware sine/cosine (v_sin_f32 /
            // v_cos_f32 take turns) of the fractional turn; the turn count carries ~1e-4 rad of
            // fp32 rounding at 1024 tokens, far below the bf16 resolution of the output
            const int hd = ep.dh / 2;
            const f32x4 ba = ld4(sbias + pc), bb = ld4(sbias + pc + 4);
#pragma unroll 2
            for (int u = 0; u < PERP; ++u) {
                const int rr = rrp0 + u * RPTP, row = grow(rr);
                if (!EXP && rr >= C::EPR) continue;
                const f32x4 va = ld4(st + rr * C::EPS + pc), vb = ld4(st + rr * C::EPS + pc + 4);
                if (row >= g.M || !rope_thread) continue;
                const int bs = sample_of(row), tok = row - bs * ep.ntok;
                // columns pc + 2q and pc + 2q + 1 hold dims pj + q and pj + q + dh/2
                const float x1[4] = {va[0] + ba[0], va[2] + ba[2], vb[0] + bb[0], vb[2] + bb[2]};
                const float x2[4] = {va[1] + ba[1], va[3] + ba[3], vb[1] + bb[1], vb[3] + bb[3]};
                float o1[4], o2[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float t = (float)tok * invt[q];
                    const float f = t - rintf(t);
                    const float sn = __builtin_amdgcn_sinf(f), cs = __builtin_amdgcn_cosf(f);
                    o1[q] = x1[q] * cs - x2[q] * sn;
                    o2[q] = x2[q] * cs + x1[q] * sn;
                }
                bf16* const dst = pbase + (((long)bs * ep.H + ph) * ep.np + tok) * ep.dh + pj;
                store_bf16x4(dst, o1);
                store_bf16x4(dst + hd, o2);
            }
        } else if (ep.kind == EP_HEADS) {
            // q/k columns without rotation, row-major (a thread stores four dims of one token)
            if (n < g.N && n < vstart) {
                const f32x4 bb = ld4(sbias + c);
                bf16* const base = proj == 0 ? qptr : kptr;
#pragma unroll 2
                for (int u = 0; u < PER; ++u) {
                    const int rr = rr0 + u * RPT, row = grow(rr);
                    if (!EXA && rr >= C::EPR) continue;
                    const f32x4 v = ld4(st + rr * C::EPS + c);
                    if (row >= g.M) continue;
                    const int bs = sample_of(row), tok = row - bs * ep.ntok;
                    float o[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) o[q] = v[q] + bb[q];
                    store_bf16x4(base + (((long)bs * ep.H + hh) * ep.np + tok) * ep.dh + j, o);
                }
            }
        }
        __syncthreads();
    }
}

// --------------------------------------------------------------------------- kernel
//
// Pipeline with two LDS stages and a ring of RD register slots: in the period between the
// barriers before the last k-steps of tiles kt - 1 and kt, the MFMAs consume tile kt (one
// stage), tile kt + 1 moves from its register slot into the other stage, and tile
// kt + 1 + RD is loaded into the freed slot, so a load has RD periods to arrive.  Small
// tiles have short periods and need RD > 1 to cover the latency of weights streamed from
// HBM.  The register -> LDS writes and the loads are interleaved one part at a time with
// the period's MFMAs (part p after MFMA slot p * SLOTS / PARTS), so neither the texture
// unit nor the LDS sees a burst and both SIMD waves keep issuing MFMAs.

template <class C, bool CONV, bool SPLIT>
__global__ __launch_bounds__(C::NT, C::OCC) void gemm_bf16_kernel(GemmArgs g, EpiParams ep) {
    static_assert(C::STAGES == 2, "two LDS stages plus the register stage");
    __shared__ __attribute__((aligned(1024))) char lds[C::LDS_BYTES];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool gated = ep.kind == EP_GATED;
    const int nt_m = (g.M - g.m_begin + C::BM - 1) / C::BM;
    const int nt_n = (g.N + C::BN - 1) / C::BN;
    // split K: workgroup b takes K range b / T of tile b % T (T tiles); a range's workgroups
    // keep the tile order of an unsplit launch
    const int split = SPLIT ? (int)blockIdx.x / (nt_m * nt_n) : 0;
    int tm, tn;
    tile_at(tile_position((int)blockIdx.x - split * nt_m * nt_n, nt_m * nt_n), nt_m, nt_n, g.band, tm, tn);
    const int m0 = g.m_begin + tm * C::BM;
    const int F = g.N / 2;

    const __amdgpu_buffer_rsrc_t ra0 = buf_rsrc(g.A0, (unsigned)((long)g.M * g.lda0 * 2));
    const __amdgpu_buffer_rsrc_t ra1 = g.A1 ? buf_rsrc(g.A1, (unsigned)((long)g.M * g.lda1 * 2)) : ra0;
    const __amdgpu_buffer_rsrc_t rb = buf_rsrc(g.B, (unsigned)((long)g.N * g.ldb * 2));

    // thread -> (row, chunk) of a stage: chunk tid % CH of rows tid / CH + p * RPP; parts
    // 0 .. AP-1 are A rows, AP .. AP+BP-1 are B rows.  LDS holds the A stages, then the B
    // stages.  The swizzle key (r / RPB) % CH of a row does not change when r moves by a
    // multiple of CH * RPB rows, so a thread's write positions (rows vr + p RPP) and fragment
    // positions (rows w0 + i 32 + lrow) are one base register plus compile-time offsets.
    constexpr int RPP = C::NT / C::CH;
    constexpr int AP = C::BM / RPP, BP = C::BN / RPP, PARTS = AP + BP;
    static_assert(C::BM % RPP == 0 && C::BN % RPP == 0, "pass split");
    static_assert(RPP % (C::CH * C::RPB) == 0 && 32 % (C::CH * C::RPB) == 0, "row-invariant swizzle key");
    constexpr int B_LDS = C::STAGES * C::A_BYTES;  // first B stage
    const int vc = tid % C::CH, vr = tid / C::CH;
    unsigned goff[PARTS];  // A rows of both A sources share the row pitch
#pragma unroll
    for (int p = 0; p < AP; ++p) goff[p] = (unsigned)((long)(m0 + vr + p * RPP) * g.lda0 * 2 + vc * 16);
    // implicit-GEMM convolution: grid position (y, x) of each A row (y << 16 | x)
    int gpos[CONV ? AP : 1];
    if constexpr (CONV) {
        const int side = g.conv_side, area = side * side;
#pragma unroll
        for (int p = 0; p < AP; ++p) {
            const int pix = (m0 + vr + p * RPP) % area;
            const int y = pix / side;
            gpos[p] = (y << 16) | (pix - y * side);
        }
    }
#pragma unroll
    for (int p = 0; p < BP; ++p) {
        const int r = vr + p * RPP;
        long gr;
        if (gated) gr = r < C::BN / 2 ? (long)tn * (C::BN / 2) + r : (long)F + tn * (C::BN / 2) + (r - C::BN / 2);
        else if (ep.kind == EP_HEADS && ep.rope) gr = rope_row((long)tn * C::BN + r, ep.dh, (long)(2 - ep.which0) * ep.d);
        else gr = (long)tn * C::BN + r;
        goff[AP + p] = (unsigned)(gr * g.ldb * 2 + vc * 16);
    }
    char* const lw = lds + vr * C::ROWB + ((vc ^ ((vr / C::RPB) % C::CH)) << 4);
    // register slot s holds the k tiles t with t % RD == s (s is a compile-time constant at
    // every call).  Tiles at or past K load zeros: their offset lies past every operand
    // buffer (sizes stay below OOB), so the descriptor's range check fails.  The main loop
    // therefore runs whole trips without a branch, the padding tiles add zero products, and
    // the compiler sees the same outstanding loads on every trip.
    const int KT = (SPLIT ? g.K / g.ksplit : g.K) / C::BK;
    const int kbase = SPLIT ? split * (g.K / g.ksplit) : 0;  // first column of the workgroup's K range
    constexpr unsigned OOB = 0xFFFFFF00u;
    u32x4 vreg[C::RD][PARTS];
    auto gload = [&](int kt, int s, int p) {
        const bool in = kt < KT;
        const int k0 = kt * C::BK;
        if (CONV && p < AP) {
            // the k tile lies inside one tap (conv_c % 64 == 0): shift the row by the tap's
            // grid offset, or load zeros (an out-of-range offset) where it leaves the grid
            const int tap = k0 / g.conv_c;
            const int c0 = k0 - tap * g.conv_c;
            const int ky = tap / 3, dy = ky - 1, dx = tap - ky * 3 - 1;
            const int yy = (gpos[p] >> 16) + dy, xx = (gpos[p] & 0xFFFF) + dx;
            const bool ok = in && (unsigned)yy < (unsigned)g.conv_side && (unsigned)xx < (unsigned)g.conv_side;
            const int shift = (dy * g.conv_side + dx) * g.lda0 * 2;
            vreg[s][p] = __builtin_amdgcn_raw_buffer_load_b128(ra0, ok ? (unsigned)((int)goff[p] + shift) : OOB,
                                                               ok ? c0 * 2 : 0, 0);
        } else if (p < AP) {
            const bool second = g.A1 && k0 >= g.K0;
            vreg[s][p] = __builtin_amdgcn_raw_buffer_load_b128(second ? ra1 : ra0, in ? goff[p] : OOB,
                                                               in ? (second ? (k0 - g.K0) * 2 : (kbase + k0) * 2) : 0, 0);
        } else {
            vreg[s][p] = __builtin_amdgcn_raw_buffer_load_b128(rb, in ? goff[p] : OOB, in ? (kbase + k0) * 2 : 0, 0);
        }
    };
    // stage and part are compile-time constants at every call
    auto lwrite = [&](int stage, int s, int p) {
        if (p < AP) *(u32x4*)(lw + stage * C::A_BYTES + p * RPP * C::ROWB) = vreg[s][p];
        else *(u32x4*)(lw + B_LDS + stage * C::B_BYTES + (p - AP) * RPP * C::ROWB) = vreg[s][p];
    };

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
    const int fkey = (lrow / C::RPB) % C::CH;
    const char* const fa = lds + (wm0 + lrow) * C::ROWB;
    const char* const fb = lds + B_LDS + (wn0 + lrow) * C::ROWB;
    auto frags = [&](int stage, int q, int buf) {
        const int sw = ((q * 2 + lhalf) ^ fkey) << 4;
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
            af[buf][i] = *(const bf16x8*)(fa + sw + stage * C::A_BYTES + i * 32 * C::ROWB);
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
            bfr[buf][j] = *(const bf16x8*)(fb + sw + stage * C::B_BYTES + j * 32 * C::ROWB);
    };
    constexpr int MPK = C::TM * C::TN, SLOTS = C::KSTEPS * MPK;
    static_assert(PARTS <= SLOTS, "part spreading");
    // MFMAs of one k-step; `part` is the k-step's position in its period.  The period moves
    // a tile from register slot S into stage ws and loads tile lt into slot S.  The compiler
    // inserts the vmcnt waits from the register dependences: vmcnt(RD * PARTS - 1) before
    // every write.
    auto mfmas = [&](int buf, int part, int ws, int lt, auto rs) {
        constexpr int S = decltype(rs)::value;
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
#pragma unroll
            for (int j = 0; j < C::TN; ++j) {
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[buf][i], bfr[buf][j], acc[i][j], 0, 0, 0);
                const int slot = part * MPK + i * C::TN + j;
                const int p = (slot * PARTS + SLOTS - 1) / SLOTS;
                if (p < PARTS && (p * SLOTS) / PARTS == slot) {
                    __builtin_amdgcn_sched_barrier(0);
                    lwrite(ws, S, p);
                    gload(lt, S, p);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
    };

    // prologue: tile 0 into stage 0, tiles 1 .. RD into the register slots (tile RD shares
    // slot 0 with tile 0).  The first period has no "last k-step of tile -1", so the parts of
    // its first slot group (write tile 1, load tile 1 + RD) are done here.
#pragma unroll
    for (int p = 0; p < PARTS; ++p) gload(0, 0, p);
    static_for<C::RD - 1>([&](auto jc) {
        constexpr int TT = decltype(jc)::value + 1;
#pragma unroll
        for (int p = 0; p < PARTS; ++p) gload(TT, TT, p);
    });
#pragma unroll
    for (int p = 0; p < PARTS; ++p) {
        lwrite(0, 0, p);
        gload(C::RD, 0, p);
    }
#pragma unroll
    for (int p = 0; p < PARTS; ++p) {
        if ((p * SLOTS) / PARTS < MPK) {
            lwrite(1, 1 % C::RD, p);
            gload(1 + C::RD, 1 % C::RD, p);
        }
    }
    __syncthreads();
    frags(0, 0, 0);
    // one k tile; jc is its position in the trip (tile kt sits in register slot J = kt % RD
    // and LDS stage st = kt % 2).  The period of tile kt (from the barrier before tile kt-1's
    // last k-step) moves tile kt + 1 into stage st ^ 1 and loads tile kt + 1 + RD, and the
    // period of tile kt + 1 starts with the last k-step
    auto iter = [&](int kt, auto jc) {
        constexpr int J = decltype(jc)::value % C::RD, st = decltype(jc)::value % 2;
#pragma unroll
        for (int q = 0; q < C::KSTEPS; ++q) {
            const int cur = q & 1, nxt = cur ^ 1;
            __builtin_amdgcn_sched_barrier(0);
            if (q + 1 < C::KSTEPS) {
                frags(st, q + 1, nxt);
            } else {
                __syncthreads();  // tile kt + 1 is in stage st ^ 1; stage st is free
                frags(st ^ 1, 0, nxt);
            }
            __builtin_amdgcn_sched_barrier(0);
            if (q + 1 < C::KSTEPS) mfmas(cur, q + 1, st ^ 1, kt + 1 + C::RD, IntC<(J + 1) % C::RD>{});
            else mfmas(cur, 0, st, kt + 2 + C::RD, IntC<(J + 2) % C::RD>{});
        }
    };
    static_assert(C::KSTEPS % 2 == 0, "fragment ring");
    constexpr int TRIP = C::RD % 2 ? 2 * C::RD : C::RD;  // whole register rings and LDS stage pairs
    for (int kt = 0; kt < KT; kt += TRIP) static_for<TRIP>([&](auto jc) { iter(kt + decltype(jc)::value, jc); });
    epilogue<C>(acc, lds, g, ep, m0, tn, wm, wn0, split);
}

// --------------------------------------------------------------------------- dispatch

namespace {
// block tiles (BM, BN); eight waves, 64-deep k tiles, two LDS stages plus RD register slots.
// Two slots on the smaller tiles: with weights streamed from HBM, one period of a 128 x 128
// tile is too short for a load to arrive (LLaDA O and W2: -17 % time with two slots); the
// 256 x 256 tile has a period twice as long and no registers to spare.  (Four waves of
// 128 x 128, one per SIMD, measured 10-20 % slower on every branch shape.)
using T256x256 = TileCfg<256, 256, 4, 2, 64, 2, 2, 1>;  // 64 x 128 wave tiles
using T256x128 = TileCfg<256, 128, 4, 2, 64, 2, 2, 2>;  // 64 x 64
using T128x256 = TileCfg<128, 256, 2, 4, 64, 2, 2, 2>;  // 64 x 64
using T128x128 = TileCfg<128, 128, 2, 4, 64, 2, 2, 2>;  // 64 x 32
using T256x192 = TileCfg<256, 192, 4, 2, 64, 2, 2, 2>;  // 64 x 96

struct Shape { int bm, bn; double rate; };
// tile id -> block shape and its per-CU throughput relative to 256 x 256 (measured on the
// branch GEMM shapes: smaller tiles move more operand bytes per FLOP through L2 and LDS)
Shape tile_shape(int tile) {
    switch (tile) {
        case 1: return {256, 256, 1.0};
        case 2: return {256, 128, 0.78};
        case 3: return {128, 256, 0.80};
        case 4: return {128, 128, 0.51};
        case 5: return {256, 192, 0.82};
        default: return {0, 0, 0.0};
    }
}
}  // namespace

// Cost of one launch of `tile` over `rows` rows in units of a 256 x 256 tile at full rate: one
// workgroup per CU, so n tiles take ceil(n / 256) rounds of tile area / per-CU rate.
// Infinite when the epilogue cannot use the tile.
static bool conv_tile(int tile) { return tile == 2 || tile == 4 || tile == 5; }

static double tile_cost(int tile, long rows, const GemmArgs& g, const EpiParams& e) {
    const Shape s = tile_shape(tile);
    if (!s.bm) return 1e300;
    if (g.conv_side > 0 && !conv_tile(tile)) return 1e300;
    if (e.kind == EP_GATED && g.N % s.bn) return 1e300;
    const long tiles = ((rows + s.bm - 1) / s.bm) * ((g.N + s.bn - 1) / s.bn);
    return (double)((tiles + 255) / 256) * s.bm * s.bn / s.rate / (256.0 * 256.0);
}

// Automatic choice: the tile with the least cost (e.g. at 1024 rows the 4096-column GEMMs run
// 128 x 128 tiles, one full round, rather than 64 large tiles).  When the rows leave a short
// tail past the last whole 256-row tile (U-ViT: 32 x 258 = 8256 = 32 x 256 + 64 rows), the
// tail can go to a second launch of 128-row tiles, so the main launch fills whole rounds
// instead of starting a third round for 64 rows; the split is taken when it is cheaper with
// the second launch charged a tenth of a round for its start-up.
GemmPlan gemm_bf16_plan(const GemmArgs& g, const EpiParams& e) {
    GemmPlan best{1, g.M, 0};
    double best_t = 1e300;
    for (int tile = 1; tile <= kGemmTiles; ++tile) {
        const double t = tile_cost(tile, g.M, g, e);
        if (t < best_t * 0.999) { best_t = t; best = GemmPlan{tile, g.M, 0}; }
    }
    const int tail = g.M % 256;
    if (g.M > 2048 && tail > 0 && tail <= 128 && g.conv_side == 0) {
        for (int tile = 1; tile <= kGemmTiles; ++tile) {
            if (tile_shape(tile).bm != 256) continue;
            const double tm = tile_cost(tile, g.M - tail, g, e);
            for (int tt = 1; tt <= kGemmTiles; ++tt) {
                if (tile_shape(tt).bm != 128) continue;
                const double t = tm + tile_cost(tt, tail, g, e) + 0.1;
                if (t < best_t * 0.97) { best_t = t; best = GemmPlan{tile, g.M - tail, tt}; }
            }
        }
    }
    return best;
}

int gemm_bf16_auto_tile(const GemmArgs& g, const EpiParams& e) { return gemm_bf16_plan(g, e).tile; }

// Two K ranges where one round of 128 x 128 tiles is the best unsplit plan of a long-K product
// and 256 x 128 tiles over half of K still fill at most one round: the larger tiles move ~1.5x
// fewer operand bytes per FLOP through the load path that bounds the small ones (LLaDA's MLP
// output GEMM, 1024 x 4096 x 12288: 128 tiles x 2 ranges).  The caller adds the two fp32
// partial products (EP_PARTIAL) to the stream itself.
int gemm_bf16_ksplit(const GemmArgs& g) {
    EpiParams e;
    e.kind = EP_RESID;
    e.d = g.N;
    const GemmPlan p = gemm_bf16_plan(g, e);
    if (p.tile != 4 || p.tail_tile || g.A1 || g.conv_side > 0 || g.K < 8192 || g.K % 128) return 1;
    const long tiles = (long)((g.M + 255) / 256) * ((g.N + 127) / 128);
    return 2 * tiles <= 256 ? 2 : 1;
}

static bool aligned(const void* p, unsigned a) { return ((uintptr_t)p % a) == 0; }

bool gemm_bf16_shape_ok(const GemmArgs& g, const EpiParams& e, int tile) {
    if (tile == 0 && e.kind == EP_PARTIAL) tile = 2;
    if (tile == 0) {
        const GemmPlan p = gemm_bf16_plan(g, e);
        if (p.tail_tile && !gemm_bf16_shape_ok(g, e, p.tail_tile)) return false;
        tile = p.tile;
    }
    if (g.m_begin != 0) return false;  // set by the dispatcher only
    // vector accesses of the loader and the epilogue: 16-byte operand rows and fp32 vectors,
    // 8-byte bf16 output groups
    if (!aligned(g.A0, 16) || !aligned(g.A1, 16) || !aligned(g.B, 16) || !aligned(e.bias, 16) ||
        !aligned(e.gate, 16) || e.gate_ld % 4 || !aligned(e.h, 16) || !aligned(e.delta, 16) ||
        !aligned(e.out, 8) || !aligned(e.hcopy, 8) || !aligned(e.q, 8) || !aligned(e.k, 8) || !aligned(e.vt, 2))
        return false;
    const Shape s = tile_shape(tile);
    if (!s.bm) return false;
    if (g.M >= (1 << 21)) return false;  // the epilogue's fp32 row -> sample split is exact below
    if (g.conv_side > 0) {
        const long area = (long)g.conv_side * g.conv_side;
        if (!conv_tile(tile) || g.A1 || g.conv_c % 64 || g.K != 9 * g.conv_c || g.lda0 != g.conv_c ||
            g.M % area || g.conv_side >= (1 << 15))
            return false;
    }
    if (!aligned(e.rowbias, 16) || e.rowbias_ld % 4) return false;
    if (g.K % 64 || (g.A1 && (g.K0 % 64 || g.lda1 != g.lda0))) return false;
    if (g.N % 4 || g.lda0 % 8 || (g.A1 && g.lda1 % 8) || g.ldb % 8) return false;  // 16-byte rows
    if (e.kind == EP_GATED && (g.N % s.bn || e.ldo % 4)) return false;
    if (e.kind == EP_ACT && e.ldo % 4) return false;
    if ((e.kind == EP_RESID || e.kind == EP_SKIP || e.kind == EP_PARTIAL) && (g.N != e.d)) return false;
    if (g.ksplit < 1 || (g.ksplit > 1) != (e.kind == EP_PARTIAL) || (g.ksplit > 1 && tile != 2)) return false;
    if (e.kind == EP_PARTIAL && (g.A1 || g.conv_side > 0 || g.K % (64 * g.ksplit) || e.gate || e.hcopy ||
                                 e.delta_mode || (long)e.part_stride < (long)g.M * g.N || e.part_stride % 4))
        return false;
    if (e.kind == EP_HEADS) {
        if (e.d % 32 || e.dh % 4) return false;  // V^T from whole 32-column MFMA blocks
        if (e.rope && e.dh % 8) return false;  // eight-column pair groups within one head
    }
    const long lim = 0xFFFFFF00L;  // 32-bit buffer ranges below the loader's out-of-range offset
    if ((long)g.M * g.lda0 * 2 > lim || (g.A1 && (long)g.M * g.lda1 * 2 > lim) || (long)g.N * g.ldb * 2 > lim)
        return false;
    return true;
}

template <class C, bool CONV = false, bool SPLIT = false>
static hipError_t run_tile(const GemmArgs& g, const EpiParams& e, hipStream_t st) {
    const int nt_m = (g.M - g.m_begin + C::BM - 1) / C::BM, nt_n = (g.N + C::BN - 1) / C::BN;
    GemmArgs ga = g;
    ga.band = tile_band(nt_m, nt_n, C::BM, C::BN);
    hipLaunchKernelGGL((gemm_bf16_kernel<C, CONV, SPLIT>), dim3(nt_m * nt_n * (SPLIT ? g.ksplit : 1)), dim3(C::NT), 0,
                       st, ga, e);
    return hipGetLastError();
}

static hipError_t launch_tile(const GemmArgs& g, const EpiParams& e, hipStream_t st, int tile) {
    if (g.conv_side > 0) {
        switch (tile) {  // implicit-GEMM convolution: the tiles with registers to spare
            case 2: return run_tile<T256x128, true>(g, e, st);
            case 4: return run_tile<T128x128, true>(g, e, st);
            case 5: return run_tile<T256x192, true>(g, e, st);
            default: return hipErrorInvalidValue;
        }
    }
    if (g.ksplit > 1) {  // K ranges (EP_PARTIAL): the 256 x 128 tiles only
        if (tile != 2) return hipErrorInvalidValue;
        return run_tile<T256x128, false, true>(g, e, st);
    }
    switch (tile) {
        case 1: return run_tile<T256x256>(g, e, st);
        case 2: return run_tile<T256x128>(g, e, st);
        case 3: return run_tile<T128x256>(g, e, st);
        case 4: return run_tile<T128x128>(g, e, st);
        case 5: return run_tile<T256x192>(g, e, st);
        default: return hipErrorInvalidValue;
    }
}

// rows [0, m_split) with the plan's tile, then the tail rows [m_split, M) with the tail tile;
// both launches index rows globally (the epilogue's sample / token split needs it)
hipError_t launch_gemm_bf16(const GemmArgs& g, const EpiParams& e, hipStream_t st, int tile) {
    if (e.kind == EP_PARTIAL && tile == 0) tile = 2;  // the split product's 256 x 128 tiles
    if (tile != 0) return launch_tile(g, e, st, tile);
    const GemmPlan p = gemm_bf16_plan(g, e);
    if (!p.tail_tile) return launch_tile(g, e, st, p.tile);
    GemmArgs gm = g;
    gm.M = p.m_split;
    const hipError_t err = launch_tile(gm, e, st, p.tile);
    if (err != hipSuccess) return err;
    GemmArgs gt = g;
    gt.m_begin = p.m_split;
    return launch_tile(gt, e, st, p.tail_tile);
}

}  // namespace sgd
