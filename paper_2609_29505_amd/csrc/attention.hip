// Fused bidirectional / cross attention (flash-style, one pass over the keys).
//
// bf16 path (MFMA 32x32x16): a wave owns 32 queries (of one key half in the split variant)
// and computes the transposed score tile S^T = K Q^T, so that one lane owns one query: the
// row maximum and row sum of the online softmax are per-lane reductions plus one exchange
// with lane ^ 32.
// The output is accumulated transposed as O^T += V^T P^T, where P^T is exactly the S^T
// accumulator layout re-packed to bf16 (the MFMA k-slots are permuted consistently on
// both operands), and V^T is read from the head-major transposed value layout written by
// the QKV GEMM epilogue.  Keys beyond nk are masked; head dims are zero-padded to a
// multiple of 32.
// fp32 path (MFMA 32x32x2 fp32): the same transposed formulation with one fp32 k-slot pair
// per MFMA; a workgroup's waves share 32 queries and take alternate 32-key blocks, and their
// partial softmax states are merged through LDS in wave order.
#include "common.h"
#include "kernels.h"
#include "tile_order.h"

namespace sgd {

// Query block and head (batch x head index) of a bf16 workgroup, from a grid of query blocks x
// heads.  The workgroups go round-robin to the XCDs in dispatch order (x fastest); they are
// renumbered so that the query blocks of one head are neighbours in the order that the XCDs
// split between them (tile_position), i.e. run on one XCD and read the head's keys and values
// through one L2 instead of one per XCD.
__device__ __forceinline__ void attn_block(int& qb, int& bh) {
    const int nqb = gridDim.x;
    const int pos = tile_position(blockIdx.y * nqb + blockIdx.x, nqb * gridDim.y);
    bh = pos / nqb;
    qb = pos - bh * nqb;
}

// {v[l], v[l ^ 32]} combined across the two 32-lane halves of the wave (one lane swap)
__device__ __forceinline__ float pair_max(float v) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float v) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Lazy rescaling: the running reference m of a lane is raised only when its block maximum
// exceeds it by more than 2^8 (checked for the whole wave at once); probabilities are then
// exp2(s - m) <= 256, exact in fp32 and in bf16's 8-bit exponent range.
constexpr float kRescaleSlack = 8.0f;

template <int DH, int NW>
__global__ __launch_bounds__(NW * 64) void attn_bf16_kernel(AttnArgs a, float scale_log2) {
    constexpr int DHP = (DH + 31) / 32 * 32;  // head dims padded to whole 32-row MFMA blocks
    constexpr int BQ = 32 * NW, BKV = 64, NT = NW * 64;
    constexpr int KS = DHP / 16, DT = DHP / 32;
    constexpr int KLDS = DHP + 8, VLDS = BKV + 8;        // padded rows: conflict-free fragment reads
    constexpr int K_CH = (BKV * (DHP / 8) + NT - 1) / NT;  // 16-byte chunks per thread per block (upper bound)
    constexpr int V_CH = (DHP * (BKV / 8) + NT - 1) / NT;
    __shared__ __attribute__((aligned(16))) bf16 sk[2][BKV * KLDS];
    __shared__ __attribute__((aligned(16))) bf16 sv[2][DHP * VLDS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int qb, bh;
    attn_block(qb, bh);
    const int b = bh / a.H, hh = bh - b * a.H;
    constexpr int dh = DH;
    const int q = qb * BQ + wave * 32 + (lane & 31);
    const int half = lane >> 5;

    const bf16* Q = (const bf16*)a.q + (long)bh * a.npq * dh;
    const bf16* K = (const bf16*)a.k + (long)bh * a.npk * dh;
    const bf16* VT = (const bf16*)a.vt + (long)bh * dh * a.npk;

    // zero the padded head dims of both buffers once (the loads below never write them)
    for (int i = tid; i < 2 * BKV * (DHP - dh); i += NT) {
        const int buf = i / (BKV * (DHP - dh)), j = i % (BKV * (DHP - dh));
        sk[buf][(j / (DHP - dh)) * KLDS + dh + j % (DHP - dh)] = f2bf(0.f);
    }
    for (int i = tid; i < 2 * (DHP - dh) * BKV; i += NT) {
        const int buf = i / ((DHP - dh) * BKV), j = i % ((DHP - dh) * BKV);
        sv[buf][(dh + j / BKV) * VLDS + j % BKV] = f2bf(0.f);
    }

    // this lane's query fragments (B operand of S^T = K Q^T)
    bf16x8 qf[KS];
    const int qrow = min(q, a.nq - 1);  // rows past nq repeat the last query: padded rows are never read
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const int c = ks * 16 + half * 8;
        if (c < dh) qf[ks] = *(const bf16x8*)(Q + (long)qrow * dh + c);
        else
            for (int e = 0; e < 8; ++e) qf[ks][e] = f2bf(0.f);
    }

    // register prefetch of one key/value block
    constexpr int kchunks = dh / 8;  // 16-byte chunks per key row
    u32x4 rk[K_CH], rv[V_CH];
    auto gload = [&](int k0) {
#pragma unroll
        for (int t = 0; t < K_CH; ++t) {
            const int i = tid + t * NT;
            if (i < BKV * kchunks) {
                const int r = i / kchunks, c = (i - r * kchunks) * 8;
                rk[t] = *(const u32x4*)(K + (long)(k0 + r) * dh + c);
            }
        }
#pragma unroll
        for (int t = 0; t < V_CH; ++t) {
            const int i = tid + t * NT;
            if (i < dh * (BKV / 8)) {
                const int r = i >> 3, c = (i & 7) * 8;
                rv[t] = *(const u32x4*)(VT + (long)r * a.npk + k0 + c);
            }
        }
    };
    auto lstore = [&](int k0, int buf) {
#pragma unroll
        for (int t = 0; t < K_CH; ++t) {
            const int i = tid + t * NT;
            if (i < BKV * kchunks) {
                const int r = i / kchunks, c = (i - r * kchunks) * 8;
                *(u32x4*)(&sk[buf][r * KLDS + c]) = rk[t];
            }
        }
#pragma unroll
        for (int t = 0; t < V_CH; ++t) {
            const int i = tid + t * NT;
            if (i < dh * (BKV / 8)) {
                const int r = i >> 3, c = (i & 7) * 8;
                bf16x8 v = __builtin_bit_cast(bf16x8, rv[t]);
                if (k0 + c + 8 > a.nk) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (k0 + c + e >= a.nk) v[e] = f2bf(0.f);
                }
                // key order inside a 16-key group: 0-3, 8-11, 4-7, 12-15, so the keys
                // {0-3, 8-11} (lanes 0-31) and {4-7, 12-15} (lanes 32-63) are contiguous
                const int g16 = c & ~15, hi8 = (c & 8) ? 4 : 0;
                bf16x4 v0, v1;
#pragma unroll
                for (int e = 0; e < 4; ++e) { v0[e] = v[e]; v1[e] = v[4 + e]; }
                *(bf16x4*)(&sv[buf][r * VLDS + g16 + hi8]) = v0;
                *(bf16x4*)(&sv[buf][r * VLDS + g16 + 8 + hi8]) = v1;
            }
        }
    };

    f32x16 o[DT];
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][r] = 0.f;
    float m = -INFINITY, lsum = 0.f;

    const int nkb = (a.nk + BKV - 1) / BKV;
    gload(0);
    __syncthreads();  // padding zeroed
    lstore(0, 0);
    __syncthreads();
    // Every load issued so far (the query fragments, block 0) has completed on the main path;
    // saying so for every path keeps the waitcnt insertion from treating the query fragments
    // as possibly in flight inside the loop, where it would wait on the loop's own key/value
    // prefetch before each score MFMA and serialise the prefetch.
    __builtin_amdgcn_s_waitcnt(0);
    for (int kb = 0; kb < nkb; ++kb) {
        const int k0 = kb * BKV;
        const int buf = kb & 1;
        if (kb + 1 < nkb) gload(k0 + BKV);  // in flight while this block computes

        f32x16 s[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int r = 0; r < 16; ++r) s[t][r] = 0.f;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                bf16x8 kf = *(const bf16x8*)(&sk[buf][(t * 32 + (lane & 31)) * KLDS + ks * 16 + half * 8]);
                s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[t], 0, 0, 0);
            }
        }
        // scale into the log2 domain (masking keys beyond nk in the tail block only), block max
        float bm = -INFINITY;
        if (k0 + BKV > a.nk) {
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = k0 + t * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
                    if (key >= a.nk) s[t][r] = -INFINITY;
                }
        }
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) bm = fmaxf(bm, s[t][r]);
        bm = pair_max(bm) * scale_log2;  // the scale is positive: max and scaling commute
        if (__builtin_amdgcn_ballot_w64(bm > m + kRescaleSlack)) {
            const float mn = fmaxf(m, bm);
            const float alpha = __builtin_amdgcn_exp2f(m - mn);
            m = mn;
            lsum *= alpha;
#pragma unroll
            for (int t = 0; t < DT; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
        }
        float ps = 0.f;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float p = __builtin_amdgcn_exp2f(fmaf(s[t][r], scale_log2, -m));
                s[t][r] = p;
                ps += p;
            }
        lsum += ps;

        // O^T += V^T P^T over the block's 64 keys, 16 at a time
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2) {
                bf16x8 pf;
#pragma unroll
                for (int e = 0; e < 8; ++e) pf[e] = f2bf(s[t][8 * k2 + e]);
                const int kc = t * 32 + 16 * k2 + half * 8;  // permuted key order (see lstore)
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
                    const bf16x8 vf = *(const bf16x8*)(&sv[buf][(dt * 32 + (lane & 31)) * VLDS + kc]);
                    o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, o[dt], 0, 0, 0);
                }
            }
        }
        if (kb + 1 < nkb) lstore(k0 + BKV, buf ^ 1);  // the other buffer: nobody reads it now
        __syncthreads();
    }

    const float l = pair_sum(lsum);
    const float inv = 1.0f / l;
    if (q < a.nq) {
        bf16* O = (bf16*)a.o + ((long)b * a.nq + q) * ((long)a.H * dh) + (long)hh * dh;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
                const int d0 = dt * 32 + g4 * 8 + half * 4;
                if (d0 < dh) {
                    bf16x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = f2bf(o[dt][g4 * 4 + e] * inv);
                    *(bf16x4*)(O + d0) = v;
                }
            }
    }
}

// The workgroup's waves form two halves of NQG waves; wave w serves query group w % NQG and
// key half w / NQG: half h takes the key blocks 2 i + h, each half with one LDS buffer (K
// block and V^T block) refilled from a register prefetch.  Splitting the keys doubles the
// waves per query range (a 1024-query, 32-head problem has only 1024 query groups of 32),
// so two waves share each SIMD and one half's softmax overlaps the other's MFMAs.  At the
// end half 1 leaves (m, partial sums, O^T) in LDS and half 0 merges them:
// O = O_0 2^(m_0 - m) + O_1 2^(m_1 - m) with m = max(m_0, m_1).
template <int DH, int NQG>
__global__ __launch_bounds__(2 * NQG * 64, 2) void attn_split_bf16_kernel(AttnArgs a, float scale_log2) {
    constexpr int DHP = (DH + 31) / 32 * 32;
    constexpr int BQ = 32 * NQG, BKV = 64, HT = NQG * 64, NT = 2 * HT;
    constexpr int KS = DHP / 16, DT = DHP / 32;
    constexpr int KLDS = DHP + 8, VLDS = BKV + 8;        // padded rows: conflict-free fragment reads
    constexpr int K_CH = (BKV * (DHP / 8) + HT - 1) / HT;  // 16-byte chunks per thread per block (upper bound)
    constexpr int V_CH = (DHP * (BKV / 8) + HT - 1) / HT;
    constexpr int HALF_BYTES = (BKV * KLDS + DHP * VLDS) * 2;
    constexpr int MERGE_BYTES = NQG * (DT * 16 + 2) * 64 * 4;  // half 1's state, lane-major
    static_assert(MERGE_BYTES <= 4 * HALF_BYTES, "merge area");
    __shared__ __attribute__((aligned(16))) char smem[4 * HALF_BYTES];  // two buffers per half

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int kh = wave / NQG, qg = wave % NQG, htid = tid - kh * HT;
    bf16* const sk0 = (bf16*)(smem + kh * 2 * HALF_BYTES);  // buffer b: sk0 + b * HALF_BYTES / 2
    constexpr int BUF = HALF_BYTES / 2;                     // bf16 elements per buffer
    constexpr int VOFF = BKV * KLDS;                        // V^T part of a buffer
    int qb, bh;
    attn_block(qb, bh);
    const int b = bh / a.H, hh = bh - b * a.H;
    constexpr int dh = DH;
    const int q = qb * BQ + qg * 32 + (lane & 31);
    const int half = lane >> 5;

    const bf16* Q = (const bf16*)a.q + (long)bh * a.npq * dh;
    const bf16* K = (const bf16*)a.k + (long)bh * a.npk * dh;
    const bf16* VT = (const bf16*)a.vt + (long)bh * dh * a.npk;

    // zero the padded head dims of this half's buffers once (the loads never write them)
#pragma unroll
    for (int bb = 0; bb < 2; ++bb) {
        bf16* const zk = sk0 + bb * BUF;
        for (int i = htid; i < BKV * (DHP - dh); i += HT) zk[(i / (DHP - dh)) * KLDS + dh + i % (DHP - dh)] = f2bf(0.f);
        for (int i = htid; i < (DHP - dh) * BKV; i += HT) zk[VOFF + (dh + i / BKV) * VLDS + i % BKV] = f2bf(0.f);
    }

    // this lane's query fragments (B operand of S^T = K Q^T)
    bf16x8 qf[KS];
    const int qrow = min(q, a.nq - 1);  // rows past nq repeat the last query: padded rows are never read
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const int c = ks * 16 + half * 8;
        if (c < dh) qf[ks] = *(const bf16x8*)(Q + (long)qrow * dh + c);
        else
            for (int e = 0; e < 8; ++e) qf[ks][e] = f2bf(0.f);
    }

    // register prefetch of one key/value block of this half
    constexpr int kchunks = dh / 8;  // 16-byte chunks per key row
    u32x4 rk[K_CH], rv[V_CH];
    auto gload = [&](int k0) {
#pragma unroll
        for (int t = 0; t < K_CH; ++t) {
            const int i = htid + t * HT;
            if (i < BKV * kchunks) {
                const int r = i / kchunks, c = (i - r * kchunks) * 8;
                rk[t] = *(const u32x4*)(K + (long)(k0 + r) * dh + c);
            }
        }
#pragma unroll
        for (int t = 0; t < V_CH; ++t) {
            const int i = htid + t * HT;
            if (i < dh * (BKV / 8)) {
                const int r = i >> 3, c = (i & 7) * 8;
                rv[t] = *(const u32x4*)(VT + (long)r * a.npk + k0 + c);
            }
        }
    };
    auto lstore = [&](int k0, int bb) {
        bf16* const sk = sk0 + bb * BUF;
        bf16* const sv = sk + VOFF;
#pragma unroll
        for (int t = 0; t < K_CH; ++t) {
            const int i = htid + t * HT;
            if (i < BKV * kchunks) {
                const int r = i / kchunks, c = (i - r * kchunks) * 8;
                *(u32x4*)(&sk[r * KLDS + c]) = rk[t];
            }
        }
#pragma unroll
        for (int t = 0; t < V_CH; ++t) {
            const int i = htid + t * HT;
            if (i < dh * (BKV / 8)) {
                const int r = i >> 3, c = (i & 7) * 8;
                bf16x8 v = __builtin_bit_cast(bf16x8, rv[t]);
                if (k0 + c + 8 > a.nk) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (k0 + c + e >= a.nk) v[e] = f2bf(0.f);
                }
                // key order inside a 16-key group: 0-3, 8-11, 4-7, 12-15, so the keys
                // {0-3, 8-11} (lanes 0-31) and {4-7, 12-15} (lanes 32-63) are contiguous
                const int g16 = c & ~15, hi8 = (c & 8) ? 4 : 0;
                bf16x4 v0, v1;
#pragma unroll
                for (int e = 0; e < 4; ++e) { v0[e] = v[e]; v1[e] = v[4 + e]; }
                *(bf16x4*)(&sv[r * VLDS + g16 + hi8]) = v0;
                *(bf16x4*)(&sv[r * VLDS + g16 + 8 + hi8]) = v1;
            }
        }
    };

    f32x16 o[DT];
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][r] = 0.f;
    float m = -INFINITY, lsum = 0.f;

    const int nkb = (a.nk + BKV - 1) / BKV;
    const int nit = (nkb + 1) / 2;  // block pairs: half h takes block 2 it + h
    // Two LDS buffers per half: iteration it computes block 2 it + kh from buffer it & 1 while
    // block 2 (it + 1) + kh moves from registers into the other buffer (read last in iteration
    // it - 1, before its closing barrier) and block 2 (it + 2) + kh is loaded into registers:
    // one barrier per iteration.
    if (kh < nkb) gload(kh * BKV);
    __syncthreads();  // padding zeroed
    if (kh < nkb) lstore(kh * BKV, 0);
    if (kh + 2 < nkb) gload((kh + 2) * BKV);
    __syncthreads();
    // Wait for every load issued so far (the query fragments, and block 2 + kh, which the first
    // iteration stores to LDS right away anyway): otherwise the waitcnt insertion treats the
    // query fragments as possibly in flight inside the loop (on paths that skip a prologue
    // store) and waits on the loop's own key/value prefetch before each score MFMA.
    __builtin_amdgcn_s_waitcnt(0);
    for (int it = 0; it < nit; ++it) {
        const int kb = 2 * it + kh;
        const int k0 = kb * BKV;
        const bool mine = kb < nkb;
        const bf16* const sk = sk0 + (it & 1) * BUF;
        const bf16* const sv = sk + VOFF;
        if (kb + 2 < nkb) {
            lstore(k0 + 2 * BKV, (it & 1) ^ 1);
            if (kb + 4 < nkb) gload(k0 + 4 * BKV);  // in flight while this block computes
        }
        if (mine) {
            f32x16 s[2];
#pragma unroll
            for (int t = 0; t < 2; ++t) {
#pragma unroll
                for (int r = 0; r < 16; ++r) s[t][r] = 0.f;
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    bf16x8 kf = *(const bf16x8*)(&sk[(t * 32 + (lane & 31)) * KLDS + ks * 16 + half * 8]);
                    s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[t], 0, 0, 0);
                }
            }
            // scale into the log2 domain (masking keys beyond nk in the tail block only), block max
            float bm = -INFINITY;
            if (k0 + BKV > a.nk) {
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int key = k0 + t * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
                        if (key >= a.nk) s[t][r] = -INFINITY;
                    }
            }
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) bm = fmaxf(bm, s[t][r]);
            bm = pair_max(bm) * scale_log2;  // the scale is positive: max and scaling commute
            if (__builtin_amdgcn_ballot_w64(bm > m + kRescaleSlack)) {
                const float mn = fmaxf(m, bm);
                const float alpha = __builtin_amdgcn_exp2f(m - mn);
                m = mn;
                lsum *= alpha;
#pragma unroll
                for (int t = 0; t < DT; ++t)
#pragma unroll
                    for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
            }
            float ps = 0.f;
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float p = __builtin_amdgcn_exp2f(fmaf(s[t][r], scale_log2, -m));
                    s[t][r] = p;
                    ps += p;
                }
            lsum += ps;

            // O^T += V^T P^T over the block's 64 keys, 16 at a time
#pragma unroll
            for (int t = 0; t < 2; ++t) {
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) {
                    bf16x8 pf;
#pragma unroll
                    for (int e = 0; e < 8; ++e) pf[e] = f2bf(s[t][8 * k2 + e]);
                    const int kc = t * 32 + 16 * k2 + half * 8;  // permuted key order (see lstore)
#pragma unroll
                    for (int dt = 0; dt < DT; ++dt) {
                        const bf16x8 vf = *(const bf16x8*)(&sv[(dt * 32 + (lane & 31)) * VLDS + kc]);
                        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, o[dt], 0, 0, 0);
                    }
                }
            }
        }
        __syncthreads();  // block it + 1 is in place; buffer it & 1 is free
    }

    // merge the two key halves through LDS (lane-major: conflict-free)
    __syncthreads();
    float* mg = (float*)smem + qg * (DT * 16 + 2) * 64;
    if (kh == 1) {
#pragma unroll
        for (int t = 0; t < DT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) mg[(t * 16 + r) * 64 + lane] = o[t][r];
        mg[DT * 16 * 64 + lane] = m;
        mg[(DT * 16 + 1) * 64 + lane] = lsum;
    }
    __syncthreads();
    if (kh == 1) return;
    {
        const float m1 = mg[DT * 16 * 64 + lane], l1 = mg[(DT * 16 + 1) * 64 + lane];
        const float mn = fmaxf(m, m1);  // half 0 always holds block 0, so mn is finite
        const float a0 = __builtin_amdgcn_exp2f(m - mn), a1 = __builtin_amdgcn_exp2f(m1 - mn);
        lsum = lsum * a0 + l1 * a1;
#pragma unroll
        for (int t = 0; t < DT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[t][r] = o[t][r] * a0 + mg[(t * 16 + r) * 64 + lane] * a1;
    }

    const float l = pair_sum(lsum);
    const float inv = 1.0f / l;
    if (q < a.nq) {
        bf16* O = (bf16*)a.o + ((long)b * a.nq + q) * ((long)a.H * dh) + (long)hh * dh;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
                const int d0 = dt * 32 + g4 * 8 + half * 4;
                if (d0 < dh) {
                    bf16x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = f2bf(o[dt][g4 * 4 + e] * inv);
                    *(bf16x4*)(O + d0) = v;
                }
            }
    }
}

// fp32 attention.  Wave w of a workgroup takes key blocks w, w + NW, ... of its 32 queries.
// Scores: S^T (32 keys x 32 queries) = K Q^T over head dims, MFMA step t contracting dims t
// (lanes 0-31) and HD + t (lanes 32-63), so each lane reads one contiguous half row of K and
// of Q.  In the accumulator lane l holds query l % 32 and keys (r / 4) * 8 + (l / 32) * 4 +
// r % 4 (register r).  Output: O^T += V^T P^T, MFMA r contracting keys (r / 4) * 8 + r % 4
// (lanes 0-31) and the same + 4 (lanes 32-63): the B operand is the lane's own score register
// r, the A operand four consecutive keys of a V^T row, one float4 per (32-dim block, r / 4).
template <int DHP, int NW>
__global__ __launch_bounds__(NW * 64) void attn_f32_kernel(AttnArgs a, float scale_log2) {
    constexpr int HD = DHP / 2, DB = DHP / 32, MS = DB * 16 + 2;  // merge record per lane
    __shared__ float mg[(NW > 1 ? NW - 1 : 1) * MS * 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int col = lane & 31, half = lane >> 5;
    const int bh = blockIdx.y, b = bh / a.H, hh = bh - b * a.H;
    const int dh = a.dh;
    const int q0 = blockIdx.x * 32;
    const float* Q = (const float*)a.q + (long)bh * a.npq * dh;
    const float* K = (const float*)a.k + (long)bh * a.npk * dh;
    const float* VT = (const float*)a.vt + (long)bh * dh * a.npk;
    // dims half * HD + t of the lane's query row (rows past nq read the last query; dims past
    // dh are zero: dh % 8 == 0, so a float4 group is wholly inside or outside)
    float qv[HD];
    {
        const float* qr = Q + (long)min(q0 + col, a.nq - 1) * dh + half * HD;
#pragma unroll
        for (int t = 0; t < HD; t += 4) {
            const f32x4 v = half * HD + t < dh ? *(const f32x4*)(qr + t) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int e = 0; e < 4; ++e) qv[t + e] = v[e];
        }
    }
    f32x16 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
    float m = -INFINITY, l = 0.f;
    const int nkb = (a.nk + 31) / 32;
    for (int kb = wave; kb < nkb; kb += NW) {
        const int k0 = kb * 32;
        f32x16 sc;
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[r] = 0.f;
        {
            // key rows k0 + col < npk (npk is a multiple of 64 and >= nk); rows past nk are masked
            const float* kr = K + (long)(k0 + col) * dh + half * HD;
#pragma unroll
            for (int t = 0; t < HD; t += 4) {
                const f32x4 v = half * HD + t < dh ? *(const f32x4*)(kr + t) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int e = 0; e < 4; ++e) sc = __builtin_amdgcn_mfma_f32_32x32x2f32(v[e], qv[t + e], sc, 0, 0, 0);
            }
        }
        f32x4 vv[DB][4];
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            const int dim = db * 32 + col;
#pragma unroll
            for (int g = 0; g < 4; ++g)
                vv[db][g] = dim < dh ? *(const f32x4*)(VT + (long)dim * a.npk + k0 + g * 8 + half * 4)
                                     : f32x4{0.f, 0.f, 0.f, 0.f};
        }
        float bm = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int key = k0 + (r >> 2) * 8 + half * 4 + (r & 3);
            sc[r] = key < a.nk ? sc[r] * scale_log2 : -INFINITY;
            bm = fmaxf(bm, sc[r]);
        }
        bm = fmaxf(bm, __shfl_xor(bm, 32, 64));  // key 0 of the block is valid: bm is finite
        const float mn = fmaxf(m, bm);
        const float alpha = __builtin_amdgcn_exp2f(m - mn);
        m = mn;
        l *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            sc[r] = __builtin_amdgcn_exp2f(sc[r] - mn);
            l += sc[r];
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int key = k0 + (r >> 2) * 8 + half * 4 + (r & 3);
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                // masked keys have p = 0, but their V^T entries may be any value (NaN included)
                const float v = key < a.nk ? vv[db][r >> 2][r & 3] : 0.f;
                o[db] = __builtin_amdgcn_mfma_f32_32x32x2f32(v, sc[r], o[db], 0, 0, 0);
            }
        }
    }
    if (NW > 1) {
        // waves 1 .. NW-1 hand (O^T, m, l) to wave 0, which merges them in wave order
        if (wave > 0) {
            float* rec = mg + (wave - 1) * MS * 64 + lane;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int r = 0; r < 16; ++r) rec[(db * 16 + r) * 64] = o[db][r];
            rec[DB * 16 * 64] = m;
            rec[(DB * 16 + 1) * 64] = l;
        }
        __syncthreads();
        if (wave > 0) return;
        for (int w = 1; w < NW; ++w) {
            const float* rec = mg + (w - 1) * MS * 64 + lane;
            const float mw = rec[DB * 16 * 64], lw = rec[(DB * 16 + 1) * 64];
            const float mn = fmaxf(m, mw);  // wave 0 holds key block 0: m and mn are finite
            const float a0 = __builtin_amdgcn_exp2f(m - mn), a1 = __builtin_amdgcn_exp2f(mw - mn);
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int r = 0; r < 16; ++r) o[db][r] = o[db][r] * a0 + rec[(db * 16 + r) * 64] * a1;
            l = l * a0 + lw * a1;
            m = mn;
        }
    }
    const int q = q0 + col;
    if (q >= a.nq) return;
    const float inv = 1.0f / (l + __shfl_xor(l, 32, 64));
    float* O = (float*)a.o + ((long)b * a.nq + q) * ((long)a.H * dh) + (long)hh * dh;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int d0 = db * 32 + g * 8 + half * 4;
            if (d0 < dh)
                *(f32x4*)(O + d0) = f32x4{o[db][g * 4] * inv, o[db][g * 4 + 1] * inv, o[db][g * 4 + 2] * inv,
                                          o[db][g * 4 + 3] * inv};
        }
}

// bf16 launch for one head dim (every loader index and padding bound a compile-time constant)
template <int DH>
static void launch_attention_bf16(const AttnArgs& a, hipStream_t st) {
    const int BH = a.B * a.H;
    const float sl2 = (float)(1.4426950408889634 / sqrt((double)DH));
    const long qg128 = (long)((a.nq + 127) / 128) * BH;  // 128-query workgroups
    const int nkb = (a.nk + 63) / 64;
    if (nkb >= 8 && qg128 < 1024) {
        // long key range, few query groups: split the keys between two wave halves
        if (qg128 >= 256)
            hipLaunchKernelGGL((attn_split_bf16_kernel<DH, 4>), dim3((a.nq + 127) / 128, BH), dim3(512), 0, st, a, sl2);
        else
            hipLaunchKernelGGL((attn_split_bf16_kernel<DH, 2>), dim3((a.nq + 63) / 64, BH), dim3(256), 0, st, a, sl2);
    } else if (qg128 < 1024) {
        // two-wave workgroups when four-wave ones would leave CUs without a second workgroup
        hipLaunchKernelGGL((attn_bf16_kernel<DH, 2>), dim3((a.nq + 63) / 64, BH), dim3(128), 0, st, a, sl2);
    } else if (DH <= 96 && nkb < 8 && a.nq > 256 && a.nq <= 288) {
        // U-ViT: 258 queries per head (256 patches + time and class tokens) in one workgroup
        // (nine waves leave 170 VGPRs a wave: head dims above 96 would spill)
        if constexpr (DH <= 96)
            hipLaunchKernelGGL((attn_bf16_kernel<DH, 9>), dim3(1, BH), dim3(576), 0, st, a, sl2);
    } else if ((a.nq + 255) / 256 * 256 == (a.nq + 127) / 128 * 128) {
        // 256-query workgroups where they add no padded queries (DiT: one workgroup per head;
        // SDXL: four): each key/value block is loaded once per 256 queries
        hipLaunchKernelGGL((attn_bf16_kernel<DH, 8>), dim3((a.nq + 255) / 256, BH), dim3(512), 0, st, a, sl2);
    } else {
        hipLaunchKernelGGL((attn_bf16_kernel<DH, 4>), dim3((a.nq + 127) / 128, BH), dim3(256), 0, st, a, sl2);
    }
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t st) {
    const int BH = a.B * a.H;
    if (dtype == 1) {
        switch (a.dh) {
#define SGD_ATTN_DH(D) \
    case D: launch_attention_bf16<D>(a, st); break;
            SGD_ATTN_DH(8) SGD_ATTN_DH(16) SGD_ATTN_DH(24) SGD_ATTN_DH(32)
            SGD_ATTN_DH(40) SGD_ATTN_DH(48) SGD_ATTN_DH(56) SGD_ATTN_DH(64)
            SGD_ATTN_DH(72) SGD_ATTN_DH(80) SGD_ATTN_DH(88) SGD_ATTN_DH(96)
            SGD_ATTN_DH(104) SGD_ATTN_DH(112) SGD_ATTN_DH(120) SGD_ATTN_DH(128)
#undef SGD_ATTN_DH
            default: return hipErrorInvalidValue;
        }
    } else {
        const float sl2 = (float)(1.4426950408889634 / sqrt((double)a.dh));
        dim3 grid((a.nq + 31) / 32, BH), block(4 * 64);
        if (a.dh <= 32) hipLaunchKernelGGL((attn_f32_kernel<32, 4>), grid, block, 0, st, a, sl2);
        else if (a.dh <= 64) hipLaunchKernelGGL((attn_f32_kernel<64, 4>), grid, block, 0, st, a, sl2);
        else if (a.dh <= 96) hipLaunchKernelGGL((attn_f32_kernel<96, 4>), grid, block, 0, st, a, sl2);
        else hipLaunchKernelGGL((attn_f32_kernel<128, 4>), grid, block, 0, st, a, sl2);
    }
    return hipGetLastError();
}

}  // namespace sgd
