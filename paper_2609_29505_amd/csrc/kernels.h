// Host-side launch functions of the HIP kernels (internal to libsgd).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sgd {

// Activation selectors for GEMM epilogues.
enum Act { ACT_NONE = 0, ACT_GELU_ERF = 1, ACT_GELU_TANH = 2, ACT_SILU = 3 };

// ---------------------------------------------------------------- GEMM
// C[M x N] = A[M x K] . B[N x K]^T with a fused epilogue.  A may come from two sources
// split along K (k < K0: A0, k >= K0: A1), which the U-ViT skip linear uses to read
// [h ; skip] without a concatenation.  Gated GEMMs read B rows [0, F) and [F, 2F) in
// pairs and write F output columns.
struct GemmArgs {
    const void* A0 = nullptr; long lda0 = 0;
    const void* A1 = nullptr; long lda1 = 0; int K0 = 0;
    const void* B = nullptr; long ldb = 0;
    int M = 0, N = 0, K = 0;  // N: product columns (gated: 2F)
    int m_begin = 0;          // first row of the launch's row tiles (rows below belong to another launch)
    int band = 0;             // bf16 GEMM tile order: row tiles per band (set by the dispatcher)
    // implicit-GEMM 3x3 convolution (bf16): A0 is the [M, conv_c] input of row-major
    // conv_side x conv_side grids (M = samples x conv_side^2), K = 9 conv_c, and A's column
    // (3 ky + kx) conv_c + c of row (sample, y, x) is input (sample, y + ky - 1, x + kx - 1, c),
    // zero outside the grid.  0: a plain GEMM.
    int conv_side = 0, conv_c = 0;
    // split K (bf16, EP_PARTIAL): workgroups [s T, (s + 1) T) of the T tiles take columns
    // [s K / ksplit, (s + 1) K / ksplit) of A and B
    int ksplit = 1;
};

enum EpKind { EP_HEADS = 0, EP_ACT = 1, EP_GATED = 2, EP_RESID = 3, EP_SKIP = 4, EP_PARTIAL = 5 };

struct EpiParams {
    int kind = EP_ACT;
    const float* bias = nullptr;
    // EP_ACT / EP_GATED: out[M x ldo] in the GEMM dtype
    void* out = nullptr; long ldo = 0; int act = 0; int F = 0;
    // EP_HEADS: q/k [B*H, Np, dh], vt [B*H, dh, Np]; column n of the product is
    // projection (which0 + n / d), head (n % d) / dh, dim n % dh
    void* q = nullptr; void* k = nullptr; void* vt = nullptr;
    int which0 = 0, ntok = 1, np = 1, H = 1, dh = 1, d = 1, rope = 0; float rope_log2_theta = 0.f;
    // EP_RESID / EP_SKIP: fp32 stream h[M x d]; delta_mode 0 none, 1 store, 2 accumulate
    // (EP_SKIP: 1 = add the cached delta to the skip output); gate[b * gate_ld + n]
    float* h = nullptr; float* delta = nullptr; int delta_mode = 0;
    const float* gate = nullptr; long gate_ld = 0; void* hcopy = nullptr;
    // EP_ACT: per-sample additive bias rowbias[sample * rowbias_ld + n] (sample = row / ntok)
    const float* rowbias = nullptr; long rowbias_ld = 0;
    // EP_PARTIAL: K range s of a split product, fp32, to h + s * part_stride ([M x d]); the bias
    // goes into range 0 only
    long part_stride = 0;
};

// dtype: 0 fp32, 1 bf16.  tile: 0 = pick automatically; 1..kGemmTiles a fixed bf16 block
// tile (1: 256x256, 2: 256x128, 3: 128x256, 4: 128x128, 5: 256x192).
constexpr int kGemmTiles = 5;
hipError_t launch_gemm(int dtype, const GemmArgs& g, const EpiParams& e, hipStream_t st, int tile = 0);
bool gemm_shape_ok(int dtype, const GemmArgs& g, const EpiParams& e, int tile = 0);
hipError_t launch_gemm_bf16(const GemmArgs& g, const EpiParams& e, hipStream_t st, int tile);
bool gemm_bf16_shape_ok(const GemmArgs& g, const EpiParams& e, int tile);
int gemm_bf16_auto_tile(const GemmArgs& g, const EpiParams& e);
// automatic tiling: rows [0, m_split) with `tile`, rows [m_split, M) (if any) with tail_tile
struct GemmPlan { int tile, m_split, tail_tile; };
GemmPlan gemm_bf16_plan(const GemmArgs& g, const EpiParams& e);
// K ranges worth splitting the [M x N] product of `g` into (1: none), when one round of
// 128 x 128 tiles is the best unsplit plan and the K ranges of larger tiles still fit one
// round; the split product runs 256 x 128 tiles (EP_PARTIAL)
int gemm_bf16_ksplit(const GemmArgs& g);

// ---------------------------------------------------------------- attention
// O[b, i, h*dh + j] = softmax_j'(q_i . k_j' / sqrt(dh)) v_j'  over keys j' < nk.
// q [BH, npq, dh], k [BH, npk, dh], vt [BH, dh, npk]; O row-major [B, nq, H*dh].
struct AttnArgs {
    const void* q; const void* k; const void* vt; void* o;
    int B, H, dh, nq, npq, nk, npk;
};
hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t st);

// ---------------------------------------------------------------- norms
constexpr int kMaxRun = 32;  // frozen units fused into one pass at most
// kind 0: RMSNorm(w), 1: LayerNorm(w, b), 2: LayerNorm (no affine) * (1 + scale_b) + shift_b.
// nfold > 0: x is the fp32 stream h of the rows and a run of frozen units ends here: the kernel
// first forms h <- ((h + fold[0]) + fold[1]) + ... (the frozen-run update, same order), writes
// it back to x, then normalises it.
struct NormArgs {
    const float* x; void* y; int M, d, kind; float eps;
    const float* w; const float* b;
    const float* shift; const float* scale; long mod_ld; int ntok;
    int nfold = 0;
    const float* fold[kMaxRun] = {};
};
// parts: the fold holds the partial products of a split residual GEMM rather than a frozen
// run's cached updates (the same additions, a kernel of its own name)
hipError_t launch_norm(int dtype, const NormArgs& a, hipStream_t st, bool parts = false);
// y = SiLU(GroupNorm(x) w + b) in bf16 for x [B, N, C] fp32 (in_bf16 = 0) or bf16; groups of
// C / groups consecutive channels (a multiple of 4) over all N positions of a sample
struct GroupNormArgs {
    const void* x; void* y; int B, N, C, groups; float eps;
    const float* w; const float* b;
};
// scratch: group_norm_scratch_bytes(B, N, groups) device bytes (per-block partial sums, stats);
// C / 4 <= 1024 threads per row block
size_t group_norm_scratch_bytes(int B, int N, int groups);
hipError_t launch_group_norm_silu(int in_bf16, const GroupNormArgs& a, void* scratch, hipStream_t st);

// ---------------------------------------------------------------- elementwise
struct FrozenRun {
    float* h; long n;  // elements
    int r;
    int snap_bf16;  // snapshot dtype: 1 bf16, 0 fp32
    const float* delta[kMaxRun];
    void* snap[kMaxRun];  // optional copies of h after adding delta[i]
};
hipError_t launch_frozen_run(const FrozenRun& f, hipStream_t st);

// h = z; U-ViT: token 0 of every sample = sinusoidal embedding of t
hipError_t launch_stream_init(const float* z, float* h, int B, int N, int d, int time_token, float t,
                              hipStream_t st);
// z = alpha z - beta h on rows [r0, r1) of every sample
hipError_t launch_state_update(float* z, const float* h, int B, int N, int d, int r0, int r1,
                               float alpha, float beta, hipStream_t st);
// x[b, :] = SiLU(emb(t) + y[b, :])  (DiT conditioning input)
hipError_t launch_cond_silu(const float* y, float* x, int B, int d, float t, hipStream_t st);
// mod[b, j] = sum_k x[b, k] W[j, k] + bias[j]  (DiT AdaLN modulation, W dtype)
hipError_t launch_adaln_mod(int dtype, const float* x, const void* W, const float* bias, float* mod,
                            int B, int d, int n_out, hipStream_t st);
// The same product for several units at once (one x, each unit its own W, bias and output):
// one launch, the unit in the grid's third dimension, each unit's tiles computed exactly as a
// single-unit launch computes them.
constexpr int kMaxModUnits = 32;
struct ModBatch {
    int n = 0;
    const void* W[kMaxModUnits] = {};
    const float* bias[kMaxModUnits] = {};
    float* mod[kMaxModUnits] = {};
};
hipError_t launch_adaln_mod_batch(int dtype, const float* x, const ModBatch& mb, int B, int d, int n_out,
                                  hipStream_t st);
// fp32 -> bf16 copy
hipError_t launch_to_bf16(const float* x, void* y, long n, hipStream_t st);

// Deterministic squared norms over rows [r0, r1) of every sample of fp32 [B, N, d] tensors:
// partial[2 b] = sum (x - y)^2 (0 unless have_y), partial[2 b + 1] = sum x^2 for the
// elements of block b (kSumBlocks blocks, fixed assignment and reduction order, fp64);
// copy (may alias y) receives x.  launch_sumsq_finish sums the partials of `count` tensors
// (partial + i * 2 kSumBlocks) into out[2 i], out[2 i + 1].
constexpr int kSumBlocks = 256;
hipError_t launch_sumsq(const float* x, const float* y, float* copy, int B, int N, int d, int r0, int r1,
                        int have_y, double* partial, hipStream_t st);
hipError_t launch_sumsq_finish(const double* partial, int count, double* out, hipStream_t st);

// ---------------------------------------------------------------- spectra (fp64)
// G = X^T X (trans = 0, X rows x cols, G cols x cols) or X X^T (trans = 1, G rows x rows)
hipError_t launch_gram(int dtype, const void* X, long rows, long cols, int trans, double* G, hipStream_t st);
// Householder tridiagonalisation of the symmetric n x n matrix A (destroyed).  diag[n],
// offd[n-1] receive the tridiagonal; work holds 5n + 8 doubles.
hipError_t launch_tridiagonalize(double* A, int n, double* diag, double* offd, double* work,
                                 hipStream_t st);
hipError_t launch_diag_copy(const double* A, int n, double* out, hipStream_t st);

}  // namespace sgd
