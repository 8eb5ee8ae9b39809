/*
 * sgd_ops.h -- single-kernel entry points of libsgd, for kernel-level parity tests and
 * microbenchmarks.  They run exactly the kernels that sgd_denoise_step launches.
 *
 * Conventions as in sgd.h: int status (SGD_OK or SGD_E_*), device pointers, enqueue on
 * hip_stream without synchronising, caller-owned buffers, no allocation.
 */
#ifndef SGD_OPS_H
#define SGD_OPS_H

#include <stdint.h>

#include "sgd.h"

#ifdef __cplusplus
extern "C" {
#endif

enum sgd_act { SGD_ACT_NONE = 0, SGD_ACT_GELU_ERF = 1, SGD_ACT_GELU_TANH = 2, SGD_ACT_SILU = 3 };

/* out[M x N] = act(A[M x K] W[N x K]^T + bias) in dtype (the branch GEMM of an MLP input
 * projection).  gated != 0: W is [2N x K] = [W_gate; W_up] and out = act(A W_gate^T +
 * b[:N]) * (A W_up^T + b[N:]).  lda/ldw/ldo are row strides in elements.  tile selects a
 * bf16 kernel variant (0 auto; 1..5 fixed block tiles, for tests and sweeps: 1 256x256,
 * 2 256x128, 3 128x256, 4 128x128, 5 256x192, rows x columns).  Shape limits (bf16): K % 64 == 0,
 * N % 4 == 0, gated N a multiple of the tile width, operand rows and bias 16-byte aligned;
 * (fp32): K % 16 == 0, N % 64 == 0. */
int sgd_op_linear(int32_t dtype, const void* A, int64_t lda, const void* W, int64_t ldw, const float* bias,
                  void* out, int64_t ldo, int32_t M, int32_t N, int32_t K, int32_t act, int32_t gated,
                  int32_t tile, void* hip_stream);

/* Attention (Sec. 3 units; the softmax(q k^T / sqrt(dh)) v of every head).  q [B*H, npq, dh],
 * k [B*H, npk, dh], vt [B*H, dh, npk] (dtype), o [B, nq, H*dh].  Keys >= nk are masked;
 * npk must be a multiple of 64 and >= nk; npq >= nq; 8 <= dh <= 128, dh % 8 == 0.  q, k, vt
 * 16-byte aligned, o 16-byte (fp32) or 8-byte (bf16) aligned. */
int sgd_op_attention(int32_t dtype, const void* q, const void* k, const void* vt, void* o, int32_t B, int32_t H,
                     int32_t dh, int32_t nq, int32_t npq, int32_t nk, int32_t npk, void* hip_stream);

/* Pre-norm of M rows of width d from fp32 x into y (dtype).  kind 0: RMSNorm with gain w;
 * 1: LayerNorm with gain w and shift b; 2: LayerNorm without affine parameters followed by
 * y * (1 + scale[r / ntok]) + shift[r / ntok] (rows of scale/shift mod_ld apart).  x, w, b,
 * shift, scale 16-byte aligned (mod_ld % 4 == 0), y 16-byte (fp32) or 8-byte (bf16) aligned. */
int sgd_op_norm(int32_t dtype, int32_t kind, const float* x, void* y, int32_t M, int32_t d, float eps,
                const float* w, const float* b, const float* shift, const float* scale, int64_t mod_ld,
                int32_t ntok, void* hip_stream);

/* The pre-norm that absorbs a frozen run (what the launcher runs when a run of frozen units
 * ends at an active unit, Sec. 3.1 frozen rule): x <- x + deltas[0] + ... + deltas[r-1],
 * added in that order and written back to x (fp32 [M x d], the residual stream), then y = the
 * pre-norm of the new x exactly as sgd_op_norm computes it.  1 <= r <= 32; deltas: r device
 * pointers (host array) to fp32 [M x d], 16-byte aligned.  Bitwise the same as
 * sgd_op_frozen_run followed by sgd_op_norm. */
int sgd_op_norm_fold(int32_t dtype, int32_t kind, float* x, void* y, int32_t M, int32_t d, float eps,
                     const float* w, const float* b, const float* shift, const float* scale, int64_t mod_ld,
                     int32_t ntok, const float* const* deltas, int32_t r, void* hip_stream);

/* Projection into attention heads (the QKV GEMM of a unit): P = A[M x K] W[n_proj*d x K]^T
 * (+ bias), column n of P belongs to projection which0 + n / d (0: q, 1: k, 2: v^T), head
 * (n % d) / dh, dim n % dh; row r is token r % ntok of sample r / ntok.  q, k are
 * [B*H, np, dh], vt is [B*H, dh, np].  rope != 0 rotates the q and k pairs (i, i + dh/2) of
 * token t by t * 10000^(-2i/dh) (rotary position embedding, the LLaDA attention; bf16 only,
 * dh a multiple of 8; any tile width).  Padded tokens (>= ntok) are not written.  tile as for
 * sgd_op_linear. */
int sgd_op_heads(int32_t dtype, const void* A, const void* W, const float* bias, void* q, void* k, void* vt,
                 int32_t M, int32_t K, int32_t n_proj, int32_t which0, int32_t ntok, int32_t np, int32_t H,
                 int32_t dh, int32_t rope, int32_t tile, void* hip_stream);

/* Residual projection of a branch (the O and W2 GEMMs): v = (A[M x K] W[N x K]^T + bias),
 * v *= gate[r / ntok] if gate != NULL (rows gate_ld apart), then h += v (fp32 [M x N]);
 * delta_mode 1 stores v into delta, 2 adds v to delta (the cached update of Sec. 3.1).  tile as
 * for sgd_op_linear. */
int sgd_op_residual(int32_t dtype, const void* A, int64_t lda, const void* W, const float* bias, float* h,
                    float* delta, int32_t delta_mode, const float* gate, int64_t gate_ld, int32_t ntok,
                    int32_t M, int32_t N, int32_t K, int32_t tile, void* hip_stream);

/* A residual projection in K ranges (the MLP output GEMM of a long-K unit, whose partial
 * products the next pre-norm adds to the stream; Sec. 3.1's update h + F(h) taken in parts):
 * parts + s * part_stride receives the fp32 [M x N] product of A's and W's columns
 * [s K / ksplit, (s + 1) K / ksplit), plus the bias in range 0, for s < ksplit.  bf16 only;
 * K a multiple of 64 ksplit, 2 <= ksplit <= 8, part_stride >= M N (a multiple of 4); 256 x 128
 * block tiles. */
int sgd_op_linear_split(int32_t dtype, const void* A, const void* W, const float* bias, float* parts,
                        int64_t part_stride, int32_t M, int32_t N, int32_t K, int32_t ksplit, void* hip_stream);

/* h <- h + delta[0] + ... + delta[r-1] elementwise over n fp32 values (n % 4 == 0), in
 * that order (the frozen-unit update of Sec. 3.1 for a run of r frozen units). */
int sgd_op_frozen_run(float* h, const float* const* deltas, int32_t r, int64_t n, void* hip_stream);

/* DiT AdaLN modulation (Sec. 4.2: conditioning keeps propagating; the per-block shift,
 * scale and gate vectors): mod[b, j] = sum_k x[b, k] W[j, k] + bias[j] for B rows of
 * x = SiLU(c) (fp32 [B x d]), W[n_out x d] of dtype (F32 or BF16), bias fp32 [n_out] or NULL,
 * mod fp32 [B x n_out].  d % 64 == 0; x, W 16-byte aligned.  fp32 accumulation of the exact
 * fp32 products x[b, k] W[j, k]. */
int sgd_op_adaln_mod(int32_t dtype, const float* x, const void* W, const float* bias, float* mod, int32_t B,
                     int32_t d, int32_t n_out, void* hip_stream);

/* SDXL UNet ResNet block: y = SiLU(GroupNorm(x) w + b) in bf16 for x [B, N, C] of dtype
 * in_dtype (the fp32 stream or a bf16 convolution output); groups of C / groups consecutive
 * channels (a multiple of 4) normalised over all N positions of a sample (biased variance,
 * eps), then the per-channel gain w and shift b (fp32 [C]).  C <= 4096.  scratch: caller
 * device memory of sgd_op_group_norm_scratch_bytes (per-block partial sums and the group
 * statistics).  x, w, b, scratch 16-byte aligned, y 8-byte aligned. */
int sgd_op_group_norm_scratch_bytes(int32_t B, int32_t N, int32_t groups, size_t* bytes);
int sgd_op_group_norm_silu(int32_t in_dtype, const void* x, void* y, int32_t B, int32_t N, int32_t C,
                           int32_t groups, float eps, const float* w, const float* b, void* scratch,
                           size_t scratch_bytes, void* hip_stream);

/* 3x3 convolution, stride 1, zero padding 1, of bf16 A [M x Cin] holding M / side^2 row-major
 * side x side grids, with the bf16 kernel W [N x 9 Cin] unfolded tap-major (column
 * (3 ky + kx) Cin + c multiplies channel c at grid offset (ky - 1, kx - 1)), as an implicit
 * GEMM on the matrix cores.  h == NULL: out [M x N] bf16 = conv + bias + rowbias[sample]
 * (rowbias fp32 [M / side^2 x N] or NULL); h != NULL: h [M x N] fp32 += conv + bias.
 * Cin % 64 == 0, N % 4 == 0.  tile: 0 auto, or 2 (256x128), 4 (128x128), 5 (256x192). */
int sgd_op_conv3x3(const void* A, const void* W, const float* bias, const float* rowbias, int32_t side, void* out,
                   float* h, int32_t M, int32_t N, int32_t Cin, int32_t tile, void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* SGD_OPS_H */
