/*
 * sgd.h -- C ABI of the scheduled denoiser step of Spectral-Guided Diffusion
 * (static spectral layer scheduling) on AMD MI355X (gfx950).
 *
 * Two operations define the method:
 *   - sgd_schedule_build: Alg. 1 (Sec. 4.1).  Every scheduled weight matrix
 *     gets its regularised Spectral Concentration Ratio (Sec. 3.2, Eq.
 *     scr-reg) and matrix score g(W) (appendix, Eq. app-matrix-score);
 *     component scores (Eqs. app-attn-score, app-xattn-score, app-mlp-score)
 *     sum to a unit score (Eq. app-block-score) that is normalised (Eq.
 *     app-score-normalization) and mapped to an integer lifetime S_l by
 *     Eq. schedule, either at a fixed tau or at an exact layer-step budget.
 *   - sgd_denoise_step: Alg. 2 (Sec. 4.2) with the residual-update semantics
 *     of Sec. 3.1.  Units with s <= S_l compute their residual branches and
 *     refresh their cached update Delta_l; units with s > S_l only add the
 *     cached Delta_l to the current residual stream.  Conditioning and
 *     skip inputs keep propagating.  The step ends with the deterministic
 *     update z <- alpha z - beta eps.
 *
 * Conventions
 *   - Every function returns an int status: SGD_OK (0) or a negative SGD_E_*
 *     code.  Nothing aborts or throws across the ABI.  sgd_last_error()
 *     returns a thread-local description of the last failure.
 *   - "Device pointer" means memory of the current HIP device.  The caller
 *     owns every buffer (weights, state, cache, workspace); handles only
 *     borrow pointers and never allocate or free device memory.
 *   - Weight matrices are row-major [out, in] (y = x W^T), dtype SGD_F32 or
 *     SGD_BF16.  Norm gains/shifts, biases, class embeddings: fp32.
 *   - Calls that take a hip_stream enqueue on it and return without a host
 *     synchronisation unless documented otherwise.  All arguments are
 *     validated before anything is enqueued: a failing call enqueues
 *     nothing.  Kernel faults surface as SGD_E_HIP on a later call.
 *   - Handles are not thread-safe; use one cache per concurrent trajectory.
 */
#ifndef SGD_H
#define SGD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------------ status */
#define SGD_OK 0
#define SGD_E_ARG (-1)         /* null pointer, bad enum, inconsistent argument   */
#define SGD_E_SHAPE (-2)       /* a size the kernels do not support              */
#define SGD_E_DTYPE (-3)       /* unsupported dtype                              */
#define SGD_E_BUDGET (-4)      /* N* < L*S_min or N* > L*T                       */
#define SGD_E_STEP (-5)        /* step != previous step + 1, or outside 1..T     */
#define SGD_E_CACHE (-6)       /* frozen unit whose cache slot was never written */
#define SGD_E_HIP (-7)         /* HIP runtime error                              */
#define SGD_E_NUMERIC (-8)     /* non-finite weights or scores                   */

enum sgd_dtype { SGD_F32 = 0, SGD_BF16 = 1 };

enum sgd_arch {
    SGD_ARCH_TINY = 0,   /* RMSNorm, MHA (no bias, no RoPE), GELU(erf) MLP             */
    SGD_ARCH_LLADA = 1,  /* RMSNorm, MHA with RoPE, SwiGLU MLP                          */
    SGD_ARCH_DIT = 2,    /* LayerNorm + AdaLN shift/scale/gate, biased MHA, GELU(tanh)  */
    SGD_ARCH_UVIT = 3,   /* LayerNorm, MHA, GELU(erf) MLP, long skips via a skip linear */
    SGD_ARCH_SDXL = 4,   /* LayerNorm, self-attn, cross-attn to a context, GEGLU MLP    */
    SGD_ARCH_SDXL_UNET = 5 /* SDXL UNet stage unit: a ResNet block (GroupNorm, SiLU, 3x3
                            * convolution + time projection, GroupNorm, SiLU, 3x3
                            * convolution) followed by the SDXL transformer block        */
};

/* What one scheduled unit is (the residual units h_l = h_{l-1} + F_l of Sec. 3.1).
 * SGD_UNIT_BLOCK: one unit per block; its branches share one lifetime and one cached update,
 *   the sum of its branch updates in execution order.
 * SGD_UNIT_BRANCH: every residual branch of a block is a unit of its own, with its own lifetime
 *   and cached update (its branch output).  Block l's branches are units l nb .. l nb + nb - 1
 *   in execution order: [ResNet block (SDXL UNet)], self-attention, [cross-attention (SDXL,
 *   SDXL UNet)], MLP; nb = 2, 3 or 4.  Its score is that branch's component of
 *   Eq. app-block-score (build the schedule from one sgd_unit per branch).
 * Schedules, active rows, cache slots, drift and replay count units: U = L (blocks) or L nb. */
enum sgd_granularity { SGD_UNIT_BLOCK = 0, SGD_UNIT_BRANCH = 1 };

/* Role of a scored matrix inside its unit (appendix "Exact Block-Level Scores"). */
enum sgd_role {
    SGD_ROLE_Q = 0, SGD_ROLE_K = 1, SGD_ROLE_V = 2, SGD_ROLE_O = 3,
    SGD_ROLE_XQ = 4, SGD_ROLE_XK = 5, SGD_ROLE_XV = 6, SGD_ROLE_XO = 7,
    SGD_ROLE_W1 = 8,   /* MLP input projection; gated MLPs: stacked [W_gate; W_up] */
    SGD_ROLE_W2 = 9,   /* MLP output projection                                  */
    SGD_ROLE_CONV = 10 /* convolution kernel unfolded to C_out x (C_in k_h k_w)   */
};

const char* sgd_last_error(void);
int sgd_version(void);

/* ---------------------------------------------------------------- schedule */

/* One scored matrix: device pointer to a row-major rows x cols matrix. */
typedef struct {
    const void* ptr;
    int64_t rows, cols;
    int32_t dtype; /* sgd_dtype */
    int32_t role;  /* sgd_role  */
} sgd_matrix;

/* One scheduled unit: its scored matrices and the attention head dimension d_h. */
typedef struct {
    const sgd_matrix* mats;
    int32_t n_mats;
    int32_t head_dim;
} sgd_unit;

/* Ranking rule of a schedule: the unit score that Eq. schedule maps to lifetimes.
 * SGD_RULE_SCR_FROB is the method (Alg. 1: g(W) = ||W||_F sqrt(rho(SCR_eta)), Eq.
 * app-matrix-score).  The others are the static baselines of Sec. "Static ranking
 * comparisons" (Table "Static rankings at matched layer-step budgets"), built at the same
 * budget reading.  A matrix rule replaces g(W) by its own statistic gamma(W) inside Eqs.
 * app-attn-score, app-xattn-score, app-mlp-score and app-conv-score, so a unit keeps the
 * same component structure:
 *   SGD_RULE_FROB         gamma = ||W||_F
 *   SGD_RULE_SPECTRAL     gamma = ||W||_2 (largest singular value)
 *   SGD_RULE_STABLE_RANK  gamma = ||W||_2^2 / ||W||_F^2, the stable rank oriented like SCR
 *                         (a concentrated spectrum ranks high; the raw stable rank ranks the
 *                         other way round)
 *   SGD_RULE_FROB_SRANK   gamma = ||W||_F ||W||_2^2 / ||W||_F^2
 *   SGD_RULE_RAW_SCR      gamma = sqrt(rho(SCR_eta)), i.e. g(W) without ||W||_F
 * Unit rules need no spectra (units may be NULL):
 *   SGD_RULE_DEPTH        raw score l + 1 (deeper units live longer)
 *   SGD_RULE_RANDOM       raw score of unit l = the (l+1)-th output of SplitMix64 (Steele,
 *                         Lea and Flood, 2014) seeded with `seed`, as (x >> 11) * 2^-53
 * Every rule's raw scores are normalised by Eq. app-score-normalization. */
enum sgd_rule {
    SGD_RULE_SCR_FROB = 0, SGD_RULE_RANDOM = 1, SGD_RULE_DEPTH = 2, SGD_RULE_FROB = 3,
    SGD_RULE_SPECTRAL = 4, SGD_RULE_STABLE_RANK = 5, SGD_RULE_FROB_SRANK = 6, SGD_RULE_RAW_SCR = 7,
    SGD_RULE_COUNT = 8
};

/* Schedule parameters (Alg. 1 inputs: T, tau, S_min; plus the budget reading).
 *   T                  horizon (denoising steps), >= 1
 *   budget_layer_steps N* >= 0 selects budget mode: Eq. schedule swept over tau, filled to
 *                      exactly N* (increments granted in increasing key j / Lambda_hat_l,
 *                      ties to the lower unit index, then the lower j)
 *   budget_pct         used when budget_layer_steps < 0 and budget_pct > 0: budget mode with
 *                      N* = floor(budget_pct * L * T / 100) (sgd_budget_layer_steps)
 *   tau                scale of Eq. schedule, > 0; tau mode when neither budget is given
 *   s_min              minimum lifetime S_min, 1..T; <= 0 selects ceil(T / 10), the smallest
 *                      integer lifetime of at least a tenth of the horizon (sgd_s_min_default)
 *   eta                regulariser of Eq. scr-reg, >= 0
 *   rule               an sgd_rule value; SGD_RULE_SCR_FROB is the method
 *   seed               SGD_RULE_RANDOM only                                                   */
typedef struct {
    int32_t T;
    int32_t budget_layer_steps;
    double tau;
    int32_t s_min;
    double eta;
    int32_t budget_pct;
    int32_t rule;
    uint64_t seed;
} sgd_sched_params;

/* Output of the schedule calls.  The caller allocates every array on the host; optional
 * arrays may be NULL.  L and T are filled in by the library; L counts the scheduled units
 * (the sgd_unit list: blocks or single branches, see sgd_granularity).
 *   lifetimes  [L]      S_l
 *   active     [T*L]    active[(s-1)*L + l] = (s <= S_l)
 *   unit_raw   [L]      raw unit score q~_l of the rule        (optional)
 *   unit_score [L]      Lambda_hat_l                           (optional)
 *   mat_stats  [6*n]    per matrix, in input order: E_k, tail energy, ||W||_F^2,
 *                       SCR_eta, g(W), ||W||_2^2               (optional)
 *   layer_steps         sum_l S_l
 *   s_min               the S_min used
 *   cut_margin          budget mode: (kappa_next - kappa_last) / kappa_last between the
 *                       first refused and the last granted increment (+inf if none)     */
typedef struct {
    int32_t L, T;
    int32_t* lifetimes;
    uint8_t* active;
    double* unit_raw;
    double* unit_score;
    double* mat_stats;
    int64_t layer_steps;
    double cut_margin;
    int32_t s_min;
} sgd_schedule;

/* Integer arithmetic of the schedule's readings, exported so that callers hold none:
 * the default minimum lifetime ceil(T / 10) for T >= 1 (0 otherwise), and the layer-step
 * ceiling N* = floor(pct * L * T / 100) of a percentage budget (SGD_E_ARG unless
 * 0 <= pct <= 100, L >= 1, T >= 1). */
int32_t sgd_s_min_default(int32_t T);
int sgd_budget_layer_steps(int32_t pct, int32_t L, int32_t T, int64_t* n_star);

/* Device scratch that sgd_schedule_build / sgd_matrix_stats need for `workers` concurrent
 * matrices (fp64 Gram of the short side plus tridiagonal work arrays per worker), for the
 * largest scored matrix of `units`.  The caller allocates it (256-byte aligned) and passes
 * it in; the library allocates no device memory. */
int sgd_schedule_workspace_bytes(const sgd_unit* units, int32_t L, int32_t workers, size_t* bytes);

/* Alg. 1: score every matrix of every unit on the GPU (fp64 Gram of the short side,
 * Householder tridiagonalisation, host implicit-QL eigenvalues), then set lifetimes.
 * Offline, once per model.  As many matrices are scored at once as the workspace holds
 * worker slots (at most 16, each with its own host thread and stream); the workspace must
 * hold at least one.  units may be NULL for SGD_RULE_DEPTH and SGD_RULE_RANDOM (then L
 * alone sizes the schedule and nothing runs on the GPU).  Synchronises hip_stream before
 * returning.  Errors: SGD_E_ARG, SGD_E_DTYPE, SGD_E_BUDGET, SGD_E_NUMERIC, SGD_E_HIP. */
int sgd_schedule_build(const sgd_unit* units, int32_t L, const sgd_sched_params* params, void* workspace,
                       size_t workspace_bytes, void* hip_stream, sgd_schedule* out);

/* Statistics of one matrix (Eq. scr-reg, Eq. app-matrix-score): out[6] =
 * {E_k, tail energy, ||W||_F^2, SCR_eta, g, ||W||_2^2}.  workspace as for
 * sgd_schedule_build with one worker.  Synchronises hip_stream. */
int sgd_matrix_stats(const sgd_matrix* m, double eta, void* workspace, size_t workspace_bytes, void* hip_stream,
                     double out[6]);

/* Host only: the rule's schedule from matrix statistics already computed, e.g. the mat_stats
 * of an earlier sgd_schedule_build (to rank the same model by several rules, or at other
 * budgets, without recomputing spectra).  units gives each matrix's role and the head
 * dimension (matrix pointers are not read); mat_stats holds 6 doubles per matrix in the
 * order of units, as sgd_schedule_build writes them.  out->mat_stats is left untouched. */
int sgd_schedule_from_stats(const sgd_unit* units, int32_t L, const double* mat_stats,
                            const sgd_sched_params* params, sgd_schedule* out);

/* Host only: lifetimes from given normalised scores Lambda_hat_l in [0, 1] (Eq. schedule
 * and the budget reading above; params->rule and seed are ignored).  unit_raw / mat_stats
 * of out are left untouched. */
int sgd_schedule_from_scores(const double* unit_score, int32_t L, const sgd_sched_params* params,
                             sgd_schedule* out);

/* Host only: a schedule with the given lifetimes (1..T each), e.g. the all-active S_l = T. */
int sgd_schedule_from_lifetimes(int32_t L, int32_t T, const int32_t* lifetimes, sgd_schedule* out);

/* ------------------------------------------------------------------- model */

/* Device pointers of one unit.  Unused entries are NULL.
 *   norm{1,2,x}_{w,b}  fp32 [d]      (DiT: none; LLaDA/tiny: gains only)
 *   w_qkv  [3d x d]   rows: W_Q, W_K, W_V        b_qkv fp32 [3d]
 *   w_o    [d x d]                                b_o   fp32 [d]
 *   w1     [F x d], gated archs [2F x d] = [W_gate; W_up]   b1 fp32 [F or 2F]
 *   w2     [d x F]                                b2    fp32 [d]
 *   w_xq   [d x d], w_xkv [2d x ctx_dim] = [W_K^x; W_V^x], w_xo [d x d], b_xo fp32 [d]  (SDXL)
 *   w_ada  [6d x d], b_ada fp32 [6d]: shift1, scale1, gate1, shift2, scale2, gate2  (DiT)
 *   w_skip [d x 2d], b_skip fp32 [d]  (U-ViT out-blocks: h <- [h ; skip] W_skip^T + b)
 *   SDXL UNet ResNet block (channels d in and out): GroupNorm gains/shifts gn{1,2}_{w,b} fp32
 *   [d]; 3x3 convolutions w_conv{1,2} [d x 9d] unfolded tap-major (column (3 ky + kx) d + c
 *   multiplies input channel c at grid offset (ky - 1, kx - 1)), b_conv{1,2} fp32 [d]; time
 *   projection w_temb [d x d], b_temb fp32 [d] applied to SiLU(emb(t) + class_emb[b])      */
typedef struct {
    const void *norm1_w, *norm1_b, *w_qkv, *b_qkv, *w_o, *b_o;
    const void *norm2_w, *norm2_b, *w1, *b1, *w2, *b2;
    const void *normx_w, *normx_b, *w_xq, *w_xkv, *w_xo, *b_xo;
    const void *w_ada, *b_ada;
    const void *w_skip, *b_skip;
    const void *gn1_w, *gn1_b, *w_conv1, *b_conv1, *w_temb, *b_temb, *gn2_w, *gn2_b, *w_conv2, *b_conv2;
} sgd_unit_weights;

/* Model description.  B samples of N tokens, width d = H * head_dim, MLP width F,
 * L units, horizon T.  Rows [update_row_begin, update_row_end) of each sample are the
 * ones the sampler updates.  class_emb: DiT per-sample class vectors fp32 [B x d].
 * ctx: SDXL context, dtype [B x ctx_len x ctx_dim].  U-ViT: L odd; units < L/2 are
 * in-blocks, unit L/2 the mid block, unit l > L/2 takes the skip of in-block L-1-l;
 * token 0 of each sample is the time token, rewritten every step.
 * SDXL UNet units: the N tokens of a sample are a row-major grid x grid latent (N = grid^2),
 * GroupNorm has `groups` groups of d / groups channels (a multiple of 4), class_emb is the
 * per-sample conditioning vector of the time projection.
 * Shape limits: d % 128 == 0, F % 64 == 0, ctx_dim % 64 == 0, head_dim in {64, 72, 128}
 * (LLaDA: 128).  Every unit weight, bias, gain and shift pointer is a device pointer,
 * 16-byte aligned (the kernels read them in 16-byte vectors; SGD_E_ARG otherwise). */
typedef struct {
    int32_t arch, dtype;
    int32_t B, N, d, H, head_dim, F, L, T;
    int32_t ctx_len, ctx_dim;
    int32_t update_row_begin, update_row_end;
    const void* class_emb;
    const void* ctx;
    const sgd_unit_weights* units; /* [L], copied by sgd_model_create */
    int32_t grid, groups;          /* SDXL UNet units only */
    int32_t granularity;           /* sgd_granularity: SGD_UNIT_BLOCK (0) or SGD_UNIT_BRANCH */
} sgd_model_desc;

typedef struct sgd_model sgd_model;
typedef struct sgd_cache sgd_cache;

int sgd_model_create(const sgd_model_desc* desc, sgd_model** out);
int sgd_model_destroy(sgd_model* model);
/* The number U of scheduled units (L, or L times the branches of a block; see sgd_granularity):
 * the L of every schedule, active row, drift record and replay result of this model. */
int sgd_model_units(const sgd_model* model, int32_t* units);

/* Bytes of scratch one sgd_denoise_step needs (device, 256-byte aligned). */
int sgd_workspace_bytes(const sgd_model* model, size_t* bytes);
/* Bytes of the per-trajectory delta cache: U fp32 [B x N x d] slots (one per scheduled unit)
 * (+ SDXL context K/V, one per block). */
int sgd_cache_bytes(const sgd_model* model, size_t* bytes);
/* Wrap a caller-owned device buffer of sgd_cache_bytes as the cache of one trajectory. */
int sgd_cache_bind(sgd_model* model, void* device_buffer, size_t bytes, sgd_cache** out);
/* Start a new trajectory on this cache: the next step must be 1; no slot is valid. */
int sgd_cache_reset(sgd_cache* cache);
int sgd_cache_destroy(sgd_cache* cache);

typedef struct {
    float alpha, beta;      /* sampler coefficients of this step                      */
    void* workspace;        /* device buffer of sgd_workspace_bytes                    */
    size_t workspace_bytes;
} sgd_step_args;

/* One network evaluation at step s (Alg. 2) followed by the sampler update.
 *   state  device fp32 [B x N x d] (z_s on entry, z_{s+1} on return; updated in place)
 *   step   s in 1..T
 *   sched  NULL runs the unscheduled forward (every unit active, cache untouched, cache
 *          may be NULL); otherwise a schedule of the model's U units (sched->L == U, see
 *          sgd_model_units) and sched->T == T
 *   cache  the trajectory's cache; steps must arrive in order 1, 2, ..., T
 * A frozen unit's slot must have been written by an earlier step of this trajectory
 * (SGD_E_CACHE).  Returns after enqueueing on hip_stream.                           */
int sgd_denoise_step(sgd_model* model, void* state, int32_t step, const sgd_schedule* sched,
                     sgd_cache* cache, const sgd_step_args* args, void* hip_stream);

/* ---------------------------------------------------------------- graphs */

/* A whole scheduled trajectory captured as one HIP graph: the executor the paper describes
 * for a static active/frozen pattern (Sec. 4.2: the pattern is known before generation, so
 * the launch sequence of every step is fixed), one graph launch per trajectory instead of
 * one launch per kernel. */
typedef struct sgd_graph sgd_graph;

/* Captures sgd_denoise_step at s = 1..T with `sched` (NULL: the unscheduled forward), each
 * with its sampler update, on hip_stream (a non-null stream; nothing runs during capture).
 *   alpha, beta  host [T]: the sampler coefficients of steps 1..T
 *   state, cache, workspace: the buffers every launch of the graph uses (their addresses are
 *                recorded); cache may be NULL when sched is NULL
 * Each sgd_graph_launch runs the T steps on `state` in place (the caller writes z_1 first)
 * and writes every cache slot before a frozen step reads it, so nothing of an earlier
 * trajectory is read.  Arguments are validated as for sgd_denoise_step; the cache is left
 * reset (host bookkeeping) after capture.  Refused (SGD_E_ARG) while kernel-class
 * profiling is on.  The graph owns no device buffer. */
int sgd_graph_capture(sgd_model* model, void* state, const sgd_schedule* sched, sgd_cache* cache,
                      const float* alpha, const float* beta, void* workspace, size_t workspace_bytes,
                      void* hip_stream, sgd_graph** out);
/* Enqueues one replay of the captured trajectory on hip_stream. */
int sgd_graph_launch(sgd_graph* graph, void* hip_stream);
int sgd_graph_destroy(sgd_graph* graph);

/* ---------------------------------------------------------- no allocation */

/* Size of the library's fixed device scratch: 96 MiB, held by every GPU the library runs on
 * until the process ends. */
#define SGD_SCRATCH_BYTES (96u * 1024u * 1024u)

/* sgd_denoise_step for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the step's workspace is
 * the library's fixed scratch instead of a caller buffer, and the call allocates nothing
 * (no hipMalloc, no hipFree).  The caller still passes the state, the schedule and the
 * cache.  A model whose sgd_workspace_bytes exceeds SGD_SCRATCH_BYTES is refused with
 * SGD_E_ARG (the LLaDA-8B-shaped workload needs about 84 MB and fits; the 8192-row
 * workloads do not).  No part of the scratch needs to start at any particular value: every
 * step writes each workspace region before reading it.  All calls on one GPU share its
 * scratch, so calls that overlap in time on one GPU (other streams, other threads) race. */
int sgd_denoise_step_noalloc(sgd_model* model, void* state, int32_t step, const sgd_schedule* sched,
                             sgd_cache* cache, float alpha, float beta, void* hip_stream);

/* -------------------------------------------------- input-aware baselines */

/* One step with an arbitrary set of active units (Alg. 2 with a per-step active set that
 * need not be nested in s).  active: host [U], nonzero = the unit computes its branch(es).
 * An active unit refreshes its cached update at every active step (except at step T, which
 * no later step reads); a frozen unit adds the update of its latest active step, which must
 * exist (SGD_E_CACHE otherwise).  Steps arrive in order 1..T on the cache, as for
 * sgd_denoise_step; the two calls may not be mixed on one trajectory. */
int sgd_denoise_step_masked(sgd_model* model, void* state, int32_t step, const uint8_t* active, sgd_cache* cache,
                            const sgd_step_args* args, void* hip_stream);

/* Device bytes of the drift record of sgd_drift_step (caller-allocated, 256-byte aligned).
 * Layout: U slots of align256(B N d 4) bytes holding each unit's fp32 input [B, N, d] of
 * the last recorded step, then U x 256 x 2 fp64 partial sums (256-byte aligned), then U x 2
 * fp64 sums: sum over the input's elements of (h_s - h_{s-1})^2 and of h_s^2 per unit
 * (U = sgd_model_units). */
int sgd_drift_bytes(const sgd_model* model, size_t* bytes);

/* One step of the causal activation-drift policy (appendix "Protocol Details", "Dynamic
 * baselines", "Causal activation drift"; Table "Static versus input-aware scheduling at
 * matched per-step active counts").  After step s-1 the policy holds, for every unit l,
 *   d_{l,s-1} = ||h_{l-1,s-1} - h_{l-1,s-2}||_2 / (||h_{l-1,s-1}||_2 + 1e-8)
 * of the unit's input h_{l-1} (the residual stream arriving at the unit, for the first unit of
 * a U-ViT out-block before its skip linear; norms over the whole [B, N, d] tensor).  Step s activates the m_s units of largest lagged drift, m_s being the
 * active count of `sched` at step s, ties to the lower unit index; step 1 is full, and at
 * step 2 no lagged drift exists (every drift counts as 0).  The step then runs as
 * sgd_denoise_step_masked and records this step's unit inputs for the next one.
 *   drift_buf   device buffer of sgd_drift_bytes, the same for a whole trajectory
 *   active_out  host [U] or NULL: the active set this step used
 *   drift_out   host [U] or NULL: the lagged drift d_{l,s-1} the choice used
 * Steps s >= 3 synchronise hip_stream first, to read the drift step s-1 recorded. */
int sgd_drift_step(sgd_model* model, void* state, int32_t step, const sgd_schedule* sched, sgd_cache* cache,
                   const sgd_step_args* args, void* drift_buf, size_t drift_bytes, uint8_t* active_out,
                   double* drift_out, void* hip_stream);

/* Oracle replay (appendix "Protocol Details", "Dynamic baselines", "Oracle replay"): a
 * non-deployable headroom search.  Parameters:
 *   tau_agree        tolerance on the relative output deviation (the paper uses 5e-3)
 *   max_layer_steps  ceiling on the active unit-steps of the whole trajectory (<= 0: U T) */
typedef struct {
    double tau_agree;
    int64_t max_layer_steps;
} sgd_replay_params;

/* Device bytes of the search's buffer (caller-allocated, 256-byte aligned): the state, two
 * output buffers and 2 U cached-update slots of B N d fp32 values each, plus the SDXL
 * context projections and reduction scratch. */
int sgd_replay_bytes(const sgd_model* model, size_t* bytes);

/* Runs the search from z_1 (device fp32 [B, N, d], not modified) along the unscheduled
 * trajectory z_{s+1} = alpha z_s - beta eps(z_s):
 *   at step s >= 2 the frozen set F (cumulative: it starts as the set of step s-1) grows
 *   greedily: every unit j not in F is evaluated frozen together with F, each frozen unit
 *   adding its update from the unscheduled evaluation of its last active step, and the
 *   deviation delta = ||eps_F+j - eps||_2 / (||eps||_2 + 1e-8) over the rows the sampler
 *   updates is measured against the unscheduled output eps(z_s); the candidate of least
 *   deviation (ties to the lower index) joins F while delta <= tau_agree, or, ignoring the
 *   tolerance, while keeping the current active count for the remaining steps would exceed
 *   the ceiling.  Step 1 is full (no update exists yet).
 *   lifetimes   host [U]: S_l = the last step before unit l joined F (T if it never did), a
 *               nested schedule for sgd_schedule_from_lifetimes
 *   evaluations host, optional: network evaluations the search ran
 *   delta_log   host [T U U] or NULL: delta of candidate j in round r of step s at
 *               [((s-1) U + r) U + j], NaN where nothing was evaluated
 * args supplies alpha, beta and the step workspace.  Synchronises hip_stream. */
int sgd_replay_search(sgd_model* model, const void* z1, const sgd_replay_params* params, const sgd_step_args* args,
                      void* replay_buf, size_t replay_bytes, int32_t* lifetimes, int64_t* evaluations,
                      double* delta_log, void* hip_stream);

/* ------------------------------------------------------------- profiling */

/* Kernel classes the launcher can time with HIP events. */
enum sgd_kernel_class {
    SGD_K_NORM = 0, SGD_K_GEMM_QKV = 1, SGD_K_ATTN = 2, SGD_K_GEMM_O = 3,
    SGD_K_GEMM_W1 = 4, SGD_K_GEMM_W2 = 5, SGD_K_FROZEN = 6, SGD_K_STATE = 7,
    SGD_K_COND = 8, SGD_K_GEMM_SKIP = 9, SGD_K_GEMM_X = 10, SGD_K_ATTN_X = 11,
    SGD_K_DRIFT = 12, SGD_K_GEMM_CONV = 13, SGD_K_GNORM = 14,
    SGD_K_FOLD = 15, /* a pre-norm that also adds the frozen run ending at its unit */
    SGD_K_NORM_PARTS = 16, /* a pre-norm that also adds a split MLP output GEMM's partials */
    SGD_K_COUNT = 17
};

/* Start timing every launch of kernel class `kclass` (or -1 to stop): the launcher records
 * a HIP event pair around each such launch on the step's stream, up to `max_launches`. */
int sgd_profile_begin(sgd_model* model, int32_t kclass, int32_t max_launches);
/* Synchronise on the recorded events and return the summed duration and launch count. */
int sgd_profile_end(sgd_model* model, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* SGD_H */
