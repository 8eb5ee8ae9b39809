// C ABI: model and cache handles, and the step launcher of the jagged denoiser step
// (Alg. 2, Sec. 4.2; residual-update semantics of Sec. 3.1).
//
// The launcher walks the units in stack order and enqueues only the kernels of active
// units.  A maximal run of consecutive frozen units becomes one bandwidth-bound kernel
// h <- h + Delta_l1 + ... + Delta_lr.  An active unit writes its cached update Delta_l
// (the sum of its branch updates, in branch order) only at its last active step s = S_l,
// because that is the update every later frozen step reads (r_l(s) = S_l).
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"
#include "kernels.h"
#include "model.h"

namespace sgd {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }
int fail(int code, const std::string& msg) {
    g_last_error = msg;
    return code;
}
int hip_fail(hipError_t e, const char* what) {
    g_last_error = std::string(what) + ": " + hipGetErrorString(e);
    return SGD_E_HIP;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace sgd

using namespace sgd;

extern "C" const char* sgd_last_error(void) { return sgd::g_last_error.c_str(); }
extern "C" int sgd_version(void) { return 1; }

namespace sgd {
bool arch_gated(int a) { return a == SGD_ARCH_LLADA || a == SGD_ARCH_SDXL || a == SGD_ARCH_SDXL_UNET; }
bool arch_cross(int a) { return a == SGD_ARCH_SDXL || a == SGD_ARCH_SDXL_UNET; }
int block_branch(int arch, int i) {
    const int first = arch == SGD_ARCH_SDXL_UNET ? BR_RESNET : BR_ATTN;
    int b = first + i;
    if (b >= BR_XATTN && !arch_cross(arch)) ++b;  // no cross-attention branch
    return b;
}
int block_branches(int arch) { return 2 + (arch == SGD_ARCH_SDXL_UNET) + arch_cross(arch); }
}  // namespace sgd

namespace {

int check_unit(const sgd_model_desc& d, const sgd_unit_weights& w, int l) {
    auto need = [&](const void* p, const char* name) -> int {
        if (!p) return fail(SGD_E_ARG, "unit " + std::to_string(l) + ": " + name + " is NULL");
        return SGD_OK;
    };
    int rc = SGD_OK;
    if ((rc = need(w.w_qkv, "w_qkv")) || (rc = need(w.w_o, "w_o")) || (rc = need(w.w1, "w1")) ||
        (rc = need(w.w2, "w2")))
        return rc;
    switch (d.arch) {
        case SGD_ARCH_TINY:
        case SGD_ARCH_LLADA:
            if ((rc = need(w.norm1_w, "norm1_w")) || (rc = need(w.norm2_w, "norm2_w"))) return rc;
            break;
        case SGD_ARCH_DIT:
            if ((rc = need(w.w_ada, "w_ada"))) return rc;
            break;
        case SGD_ARCH_UVIT:
        case SGD_ARCH_SDXL:
        case SGD_ARCH_SDXL_UNET:
            if ((rc = need(w.norm1_w, "norm1_w")) || (rc = need(w.norm1_b, "norm1_b")) ||
                (rc = need(w.norm2_w, "norm2_w")) || (rc = need(w.norm2_b, "norm2_b")))
                return rc;
            break;
    }
    if (d.arch == SGD_ARCH_SDXL_UNET) {
        if ((rc = need(w.gn1_w, "gn1_w")) || (rc = need(w.gn1_b, "gn1_b")) || (rc = need(w.w_conv1, "w_conv1")) ||
            (rc = need(w.b_conv1, "b_conv1")) || (rc = need(w.w_temb, "w_temb")) || (rc = need(w.b_temb, "b_temb")) ||
            (rc = need(w.gn2_w, "gn2_w")) || (rc = need(w.gn2_b, "gn2_b")) || (rc = need(w.w_conv2, "w_conv2")) ||
            (rc = need(w.b_conv2, "b_conv2")))
            return rc;
    }
    if (d.arch == SGD_ARCH_UVIT && l > d.L / 2 && (rc = need(w.w_skip, "w_skip"))) return rc;
    if (arch_cross(d.arch)) {
        if ((rc = need(w.normx_w, "normx_w")) || (rc = need(w.normx_b, "normx_b")) || (rc = need(w.w_xq, "w_xq")) ||
            (rc = need(w.w_xkv, "w_xkv")) || (rc = need(w.w_xo, "w_xo")))
            return rc;
    }
    // the kernels read weights, biases, gains and shifts in 16-byte vectors
    const void* ptrs[] = {w.norm1_w, w.norm1_b, w.w_qkv, w.b_qkv, w.w_o, w.b_o, w.norm2_w, w.norm2_b, w.w1, w.b1,
                          w.w2, w.b2, w.normx_w, w.normx_b, w.w_xq, w.w_xkv, w.w_xo, w.b_xo, w.w_ada, w.b_ada,
                          w.w_skip, w.b_skip, w.gn1_w, w.gn1_b, w.w_conv1, w.b_conv1, w.w_temb, w.b_temb,
                          w.gn2_w, w.gn2_b, w.w_conv2, w.b_conv2};
    for (const void* p : ptrs)
        if ((uintptr_t)p % 16) return fail(SGD_E_ARG, "unit " + std::to_string(l) + ": weights must be 16-byte aligned");
    return SGD_OK;
}

}  // namespace

extern "C" int sgd_model_create(const sgd_model_desc* desc, sgd_model** out) {
    if (!desc || !out || !desc->units) return fail(SGD_E_ARG, "NULL argument");
    const sgd_model_desc& d = *desc;
    if (d.arch < SGD_ARCH_TINY || d.arch > SGD_ARCH_SDXL_UNET) return fail(SGD_E_ARG, "unknown arch");
    if (d.dtype != SGD_F32 && d.dtype != SGD_BF16) return fail(SGD_E_DTYPE, "dtype must be F32 or BF16");
    if (d.dtype == SGD_F32 && (arch_gated(d.arch) || d.arch == SGD_ARCH_LLADA))
        return fail(SGD_E_DTYPE, "fp32 is supported for the tiny, DiT and U-ViT architectures");
    if (d.B < 1 || d.N < 1 || d.L < 1 || d.T < 1 || d.H < 1 || d.head_dim < 1)
        return fail(SGD_E_SHAPE, "B, N, L, T, H, head_dim must be >= 1");
    if (d.d != d.H * d.head_dim) return fail(SGD_E_SHAPE, "d must equal H * head_dim");
    if (d.d % 128) return fail(SGD_E_SHAPE, "d must be a multiple of 128");
    if (d.F < 64 || d.F % 64 || (!arch_gated(d.arch) && d.F % 128))
        return fail(SGD_E_SHAPE, "F must be a multiple of 128 (gated MLPs: 64)");
    if (d.head_dim != 64 && d.head_dim != 72 && d.head_dim != 128) return fail(SGD_E_SHAPE, "head_dim must be 64, 72 or 128");
    if (d.arch == SGD_ARCH_LLADA && d.head_dim != 128) return fail(SGD_E_SHAPE, "rotary heads need head_dim 128");
    if (d.update_row_begin < 0 || d.update_row_end > d.N || d.update_row_begin > d.update_row_end)
        return fail(SGD_E_ARG, "update rows outside [0, N]");
    if ((d.arch == SGD_ARCH_DIT || d.arch == SGD_ARCH_SDXL_UNET) && !d.class_emb)
        return fail(SGD_E_ARG, "DiT and SDXL UNet units need class_emb");
    if (d.arch == SGD_ARCH_SDXL_UNET) {
        if (d.grid < 1 || (long)d.grid * d.grid != d.N) return fail(SGD_E_SHAPE, "SDXL UNet units need N = grid^2");
        if (d.groups < 1 || d.d % d.groups || (d.d / d.groups) % 4 || d.d > 4096)
            return fail(SGD_E_SHAPE, "GroupNorm groups must split d (<= 4096) into multiples of 4 channels");
    }
    if (d.arch == SGD_ARCH_UVIT && (d.L % 2 == 0 || d.L < 3)) return fail(SGD_E_SHAPE, "U-ViT needs an odd L >= 3");
    if (d.arch == SGD_ARCH_UVIT && d.N < 2) return fail(SGD_E_SHAPE, "U-ViT needs the time and class tokens");
    if (arch_cross(d.arch)) {
        if (!d.ctx) return fail(SGD_E_ARG, "SDXL needs ctx");
        if (d.ctx_len < 1 || d.ctx_dim < 64 || d.ctx_dim % 64) return fail(SGD_E_SHAPE, "ctx_len >= 1, ctx_dim % 64 == 0");
    }
    if ((long)d.B * d.N * d.d >= (1L << 31)) return fail(SGD_E_SHAPE, "B * N * d must stay below 2^31");
    if (d.granularity != SGD_UNIT_BLOCK && d.granularity != SGD_UNIT_BRANCH)
        return fail(SGD_E_ARG, "granularity must be SGD_UNIT_BLOCK or SGD_UNIT_BRANCH");
    for (int l = 0; l < d.L; ++l) {
        int rc = check_unit(d, d.units[l], l);
        if (rc) return rc;
    }
    sgd_model* m = new sgd_model();
    m->d = d;
    m->u.assign(d.units, d.units + d.L);
    m->d.units = nullptr;
    m->dt = d.dtype == SGD_BF16 ? 1 : 0;
    m->es = m->dt ? 2 : 4;
    m->np = (d.N + 63) / 64 * 64;
    m->npc = arch_cross(d.arch) ? (d.ctx_len + 63) / 64 * 64 : 64;
    m->M = (long)d.B * d.N;
    m->nb = d.granularity == SGD_UNIT_BRANCH ? block_branches(d.arch) : 1;
    m->nu = d.L * m->nb;
    const size_t Md = (size_t)m->M * d.d;
    const size_t heads = (size_t)d.B * d.H * m->np * d.head_dim;
    const size_t cheads = (size_t)d.B * d.H * m->npc * d.head_dim;
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t r = o; o = align256(o + bytes); return r; };
    m->w_h = take(Md * 4);
    m->w_xb = take(Md * m->es);
    m->w_q = take(heads * m->es);
    m->w_k = take(heads * m->es);
    m->w_vt = take(heads * m->es);
    m->w_ob = take(Md * m->es);
    m->w_hid = take((size_t)m->M * d.F * m->es);
    const bool cond = d.arch == SGD_ARCH_DIT || d.arch == SGD_ARCH_SDXL_UNET;
    m->w_siluc = take(cond ? (size_t)d.B * d.d * 4 : 0);
    // one modulation slot per block: a step computes every needed block's in one launch
    m->mod_slot = cond ? align256((size_t)d.B * (d.arch == SGD_ARCH_DIT ? 6 : 1) * d.d * 4) : 0;
    m->w_mod = take(m->mod_slot * d.L);
    m->w_hb = take(d.arch == SGD_ARCH_UVIT ? 2 * Md * m->es : 0);
    m->w_skip = take(d.arch == SGD_ARCH_UVIT ? (size_t)(d.L / 2) * align256(Md * m->es) : 0);
    m->ckv_unit = align256(2 * cheads * m->es);
    m->w_ckv = take(arch_cross(d.arch) ? m->ckv_unit : 0);
    m->w_gn = take(d.arch == SGD_ARCH_SDXL_UNET ? group_norm_scratch_bytes(d.B, d.N, d.groups) : 0);
    m->w_total = o;
    if (m->dt == 1) {
        GemmArgs g;
        g.M = (int)m->M; g.N = d.d; g.K = d.F; g.lda0 = d.F; g.ldb = d.F;
        const int ks = gemm_bf16_ksplit(g);
        m->part_bytes = align256(Md * 4);
        if (ks > 1 && m->w_q + ks * m->part_bytes <= m->w_hid) m->w2_ksplit = ks;
    }
    o = 0;
    m->c_delta = take((size_t)m->nu * align256(Md * 4));
    m->c_ctx = take(arch_cross(d.arch) ? (size_t)d.L * m->ckv_unit : 0);
    m->c_total = o;
    *out = m;
    return SGD_OK;
}

extern "C" int sgd_model_destroy(sgd_model* m) {
    if (!m) return fail(SGD_E_ARG, "NULL model");
    for (hipEvent_t e : m->prof_ev) (void)hipEventDestroy(e);
    delete m;
    return SGD_OK;
}

extern "C" int sgd_model_units(const sgd_model* m, int32_t* units) {
    if (!m || !units) return fail(SGD_E_ARG, "NULL argument");
    *units = m->nu;
    return SGD_OK;
}

extern "C" int sgd_workspace_bytes(const sgd_model* m, size_t* bytes) {
    if (!m || !bytes) return fail(SGD_E_ARG, "NULL argument");
    *bytes = m->w_total;
    return SGD_OK;
}

extern "C" int sgd_cache_bytes(const sgd_model* m, size_t* bytes) {
    if (!m || !bytes) return fail(SGD_E_ARG, "NULL argument");
    *bytes = m->c_total;
    return SGD_OK;
}

extern "C" int sgd_cache_bind(sgd_model* m, void* buf, size_t bytes, sgd_cache** out) {
    if (!m || !buf || !out) return fail(SGD_E_ARG, "NULL argument");
    if (bytes < m->c_total) return fail(SGD_E_ARG, "cache buffer smaller than sgd_cache_bytes");
    if ((uintptr_t)buf % 256) return fail(SGD_E_ARG, "cache buffer must be 256-byte aligned");
    sgd_cache* c = new sgd_cache();
    c->m = m;
    c->base = (char*)buf;
    c->bytes = bytes;
    c->last_step = 0;
    c->written.assign(m->nu, 0);
    c->ctx_valid = false;
    *out = c;
    return SGD_OK;
}

extern "C" int sgd_cache_reset(sgd_cache* c) {
    if (!c) return fail(SGD_E_ARG, "NULL cache");
    c->last_step = 0;
    std::fill(c->written.begin(), c->written.end(), 0);
    c->ctx_valid = false;
    return SGD_OK;
}

extern "C" int sgd_cache_destroy(sgd_cache* c) {
    if (!c) return fail(SGD_E_ARG, "NULL cache");
    delete c;
    return SGD_OK;
}

extern "C" int sgd_profile_begin(sgd_model* m, int32_t kclass, int32_t max_launches) {
    if (!m) return fail(SGD_E_ARG, "NULL model");
    if (kclass >= SGD_K_COUNT || kclass < -1) return fail(SGD_E_ARG, "unknown kernel class");
    for (hipEvent_t e : m->prof_ev) (void)hipEventDestroy(e);
    m->prof_ev.clear();
    m->prof_class = -1;
    m->prof_n = 0;
    if (kclass < 0) return SGD_OK;
    if (max_launches < 1 || max_launches > (1 << 16)) return fail(SGD_E_ARG, "max_launches must lie in 1..65536");
    m->prof_ev.resize(2 * (size_t)max_launches);
    for (auto& e : m->prof_ev) SGD_HIP_TRY(hipEventCreate(&e));
    m->prof_class = kclass;
    m->prof_max = max_launches;
    return SGD_OK;
}

extern "C" int sgd_profile_end(sgd_model* m, double* total_ms, int64_t* launches) {
    if (!m || !total_ms || !launches) return fail(SGD_E_ARG, "NULL argument");
    double tot = 0.0;
    for (int i = 0; i < m->prof_n; ++i) {
        SGD_HIP_TRY(hipEventSynchronize(m->prof_ev[2 * i + 1]));
        float ms = 0.f;
        SGD_HIP_TRY(hipEventElapsedTime(&ms, m->prof_ev[2 * i], m->prof_ev[2 * i + 1]));
        tot += ms;
    }
    *total_ms = tot;
    *launches = m->prof_n;
    m->prof_class = -1;
    m->prof_n = 0;
    return SGD_OK;
}

// ---------------------------------------------------------------------------- step

namespace {

struct Step {
    sgd_model* m;
    hipStream_t st;
    char* ws;
    hipError_t err = hipSuccess;

    template <typename F>
    void run(int kclass, F&& f) {
        if (err != hipSuccess) return;
        const bool prof = m->prof_class == kclass && m->prof_n < m->prof_max;
        if (prof) err = hipEventRecord(m->prof_ev[2 * m->prof_n], st);
        if (err == hipSuccess) err = f();
        if (prof && err == hipSuccess) {
            err = hipEventRecord(m->prof_ev[2 * m->prof_n + 1], st);
            m->prof_n++;
        }
    }
};

}  // namespace

namespace sgd {

// Shape check of every GEMM the step launches (nothing is enqueued on failure).
int check_step_shapes(const sgd_model* m) {
    const sgd_model_desc& d = m->d;
    const bool gated = arch_gated(d.arch);
    GemmArgs g;
    EpiParams e;
    g.M = (int)m->M; g.K = d.d; g.N = 3 * d.d; e.kind = EP_HEADS; e.rope = d.arch == SGD_ARCH_LLADA; e.dh = d.head_dim;
    e.d = d.d;
    bool ok = gemm_shape_ok(m->dt, g, e);
    e.rope = 0; e.kind = EP_RESID; g.N = d.d; ok = ok && gemm_shape_ok(m->dt, g, e);
    e.kind = gated ? EP_GATED : EP_ACT; g.N = gated ? 2 * d.F : d.F; ok = ok && gemm_shape_ok(m->dt, g, e);
    e.kind = EP_RESID; g.N = d.d; g.K = d.F; ok = ok && gemm_shape_ok(m->dt, g, e);
    if (m->w2_ksplit > 1) {
        GemmArgs gs = g;
        gs.ksplit = m->w2_ksplit;
        EpiParams es = e;
        es.kind = EP_PARTIAL; es.part_stride = (long)(m->part_bytes / 4);
        ok = ok && gemm_shape_ok(m->dt, gs, es);
    }
    if (d.arch == SGD_ARCH_SDXL_UNET) {
        g.K = 9 * d.d; g.lda0 = d.d; g.ldb = 9 * d.d; g.conv_side = d.grid; g.conv_c = d.d;
        ok = ok && gemm_shape_ok(m->dt, g, e);
        e.kind = EP_ACT; e.ldo = d.d; ok = ok && gemm_shape_ok(m->dt, g, e);
    }
    if (!ok) return fail(SGD_E_SHAPE, "GEMM shapes not supported by the kernels");
    return SGD_OK;
}

// One network evaluation at step `step` (Alg. 2) as the plan describes it: the units in
// stack order, active ones computing every branch, maximal runs of frozen ones adding their
// cached updates in one pass; then the sampler update (or h_L left in the stream buffer).
// Arguments are validated by the callers.
int run_step(sgd_model* m, void* state, int step, const StepPlan& plan, const sgd_step_args* args,
             hipStream_t stream) {
    const sgd_model_desc& d = m->d;
    Step S{m, stream, (char*)args->workspace};
    const int dt = m->dt;
    const long M = m->M;
    const int L = d.L;
    const int dd = d.d, F = d.F, H = d.H, dh = d.head_dim, N = d.N;
    const size_t Md = (size_t)M * dd;
    const uint8_t* act = plan.act;
    float* h = plan.h ? plan.h : (float*)(S.ws + m->w_h);
    void* xb = S.ws + m->w_xb;
    void* qb = S.ws + m->w_q;
    void* kb = S.ws + m->w_k;
    void* vtb = S.ws + m->w_vt;
    void* ob = S.ws + m->w_ob;
    void* hid = S.ws + m->w_hid;
    float* siluc = (float*)(S.ws + m->w_siluc);
    auto hb = [&](int i) { return (void*)(S.ws + m->w_hb + i * Md * m->es); };
    auto skipbuf = [&](int i) { return (void*)(S.ws + m->w_skip + (size_t)i * align256(Md * m->es)); };
    const bool uvit = d.arch == SGD_ARCH_UVIT, dit = d.arch == SGD_ARCH_DIT, sdxl = arch_cross(d.arch);
    const bool unet = d.arch == SGD_ARCH_SDXL_UNET;
    const int half = L / 2;
    const float t = (float)(1000.0 * (double)(d.T - step + 1) / (double)d.T);
    const int norm_kind = (d.arch == SGD_ARCH_TINY || d.arch == SGD_ARCH_LLADA) ? 0 : dit ? 2 : 1;
    const float norm_eps = dit ? 1e-6f : 1e-5f;
    const bool gated = arch_gated(d.arch);
    const int mlp_act = d.arch == SGD_ARCH_LLADA ? ACT_SILU : dit ? ACT_GELU_TANH : ACT_GELU_ERF;
    const DriftRec* dr = plan.drift;

    // ---- stream set-up and per-step conditioning
    S.run(SGD_K_STATE, [&] { return launch_stream_init((const float*)state, h, d.B, N, dd, uvit ? 1 : 0, t, S.st); });
    if (dit || unet)
        S.run(SGD_K_COND, [&] { return launch_cond_silu((const float*)d.class_emb, siluc, d.B, dd, t, S.st); });

    // SDXL: context keys/values are step-invariant; a trajectory computes them once into its
    // cache, an unscheduled evaluation per active unit into the workspace.
    const size_t cheads = (size_t)d.B * H * m->npc * dh;
    auto ctx_kv = [&](int l, char* dst) {
        GemmArgs g;
        g.A0 = d.ctx; g.lda0 = d.ctx_dim; g.B = m->u[l].w_xkv; g.ldb = d.ctx_dim;
        g.M = d.B * d.ctx_len; g.N = 2 * dd; g.K = d.ctx_dim;
        EpiParams e;
        e.kind = EP_HEADS; e.which0 = 1; e.k = dst; e.vt = dst + cheads * m->es;
        e.ntok = d.ctx_len; e.np = m->npc; e.H = H; e.dh = dh; e.d = dd;
        S.run(SGD_K_GEMM_X, [&] { return launch_gemm(dt, g, e, S.st); });
    };
    if (sdxl && plan.ckv && plan.ckv_fill)
        for (int l = 0; l < L; ++l) ctx_kv(l, plan.ckv + (size_t)l * m->ckv_unit);

    // block l's modulation (DiT: AdaLN shift, scale and gate of both branches; UNet: the ResNet
    // branch's time projection) for every block whose consumer runs this step, in one launch
    // per kMaxModUnits blocks instead of one per block
    auto mod_of = [&](int l) { return (float*)(S.ws + m->w_mod + (size_t)l * m->mod_slot); };
    if (dit || unet) {
        ModBatch mb;
        auto flush = [&] {
            if (!mb.n) return;
            S.run(SGD_K_COND, [&] {
                return launch_adaln_mod_batch(dt, siluc, mb, d.B, dd, dit ? 6 * dd : dd, S.st);
            });
            mb.n = 0;
        };
        for (int l = 0; l < L; ++l) {
            bool need = false;  // DiT: any unit of the block; UNet: its ResNet branch (the first)
            for (int k = 0; k < (dit ? m->nb : 1); ++k) need = need || act[l * m->nb + k];
            if (!need) continue;
            mb.W[mb.n] = dit ? m->u[l].w_ada : m->u[l].w_temb;
            mb.bias[mb.n] = (const float*)(dit ? m->u[l].b_ada : m->u[l].b_temb);
            mb.mod[mb.n] = mod_of(l);
            if (++mb.n == kMaxModUnits) flush();
        }
        flush();
    }

    // a frozen run that ends at an active unit is added by that unit's first norm kernel
    // (same additions, same order) instead of a pass of its own
    std::vector<const float*> fold;
    bool fold_parts = false;  // fold holds a split MLP output GEMM's partial products
    auto norm = [&](const float* w, const float* b, const float* shift, const float* scale) {
        NormArgs a{h, xb, (int)M, dd, norm_kind, norm_eps, w, b, shift, scale, 6L * dd, N};
        a.nfold = (int)fold.size();
        for (int i = 0; i < a.nfold; ++i) a.fold[i] = fold[i];
        const int kclass = fold.empty() ? SGD_K_NORM : fold_parts ? SGD_K_NORM_PARTS : SGD_K_FOLD;
        const bool parts = fold_parts;
        fold.clear();
        fold_parts = false;
        S.run(kclass, [&] { return launch_norm(dt, a, S.st, parts); });
    };
    auto resid = [&](int kclass, const void* A, long lda, int K, const void* W, const void* bias, const float* gate,
                     float* dlt, int dmode, void* hcopy) {
        GemmArgs g;
        g.A0 = A; g.lda0 = lda; g.B = W; g.ldb = K; g.M = (int)M; g.N = dd; g.K = K;
        EpiParams e;
        e.kind = EP_RESID; e.bias = (const float*)bias; e.h = h; e.d = dd; e.delta = dlt; e.delta_mode = dmode;
        e.gate = gate; e.gate_ld = 6L * dd; e.ntok = N; e.hcopy = hcopy;
        S.run(kclass, [&] { return launch_gemm(dt, g, e, S.st); });
    };
    auto attention = [&](const void* q, const void* k, const void* vt, int nk, int npk, int kclass) {
        AttnArgs a{q, k, vt, ob, d.B, H, dh, N, m->np, nk, npk};
        S.run(kclass, [&] { return launch_attention(dt, a, S.st); });
    };
    // the input-aware baseline: this unit's input against the previous recorded step's
    auto record_drift = [&](int l) {
        if (!dr) return;
        S.run(SGD_K_DRIFT, [&] {
            return launch_sumsq(h, dr->prev + (size_t)l * (align256(Md * 4) / 4), dr->prev + (size_t)l * (align256(Md * 4) / 4),
                                d.B, N, dd, 0, N, dr->have_prev ? 1 : 0, dr->partial + (size_t)l * kSumBlocks * 2, S.st);
        });
    };

    int hb_cur = 0;
    // where block l's output copy (for a long skip or the next out-block) goes, or NULL
    auto out_copy = [&](int l) -> void* {
        if (!uvit) return nullptr;
        if (l < half) return skipbuf(l);
        if (l + 1 < L) return hb(hb_cur);
        return nullptr;
    };

    // scheduled units: blocks (nb = 1: a unit runs every branch of its block) or single
    // branches (nb = the block's branch count: unit u is branch u % nb of block u / nb)
    const int nb = m->nb, nu = m->nu;
    auto branch_of = [&](int u) { return nb == 1 ? -1 : block_branch(d.arch, u % nb); };
    auto last_of_block = [&](int u) { return u % nb == nb - 1; };
    // a U-ViT out-block's first unit: its skip linear reads h before anything else
    auto out_start = [&](int u) { return uvit && u / nb > half && u % nb == 0; };

    int u = 0;
    while (u < nu && S.err == hipSuccess) {
        const int l = u / nb;
        const sgd_unit_weights& w = m->u[l];
        if (out_start(u)) {
            // U-ViT skip linear (always executed): h <- [h ; skip] W_skip^T + b; a frozen block
            // unit's cached update is added in the same epilogue
            record_drift(u);
            const bool frozen_block = nb == 1 && !act[u];
            GemmArgs g;
            g.A0 = hb(hb_cur); g.lda0 = dd; g.A1 = skipbuf(L - 1 - l); g.lda1 = dd; g.K0 = dd;
            g.B = w.w_skip; g.ldb = 2L * dd; g.M = (int)M; g.N = dd; g.K = 2 * dd;
            hb_cur ^= 1;
            EpiParams e;
            e.kind = EP_SKIP; e.bias = (const float*)w.b_skip; e.h = h; e.d = dd;
            if (frozen_block) { e.delta = (float*)plan.dread[u]; e.delta_mode = 1; e.hcopy = out_copy(l); }
            S.run(SGD_K_GEMM_SKIP, [&] { return launch_gemm(dt, g, e, S.st); });
            if (frozen_block) { ++u; continue; }
        } else if (act[u]) {
            record_drift(u);
        }
        if (!act[u]) {
            // maximal run of frozen units that crosses no skip linear (single units while drift
            // is recorded: each unit's input is measured before its update)
            FrozenRun fr{};
            fr.h = h; fr.n = (long)Md; fr.r = 0; fr.snap_bf16 = dt;
            const int cap = dr ? 1 : kMaxRun;
            if (dr && !out_start(u)) record_drift(u);
            bool snaps = false;
            do {
                fr.delta[fr.r] = plan.dread[u];
                fr.snap[fr.r] = last_of_block(u) ? out_copy(u / nb) : nullptr;
                snaps = snaps || fr.snap[fr.r];
                fr.r++;
                ++u;
            } while (u < nu && !act[u] && !out_start(u) && fr.r < cap);
            // handed to the next unit's first norm when that unit computes and starts with one
            // (not a U-ViT out-block, whose skip linear reads h first; not a UNet ResNet
            // branch, which starts with GroupNorm), and no unit of the run copies h out
            const bool next_norm = u < nu && act[u] && !out_start(u) &&
                                   !(unet && (nb == 1 || branch_of(u) == BR_RESNET));
            if (!dr && !snaps && next_norm) {
                fold.assign(fr.delta, fr.delta + fr.r);
                continue;
            }
            S.run(SGD_K_FROZEN, [&] { return launch_frozen_run(fr, S.st); });
            continue;
        }
        // ---- active unit: its branch, or every branch of its block, in order
        float* dl = plan.dwrite ? plan.dwrite[u] : nullptr;
        // cached-update mode of a branch's residual epilogue: a block unit stores its first
        // branch's update and adds the later ones; a branch unit stores its own
        bool first = true;
        auto dmode = [&]() { const int r = dl ? (first || nb > 1 ? 1 : 2) : 0; first = false; return r; };
        const float* mod_l = dit ? mod_of(l) : nullptr;
        const int br = branch_of(u);
        if (unet && (br < 0 || br == BR_RESNET)) {
            // ResNet block: GroupNorm + SiLU, 3x3 convolution (+ bias + the block's time
            // projection, computed with the step's modulations) into the hidden buffer,
            // GroupNorm + SiLU, 3x3 convolution added to the stream
            GroupNormArgs gn{h, xb, d.B, N, dd, d.groups, 1e-5f, (const float*)w.gn1_w, (const float*)w.gn1_b};
            S.run(SGD_K_GNORM, [&] { return launch_group_norm_silu(0, gn, S.ws + m->w_gn, S.st); });
            GemmArgs g;
            g.A0 = xb; g.lda0 = dd; g.B = w.w_conv1; g.ldb = 9L * dd; g.M = (int)M; g.N = dd; g.K = 9 * dd;
            g.conv_side = d.grid; g.conv_c = dd;
            EpiParams e;
            e.kind = EP_ACT; e.bias = (const float*)w.b_conv1; e.out = hid; e.ldo = dd; e.act = ACT_NONE;
            e.rowbias = mod_of(l); e.rowbias_ld = dd; e.ntok = N;
            S.run(SGD_K_GEMM_CONV, [&] { return launch_gemm(dt, g, e, S.st); });
            GroupNormArgs gn2{hid, xb, d.B, N, dd, d.groups, 1e-5f, (const float*)w.gn2_w, (const float*)w.gn2_b};
            S.run(SGD_K_GNORM, [&] { return launch_group_norm_silu(1, gn2, S.ws + m->w_gn, S.st); });
            GemmArgs g2 = g;
            g2.B = w.w_conv2;
            EpiParams e2;
            e2.kind = EP_RESID; e2.bias = (const float*)w.b_conv2; e2.h = h; e2.d = dd; e2.delta = dl;
            e2.delta_mode = dmode(); e2.ntok = N;
            S.run(SGD_K_GEMM_CONV, [&] { return launch_gemm(dt, g2, e2, S.st); });
        }
        if (br < 0 || br == BR_ATTN) {
            norm((const float*)w.norm1_w, (const float*)w.norm1_b, mod_l, mod_l ? mod_l + dd : nullptr);
            GemmArgs g;
            g.A0 = xb; g.lda0 = dd; g.B = w.w_qkv; g.ldb = dd; g.M = (int)M; g.N = 3 * dd; g.K = dd;
            EpiParams e;
            e.kind = EP_HEADS; e.bias = (const float*)w.b_qkv; e.q = qb; e.k = kb; e.vt = vtb;
            e.ntok = N; e.np = m->np; e.H = H; e.dh = dh; e.d = dd;
            e.rope = d.arch == SGD_ARCH_LLADA; e.rope_log2_theta = (float)std::log2(10000.0);
            S.run(SGD_K_GEMM_QKV, [&] { return launch_gemm(dt, g, e, S.st); });
            attention(qb, kb, vtb, N, m->np, SGD_K_ATTN);
            resid(SGD_K_GEMM_O, ob, dd, dd, w.w_o, w.b_o, mod_l ? mod_l + 2 * dd : nullptr, dl, dmode(), nullptr);
        }
        if (sdxl && (br < 0 || br == BR_XATTN)) {
            char* ckv = plan.ckv ? plan.ckv + (size_t)l * m->ckv_unit : S.ws + m->w_ckv;
            if (!plan.ckv) ctx_kv(l, ckv);
            norm((const float*)w.normx_w, (const float*)w.normx_b, nullptr, nullptr);
            GemmArgs g;
            g.A0 = xb; g.lda0 = dd; g.B = w.w_xq; g.ldb = dd; g.M = (int)M; g.N = dd; g.K = dd;
            EpiParams e;
            e.kind = EP_HEADS; e.q = qb; e.ntok = N; e.np = m->np; e.H = H; e.dh = dh; e.d = dd;
            S.run(SGD_K_GEMM_X, [&] { return launch_gemm(dt, g, e, S.st); });
            attention(qb, ckv, ckv + cheads * m->es, d.ctx_len, m->npc, SGD_K_ATTN_X);
            resid(SGD_K_GEMM_X, ob, dd, dd, w.w_xo, w.b_xo, nullptr, dl, dmode(), nullptr);
        }
        if (br < 0 || br == BR_MLP) {
            norm((const float*)w.norm2_w, (const float*)w.norm2_b, mod_l ? mod_l + 3 * dd : nullptr,
                 mod_l ? mod_l + 4 * dd : nullptr);
            GemmArgs g;
            g.A0 = xb; g.lda0 = dd; g.B = w.w1; g.ldb = dd; g.M = (int)M; g.N = gated ? 2 * F : F; g.K = dd;
            EpiParams e;
            e.kind = gated ? EP_GATED : EP_ACT; e.bias = (const float*)w.b1; e.out = hid; e.ldo = F; e.act = mlp_act;
            e.F = F;
            S.run(SGD_K_GEMM_W1, [&] { return launch_gemm(dt, g, e, S.st); });
            // the MLP is a block's last branch: the block's output copy goes with it
            const float* gate2 = mod_l ? mod_l + 5 * dd : nullptr;
            const int dm2 = dmode();
            void* copy2 = out_copy(l);
            // K ranges of the split product go into fp32 partials that the next unit's pre-norm
            // adds to h in range order: only when that unit computes and reads h first through
            // its pre-norm, and this step has no gate, cached-update store, copy or drift record
            const bool next_norm = u + 1 < nu && act[u + 1] && !out_start(u + 1) &&
                                   !(unet && (nb == 1 || branch_of(u + 1) == BR_RESNET));
            if (m->w2_ksplit > 1 && !gate2 && !dm2 && !copy2 && !dr && next_norm) {
                GemmArgs g2;
                g2.A0 = hid; g2.lda0 = F; g2.B = w.w2; g2.ldb = F; g2.M = (int)M; g2.N = dd; g2.K = F;
                g2.ksplit = m->w2_ksplit;
                EpiParams e2;
                e2.kind = EP_PARTIAL; e2.bias = (const float*)w.b2; e2.h = (float*)(S.ws + m->w_q); e2.d = dd;
                e2.part_stride = (long)(m->part_bytes / 4);
                S.run(SGD_K_GEMM_W2, [&] { return launch_gemm(dt, g2, e2, S.st); });
                for (int s2 = 0; s2 < m->w2_ksplit; ++s2) fold.push_back((const float*)(S.ws + m->w_q + s2 * m->part_bytes));
                fold_parts = true;
            } else {
                resid(SGD_K_GEMM_W2, hid, F, F, w.w2, w.b2, gate2, dl, dm2, copy2);
            }
        }
        ++u;
    }
    if (dr && dr->have_prev) S.run(SGD_K_DRIFT, [&] { return launch_sumsq_finish(dr->partial, nu, dr->sums, S.st); });
    if (plan.sampler)
        S.run(SGD_K_STATE, [&] {
            return launch_state_update((float*)state, h, d.B, N, dd, d.update_row_begin, d.update_row_end, args->alpha,
                                       args->beta, S.st);
        });
    if (S.err != hipSuccess) return hip_fail(S.err, "enqueue");
    return SGD_OK;
}

int check_step_args(const sgd_model* m, void* state, int32_t step, const sgd_step_args* args) {
    if (!m || !state || !args) return fail(SGD_E_ARG, "NULL argument");
    if (!args->workspace || args->workspace_bytes < m->w_total) return fail(SGD_E_ARG, "workspace missing or too small");
    if ((uintptr_t)args->workspace % 256) return fail(SGD_E_ARG, "workspace must be 256-byte aligned");
    if ((uintptr_t)state % 16) return fail(SGD_E_ARG, "state must be 16-byte aligned");
    if (step < 1 || step > m->d.T) return fail(SGD_E_STEP, "step outside 1..T");
    return check_step_shapes(m);
}

int check_cache(const sgd_model* m, const sgd_cache* cache, int32_t step) {
    if (!cache) return fail(SGD_E_ARG, "a scheduled step needs a cache");
    if (cache->m != m) return fail(SGD_E_ARG, "cache bound to another model");
    if (step != cache->last_step + 1) return fail(SGD_E_STEP, "steps must arrive in order 1, 2, ..., T");
    return SGD_OK;
}

float* cache_delta(const sgd_model* m, const sgd_cache* c, int l) {
    return (float*)(c->base + m->c_delta + (size_t)l * align256((size_t)m->M * m->d.d * 4));
}

// The masked step shared by sgd_denoise_step_masked and the drift policy: active units
// refresh their cached update (except at the last step, which no later step reads).
int masked_step(sgd_model* m, void* state, int32_t step, const uint8_t* row, sgd_cache* cache,
                const sgd_step_args* args, const DriftRec* drift, hipStream_t st) {
    const int L = m->nu;  // scheduled units
    std::vector<const float*> dread(L, nullptr);
    std::vector<float*> dwrite(L, nullptr);
    std::vector<uint8_t> act(L);
    for (int l = 0; l < L; ++l) {
        act[l] = row[l] ? 1 : 0;
        if (!act[l] && !cache->written[l])
            return fail(SGD_E_CACHE, "unit " + std::to_string(l) + " is frozen but its cache slot was never written");
        dread[l] = cache_delta(m, cache, l);
        if (act[l] && step < m->d.T) dwrite[l] = cache_delta(m, cache, l);
    }
    StepPlan plan;
    plan.act = act.data();
    plan.dread = dread.data();
    plan.dwrite = dwrite.data();
    plan.ckv = arch_cross(m->d.arch) ? cache->base + m->c_ctx : nullptr;
    plan.ckv_fill = arch_cross(m->d.arch) && !cache->ctx_valid;
    plan.drift = drift;
    int rc = run_step(m, state, step, plan, args, st);
    if (rc) return rc;
    cache->last_step = step;
    for (int l = 0; l < L; ++l)
        if (dwrite[l]) cache->written[l] = 1;
    if (arch_cross(m->d.arch)) cache->ctx_valid = true;
    return SGD_OK;
}

}  // namespace sgd

extern "C" int sgd_denoise_step(sgd_model* m, void* state, int32_t step, const sgd_schedule* sched,
                                sgd_cache* cache, const sgd_step_args* args, void* hip_stream) {
    int rc = check_step_args(m, state, step, args);
    if (rc) return rc;
    const sgd_model_desc& d = m->d;
    const int L = m->nu;  // scheduled units
    std::vector<uint8_t> act(L, 1);
    std::vector<int> life(L, d.T);
    std::vector<const float*> dread(L, nullptr);
    std::vector<float*> dwrite(L, nullptr);
    if (sched) {
        if ((rc = check_cache(m, cache, step))) return rc;
        if (sched->L != L || sched->T != d.T || !sched->lifetimes || !sched->active)
            return fail(SGD_E_ARG, "schedule does not match the model");
        for (int l = 0; l < L; ++l) {
            life[l] = sched->lifetimes[l];
            act[l] = sched->active[(size_t)(step - 1) * L + l];
            if (life[l] < 1 || life[l] > d.T) return fail(SGD_E_ARG, "lifetime outside 1..T");
            if ((act[l] != 0) != (step <= life[l])) return fail(SGD_E_ARG, "active mask disagrees with lifetimes");
            if (!act[l] && !cache->written[l])
                return fail(SGD_E_CACHE, "unit " + std::to_string(l) + " is frozen but its cache slot was never written");
            dread[l] = cache_delta(m, cache, l);
            // the update every later frozen step reads is the one of the last active step
            if (step == life[l] && life[l] < d.T) dwrite[l] = cache_delta(m, cache, l);
        }
    }
    StepPlan plan;
    plan.act = act.data();
    plan.dread = dread.data();
    plan.dwrite = dwrite.data();
    plan.ckv = arch_cross(d.arch) && sched ? cache->base + m->c_ctx : nullptr;
    plan.ckv_fill = arch_cross(d.arch) && sched && !cache->ctx_valid;
    rc = run_step(m, state, step, plan, args, (hipStream_t)hip_stream);
    if (rc) return rc;
    if (sched) {
        cache->last_step = step;
        for (int u = 0; u < L; ++u)
            if (step == life[u]) cache->written[u] = 1;
        if (arch_cross(d.arch)) cache->ctx_valid = true;
    }
    return SGD_OK;
}

// ---------------------------------------------------------------------------- graphs

struct sgd_graph {
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
};

extern "C" int sgd_graph_capture(sgd_model* m, void* state, const sgd_schedule* sched, sgd_cache* cache,
                                 const float* alpha, const float* beta, void* workspace, size_t workspace_bytes,
                                 void* hip_stream, sgd_graph** out) {
    if (!m || !state || !alpha || !beta || !out) return fail(SGD_E_ARG, "NULL argument");
    if (!hip_stream) return fail(SGD_E_ARG, "capture needs a non-null stream");
    if (m->prof_class >= 0) return fail(SGD_E_ARG, "kernel-class profiling is on");
    if (sched && !cache) return fail(SGD_E_ARG, "a scheduled trajectory needs a cache");
    if (cache && cache->m != m) return fail(SGD_E_ARG, "cache bound to another model");
    sgd_step_args a{alpha[0], beta[0], workspace, workspace_bytes};
    int rc = check_step_args(m, state, 1, &a);  // before capture: nothing to unwind
    if (rc) return rc;
    hipStream_t st = (hipStream_t)hip_stream;
    if (cache) sgd_cache_reset(cache);
    hipError_t e = hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) return hip_fail(e, "hipStreamBeginCapture");
    for (int s = 1; s <= m->d.T && rc == SGD_OK; ++s) {
        a.alpha = alpha[s - 1];
        a.beta = beta[s - 1];
        rc = sgd_denoise_step(m, state, s, sched, sched ? cache : nullptr, &a, hip_stream);
    }
    hipGraph_t g = nullptr;
    e = hipStreamEndCapture(st, &g);
    if (cache) sgd_cache_reset(cache);
    if (rc != SGD_OK || e != hipSuccess) {
        if (g) (void)hipGraphDestroy(g);
        return rc != SGD_OK ? rc : hip_fail(e, "hipStreamEndCapture");
    }
    hipGraphExec_t ex = nullptr;
    e = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    if (e != hipSuccess) {
        (void)hipGraphDestroy(g);
        return hip_fail(e, "hipGraphInstantiate");
    }
    *out = new sgd_graph{g, ex};
    return SGD_OK;
}

extern "C" int sgd_graph_launch(sgd_graph* g, void* hip_stream) {
    if (!g) return fail(SGD_E_ARG, "NULL graph");
    hipError_t e = hipGraphLaunch(g->exec, (hipStream_t)hip_stream);
    return e == hipSuccess ? SGD_OK : hip_fail(e, "hipGraphLaunch");
}

extern "C" int sgd_graph_destroy(sgd_graph* g) {
    if (!g) return fail(SGD_E_ARG, "NULL graph");
    if (g->exec) (void)hipGraphExecDestroy(g->exec);
    if (g->graph) (void)hipGraphDestroy(g->graph);
    delete g;
    return SGD_OK;
}

extern "C" int sgd_denoise_step_masked(sgd_model* m, void* state, int32_t step, const uint8_t* active,
                                       sgd_cache* cache, const sgd_step_args* args, void* hip_stream) {
    int rc = check_step_args(m, state, step, args);
    if (rc) return rc;
    if (!active) return fail(SGD_E_ARG, "NULL active row");
    if ((rc = check_cache(m, cache, step))) return rc;
    return masked_step(m, state, step, active, cache, args, nullptr, (hipStream_t)hip_stream);
}

// ---------------------------------------------------------------------------- no allocation

// The allocation-free step: its workspace is this file-scope device array instead of a
// caller buffer.  Each GPU the library runs on holds its own copy until the process ends;
// host code never uses the array's name as an address (it is a host-side stand-in), only
// the per-device address hipGetSymbolAddress returns.
static __device__ __align__(256) char scratch[SGD_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// The current device's address of `scratch`, looked up once per device (that device current).
int scratch_address(void** out) {
    int dev = 0;
    SGD_HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(SGD_E_ARG, "device index beyond the scratch table");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) return fail(SGD_E_HIP, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return SGD_OK;
}
}  // namespace

extern "C" int sgd_denoise_step_noalloc(sgd_model* m, void* state, int32_t step, const sgd_schedule* sched,
                                        sgd_cache* cache, float alpha, float beta, void* hip_stream) {
    if (!m) return fail(SGD_E_ARG, "NULL model");
    if (m->w_total > (size_t)SGD_SCRATCH_BYTES)
        return fail(SGD_E_ARG, "the model's step workspace (" + std::to_string(m->w_total) +
                                   " bytes) exceeds the fixed scratch of " + std::to_string((size_t)SGD_SCRATCH_BYTES) +
                                   " bytes; use sgd_denoise_step with a workspace");
    void* ws = nullptr;
    int rc = scratch_address(&ws);
    if (rc) return rc;
    sgd_step_args a;
    a.alpha = alpha;
    a.beta = beta;
    a.workspace = ws;
    a.workspace_bytes = (size_t)SGD_SCRATCH_BYTES;
    return sgd_denoise_step(m, state, step, sched, cache, &a, hip_stream);
}

// ---------------------------------------------------------------------------- single ops

#include "../../include/sgd_ops.h"

extern "C" int sgd_op_linear(int32_t dtype, const void* A, int64_t lda, const void* W, int64_t ldw,
                             const float* bias, void* out, int64_t ldo, int32_t M, int32_t N, int32_t K,
                             int32_t act, int32_t gated, int32_t tile, void* hip_stream) {
    if (!A || !W || !out) return fail(SGD_E_ARG, "NULL argument");
    if (dtype != SGD_F32 && dtype != SGD_BF16) return fail(SGD_E_DTYPE, "dtype must be F32 or BF16");
    if (act < 0 || act > 3 || tile < 0 || tile > kGemmTiles) return fail(SGD_E_ARG, "bad act or tile");
    if (gated && dtype != SGD_BF16) return fail(SGD_E_DTYPE, "gated GEMMs are bf16 only");
    GemmArgs g;
    g.A0 = A; g.lda0 = lda; g.B = W; g.ldb = ldw; g.M = M; g.N = gated ? 2 * N : N; g.K = K;
    EpiParams e;
    e.kind = gated ? EP_GATED : EP_ACT; e.bias = bias; e.out = out; e.ldo = ldo; e.act = act; e.F = N;
    const int dt = dtype == SGD_BF16 ? 1 : 0;
    if (!gemm_shape_ok(dt, g, e, tile)) return fail(SGD_E_SHAPE, "GEMM shape not supported");
    SGD_HIP_TRY(launch_gemm(dt, g, e, (hipStream_t)hip_stream, tile));
    return SGD_OK;
}

extern "C" int sgd_op_linear_split(int32_t dtype, const void* A, const void* W, const float* bias, float* parts,
                                   int64_t part_stride, int32_t M, int32_t N, int32_t K, int32_t ksplit,
                                   void* hip_stream) {
    if (!A || !W || !parts) return fail(SGD_E_ARG, "NULL argument");
    if (dtype != SGD_BF16) return fail(SGD_E_DTYPE, "split products are bf16 only");
    if (ksplit < 2 || ksplit > 8) return fail(SGD_E_ARG, "2 <= ksplit <= 8");
    GemmArgs g;
    g.A0 = A; g.lda0 = K; g.B = W; g.ldb = K; g.M = M; g.N = N; g.K = K; g.ksplit = ksplit;
    EpiParams e;
    e.kind = EP_PARTIAL; e.bias = bias; e.h = parts; e.d = N; e.part_stride = part_stride;
    if (!gemm_shape_ok(1, g, e)) return fail(SGD_E_SHAPE, "GEMM shape not supported");
    SGD_HIP_TRY(launch_gemm(1, g, e, (hipStream_t)hip_stream));
    return SGD_OK;
}

extern "C" int sgd_op_heads(int32_t dtype, const void* A, const void* W, const float* bias, void* q, void* k,
                            void* vt, int32_t M, int32_t K, int32_t n_proj, int32_t which0, int32_t ntok, int32_t np,
                            int32_t H, int32_t dh, int32_t rope, int32_t tile, void* hip_stream) {
    if (tile < 0 || tile > kGemmTiles) return fail(SGD_E_ARG, "bad tile");
    if (!A || !W || (which0 == 0 && !q) || (which0 + n_proj > 1 && !k) || (which0 + n_proj > 2 && !vt))
        return fail(SGD_E_ARG, "NULL argument");
    if (dtype != SGD_F32 && dtype != SGD_BF16) return fail(SGD_E_DTYPE, "dtype must be F32 or BF16");
    if (n_proj < 1 || which0 < 0 || which0 + n_proj > 3 || ntok < 1 || np < ntok || M % ntok || H < 1 || dh < 1)
        return fail(SGD_E_SHAPE, "bad heads shape");
    GemmArgs g;
    g.A0 = A; g.lda0 = K; g.B = W; g.ldb = K; g.M = M; g.N = n_proj * H * dh; g.K = K;
    EpiParams e;
    e.kind = EP_HEADS; e.bias = bias; e.q = q; e.k = k; e.vt = vt; e.which0 = which0; e.ntok = ntok; e.np = np;
    e.H = H; e.dh = dh; e.d = H * dh; e.rope = rope; e.rope_log2_theta = (float)std::log2(10000.0);
    const int dt = dtype == SGD_BF16 ? 1 : 0;
    if (!gemm_shape_ok(dt, g, e, tile)) return fail(SGD_E_SHAPE, "GEMM shape not supported");
    SGD_HIP_TRY(launch_gemm(dt, g, e, (hipStream_t)hip_stream, tile));
    return SGD_OK;
}

extern "C" int sgd_op_residual(int32_t dtype, const void* A, int64_t lda, const void* W, const float* bias, float* h,
                               float* delta, int32_t delta_mode, const float* gate, int64_t gate_ld, int32_t ntok,
                               int32_t M, int32_t N, int32_t K, int32_t tile, void* hip_stream) {
    if (tile < 0 || tile > kGemmTiles) return fail(SGD_E_ARG, "bad tile");
    if (!A || !W || !h || (delta_mode && !delta)) return fail(SGD_E_ARG, "NULL argument");
    if (dtype != SGD_F32 && dtype != SGD_BF16) return fail(SGD_E_DTYPE, "dtype must be F32 or BF16");
    if (delta_mode < 0 || delta_mode > 2 || ntok < 1) return fail(SGD_E_ARG, "bad delta_mode or ntok");
    GemmArgs g;
    g.A0 = A; g.lda0 = lda; g.B = W; g.ldb = K; g.M = M; g.N = N; g.K = K;
    EpiParams e;
    e.kind = EP_RESID; e.bias = bias; e.h = h; e.d = N; e.delta = delta; e.delta_mode = delta_mode; e.gate = gate;
    e.gate_ld = gate_ld; e.ntok = ntok;
    const int dt = dtype == SGD_BF16 ? 1 : 0;
    if (!gemm_shape_ok(dt, g, e, tile)) return fail(SGD_E_SHAPE, "GEMM shape not supported");
    SGD_HIP_TRY(launch_gemm(dt, g, e, (hipStream_t)hip_stream, tile));
    return SGD_OK;
}

extern "C" int sgd_op_attention(int32_t dtype, const void* q, const void* k, const void* vt, void* o, int32_t B,
                                int32_t H, int32_t dh, int32_t nq, int32_t npq, int32_t nk, int32_t npk,
                                void* hip_stream) {
    if (!q || !k || !vt || !o) return fail(SGD_E_ARG, "NULL argument");
    if (dtype != SGD_F32 && dtype != SGD_BF16) return fail(SGD_E_DTYPE, "dtype must be F32 or BF16");
    if (B < 1 || H < 1 || nq < 1 || nk < 1 || npq < nq || npk < nk || npk % 64 || dh < 8 || dh > 128 || dh % 8)
        return fail(SGD_E_SHAPE, "attention shape not supported");
    if ((uintptr_t)q % 16 || (uintptr_t)k % 16 || (uintptr_t)vt % 16 || (uintptr_t)o % (dtype == SGD_F32 ? 16 : 8))
        return fail(SGD_E_ARG, "attention operands must be 16-byte aligned (bf16 output: 8)");
    AttnArgs a{q, k, vt, o, B, H, dh, nq, npq, nk, npk};
    SGD_HIP_TRY(launch_attention(dtype == SGD_BF16 ? 1 : 0, a, (hipStream_t)hip_stream));
    return SGD_OK;
}

extern "C" int sgd_op_norm(int32_t dtype, int32_t kind, const float* x, void* y, int32_t M, int32_t d, float eps,
                           const float* w, const float* b, const float* shift, const float* scale, int64_t mod_ld,
                           int32_t ntok, void* hip_stream) {
    if (!x || !y) return fail(SGD_E_ARG, "NULL argument");
    if (dtype != SGD_F32 && dtype != SGD_BF16) return fail(SGD_E_DTYPE, "dtype must be F32 or BF16");
    if (kind < 0 || kind > 2 || M < 1 || d < 4 || d % 4 || d > 8192) return fail(SGD_E_SHAPE, "norm shape not supported");
    if ((kind == 0 && !w) || (kind == 1 && (!w || !b)) || (kind == 2 && (!shift || !scale || ntok < 1)))
        return fail(SGD_E_ARG, "missing norm parameters");
    if ((uintptr_t)x % 16 || (uintptr_t)w % 16 || (uintptr_t)b % 16 || (uintptr_t)shift % 16 || (uintptr_t)scale % 16 ||
        mod_ld % 4 || (uintptr_t)y % (dtype == SGD_BF16 ? 8 : 16))
        return fail(SGD_E_ARG, "norm operands must be 16-byte aligned (bf16 output: 8)");
    NormArgs a{x, y, M, d, kind, eps, w, b, shift, scale, mod_ld, ntok};
    SGD_HIP_TRY(launch_norm(dtype == SGD_BF16 ? 1 : 0, a, (hipStream_t)hip_stream));
    return SGD_OK;
}

extern "C" int sgd_op_norm_fold(int32_t dtype, int32_t kind, float* x, void* y, int32_t M, int32_t d, float eps,
                                const float* w, const float* b, const float* shift, const float* scale, int64_t mod_ld,
                                int32_t ntok, const float* const* deltas, int32_t r, void* hip_stream) {
    if (!x || !y || !deltas) return fail(SGD_E_ARG, "NULL argument");
    if (dtype != SGD_F32 && dtype != SGD_BF16) return fail(SGD_E_DTYPE, "dtype must be F32 or BF16");
    if (kind < 0 || kind > 2 || M < 1 || d < 4 || d % 4 || d > 8192) return fail(SGD_E_SHAPE, "norm shape not supported");
    if (r < 1 || r > kMaxRun) return fail(SGD_E_ARG, "1 <= r <= 32 cached updates");
    if ((kind == 0 && !w) || (kind == 1 && (!w || !b)) || (kind == 2 && (!shift || !scale || ntok < 1)))
        return fail(SGD_E_ARG, "missing norm parameters");
    if ((uintptr_t)x % 16 || (uintptr_t)w % 16 || (uintptr_t)b % 16 || (uintptr_t)shift % 16 || (uintptr_t)scale % 16 ||
        mod_ld % 4 || (uintptr_t)y % (dtype == SGD_BF16 ? 8 : 16))
        return fail(SGD_E_ARG, "norm operands must be 16-byte aligned (bf16 output: 8)");
    NormArgs a{x, y, M, d, kind, eps, w, b, shift, scale, mod_ld, ntok};
    a.nfold = r;
    for (int i = 0; i < r; ++i) {
        if (!deltas[i] || (uintptr_t)deltas[i] % 16) return fail(SGD_E_ARG, "NULL or misaligned delta");
        a.fold[i] = deltas[i];
    }
    SGD_HIP_TRY(launch_norm(dtype == SGD_BF16 ? 1 : 0, a, (hipStream_t)hip_stream));
    return SGD_OK;
}

extern "C" int sgd_op_frozen_run(float* h, const float* const* deltas, int32_t r, int64_t n, void* hip_stream) {
    if (!h || !deltas || r < 1 || r > kMaxRun || n < 4 || n % 4) return fail(SGD_E_ARG, "bad frozen-run arguments");
    FrozenRun f{};
    f.h = h; f.n = n; f.r = r; f.snap_bf16 = 1;
    for (int i = 0; i < r; ++i) {
        if (!deltas[i]) return fail(SGD_E_ARG, "NULL delta");
        f.delta[i] = deltas[i];
        f.snap[i] = nullptr;
    }
    SGD_HIP_TRY(launch_frozen_run(f, (hipStream_t)hip_stream));
    return SGD_OK;
}

extern "C" int sgd_op_adaln_mod(int32_t dtype, const float* x, const void* W, const float* bias, float* mod,
                                int32_t B, int32_t d, int32_t n_out, void* hip_stream) {
    if (!x || !W || !mod) return fail(SGD_E_ARG, "NULL argument");
    if (dtype != SGD_F32 && dtype != SGD_BF16) return fail(SGD_E_DTYPE, "dtype must be F32 or BF16");
    if (B < 1 || n_out < 1 || d < 64 || d % 64) return fail(SGD_E_SHAPE, "modulation shape not supported");
    if ((uintptr_t)x % 16 || (uintptr_t)W % 16) return fail(SGD_E_ARG, "x and W must be 16-byte aligned");
    SGD_HIP_TRY(launch_adaln_mod(dtype == SGD_BF16 ? 1 : 0, x, W, bias, mod, B, d, n_out, (hipStream_t)hip_stream));
    return SGD_OK;
}

extern "C" int sgd_op_group_norm_scratch_bytes(int32_t B, int32_t N, int32_t groups, size_t* bytes) {
    if (!bytes || B < 1 || N < 1 || groups < 1) return fail(SGD_E_ARG, "bad arguments");
    *bytes = group_norm_scratch_bytes(B, N, groups);
    return SGD_OK;
}

extern "C" int sgd_op_group_norm_silu(int32_t in_dtype, const void* x, void* y, int32_t B, int32_t N, int32_t C,
                                      int32_t groups, float eps, const float* w, const float* b, void* scratch,
                                      size_t scratch_bytes, void* hip_stream) {
    if (!x || !y || !w || !b || !scratch) return fail(SGD_E_ARG, "NULL argument");
    if (in_dtype != SGD_F32 && in_dtype != SGD_BF16) return fail(SGD_E_DTYPE, "dtype must be F32 or BF16");
    if (B < 1 || N < 1 || groups < 1 || C % groups || (C / groups) % 4 || C > 4096)
        return fail(SGD_E_SHAPE, "group shape not supported");
    if (scratch_bytes < group_norm_scratch_bytes(B, N, groups)) return fail(SGD_E_ARG, "scratch too small");
    if ((uintptr_t)x % 16 || (uintptr_t)w % 16 || (uintptr_t)b % 16 || (uintptr_t)y % 8 || (uintptr_t)scratch % 16)
        return fail(SGD_E_ARG, "operands must be 16-byte aligned (output: 8)");
    GroupNormArgs a{x, y, B, N, C, groups, eps, w, b};
    SGD_HIP_TRY(launch_group_norm_silu(in_dtype == SGD_BF16 ? 1 : 0, a, scratch, (hipStream_t)hip_stream));
    return SGD_OK;
}

extern "C" int sgd_op_conv3x3(const void* A, const void* W, const float* bias, const float* rowbias, int32_t side,
                              void* out, float* h, int32_t M, int32_t N, int32_t Cin, int32_t tile, void* hip_stream) {
    if (!A || !W || (!out && !h)) return fail(SGD_E_ARG, "NULL argument");
    if (side < 1 || M < 1 || N < 1 || Cin < 1) return fail(SGD_E_SHAPE, "bad convolution shape");
    if (tile < 0 || tile > kGemmTiles) return fail(SGD_E_ARG, "bad tile");
    GemmArgs g;
    g.A0 = A; g.lda0 = Cin; g.B = W; g.ldb = 9L * Cin; g.M = M; g.N = N; g.K = 9 * Cin;
    g.conv_side = side; g.conv_c = Cin;
    EpiParams e;
    e.bias = bias; e.ntok = side * side;
    if (h) {
        e.kind = EP_RESID; e.h = h; e.d = N;
    } else {
        e.kind = EP_ACT; e.out = out; e.ldo = N; e.act = ACT_NONE; e.rowbias = rowbias; e.rowbias_ld = N;
    }
    if (!gemm_shape_ok(1, g, e, tile)) return fail(SGD_E_SHAPE, "convolution shape not supported");
    SGD_HIP_TRY(launch_gemm(1, g, e, (hipStream_t)hip_stream, tile));
    return SGD_OK;
}
