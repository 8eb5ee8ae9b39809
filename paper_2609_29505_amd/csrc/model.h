// Model and cache handles and the shared step launcher (internal to libsgd).
#pragma once

#include <hip/hip_runtime.h>

#include <vector>

#include "../../include/sgd.h"

struct sgd_model {
    sgd_model_desc d;
    std::vector<sgd_unit_weights> u;
    int dt = 1;       // 0 fp32, 1 bf16
    size_t es = 2;    // element bytes of activations
    int np = 64;      // tokens padded to 64
    int npc = 64;     // context tokens padded to 64
    long M = 0;
    int nb = 1;       // scheduled units per block (1, or the block's branches)
    int nu = 0;       // scheduled units: L nb
    // workspace layout
    size_t w_h, w_xb, w_q, w_k, w_vt, w_ob, w_hid, w_siluc, w_mod, w_hb, w_skip, w_ckv, w_gn, w_total;
    size_t mod_slot = 0;  // bytes of one block's modulation in the workspace
    // MLP output GEMM in K ranges (1: unsplit); partial s at workspace offset w_q + s * part_bytes,
    // in the q / k / V^T / attention-output buffers, which no kernel reads between that GEMM and
    // the next unit's QKV GEMM
    int w2_ksplit = 1;
    size_t part_bytes = 0;
    // cache layout
    size_t c_delta, c_ctx, c_total;
    size_t ckv_unit;  // bytes of one unit's context K and V^T
    // profiling
    int prof_class = -1;
    int prof_max = 0;
    int prof_n = 0;
    std::vector<hipEvent_t> prof_ev;
};

struct sgd_cache {
    sgd_model* m;
    char* base;
    size_t bytes;
    int last_step;
    std::vector<int> written;
    bool ctx_valid;
};

namespace sgd {

size_t align256(size_t x);
bool arch_gated(int arch);
bool arch_cross(int arch);  // SDXL-style units with a cross-attention branch
// residual branches of a block, in execution order
enum Branch { BR_RESNET = 0, BR_ATTN = 1, BR_XATTN = 2, BR_MLP = 3 };
int block_branches(int arch);         // branches per block: 2, 3 or 4
int block_branch(int arch, int i);    // the i-th branch of a block (Branch)

// Drift recording of one step (the input-aware baseline): for every unit, the squared norm
// of the change of its input since the previous recorded step and the squared norm of the
// input, as per-block partial sums; the inputs then replace the previous ones.
struct DriftRec {
    float* prev = nullptr;      // [L] slots of align256(M d 4) bytes: the previous step's unit inputs
    double* partial = nullptr;  // [L][kSumBlocks][2]
    double* sums = nullptr;     // [L][2]: sum (h - prev)^2, sum h^2
    bool have_prev = false;     // false at the first recorded step: snapshots only
};

// What one network evaluation does beyond the branch kernels.
struct StepPlan {
    const uint8_t* act = nullptr;         // [L] 1 = the unit computes its branches
    const float* const* dread = nullptr;  // [L] cached update a frozen unit adds
    float* const* dwrite = nullptr;       // [L] where an active unit stores its update (NULL: none)
    char* ckv = nullptr;                  // SDXL context K/V per unit (stride ckv_unit); NULL: per active unit
    bool ckv_fill = false;                // compute every unit's context K/V into ckv first
    float* h = nullptr;                   // residual stream buffer (NULL: the workspace's); holds h_L at the end
    bool sampler = true;                  // z <- alpha z - beta h_L on the update rows
    const DriftRec* drift = nullptr;      // record drift (NULL: no)
};

int check_step_shapes(const sgd_model* m);
int check_step_args(const sgd_model* m, void* state, int32_t step, const sgd_step_args* args);
int check_cache(const sgd_model* m, const sgd_cache* cache, int32_t step);
float* cache_delta(const sgd_model* m, const sgd_cache* c, int l);
int run_step(sgd_model* m, void* state, int step, const StepPlan& plan, const sgd_step_args* args, hipStream_t st);
int masked_step(sgd_model* m, void* state, int32_t step, const uint8_t* row, sgd_cache* cache,
                const sgd_step_args* args, const DriftRec* drift, hipStream_t st);

}  // namespace sgd
