// The input-aware baselines of the appendix "Protocol Details", "Dynamic baselines", on
// the same launcher as the static schedule:
//   - the causal activation-drift policy (sgd_drift_step): at step s, the m_s units whose
//     input changed most between steps s-2 and s-1 (relative to its norm) compute, where
//     m_s is the static schedule's active count; the first step is full;
//   - oracle replay (sgd_replay_search): on the recorded unscheduled trajectory, a greedy,
//     cumulative search for frozen units whose reuse keeps the denoiser output within a
//     tolerance of the unscheduled one, under a ceiling on active layer-steps.
// Both run units in non-nested patterns, so an active unit refreshes its cached update at
// every active step (Alg. 2) and a frozen unit adds the update of its latest active step.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <string>
#include <vector>

#include "internal.h"
#include "kernels.h"
#include "model.h"

using namespace sgd;

namespace {

size_t slot_bytes(const sgd_model* m) { return align256((size_t)m->M * m->d.d * 4); }

// drift buffer: [U] unit-input slots, [U][kSumBlocks][2] partial sums, [U][2] sums (U scheduled units)
struct DriftLayout {
    size_t prev, partial, sums, total;
};
DriftLayout drift_layout(const sgd_model* m) {
    DriftLayout o;
    const int L = m->nu;
    o.prev = 0;
    o.partial = (size_t)L * slot_bytes(m);
    o.sums = o.partial + align256((size_t)L * kSumBlocks * 2 * sizeof(double));
    o.total = o.sums + align256((size_t)L * 2 * sizeof(double));
    return o;
}

// the m largest drifts, ties to the lower index
void top_m(const std::vector<double>& dr, int m, uint8_t* row) {
    const int L = (int)dr.size();
    std::vector<int> idx(L);
    for (int l = 0; l < L; ++l) idx[l] = l;
    std::stable_sort(idx.begin(), idx.end(), [&](int a, int b) { return dr[a] > dr[b]; });
    for (int l = 0; l < L; ++l) row[l] = 0;
    for (int i = 0; i < m && i < L; ++i) row[idx[i]] = 1;
}

}  // namespace

extern "C" int sgd_drift_bytes(const sgd_model* m, size_t* bytes) {
    if (!m || !bytes) return fail(SGD_E_ARG, "NULL argument");
    *bytes = drift_layout(m).total;
    return SGD_OK;
}

extern "C" int sgd_drift_step(sgd_model* m, void* state, int32_t step, const sgd_schedule* sched, sgd_cache* cache,
                              const sgd_step_args* args, void* drift_buf, size_t drift_bytes, uint8_t* active_out,
                              double* drift_out, void* hip_stream) {
    int rc = check_step_args(m, state, step, args);
    if (rc) return rc;
    if ((rc = check_cache(m, cache, step))) return rc;
    const int L = m->nu, T = m->d.T;  // scheduled units
    if (!sched || sched->L != L || sched->T != T || !sched->active)
        return fail(SGD_E_ARG, "schedule does not match the model");
    const DriftLayout lay = drift_layout(m);
    if (!drift_buf || drift_bytes < lay.total) return fail(SGD_E_ARG, "drift buffer missing or smaller than sgd_drift_bytes");
    if ((uintptr_t)drift_buf % 256) return fail(SGD_E_ARG, "drift buffer must be 256-byte aligned");
    hipStream_t st = (hipStream_t)hip_stream;
    char* base = (char*)drift_buf;
    int m_s = 0;
    for (int l = 0; l < L; ++l) m_s += sched->active[(size_t)(step - 1) * L + l] ? 1 : 0;
    // the lagged drift d_{l,s-1}: recorded by step s-1 from its inputs and those of step s-2
    std::vector<double> dr(L, 0.0);
    if (step >= 3) {
        std::vector<double> sums(2 * L);
        SGD_HIP_TRY(hipMemcpyAsync(sums.data(), base + lay.sums, 2 * L * sizeof(double), hipMemcpyDeviceToHost, st));
        SGD_HIP_TRY(hipStreamSynchronize(st));
        for (int l = 0; l < L; ++l) dr[l] = std::sqrt(sums[2 * l]) / (std::sqrt(sums[2 * l + 1]) + 1e-8);
    }
    std::vector<uint8_t> row(L, 1);
    if (step > 1) top_m(dr, m_s, row.data());
    DriftRec rec;
    rec.prev = (float*)(base + lay.prev);
    rec.partial = (double*)(base + lay.partial);
    rec.sums = (double*)(base + lay.sums);
    rec.have_prev = step >= 2;
    // the last step's drift would never be used
    rc = masked_step(m, state, step, row.data(), cache, args, step < T ? &rec : nullptr, st);
    if (rc) return rc;
    if (active_out) std::memcpy(active_out, row.data(), L);
    if (drift_out) std::memcpy(drift_out, dr.data(), L * sizeof(double));
    return SGD_OK;
}

// ---------------------------------------------------------------------------- oracle replay

namespace {

// replay buffer: z, h of the unscheduled evaluation, h of a candidate, 2 U update slots (U
// scheduled units), SDXL context K/V (one per block), [U][kSumBlocks][2] partial sums, [U][2] sums
struct ReplayLayout {
    size_t z, href, hcand, slots, ckv, partial, sums, total;
};
ReplayLayout replay_layout(const sgd_model* m) {
    ReplayLayout o;
    const int L = m->nu;
    const size_t sb = slot_bytes(m);
    o.z = 0;
    o.href = sb;
    o.hcand = 2 * sb;
    o.slots = 3 * sb;
    o.ckv = o.slots + 2 * (size_t)L * sb;
    o.partial = o.ckv + (arch_cross(m->d.arch) ? (size_t)m->d.L * m->ckv_unit : 0);
    o.sums = o.partial + align256((size_t)L * kSumBlocks * 2 * sizeof(double));
    o.total = o.sums + align256((size_t)L * 2 * sizeof(double));
    return o;
}

}  // namespace

extern "C" int sgd_replay_bytes(const sgd_model* m, size_t* bytes) {
    if (!m || !bytes) return fail(SGD_E_ARG, "NULL argument");
    *bytes = replay_layout(m).total;
    return SGD_OK;
}

extern "C" int sgd_replay_search(sgd_model* m, const void* z1, const sgd_replay_params* p, const sgd_step_args* args,
                                 void* replay_buf, size_t replay_bytes, int32_t* lifetimes, int64_t* evaluations,
                                 double* delta_log, void* hip_stream) {
    if (!m || !z1 || !p || !args || !lifetimes) return fail(SGD_E_ARG, "NULL argument");
    const ReplayLayout lay = replay_layout(m);
    if (!replay_buf || replay_bytes < lay.total) return fail(SGD_E_ARG, "replay buffer missing or smaller than sgd_replay_bytes");
    if ((uintptr_t)replay_buf % 256 || (uintptr_t)z1 % 16) return fail(SGD_E_ARG, "replay buffer must be 256-byte aligned");
    if (!(p->tau_agree >= 0) || !std::isfinite(p->tau_agree)) return fail(SGD_E_ARG, "tau_agree must be finite and >= 0");
    char* base = (char*)replay_buf;
    int rc = check_step_args(m, base + lay.z, 1, args);
    if (rc) return rc;
    const sgd_model_desc& d = m->d;
    const int L = m->nu, T = d.T;  // scheduled units
    const int64_t ceiling = p->max_layer_steps > 0 ? p->max_layer_steps : (int64_t)L * T;
    if (ceiling < L) return fail(SGD_E_BUDGET, "the ceiling is below one full first step");
    hipStream_t st = (hipStream_t)hip_stream;
    const size_t sb = slot_bytes(m);
    float* z = (float*)(base + lay.z);
    float* href = (float*)(base + lay.href);
    float* hcand = (float*)(base + lay.hcand);
    double* partial = (double*)(base + lay.partial);
    double* sums_dev = (double*)(base + lay.sums);
    auto slot = [&](int i) { return (float*)(base + lay.slots + (size_t)i * sb); };
    // cur[l]: slot holding unit l's update of its latest active step; nxt[l]: scratch slot
    std::vector<int> cur(L), nxt(L);
    for (int l = 0; l < L; ++l) { cur[l] = l; nxt[l] = L + l; }
    const size_t Md = (size_t)m->M * d.d;
    SGD_HIP_TRY(hipMemcpyAsync(z, z1, Md * 4, hipMemcpyDeviceToDevice, st));
    if (delta_log)
        for (size_t i = 0; i < (size_t)T * L * L; ++i) delta_log[i] = std::numeric_limits<double>::quiet_NaN();
    std::vector<uint8_t> frozen(L, 0), act(L, 1);
    std::vector<const float*> dread(L);
    std::vector<float*> dwrite(L);
    std::vector<double> sums(2 * L);
    int64_t evals = 0, spent = 0;
    for (int l = 0; l < L; ++l) lifetimes[l] = T;
    const int r0 = d.update_row_begin, r1 = d.update_row_end;
    for (int s = 1; s <= T; ++s) {
        // 1. the unscheduled evaluation at z_s: reference output and every unit's update
        StepPlan full;
        std::fill(act.begin(), act.end(), 1);
        for (int l = 0; l < L; ++l) dwrite[l] = slot(nxt[l]);
        full.act = act.data();
        full.dread = dread.data();
        full.dwrite = dwrite.data();
        full.ckv = arch_cross(d.arch) ? base + lay.ckv : nullptr;
        full.ckv_fill = s == 1;
        full.h = href;
        full.sampler = false;
        if ((rc = run_step(m, z, s, full, args, st))) return rc;
        ++evals;
        // 2. greedy growth of the cumulative frozen set (no cache exists at step 1)
        int nfrozen = 0;
        for (int l = 0; l < L; ++l) nfrozen += frozen[l];
        for (int round = 0; s > 1 && nfrozen < L; ++round) {
            std::vector<int> cand;
            for (int l = 0; l < L; ++l)
                if (!frozen[l]) cand.push_back(l);
            for (int j : cand) {
                StepPlan pl;
                for (int l = 0; l < L; ++l) {
                    act[l] = (frozen[l] || l == j) ? 0 : 1;
                    dread[l] = slot(cur[l]);
                }
                pl.act = act.data();
                pl.dread = dread.data();
                pl.dwrite = nullptr;
                pl.ckv = arch_cross(d.arch) ? base + lay.ckv : nullptr;
                pl.h = hcand;
                pl.sampler = false;
                if ((rc = run_step(m, z, s, pl, args, st))) return rc;
                ++evals;
                SGD_HIP_TRY(launch_sumsq(href, hcand, nullptr, d.B, d.N, d.d, r0, r1, 1,
                                         partial + (size_t)j * 2 * kSumBlocks, st));
            }
            SGD_HIP_TRY(launch_sumsq_finish(partial, L, sums_dev, st));
            SGD_HIP_TRY(hipMemcpyAsync(sums.data(), sums_dev, 2 * L * sizeof(double), hipMemcpyDeviceToHost, st));
            SGD_HIP_TRY(hipStreamSynchronize(st));
            int best = -1;
            double best_dev = std::numeric_limits<double>::infinity();
            for (int j : cand) {
                const double dev = std::sqrt(sums[2 * j]) / (std::sqrt(sums[2 * j + 1]) + 1e-8);
                if (delta_log && round < L) delta_log[((size_t)(s - 1) * L + round) * L + j] = dev;
                if (dev < best_dev) { best_dev = dev; best = j; }
            }
            // the tolerance, or the ceiling if the active layer-steps still planned exceed it
            const int64_t planned = spent + (int64_t)(T - s + 1) * (L - nfrozen);
            if (best < 0 || (best_dev > p->tau_agree && planned <= ceiling)) break;
            frozen[best] = 1;
            lifetimes[best] = s - 1;
            ++nfrozen;
        }
        spent += L - nfrozen;
        // 3. units still active keep this step's update; frozen ones keep the one of S_l
        for (int l = 0; l < L; ++l)
            if (!frozen[l]) std::swap(cur[l], nxt[l]);
        // 4. z_{s+1} from the unscheduled output: the search runs on the recorded trajectory
        SGD_HIP_TRY(launch_state_update(z, href, d.B, d.N, d.d, r0, r1, args->alpha, args->beta, st));
    }
    SGD_HIP_TRY(hipStreamSynchronize(st));
    if (evaluations) *evaluations = evals;
    return SGD_OK;
}
