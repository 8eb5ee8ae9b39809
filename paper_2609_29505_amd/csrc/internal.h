// Host-side internals shared by the C ABI translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <string>

#include "../../include/sgd.h"

namespace sgd {

void set_error(const std::string& msg);
int fail(int code, const std::string& msg);
int hip_fail(hipError_t e, const char* what);

#define SGD_HIP_TRY(expr)                                 \
    do {                                                  \
        hipError_t _e = (expr);                           \
        if (_e != hipSuccess) return hip_fail(_e, #expr); \
    } while (0)

// Lifetimes from normalised scores (Eq. schedule; budget mode sweeps tau).  Fills
// lifetimes, active, layer_steps, cut_margin of `out`.
int lifetimes_from_scores(const double* score, int L, const sgd_sched_params* p, sgd_schedule* out);

}  // namespace sgd
