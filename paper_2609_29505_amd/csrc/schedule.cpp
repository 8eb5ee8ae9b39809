// Schedule construction (Alg. 1, Sec. 4.1) behind sgd_schedule_build.
//
// Per scored matrix W (m x n, d = min(m, n)): the fp64 Gram matrix of the short side on
// the GPU, its Householder tridiagonal form on the GPU, and the eigenvalues of that
// tridiagonal matrix on the host (implicit symmetric QR with Wilkinson shift, Golub & Van
// Loan Sec. 8.3).  The eigenvalues are the squared singular values sigma_i^2, from which
//   E_k = sum_{i<=k} sigma_i^2, k = min(d, max(1, floor(d/10)))
//   SCR_eta = log((E_k + eta F) / (tail + eta F)), F = ||W||_F^2 = trace of the Gram
//   g(W) = sqrt(F) sqrt(rho), rho = (E_k + eta F) / (E_k + tail + 2 eta F)
// (Eq. scr-reg; Eq. app-matrix-score with rho(u) = e^u / (1 + e^u) evaluated at u = SCR).
// Unit scores combine g by Eqs. app-attn-score / app-xattn-score / app-mlp-score /
// app-conv-score, sum per unit (Eq. app-block-score) and normalise with eps = 1e-12
// (Eq. app-score-normalization).  Lifetimes follow Eq. schedule.
#include <algorithm>
#include <atomic>
#include <cfloat>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <mutex>
#include <thread>
#include <tuple>
#include <vector>

#include "internal.h"
#include "kernels.h"

namespace sgd {

// ---------------------------------------------------------------------------- eigenvalues

// One implicit symmetric QR step on the unreduced block [lo, hi] of the tridiagonal
// matrix with diagonal a and subdiagonal b (b[i] = T[i+1][i]).  The shift is the
// eigenvalue of the trailing 2 x 2 block closer to its last diagonal entry.  Rotations
// R = [[c, s], [-s, c]] act on rows/columns (k, k+1); the first is chosen from the
// shifted first column, the others chase the bulge T[k+1][k-1] down the band.
static void qr_step(double* a, double* b, int lo, int hi) {
    const double dd = 0.5 * (a[hi - 1] - a[hi]);
    const double bn = b[hi - 1];
    const double den = dd + std::copysign(std::hypot(dd, bn), dd == 0.0 ? 1.0 : dd);
    const double mu = a[hi] - (den != 0.0 ? bn * bn / den : 0.0);
    double x = a[lo] - mu, z = b[lo];
    for (int k = lo; k < hi; ++k) {
        const double r = std::hypot(x, z);
        const double c = r == 0.0 ? 1.0 : x / r;
        const double s = r == 0.0 ? 0.0 : z / r;
        if (k > lo) b[k - 1] = r;
        const double ak = a[k], ak1 = a[k + 1], bk = b[k];
        a[k] = c * c * ak + 2.0 * c * s * bk + s * s * ak1;
        a[k + 1] = s * s * ak - 2.0 * c * s * bk + c * c * ak1;
        b[k] = c * s * (ak1 - ak) + (c * c - s * s) * bk;
        if (k + 1 < hi) {
            z = s * b[k + 1];
            b[k + 1] = c * b[k + 1];
            x = b[k];
        }
    }
}

// Eigenvalues of the symmetric tridiagonal (a, b); a is overwritten with them (unsorted).
static bool tridiag_eigenvalues(std::vector<double>& a, std::vector<double>& b) {
    const int n = (int)a.size();
    if (n <= 1) return true;
    double anorm = 0.0;
    for (int i = 0; i < n; ++i) anorm = std::max(anorm, std::fabs(a[i]) + (i ? std::fabs(b[i - 1]) : 0.0) +
                                                            (i + 1 < n ? std::fabs(b[i]) : 0.0));
    const double eps = DBL_EPSILON;
    const double floor_tol = 1e-3 * eps * anorm;
    auto negligible = [&](int i) { return std::fabs(b[i]) <= eps * (std::fabs(a[i]) + std::fabs(a[i + 1])) + floor_tol; };
    int hi = n - 1, iter = 0;
    while (hi > 0) {
        if (negligible(hi - 1)) {
            b[hi - 1] = 0.0;
            --hi;
            iter = 0;
            continue;
        }
        int lo = hi - 1;
        while (lo > 0 && !negligible(lo - 1)) --lo;
        if (lo > 0) b[lo - 1] = 0.0;
        if (++iter > 200) return false;
        qr_step(a.data(), b.data(), lo, hi);
    }
    return true;
}

struct MatStats {
    double e_top = 0, e_tail = 0, frob = 0, scr = 0, g = 0, sigma1_sq = 0;
};

static int rank_k(long m, long n) {
    const long d = std::min(m, n);
    return (int)std::min<long>(d, std::max<long>(1, d / 10));
}

static MatStats stats_from_eigs(std::vector<double>& lam, double frob, int k, double eta) {
    for (double& v : lam) v = std::max(v, 0.0);
    std::sort(lam.begin(), lam.end(), [](double x, double y) { return x > y; });
    MatStats s;
    for (size_t i = 0; i < lam.size(); ++i) (i < (size_t)k ? s.e_top : s.e_tail) += lam[i];
    s.frob = frob;
    const double A = s.e_top + eta * frob, B = s.e_tail + eta * frob;
    s.scr = B > 0 ? std::log(A / B) : std::numeric_limits<double>::infinity();
    const double rho = (A + B) > 0 ? A / (A + B) : 0.0;
    s.g = std::sqrt(frob) * std::sqrt(rho);
    s.sigma1_sq = lam.empty() ? 0.0 : lam[0];
    return s;
}

// ---------------------------------------------------------------------------- GPU driver

struct MatJob {
    const sgd_matrix* m;
    MatStats out;
};

static int validate_matrix(const sgd_matrix* m) {
    if (!m || !m->ptr) return fail(SGD_E_ARG, "matrix pointer is NULL");
    if (m->rows < 1 || m->cols < 1) return fail(SGD_E_SHAPE, "matrix has an empty dimension");
    if (std::min(m->rows, m->cols) > 16384) return fail(SGD_E_SHAPE, "matrix short side above 16384");
    if (m->dtype != SGD_F32 && m->dtype != SGD_BF16) return fail(SGD_E_DTYPE, "matrix dtype must be F32 or BF16");
    if (m->role < SGD_ROLE_Q || m->role > SGD_ROLE_CONV) return fail(SGD_E_ARG, "unknown matrix role");
    return SGD_OK;
}

// Device doubles one worker needs for matrices whose short side is at most n: the Gram
// matrix, the diagonal, the off-diagonal, the Householder work array and the Gram's
// diagonal (for ||W||_F^2), each rounded up to 256 bytes.
static size_t worker_bytes(long n) {
    auto a = [](size_t b) { return (b + 255) & ~(size_t)255; };
    return a((size_t)n * n * 8) + 3 * a((size_t)n * 8) + a((size_t)(5 * n + 8) * 8);
}

// Score every job with a pool of host workers, each driving its own stream and one slot of
// the caller's workspace.
static int run_stats(std::vector<MatJob>& jobs, double eta, char* ws, size_t ws_bytes, hipStream_t user_stream) {
    if (jobs.empty()) return SGD_OK;
    int dev = 0;
    SGD_HIP_TRY(hipGetDevice(&dev));
    SGD_HIP_TRY(hipStreamSynchronize(user_stream));
    long nmax = 0;
    for (auto& j : jobs) nmax = std::max(nmax, std::min(j.m->rows, j.m->cols));
    const size_t per = worker_bytes(nmax);
    if (!ws || ws_bytes < per) return fail(SGD_E_ARG, "schedule workspace smaller than one worker slot");
    if ((uintptr_t)ws % 256) return fail(SGD_E_ARG, "schedule workspace must be 256-byte aligned");
    unsigned hc = std::thread::hardware_concurrency();
    int nw = (int)std::min<size_t>(jobs.size(), std::max(1u, std::min(hc ? hc : 1u, 16u)));
    nw = (int)std::min<size_t>(nw, ws_bytes / per);

    std::atomic<size_t> next{0};
    std::mutex emu;
    int first_err = SGD_OK;
    std::string err_msg;
    auto record = [&](int code, const std::string& msg) {
        std::lock_guard<std::mutex> lk(emu);
        if (first_err == SGD_OK) { first_err = code; err_msg = msg; }
    };
    auto worker = [&](int slot) {
        if (hipSetDevice(dev) != hipSuccess) { record(SGD_E_HIP, "hipSetDevice failed in a worker"); return; }
        hipStream_t st = nullptr;
        auto a = [](size_t b) { return (b + 255) & ~(size_t)255; };
        char* base = ws + (size_t)slot * per;
        double* G = (double*)base;
        double* dg = (double*)(base + a((size_t)nmax * nmax * 8));
        double* od = (double*)((char*)dg + a((size_t)nmax * 8));
        double* trace = (double*)((char*)od + a((size_t)nmax * 8));
        double* work = (double*)((char*)trace + a((size_t)nmax * 8));
        hipError_t e = hipStreamCreateWithFlags(&st, hipStreamNonBlocking);
        if (e != hipSuccess) {
            record(SGD_E_HIP, std::string("worker stream: ") + hipGetErrorString(e));
            return;
        }
        std::vector<double> ha, hb, htr;
        for (;;) {
            const size_t i = next.fetch_add(1);
            if (i >= jobs.size()) break;
            {
                std::lock_guard<std::mutex> lk(emu);
                if (first_err != SGD_OK) break;
            }
            const sgd_matrix* m = jobs[i].m;
            const int trans = m->cols > m->rows ? 1 : 0;  // Gram of the short side
            const int n = (int)std::min(m->rows, m->cols);
            e = launch_gram(m->dtype, m->ptr, m->rows, m->cols, trans, G, st);
            if (e == hipSuccess) e = launch_diag_copy(G, n, trace, st);
            if (e == hipSuccess) e = launch_tridiagonalize(G, n, dg, od, work, st);
            ha.assign(n, 0.0);
            hb.assign(n > 1 ? n - 1 : 0, 0.0);
            htr.assign(n, 0.0);
            if (e == hipSuccess) e = hipMemcpyAsync(ha.data(), dg, n * sizeof(double), hipMemcpyDeviceToHost, st);
            if (e == hipSuccess && n > 1)
                e = hipMemcpyAsync(hb.data(), od, (n - 1) * sizeof(double), hipMemcpyDeviceToHost, st);
            if (e == hipSuccess) e = hipMemcpyAsync(htr.data(), trace, n * sizeof(double), hipMemcpyDeviceToHost, st);
            if (e == hipSuccess) e = hipStreamSynchronize(st);
            if (e != hipSuccess) {
                record(SGD_E_HIP, std::string("spectral kernels: ") + hipGetErrorString(e));
                break;
            }
            double frob = 0.0;
            for (double v : htr) frob += v;
            bool finite = std::isfinite(frob);
            for (double v : ha) finite = finite && std::isfinite(v);
            for (double v : hb) finite = finite && std::isfinite(v);
            if (!finite) {
                record(SGD_E_NUMERIC, "non-finite weights in a scored matrix");
                break;
            }
            if (!tridiag_eigenvalues(ha, hb)) {
                record(SGD_E_NUMERIC, "tridiagonal eigenvalue iteration did not converge");
                break;
            }
            jobs[i].out = stats_from_eigs(ha, frob, rank_k(m->rows, m->cols), eta);
        }
        (void)hipStreamDestroy(st);
    };
    std::vector<std::thread> th;
    for (int w = 0; w < nw; ++w) th.emplace_back(worker, w);
    for (auto& t : th) t.join();
    if (first_err != SGD_OK) return fail(first_err, err_msg);
    return SGD_OK;
}

// ---------------------------------------------------------------------------- lifetimes

// The parameters with the library's defaults applied: S_min <= 0 -> ceil(T / 10); a
// percentage budget -> N* = floor(pct L T / 100).  Validates the result.
static int resolve_params(const sgd_sched_params* p, int L, sgd_sched_params* r) {
    if (!p) return fail(SGD_E_ARG, "params is NULL");
    if (L < 1) return fail(SGD_E_ARG, "L must be >= 1");
    if (p->T < 1) return fail(SGD_E_ARG, "T must be >= 1");
    *r = *p;
    if (r->s_min <= 0) r->s_min = sgd_s_min_default(p->T);
    if (r->s_min > p->T) return fail(SGD_E_ARG, "s_min must lie in 1..T");
    if (r->budget_layer_steps < 0 && r->budget_pct > 0) {
        if (r->budget_pct > 100) return fail(SGD_E_ARG, "budget_pct must lie in 1..100");
        const int64_t n = (int64_t)r->budget_pct * L * p->T / 100;
        if (n > INT32_MAX) return fail(SGD_E_ARG, "budget above 2^31 layer-steps");
        r->budget_layer_steps = (int32_t)n;
    }
    if (r->budget_layer_steps < 0 && !(r->tau > 0)) return fail(SGD_E_ARG, "tau must be > 0 in tau mode");
    if (!(r->eta >= 0) || !std::isfinite(r->eta)) return fail(SGD_E_ARG, "eta must be finite and >= 0");
    if (r->rule < 0 || r->rule >= SGD_RULE_COUNT) return fail(SGD_E_ARG, "unknown ranking rule");
    if (r->budget_layer_steps >= 0) {
        const long lo = (long)L * r->s_min, hi = (long)L * p->T;
        if (r->budget_layer_steps < lo || r->budget_layer_steps > hi)
            return fail(SGD_E_BUDGET, "budget outside [L*s_min, L*T]");
    }
    return SGD_OK;
}

int lifetimes_from_scores(const double* score, int L, const sgd_sched_params* p, sgd_schedule* out) {
    const int T = p->T;
    std::vector<int> S(L, p->s_min);
    double margin = std::numeric_limits<double>::infinity();
    if (p->budget_layer_steps < 0) {
        for (int l = 0; l < L; ++l) {
            const double v = std::ceil((double)T * std::min(1.0, score[l] / p->tau));
            S[l] = std::max(p->s_min, (int)v);
        }
    } else {
        struct Ev { double key; int l, j; };
        std::vector<Ev> ev;
        ev.reserve((size_t)L * (T - p->s_min));
        for (int l = 0; l < L; ++l)
            for (int j = p->s_min; j < T; ++j)
                ev.push_back({score[l] > 0 ? (double)j / score[l] : std::numeric_limits<double>::infinity(), l, j});
        std::sort(ev.begin(), ev.end(), [](const Ev& x, const Ev& y) {
            return std::tie(x.key, x.l, x.j) < std::tie(y.key, y.l, y.j);
        });
        const long grant = (long)p->budget_layer_steps - (long)L * p->s_min;
        for (long i = 0; i < grant; ++i) S[ev[i].l] += 1;
        if (grant > 0 && grant < (long)ev.size()) {
            const double last = ev[grant - 1].key, nxt = ev[grant].key;
            if (std::isfinite(last) && last > 0 && std::isfinite(nxt)) margin = (nxt - last) / last;
        }
    }
    out->L = L;
    out->T = T;
    long total = 0;
    for (int l = 0; l < L; ++l) total += S[l];
    if (out->lifetimes)
        for (int l = 0; l < L; ++l) out->lifetimes[l] = S[l];
    if (out->active)
        for (int s = 1; s <= T; ++s)
            for (int l = 0; l < L; ++l) out->active[(size_t)(s - 1) * L + l] = (uint8_t)(s <= S[l]);
    out->layer_steps = total;
    out->cut_margin = margin;
    out->s_min = p->s_min;
    return SGD_OK;
}

// SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number generators",
// OOPSLA 2014): output i of the stream seeded with `seed` mixes seed + i * golden gamma.
static uint64_t splitmix64(uint64_t seed, uint64_t i) {
    uint64_t z = seed + i * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Matrix statistic of a ranking rule (g(W) for the method).
static double rule_stat(const MatStats& s, int rule) {
    switch (rule) {
        case SGD_RULE_FROB: return std::sqrt(s.frob);
        case SGD_RULE_SPECTRAL: return std::sqrt(s.sigma1_sq);
        case SGD_RULE_STABLE_RANK: return s.frob > 0 ? s.sigma1_sq / s.frob : 0.0;
        case SGD_RULE_FROB_SRANK: return s.frob > 0 ? std::sqrt(s.frob) * (s.sigma1_sq / s.frob) : 0.0;
        case SGD_RULE_RAW_SCR: {
            const double g = s.g, f = std::sqrt(s.frob);
            return f > 0 ? g / f : 0.0;
        }
        default: return s.g;
    }
}

}  // namespace sgd

using namespace sgd;

// Unit raw scores of the rule from the matrices' statistics (Eqs. app-attn-score,
// app-xattn-score, app-mlp-score, app-conv-score, app-block-score with the rule's statistic
// in place of g), normalised (Eq. app-score-normalization) and mapped to lifetimes.
static int rank_units(const sgd_unit* units, int L, const std::vector<MatStats>& st, const sgd_sched_params& p,
                      sgd_schedule* out) {
    std::vector<double> raw(L, 0.0);
    if (p.rule == SGD_RULE_DEPTH) {
        for (int l = 0; l < L; ++l) raw[l] = (double)(l + 1);
    } else if (p.rule == SGD_RULE_RANDOM) {
        for (int l = 0; l < L; ++l) raw[l] = (double)(splitmix64(p.seed, (uint64_t)l + 1) >> 11) * 0x1.0p-53;
    } else {
        size_t ji = 0;
        for (int l = 0; l < L; ++l) {
            const sgd_unit& u = units[l];
            double g[SGD_ROLE_CONV + 1];
            bool have[SGD_ROLE_CONV + 1] = {};
            double conv = 0.0;
            for (int i = 0; i < u.n_mats; ++i, ++ji) {
                const int r = u.mats[i].role;
                const double v = rule_stat(st[ji], p.rule);
                if (r == SGD_ROLE_CONV) { conv += v; continue; }
                have[r] = true;
                g[r] = v;
            }
            const double sdh = std::sqrt((double)u.head_dim);
            double q = 0.0;
            if (have[SGD_ROLE_Q] && have[SGD_ROLE_K] && have[SGD_ROLE_V] && have[SGD_ROLE_O])
                q += g[SGD_ROLE_O] * g[SGD_ROLE_V] * (1.0 + g[SGD_ROLE_Q] * g[SGD_ROLE_K] / sdh);
            if (have[SGD_ROLE_XQ] && have[SGD_ROLE_XK] && have[SGD_ROLE_XV] && have[SGD_ROLE_XO])
                q += g[SGD_ROLE_XO] * g[SGD_ROLE_XV] * (1.0 + g[SGD_ROLE_XQ] * g[SGD_ROLE_XK] / sdh);
            if (have[SGD_ROLE_W1] && have[SGD_ROLE_W2]) q += g[SGD_ROLE_W2] * g[SGD_ROLE_W1];
            q += conv;
            raw[l] = q;
        }
    }
    double mx = 0.0;
    for (double v : raw) {
        if (!std::isfinite(v)) return fail(SGD_E_NUMERIC, "non-finite unit score");
        mx = std::max(mx, v);
    }
    std::vector<double> score(L);
    for (int l = 0; l < L; ++l) score[l] = raw[l] / (mx + 1e-12);
    int rc = lifetimes_from_scores(score.data(), L, &p, out);
    if (rc) return rc;
    if (out->unit_raw) std::memcpy(out->unit_raw, raw.data(), L * sizeof(double));
    if (out->unit_score) std::memcpy(out->unit_score, score.data(), L * sizeof(double));
    if (out->mat_stats)
        for (size_t i = 0; i < st.size(); ++i) {
            const MatStats& m = st[i];
            double* o = out->mat_stats + 6 * i;
            o[0] = m.e_top; o[1] = m.e_tail; o[2] = m.frob; o[3] = m.scr; o[4] = m.g; o[5] = m.sigma1_sq;
        }
    return SGD_OK;
}

extern "C" int32_t sgd_s_min_default(int32_t T) { return T >= 1 ? (T + 9) / 10 : 0; }

extern "C" int sgd_budget_layer_steps(int32_t pct, int32_t L, int32_t T, int64_t* n_star) {
    if (!n_star) return fail(SGD_E_ARG, "NULL argument");
    if (pct < 0 || pct > 100 || L < 1 || T < 1) return fail(SGD_E_ARG, "need 0 <= pct <= 100, L >= 1, T >= 1");
    *n_star = (int64_t)pct * L * T / 100;
    return SGD_OK;
}

extern "C" int sgd_schedule_from_scores(const double* unit_score, int32_t L, const sgd_sched_params* params,
                                        sgd_schedule* out) {
    if (!unit_score || !out || !out->lifetimes || !out->active) return fail(SGD_E_ARG, "NULL argument");
    sgd_sched_params p;
    int rc = resolve_params(params, L, &p);
    if (rc) return rc;
    for (int l = 0; l < L; ++l)
        if (!std::isfinite(unit_score[l]) || unit_score[l] < 0) return fail(SGD_E_NUMERIC, "scores must be finite and >= 0");
    rc = lifetimes_from_scores(unit_score, L, &p, out);
    if (rc) return rc;
    if (out->unit_score)
        for (int l = 0; l < L; ++l) out->unit_score[l] = unit_score[l];
    return SGD_OK;
}

extern "C" int sgd_schedule_from_lifetimes(int32_t L, int32_t T, const int32_t* lifetimes, sgd_schedule* out) {
    if (!lifetimes || !out || !out->lifetimes || !out->active) return fail(SGD_E_ARG, "NULL argument");
    if (L < 1 || T < 1) return fail(SGD_E_ARG, "L and T must be >= 1");
    long total = 0;
    int smin = T;
    for (int l = 0; l < L; ++l) {
        if (lifetimes[l] < 1 || lifetimes[l] > T) return fail(SGD_E_ARG, "lifetimes must lie in 1..T");
        total += lifetimes[l];
        smin = std::min(smin, (int)lifetimes[l]);
    }
    out->L = L;
    out->T = T;
    for (int l = 0; l < L; ++l) out->lifetimes[l] = lifetimes[l];
    for (int s = 1; s <= T; ++s)
        for (int l = 0; l < L; ++l) out->active[(size_t)(s - 1) * L + l] = (uint8_t)(s <= lifetimes[l]);
    out->layer_steps = total;
    out->cut_margin = std::numeric_limits<double>::infinity();
    out->s_min = smin;
    return SGD_OK;
}

extern "C" int sgd_schedule_workspace_bytes(const sgd_unit* units, int32_t L, int32_t workers, size_t* bytes) {
    if (!bytes || (!units && L > 0)) return fail(SGD_E_ARG, "NULL argument");
    if (workers < 1 || workers > 16) return fail(SGD_E_ARG, "workers must lie in 1..16");
    long nmax = 0;
    for (int l = 0; l < L; ++l) {
        if (units[l].n_mats > 0 && !units[l].mats) return fail(SGD_E_ARG, "unit without matrices");
        for (int i = 0; i < units[l].n_mats; ++i)
            nmax = std::max<long>(nmax, std::min(units[l].mats[i].rows, units[l].mats[i].cols));
    }
    *bytes = nmax > 0 ? (size_t)workers * worker_bytes(nmax) : 0;
    return SGD_OK;
}

extern "C" int sgd_matrix_stats(const sgd_matrix* m, double eta, void* workspace, size_t workspace_bytes,
                                void* hip_stream, double out[6]) {
    if (!out) return fail(SGD_E_ARG, "out is NULL");
    int rc = validate_matrix(m);
    if (rc) return rc;
    if (!(eta >= 0) || !std::isfinite(eta)) return fail(SGD_E_ARG, "eta must be finite and >= 0");
    std::vector<MatJob> jobs{{m, {}}};
    rc = run_stats(jobs, eta, (char*)workspace, workspace_bytes, (hipStream_t)hip_stream);
    if (rc) return rc;
    const MatStats& s = jobs[0].out;
    out[0] = s.e_top; out[1] = s.e_tail; out[2] = s.frob; out[3] = s.scr; out[4] = s.g; out[5] = s.sigma1_sq;
    return SGD_OK;
}

extern "C" int sgd_schedule_build(const sgd_unit* units, int32_t L, const sgd_sched_params* params, void* workspace,
                                  size_t workspace_bytes, void* hip_stream, sgd_schedule* out) {
    if (!out || !out->lifetimes || !out->active) return fail(SGD_E_ARG, "NULL argument");
    sgd_sched_params p;
    int rc = resolve_params(params, L, &p);
    if (rc) return rc;
    const bool unit_rule = p.rule == SGD_RULE_DEPTH || p.rule == SGD_RULE_RANDOM;
    if (!units && !unit_rule) return fail(SGD_E_ARG, "units is NULL");
    std::vector<MatJob> jobs;
    if (units) {
        for (int l = 0; l < L; ++l) {
            const sgd_unit& u = units[l];
            if (u.n_mats < 1 || !u.mats) return fail(SGD_E_ARG, "unit without matrices");
            if (u.head_dim < 1) return fail(SGD_E_ARG, "head_dim must be >= 1");
            bool seen[SGD_ROLE_CONV + 1] = {};
            for (int i = 0; i < u.n_mats; ++i) {
                rc = validate_matrix(&u.mats[i]);
                if (rc) return rc;
                const int r = u.mats[i].role;
                if (r != SGD_ROLE_CONV && seen[r]) return fail(SGD_E_ARG, "a unit lists the same role twice");
                seen[r] = true;
                jobs.push_back({&u.mats[i], {}});
            }
        }
    }
    // unit rules only rank units; spectra are computed when matrices are given (mat_stats)
    if (!unit_rule || (units && out->mat_stats)) {
        rc = run_stats(jobs, p.eta, (char*)workspace, workspace_bytes, (hipStream_t)hip_stream);
        if (rc) return rc;
    }
    std::vector<MatStats> st(jobs.size());
    for (size_t i = 0; i < jobs.size(); ++i) st[i] = jobs[i].out;
    return rank_units(units, L, st, p, out);
}

extern "C" int sgd_schedule_from_stats(const sgd_unit* units, int32_t L, const double* mat_stats,
                                       const sgd_sched_params* params, sgd_schedule* out) {
    if (!units || !mat_stats || !out || !out->lifetimes || !out->active) return fail(SGD_E_ARG, "NULL argument");
    sgd_sched_params p;
    int rc = resolve_params(params, L, &p);
    if (rc) return rc;
    std::vector<MatStats> st;
    for (int l = 0; l < L; ++l) {
        const sgd_unit& u = units[l];
        if (u.n_mats < 1 || !u.mats) return fail(SGD_E_ARG, "unit without matrices");
        if (u.head_dim < 1) return fail(SGD_E_ARG, "head_dim must be >= 1");
        bool seen[SGD_ROLE_CONV + 1] = {};
        for (int i = 0; i < u.n_mats; ++i) {
            const int r = u.mats[i].role;
            if (r < SGD_ROLE_Q || r > SGD_ROLE_CONV) return fail(SGD_E_ARG, "unknown matrix role");
            if (r != SGD_ROLE_CONV && seen[r]) return fail(SGD_E_ARG, "a unit lists the same role twice");
            seen[r] = true;
            const double* o = mat_stats + 6 * st.size();
            MatStats m;
            m.e_top = o[0]; m.e_tail = o[1]; m.frob = o[2]; m.scr = o[3]; m.g = o[4]; m.sigma1_sq = o[5];
            for (int c = 0; c < 6; ++c)
                if (!std::isfinite(o[c]) && c != 3) return fail(SGD_E_NUMERIC, "non-finite matrix statistic");
            st.push_back(m);
        }
    }
    double* keep = out->mat_stats;
    out->mat_stats = nullptr;  // the statistics are inputs here
    rc = rank_units(units, L, st, p, out);
    out->mat_stats = keep;
    return rc;
}
