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
    double e_top = 0, e_tail = 0, frob = 0, scr = 0, g = 0;
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

// Score every job with a pool of host workers, each driving its own stream.
static int run_stats(std::vector<MatJob>& jobs, double eta, hipStream_t user_stream) {
    if (jobs.empty()) return SGD_OK;
    int dev = 0;
    SGD_HIP_TRY(hipGetDevice(&dev));
    SGD_HIP_TRY(hipStreamSynchronize(user_stream));
    long nmax = 0;
    for (auto& j : jobs) nmax = std::max(nmax, std::min(j.m->rows, j.m->cols));
    unsigned hc = std::thread::hardware_concurrency();
    int nw = (int)std::min<size_t>(jobs.size(), std::max(1u, std::min(hc ? hc : 1u, 16u)));
    // keep the Gram buffers within a few GB
    const double gbytes = (double)nmax * nmax * 8.0;
    while (nw > 1 && gbytes * nw > 4.0e9) --nw;

    std::atomic<size_t> next{0};
    std::mutex emu;
    int first_err = SGD_OK;
    std::string err_msg;
    auto record = [&](int code, const std::string& msg) {
        std::lock_guard<std::mutex> lk(emu);
        if (first_err == SGD_OK) { first_err = code; err_msg = msg; }
    };
    auto worker = [&]() {
        if (hipSetDevice(dev) != hipSuccess) { record(SGD_E_HIP, "hipSetDevice failed in a worker"); return; }
        hipStream_t st = nullptr;
        double *G = nullptr, *dg = nullptr, *od = nullptr, *work = nullptr, *trace = nullptr;
        auto cleanup = [&]() {
            if (G) (void)hipFree(G);
            if (dg) (void)hipFree(dg);
            if (od) (void)hipFree(od);
            if (work) (void)hipFree(work);
            if (trace) (void)hipFree(trace);
            if (st) (void)hipStreamDestroy(st);
        };
        hipError_t e = hipStreamCreateWithFlags(&st, hipStreamNonBlocking);
        if (e == hipSuccess) e = hipMalloc(&G, (size_t)nmax * nmax * sizeof(double));
        if (e == hipSuccess) e = hipMalloc(&dg, (size_t)nmax * sizeof(double));
        if (e == hipSuccess) e = hipMalloc(&od, (size_t)nmax * sizeof(double));
        if (e == hipSuccess) e = hipMalloc(&work, (size_t)(5 * nmax + 8) * sizeof(double));
        if (e == hipSuccess) e = hipMalloc(&trace, (size_t)nmax * sizeof(double));
        if (e != hipSuccess) {
            record(SGD_E_HIP, std::string("spectral workspace: ") + hipGetErrorString(e));
            cleanup();
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
        cleanup();
    };
    std::vector<std::thread> th;
    for (int w = 0; w < nw; ++w) th.emplace_back(worker);
    for (auto& t : th) t.join();
    if (first_err != SGD_OK) return fail(first_err, err_msg);
    return SGD_OK;
}

// ---------------------------------------------------------------------------- lifetimes

static int check_params(const sgd_sched_params* p, int L) {
    if (!p) return fail(SGD_E_ARG, "params is NULL");
    if (L < 1) return fail(SGD_E_ARG, "L must be >= 1");
    if (p->T < 1) return fail(SGD_E_ARG, "T must be >= 1");
    if (p->s_min < 1 || p->s_min > p->T) return fail(SGD_E_ARG, "s_min must lie in 1..T");
    if (p->budget_layer_steps < 0 && !(p->tau > 0)) return fail(SGD_E_ARG, "tau must be > 0 in tau mode");
    if (!(p->eta >= 0) || !std::isfinite(p->eta)) return fail(SGD_E_ARG, "eta must be finite and >= 0");
    if (p->budget_layer_steps >= 0) {
        const long lo = (long)L * p->s_min, hi = (long)L * p->T;
        if (p->budget_layer_steps < lo || p->budget_layer_steps > hi)
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
    return SGD_OK;
}

}  // namespace sgd

using namespace sgd;

extern "C" int sgd_schedule_from_scores(const double* unit_score, int32_t L, const sgd_sched_params* params,
                                        sgd_schedule* out) {
    if (!unit_score || !out || !out->lifetimes || !out->active) return fail(SGD_E_ARG, "NULL argument");
    int rc = check_params(params, L);
    if (rc) return rc;
    for (int l = 0; l < L; ++l)
        if (!std::isfinite(unit_score[l]) || unit_score[l] < 0) return fail(SGD_E_NUMERIC, "scores must be finite and >= 0");
    rc = lifetimes_from_scores(unit_score, L, params, out);
    if (rc) return rc;
    if (out->unit_score)
        for (int l = 0; l < L; ++l) out->unit_score[l] = unit_score[l];
    return SGD_OK;
}

extern "C" int sgd_schedule_from_lifetimes(int32_t L, int32_t T, const int32_t* lifetimes, sgd_schedule* out) {
    if (!lifetimes || !out || !out->lifetimes || !out->active) return fail(SGD_E_ARG, "NULL argument");
    if (L < 1 || T < 1) return fail(SGD_E_ARG, "L and T must be >= 1");
    long total = 0;
    for (int l = 0; l < L; ++l) {
        if (lifetimes[l] < 1 || lifetimes[l] > T) return fail(SGD_E_ARG, "lifetimes must lie in 1..T");
        total += lifetimes[l];
    }
    out->L = L;
    out->T = T;
    for (int l = 0; l < L; ++l) out->lifetimes[l] = lifetimes[l];
    for (int s = 1; s <= T; ++s)
        for (int l = 0; l < L; ++l) out->active[(size_t)(s - 1) * L + l] = (uint8_t)(s <= lifetimes[l]);
    out->layer_steps = total;
    out->cut_margin = std::numeric_limits<double>::infinity();
    return SGD_OK;
}

extern "C" int sgd_matrix_stats(const sgd_matrix* m, double eta, void* hip_stream, double out[5]) {
    if (!out) return fail(SGD_E_ARG, "out is NULL");
    int rc = validate_matrix(m);
    if (rc) return rc;
    if (!(eta >= 0) || !std::isfinite(eta)) return fail(SGD_E_ARG, "eta must be finite and >= 0");
    std::vector<MatJob> jobs{{m, {}}};
    rc = run_stats(jobs, eta, (hipStream_t)hip_stream);
    if (rc) return rc;
    const MatStats& s = jobs[0].out;
    out[0] = s.e_top; out[1] = s.e_tail; out[2] = s.frob; out[3] = s.scr; out[4] = s.g;
    return SGD_OK;
}

extern "C" int sgd_schedule_build(const sgd_unit* units, int32_t L, const sgd_sched_params* params,
                                  void* hip_stream, sgd_schedule* out) {
    if (!units || !out || !out->lifetimes || !out->active) return fail(SGD_E_ARG, "NULL argument");
    int rc = check_params(params, L);
    if (rc) return rc;
    std::vector<MatJob> jobs;
    for (int l = 0; l < L; ++l) {
        const sgd_unit& u = units[l];
        if (u.n_mats < 1 || !u.mats) return fail(SGD_E_ARG, "unit without matrices");
        if (u.head_dim < 1) return fail(SGD_E_ARG, "head_dim must be >= 1");
        for (int i = 0; i < u.n_mats; ++i) {
            rc = validate_matrix(&u.mats[i]);
            if (rc) return rc;
            jobs.push_back({&u.mats[i], {}});
        }
    }
    rc = run_stats(jobs, params->eta, (hipStream_t)hip_stream);
    if (rc) return rc;
    // combine: component scores -> unit raw score -> normalised score
    std::vector<double> raw(L, 0.0);
    size_t ji = 0;
    for (int l = 0; l < L; ++l) {
        const sgd_unit& u = units[l];
        double g[SGD_ROLE_CONV + 1];
        bool have[SGD_ROLE_CONV + 1] = {};
        double conv = 0.0;
        for (int i = 0; i < u.n_mats; ++i, ++ji) {
            const int r = u.mats[i].role;
            if (r == SGD_ROLE_CONV) { conv += jobs[ji].out.g; continue; }
            if (have[r]) return fail(SGD_E_ARG, "a unit lists the same role twice");
            have[r] = true;
            g[r] = jobs[ji].out.g;
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
    double mx = 0.0;
    for (double v : raw) {
        if (!std::isfinite(v)) return fail(SGD_E_NUMERIC, "non-finite unit score");
        mx = std::max(mx, v);
    }
    std::vector<double> score(L);
    for (int l = 0; l < L; ++l) score[l] = raw[l] / (mx + 1e-12);
    rc = lifetimes_from_scores(score.data(), L, params, out);
    if (rc) return rc;
    if (out->unit_raw) std::memcpy(out->unit_raw, raw.data(), L * sizeof(double));
    if (out->unit_score) std::memcpy(out->unit_score, score.data(), L * sizeof(double));
    if (out->mat_stats)
        for (size_t i = 0; i < jobs.size(); ++i) {
            const MatStats& s = jobs[i].out;
            double* o = out->mat_stats + 5 * i;
            o[0] = s.e_top; o[1] = s.e_tail; o[2] = s.frob; o[3] = s.scr; o[4] = s.g;
        }
    return SGD_OK;
}
