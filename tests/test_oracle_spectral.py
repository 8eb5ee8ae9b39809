"""Pins for the oracle's spectral scores (Sec. 3.2 Eq. scr-reg, Lemma "Spectral energy
sandwich", appendix "Exact Block-Level Scores").

Each test fixes the oracle against something other than itself: a closed
form, an invariant the mathematics guarantees, or brute force.
"""
import math

import numpy as np
import pytest

import synth
from oracle import spectral as sp


def harmonic(n, p):
    return math.fsum(i ** (-p) for i in range(1, n + 1))


def planted64(seed, m, n):
    rng = np.random.default_rng(seed)
    w, pl = synth.planted_matrix(rng, m, n, np.float64)
    return w, pl


# ---------------------------------------------------------------- rank k

@pytest.mark.parametrize("m,n,k", [(1, 1, 1), (1, 50, 1), (5, 3, 1), (9, 9, 1), (10, 10, 1),
                                   (19, 40, 1), (20, 20, 2), (256, 1024, 25), (4096, 4096, 409),
                                   (1152, 4608, 115), (1024, 2048, 102), (1280, 1280, 128)])
def test_rank_k(m, n, k):
    # k = min(d, max(1, floor(0.1 d))), d = min(m, n)
    assert sp.rank_k(m, n) == k


# ---------------------------------------------------------------- closed forms

@pytest.mark.parametrize("seed,m,n", [(0, 256, 256), (1, 300, 200), (2, 200, 700), (3, 640, 640)])
def test_planted_closed_form(seed, m, n):
    """Planted s_i ~ i^-a with ||W||_F^2 = c^2 d: E_k / F = H_k(2a) / H_d(2a)."""
    w, pl = planted64(seed, m, n)
    d = min(m, n)
    k = max(1, d // 10)
    rho0 = harmonic(k, 2 * pl.a) / harmonic(d, 2 * pl.a)
    st = sp.matrix_stats(w, eta=0.0)
    assert st.frob_sq == pytest.approx(pl.c ** 2 * d, rel=1e-12)
    assert st.energy_top / st.frob_sq == pytest.approx(rho0, rel=1e-11)
    assert st.scr == pytest.approx(math.log(rho0 / (1 - rho0)), rel=1e-9, abs=1e-10)
    assert st.g == pytest.approx(math.sqrt(st.frob_sq * rho0), rel=1e-11)
    eta = 1e-6
    st = sp.matrix_stats(w, eta=eta)
    F = pl.c ** 2 * d
    A = F * rho0 + eta * F
    B = F * (1 - rho0) + eta * F
    assert st.scr == pytest.approx(math.log(A / B), rel=1e-9, abs=1e-10)


def test_appendix_values_golden():
    """Closed-form rho_0 and SCR values for the planted spectra (tests/golden/planted_scr.txt)."""
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "planted_scr.txt")
    rows = [l.split() for l in open(path) if l.strip() and not l.startswith("#")]
    assert rows
    for d, k, a, rho0, scr0, scr_eta in rows:
        d, k, a = int(d), int(k), float(a)
        assert sp.rank_k(d, d) == k
        r = harmonic(k, 2 * a) / harmonic(d, 2 * a)
        assert r == pytest.approx(float(rho0), rel=1e-11)
        assert math.log(r / (1 - r)) == pytest.approx(float(scr0), rel=1e-8)
        # and the oracle on an explicit diagonal matrix with that spectrum
        s = np.arange(1, d + 1, dtype=np.float64) ** (-a)
        st = sp.matrix_stats(np.diag(s), eta=1e-6)
        assert st.scr == pytest.approx(float(scr_eta), rel=1e-8)


def test_rank_one_regularised():
    """Rank one: tail = 0, so SCR_eta = log((1 + eta) / eta)."""
    rng = np.random.default_rng(5)
    w = np.outer(rng.standard_normal(40), rng.standard_normal(30))
    for eta in (1e-6, 1e-3, 0.5):
        st = sp.matrix_stats(w, eta=eta)
        assert st.scr == pytest.approx(math.log((1 + eta) / eta), rel=1e-9)


def test_identity_rho_is_k_over_d():
    for d in (1, 7, 10, 64, 257):
        st = sp.matrix_stats(np.eye(d), eta=0.0)
        k = sp.rank_k(d, d)
        if k < d:
            assert st.energy_top / st.frob_sq == pytest.approx(k / d, rel=1e-12)
            assert st.g == pytest.approx(math.sqrt(k), rel=1e-12)
        else:  # d = 1: everything is in the head, B = 0
            assert st.g == pytest.approx(1.0, rel=1e-12)


def test_vector_edge_case_d1():
    """d = 1 (a row vector): k = 1, the tail is empty and only eta keeps SCR finite."""
    w = np.arange(1.0, 6.0)[None, :]
    st = sp.matrix_stats(w, eta=1e-6)
    assert st.k == 1 and st.energy_tail == 0.0
    assert st.scr == pytest.approx(math.log((1 + 1e-6) / 1e-6), rel=1e-9)


# ---------------------------------------------------------------- invariants

def test_sandwich():
    """||W||_F sqrt(rho/k) <= ||W||_2 <= ||W||_F sqrt(rho)  (eta = 0)."""
    rng = np.random.default_rng(11)
    mats = [rng.standard_normal((50, 80)), rng.standard_normal((120, 33)) ** 3]
    mats += [planted64(s, 90, 70)[0] for s in range(3)]
    for w in mats:
        st = sp.matrix_stats(w, eta=0.0)
        s1 = np.linalg.norm(w, 2)
        assert st.g / math.sqrt(st.k) <= s1 * (1 + 1e-12)
        assert s1 <= st.g * (1 + 1e-12)


def test_scale_and_orthogonal_invariance():
    rng = np.random.default_rng(12)
    w = rng.standard_normal((60, 45))
    base = sp.matrix_stats(w, eta=1e-6)
    scaled = sp.matrix_stats(-3.5 * w, eta=1e-6)
    assert scaled.scr == pytest.approx(base.scr, rel=1e-11)
    assert scaled.g == pytest.approx(3.5 * base.g, rel=1e-11)
    q, _ = np.linalg.qr(rng.standard_normal((60, 60)))
    rot = sp.matrix_stats(q @ w, eta=1e-6)
    assert rot.scr == pytest.approx(base.scr, rel=1e-10)
    assert rot.g == pytest.approx(base.g, rel=1e-11)
    tr = sp.matrix_stats(w.T, eta=1e-6)
    assert tr.scr == pytest.approx(base.scr, rel=1e-11)


# ---------------------------------------------------------------- brute-force SVD

def jacobi_singular_values(a):
    """One-sided Jacobi (Hestenes) SVD: rotate column pairs until orthogonal."""
    u = np.array(a, dtype=np.float64)
    if u.shape[0] < u.shape[1]:
        u = u.T.copy()
    n = u.shape[1]
    for _ in range(60):
        off = 0.0
        for i in range(n - 1):
            for j in range(i + 1, n):
                alpha = float(u[:, i] @ u[:, i])
                beta = float(u[:, j] @ u[:, j])
                gamma = float(u[:, i] @ u[:, j])
                if abs(gamma) < 1e-300:
                    continue
                off = max(off, abs(gamma) / math.sqrt(alpha * beta))
                zeta = (beta - alpha) / (2 * gamma)
                t = math.copysign(1.0, zeta) / (abs(zeta) + math.sqrt(1 + zeta * zeta))
                c = 1 / math.sqrt(1 + t * t)
                s = c * t
                ui = u[:, i].copy()
                u[:, i] = c * ui - s * u[:, j]
                u[:, j] = s * ui + c * u[:, j]
        if off < 1e-15:
            break
    return np.sort(np.linalg.norm(u, axis=0))[::-1]


def test_two_by_two_analytic():
    rng = np.random.default_rng(3)
    for _ in range(20):
        a, b, c, d = rng.standard_normal(4)
        # sigma_{1,2} = (sqrt((a+d)^2 + (c-b)^2) +- sqrt((a-d)^2 + (b+c)^2)) / 2
        p = math.hypot(a + d, c - b)
        q = math.hypot(a - d, b + c)
        s = sorted([(p + q) / 2, abs(p - q) / 2], reverse=True)
        lam = sp.singular_values_sq(np.array([[a, b], [c, d]]))
        assert np.allclose(np.sqrt(lam), s, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("shape", [(3, 3), (5, 8), (8, 4), (7, 7)])
def test_jacobi_vs_oracle(shape):
    rng = np.random.default_rng(sum(shape))
    w = rng.standard_normal(shape)
    ref = jacobi_singular_values(w)
    lam = sp.singular_values_sq(w)
    assert np.allclose(np.sqrt(lam), ref, rtol=1e-12, atol=1e-13)


def test_gram_branch_matches_svd_branch():
    """d > 1024 uses the Gram eigenvalues; compare with the SVD branch on the same matrix."""
    w, pl = planted64(21, 1040, 1100)
    lam = sp.singular_values_sq(w)
    assert np.allclose(lam, pl.s ** 2, rtol=1e-9, atol=1e-12 * pl.s[0] ** 2)


# ---------------------------------------------------------------- component scores

def _unit(rng, d, roles):
    return {r: rng.standard_normal((d if r != "w1" else 2 * d, d if r != "w2" else 2 * d)) for r in roles}


def test_q_attn_structure():
    """Degree one in W_O and W_V, affine in g(W_Q) g(W_K) with slope g_O g_V / sqrt(d_h)."""
    rng = np.random.default_rng(7)
    m = _unit(rng, 24, ("q", "k", "v", "o"))
    base = sp.unit_score(m, head_dim=4).raw
    for role in ("o", "v"):
        mm = dict(m)
        mm[role] = 2.5 * m[role]
        assert sp.unit_score(mm, head_dim=4).raw == pytest.approx(2.5 * base, rel=1e-12)
    g = {r: sp.matrix_stats(m[r]).g for r in m}
    outer = g["o"] * g["v"]
    for role in ("q", "k"):
        mm = dict(m)
        mm[role] = 3.0 * m[role]
        # scaling W_Q (or W_K) by 3 triples only the score-path term
        assert sp.unit_score(mm, head_dim=4).raw - outer == pytest.approx(3.0 * (base - outer), rel=1e-11)
    # the score-path term falls as 1 / sqrt(d_h)
    t4 = sp.unit_score(m, head_dim=4).raw - outer
    t16 = sp.unit_score(m, head_dim=16).raw - outer
    assert t4 / t16 == pytest.approx(2.0, rel=1e-12)
    # lower bound from the sandwich: every g >= spectral norm
    s = {r: np.linalg.norm(m[r], 2) for r in m}
    assert base >= s["o"] * s["v"] * (1 + s["q"] * s["k"] / 2.0)


def test_q_mlp_and_block_sum():
    rng = np.random.default_rng(8)
    d = 16
    attn = {r: rng.standard_normal((d, d)) for r in ("q", "k", "v", "o")}
    xattn = {r: rng.standard_normal((d, d)) for r in ("xq", "xk", "xv", "xo")}
    mlp = {"w1": rng.standard_normal((40, d)), "w2": rng.standard_normal((d, 40))}
    q_a = sp.unit_score(attn, 4).raw
    q_x = sp.unit_score({"q": xattn["xq"], "k": xattn["xk"], "v": xattn["xv"], "o": xattn["xo"]}, 4).raw
    q_m = sp.unit_score(mlp, 4).raw
    # q_mlp is bilinear in (W1, W2)
    mm = dict(mlp)
    mm["w1"] = 2 * mlp["w1"]
    mm["w2"] = 3 * mlp["w2"]
    assert sp.unit_score(mm, 4).raw == pytest.approx(6 * q_m, rel=1e-12)
    # the block score sums its components
    full = sp.unit_score({**attn, **xattn, **mlp}, 4).raw
    assert full == pytest.approx(q_a + q_x + q_m, rel=1e-12)


def test_normalise():
    raw = [3.0, 1.5, 0.0, 2.9999]
    lam = sp.normalise(raw)
    assert lam.max() < 1.0 and 1.0 - lam.max() == pytest.approx(1e-12 / 3.0, rel=1e-3)
    assert lam[1] / lam[0] == pytest.approx(0.5, rel=1e-15)
    assert lam[2] == 0.0
