"""C-ABI tests that need no GPU: the library loads, exports what include/sgd.h declares,
and its host-side schedule logic matches the oracle bit for bit."""
import os
import re

import numpy as np
import pytest

from oracle import schedule as osch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

P = pytest.importorskip("paper_2609_29505_amd")


def _lib_or_skip():
    if not os.path.exists(P.lib_path):
        pytest.skip("libsgd.so not built")
    return P.lib()


def test_exports_match_header():
    _lib_or_skip()
    import subprocess
    hdr = open(os.path.join(ROOT, "include", "sgd.h")).read() + open(os.path.join(ROOT, "include", "sgd_ops.h")).read()
    declared = set(re.findall(r"\b(sgd_[a-z_0-9]+)\s*\(", hdr))
    out = subprocess.run(["nm", "-D", "--defined-only", P.lib_path], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (sgd_[a-z_0-9]+)\b", out))
    assert declared, "no declarations found"
    assert declared <= exported, f"declared but not exported: {declared - exported}"
    assert set(P.binding.EXPORTS) <= exported


def test_version():
    assert _lib_or_skip().sgd_version() == 1


@pytest.mark.parametrize("seed", range(40))
def test_budget_lifetimes_match_oracle(seed):
    _lib_or_skip()
    rng = np.random.default_rng(seed)
    L, T = int(rng.integers(1, 40)), int(rng.integers(1, 101))
    smin = osch.s_min_default(T)
    lam = rng.random(L)
    if seed % 5 == 0:
        lam[rng.integers(0, L)] = 0.0
    if seed % 7 == 0 and L > 2:
        lam[1] = lam[0]  # a tie
    n = int(rng.integers(L * smin, L * T + 1))
    ref = osch.lifetimes_budget(lam, T, n, smin)
    got = P.schedule_from_scores(lam, T, budget=n, s_min=smin)
    assert np.array_equal(got.lifetimes, ref.lifetimes)
    assert got.layer_steps == ref.layer_steps == n
    assert np.array_equal(got.active, osch.active_mask(ref.lifetimes, T))
    if np.isfinite(ref.cut_margin):
        assert got.cut_margin == ref.cut_margin
    else:
        assert not np.isfinite(got.cut_margin)


@pytest.mark.parametrize("tau", [0.25, 0.5, 1.0, 2.0])
def test_tau_lifetimes_match_oracle(tau):
    _lib_or_skip()
    rng = np.random.default_rng(int(tau * 100))
    lam = rng.random(50)
    lam[3] = tau * 7 / 20  # exactly on a breakpoint
    ref = osch.lifetimes_tau(lam, 20, tau, 2)
    got = P.schedule_from_scores(lam, 20, tau=tau, s_min=2)
    assert np.array_equal(got.lifetimes, ref)


def test_from_lifetimes_and_errors():
    _lib_or_skip()
    s = P.schedule_from_lifetimes([3, 1, 5], 5)
    assert s.layer_steps == 9
    assert np.array_equal(s.active, osch.active_mask([3, 1, 5], 5))
    with pytest.raises(P.SgdError) as e:
        P.schedule_from_lifetimes([0, 1], 5)
    assert e.value.code == -1
    with pytest.raises(P.SgdError) as e:
        P.schedule_from_scores([0.5, 0.2], 10, budget=1)
    assert e.value.code == -4
    with pytest.raises(P.SgdError) as e:
        P.schedule_from_scores([0.5, float("nan")], 10, budget=10)
    assert e.value.code == -8
    with pytest.raises(P.SgdError) as e:
        P.schedule_from_scores([0.5, 0.2], 10, tau=-1.0)
    assert e.value.code == -1


def test_library_defaults_match_oracle_readings():
    """The minimum-lifetime default and the percentage budget live in the library; they
    equal the oracle's readings (ceil(T / 10); floor(pct L T / 100))."""
    _lib_or_skip()
    for T in range(1, 201):
        assert P.s_min_default(T) == osch.s_min_default(T)
    rng = np.random.default_rng(0)
    for _ in range(300):
        pct, L, T = int(rng.integers(0, 101)), int(rng.integers(1, 64)), int(rng.integers(1, 201))
        assert P.budget_layer_steps(pct, L, T) == osch.budget_layer_steps(pct, L, T)
    with pytest.raises(P.SgdError):
        P.budget_layer_steps(101, 4, 10)


@pytest.mark.parametrize("seed", range(10))
def test_default_s_min_and_pct_budget(seed):
    """s_min = 0 and a percentage budget: the library applies its defaults."""
    _lib_or_skip()
    rng = np.random.default_rng(100 + seed)
    L, T = int(rng.integers(2, 40)), int(rng.integers(10, 101))
    lam = rng.random(L)
    pct = int(rng.integers(35, 100))
    n = osch.budget_layer_steps(pct, L, T)
    ref = osch.lifetimes_budget(lam, T, n, osch.s_min_default(T))
    got = P.schedule_from_scores(lam, T, budget_pct=pct)  # s_min None -> 0 -> library default
    assert got.s_min == osch.s_min_default(T)
    assert np.array_equal(got.lifetimes, ref.lifetimes)
    assert got.layer_steps == n


@pytest.mark.parametrize("rule", ["depth", "random"])
def test_unit_rules_build_without_spectra(rule):
    """The depth and random rankings (Sec. "Static ranking comparisons") need no weights:
    sgd_schedule_build runs them on the host, bit for bit the oracle's lifetimes."""
    _lib_or_skip()
    from oracle import rules as ru
    for L, T, pct in ((4, 10, 50), (32, 64, 35), (28, 50, 50), (7, 13, 70)):
        n = osch.budget_layer_steps(pct, L, T)
        got = P.schedule_build(None, None, T, budget_pct=pct, rule=rule, seed=99, L=L)
        ref = ru.lifetimes(rule, [], 1, T, n, osch.s_min_default(T), seed=99, L=L)
        assert np.array_equal(got.lifetimes, ref.lifetimes), (rule, L, T)
        assert np.array_equal(got.unit_raw, ru.raw_scores(rule, [], 1, seed=99, L=L))
        assert got.layer_steps == n


@pytest.mark.parametrize("rule", ["scr_frob", "frob", "spectral", "stable_rank", "frob_srank", "raw_scr"])
def test_rule_schedules_from_stats_match_oracle(rule):
    """Every matrix rule from given statistics (no GPU): the library's unit scores and
    lifetimes against the oracle's rules on the same statistics, bit for bit."""
    _lib_or_skip()
    from oracle import rules as ru
    from oracle import spectral as sp
    rng = np.random.default_rng(7)
    L, T, dh = 9, 30, 64
    roles, rows, stats = [], [], []
    for l in range(L):
        rl = ["q", "k", "v", "o", "w1", "w2"] + (["xq", "xk", "xv", "xo"] if l % 3 == 0 else [])
        u = {}
        for r in rl:
            ev = np.sort(rng.random(40) ** (3 * rng.random()))[::-1] * rng.uniform(0.5, 4)
            k = 4
            F = float(ev.sum())
            a, b = ev[:k].sum() + 1e-6 * F, ev[k:].sum() + 1e-6 * F
            st = sp.MatrixStats(40, 40, k, float(ev[:k].sum()), float(ev[k:].sum()), F, float(np.log(a / b)),
                                float(np.sqrt(F) * np.sqrt(a / (a + b))), float(ev[0]))
            u[r] = st
            rows.append([st.energy_top, st.energy_tail, st.frob_sq, st.scr, st.g, st.sigma1_sq])
        roles.append(rl)
        stats.append(u)
    for pct in (35, 50, 70):
        n = osch.budget_layer_steps(pct, L, T)
        ref = ru.lifetimes(rule, stats, dh, T, n, osch.s_min_default(T))
        got = P.schedule_from_stats(roles, [dh] * L, np.array(rows), T, budget_pct=pct, rule=rule)
        assert np.array_equal(got.unit_raw, ru.raw_scores(rule, stats, dh))
        assert np.array_equal(got.lifetimes, ref.lifetimes)


@pytest.mark.parametrize("arch,nb", [("tiny", 2), ("llada", 2), ("dit", 2), ("uvit", 2), ("sdxl", 3), ("sdxl_unet", 4)])
def test_model_units_by_granularity(arch, nb):
    """sgd_model_create validates and lays out without touching device memory, so the unit count
    and the cache size of both granularities are checked here with stand-in pointers (never
    dereferenced): L block units, or L nb branch units with one cache slot each."""
    import ctypes as C
    lib = _lib_or_skip()
    b = P.binding
    L, B, N, d, H, dh, F = (3 if arch == "uvit" else 2), 1, 64, 256, 2, 128, 512
    fake = 1 << 20  # 1 MiB-aligned stand-in address
    cw = (b.sgd_unit_weights * L)()
    for l in range(L):
        for name in b._W_FIELDS:
            setattr(cw[l], name, fake)

    def create(granularity):
        dsc = b.sgd_model_desc()
        dsc.arch, dsc.dtype = b.SGD_ARCH[arch], b.SGD_BF16
        dsc.B, dsc.N, dsc.d, dsc.H, dsc.head_dim, dsc.F, dsc.L, dsc.T = B, N, d, H, dh, F, L, 10
        dsc.ctx_len, dsc.ctx_dim = 77, 256
        dsc.update_row_begin, dsc.update_row_end = 0, N
        dsc.class_emb, dsc.ctx = fake, fake
        dsc.units = C.cast(cw, C.POINTER(b.sgd_unit_weights))
        dsc.grid, dsc.groups = 8, 32
        dsc.granularity = granularity
        h = C.c_void_p()
        rc = lib.sgd_model_create(C.byref(dsc), C.byref(h))
        return rc, h

    sizes = {}
    for g, units in ((b.SGD_UNIT["block"], L), (b.SGD_UNIT["branch"], L * nb)):
        rc, h = create(g)
        assert rc == 0, lib.sgd_last_error()
        nu, cb = C.c_int32(), C.c_size_t()
        assert lib.sgd_model_units(h, C.byref(nu)) == 0 and nu.value == units
        assert lib.sgd_cache_bytes(h, C.byref(cb)) == 0
        sizes[g] = cb.value
        assert lib.sgd_model_destroy(h) == 0
    slot = B * N * d * 4  # one fp32 [B, N, d] update, 256-byte aligned already
    assert sizes[1] - sizes[0] == (nb - 1) * L * slot
    rc, _ = create(2)
    assert rc == -1 and b"granularity" in lib.sgd_last_error()


@pytest.mark.parametrize("field,value,code,words", [
    ("B", 0, -2, b">= 1"), ("N", 0, -2, b">= 1"), ("L", 0, -2, b">= 1"), ("T", 0, -2, b">= 1"),
    ("d", 384, -2, b"H * head_dim"), ("head_dim", 96, -2, b"head_dim"), ("F", 100, -2, b"F must"),
    ("dtype", 7, -3, b"dtype"), ("granularity", -1, -1, b"granularity"),
    ("N", 1 << 23, -2, b"2^31")])  # B N d = 2^31: past the largest stream the kernels index
def test_model_create_refuses_bad_shapes(field, value, code, words):
    """Empty and unsupported model shapes are refused on the host with their error code and a
    message naming the constraint, before any device memory is touched (stand-in pointers)."""
    import ctypes as C
    lib = _lib_or_skip()
    b = P.binding
    L, B, N, d, H, dh, F = 2, 1, 64, 256, 2, 128, 512
    fake = 1 << 20
    cw = (b.sgd_unit_weights * L)()
    for l in range(L):
        for name in b._W_FIELDS:
            setattr(cw[l], name, fake)
    dsc = b.sgd_model_desc()
    dsc.arch, dsc.dtype = b.SGD_ARCH["tiny"], b.SGD_BF16
    dsc.B, dsc.N, dsc.d, dsc.H, dsc.head_dim, dsc.F, dsc.L, dsc.T = B, N, d, H, dh, F, L, 10
    dsc.update_row_begin, dsc.update_row_end = 0, N
    dsc.class_emb, dsc.ctx = fake, fake
    dsc.units = C.cast(cw, C.POINTER(b.sgd_unit_weights))
    h = C.c_void_p()
    assert lib.sgd_model_create(C.byref(dsc), C.byref(h)) == 0, lib.sgd_last_error()
    assert lib.sgd_model_destroy(h) == 0
    setattr(dsc, field, value)
    if field == "head_dim":  # keep d = H head_dim a multiple of 128 so the head-dim check is reached
        dsc.H, dsc.d = 4, 4 * value
    rc = lib.sgd_model_create(C.byref(dsc), C.byref(h))
    assert rc == code, (field, rc, lib.sgd_last_error())
    assert words in lib.sgd_last_error(), lib.sgd_last_error()
