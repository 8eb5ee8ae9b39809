"""Full-size GPU checks: every workload at its real shape, in the launch configuration
bench.py times.

* Step parity, teacher-forced: step 1 (every unit active) and step 2 with every other unit
  frozen (lifetimes 1 / T) match the oracle at the per-step bar (2e-2 bf16, 1e-4 fp32); step 1
  run twice gives bitwise the same state.
* Schedule: every matrix's statistics and every unit's score against the oracle's stored
  full-size values, lifetimes and masks bit for bit, for the method and every ranking rule.
"""
import os
import time

import numpy as np
import pytest

import synth
from oracle import model as om
from oracle import schedule as osch
from oracle import spectral as osp
from oracle.numerics import decode

from helpers import TOL, load_fullsize_golden, rel_err

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

FULL = ["tiny", "dit", "uvit", "sdxl", "llada", "sdxl_unet"]


def progress(msg):
    """Progress lines for long full-size cases, also appended to a log file in the directory
    SGD_PROGRESS_DIR names (for runners that watch files rather than captured output)."""
    d = os.environ.get("SGD_PROGRESS_DIR", "")
    line = f"[{time.strftime('%H:%M:%S')}] {msg}\n"
    if d and os.path.isdir(d):
        with open(os.path.join(d, "fullsize_progress.log"), "a") as f:
            f.write(line)
    print(line, end="", flush=True)


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_29505_amd as P
    P.lib()
    return P


def load(name):
    cfg = synth.get_config(name)
    progress(f"{name}: generating weights")
    w = synth.model_weights(cfg, workers=min(16, os.cpu_count() or 1),
                            progress=lambda u: None)
    return cfg, w, synth.inputs(cfg)


@pytest.mark.parametrize("name", FULL)
def test_fullsize_step_parity(P, name):
    import torch
    cfg, w, x = load(name)
    dm = P.DeviceModel(cfg, w, x)
    T, L = cfg.T, cfg.L
    S = np.array([1 if l % 2 == 0 else T for l in range(L)])
    mask = osch.active_mask(S, T)
    sched = P.schedule_from_lifetimes(S, T)
    # GPU: step 1 from z0; step 2 from the oracle's z_2 with the GPU's own cache
    m = om.Model(cfg, w, x, lazy=(cfg.name == "llada"))
    cross = [m.cross_kv(u) for u in m.units] if cfg.arch in om.CROSS_ARCHS else None
    cache = P.Cache(dm)
    cache.reset()
    z = torch.from_numpy(x["z"].copy()).cuda()
    dm.step(z, 1, sched, cache)
    g1 = z.cpu().numpy().astype(np.float64)
    # the same step again on a fresh cache: bitwise the same state (no order-dependent sums,
    # e.g. in the split-K exchange of the long-K MLP output GEMM)
    cache_b = P.Cache(dm)
    cache_b.reset()
    zb = torch.from_numpy(x["z"].copy()).cuda()
    dm.step(zb, 1, sched, cache_b)
    assert np.array_equal(zb.cpu().numpy(), z.cpu().numpy())
    del cache_b, zb
    progress(f"{name}: oracle step 1")
    oc = {}
    eps1 = om.denoise_step(m, x["z"], 1, mask[0], oc, cross)
    z1 = om.sampler_update(cfg, np.asarray(x["z"], np.float64), eps1, 1)
    e1 = rel_err(g1, z1)
    z.copy_(torch.from_numpy(z1.astype(np.float32)))
    dm.step(z, 2, sched, cache)
    g2 = z.cpu().numpy().astype(np.float64)
    progress(f"{name}: oracle step 2 ({int((1 - mask[1]).sum())} of {L} units frozen)")
    eps2 = om.denoise_step(m, z1, 2, mask[1], oc, cross)
    z2 = om.sampler_update(cfg, z1, eps2, 2)
    e2 = rel_err(g2, z2)
    progress(f"{name}: step 1 error {e1:.3e}, step 2 error {e2:.3e}")
    assert np.isfinite(g2).all()
    assert e1 <= TOL[cfg.dtype] and e2 <= TOL[cfg.dtype], (e1, e2)
    dm.close()


def test_fullsize_late_step_real_schedule(P):
    """The LLaDA-8B-shaped workload at step 40 of its 35 % schedule (the oracle's lifetimes from
    the stored full-size scores): four active units, frozen runs of 16, 3, 6 and 1 units folded
    into the next pre-norm and a run of 2 at the end of the stack on its own.  The GPU runs steps
    1-39 itself; step 40 from its own state and cached updates against the oracle's step 40 on
    the same state and the same cached updates (2e-2 on the state and on the network output,
    recovered from the sampler update on the rows it owns)."""
    import torch
    name = "llada"
    cfg, w, x = load(name)
    T, L = cfg.T, cfg.L
    pct, s0 = min(cfg.budgets), 40
    _, graw = load_fullsize_golden(name)
    bs = osch.lifetimes_budget(osp.normalise(graw), T, osch.budget_layer_steps(pct, L, T), osch.s_min_default(T))
    S = np.asarray(bs.lifetimes)
    mask = osch.active_mask(S, T)
    assert 2 <= int(mask[s0 - 1].sum()) <= L // 4  # mostly frozen at this step
    dm = P.DeviceModel(cfg, w, x)
    sched = P.schedule_from_lifetimes(S, T)
    assert np.array_equal(sched.lifetimes, S)
    cache = P.Cache(dm)
    cache.reset()
    z = torch.from_numpy(x["z"].copy()).cuda()
    progress(f"{name}: GPU steps 1-{s0 - 1} of the {pct} % schedule")
    for s in range(1, s0):
        dm.step(z, s, sched, cache)
    torch.cuda.synchronize()
    zin = z.cpu().numpy().astype(np.float64)
    slot = (cfg.M * cfg.d * 4 + 255) // 256 * 256
    deltas = {u: cache.buf[u * slot: u * slot + cfg.M * cfg.d * 4].view(torch.float32).cpu().numpy()
              .astype(np.float64).reshape(zin.shape) for u in range(L) if not mask[s0 - 1][u]}
    dm.step(z, s0, sched, cache)
    g = z.cpu().numpy().astype(np.float64)
    dm.close()
    progress(f"{name}: oracle step {s0} ({int(mask[s0 - 1].sum())} of {L} units active)")
    m = om.Model(cfg, w, x, lazy=True)
    eps = om.denoise_step(m, zin, s0, mask[s0 - 1], deltas)
    ref = om.sampler_update(cfg, zin, eps, s0)
    e = rel_err(g, ref)
    # the network output itself, recovered from the update z - eps / T on the sampler's rows
    r0, r1 = cfg.update_rows
    e_eps = rel_err(T * (zin[:, r0:r1] - g[:, r0:r1]), eps[:, r0:r1])
    progress(f"{name}: step {s0} error {e:.3e}, network output error {e_eps:.3e}")
    assert e <= TOL[cfg.dtype] and e_eps <= TOL[cfg.dtype], (e, e_eps)


@pytest.mark.parametrize("name", FULL)
def test_fullsize_schedule(P, name):
    """The GPU's scores and schedules at full size against the oracle's stored statistics
    (tests/golden/fullsize_<workload>.txt, written by the oracle alone): every matrix's E_k,
    tail, ||W||_F^2, ||W||_2^2 and g, every unit's raw score to 1e-10, and the lifetimes and
    mask bit for bit at every budget, for the method and for every static ranking rule."""
    from oracle import rules as ru
    cfg, w, x = load(name)
    dm = P.DeviceModel(cfg, w, x)
    T, L = cfg.T, cfg.L
    smin = osch.s_min_default(T)
    units = dm.scored_units()
    gstats, graw = load_fullsize_golden(name)
    progress(f"{name}: schedule build on the GPU")
    sched = P.schedule_build(units, [cfg.dh] * L, T, budget_pct=min(cfg.budgets))
    assert sched.s_min == smin
    # every matrix against the oracle's statistics
    row = 0
    for l, mats in enumerate(units):
        nconv = 0
        for role, _ in mats:
            if role == "conv":  # the unit's convolutions, in order
                nconv += 1
                role = f"conv{nconv}"
            ref = gstats[l][role]
            got = sched.mat_stats[row]
            row += 1
            F = ref.frob_sq
            assert got[2] == pytest.approx(F, rel=1e-12), (l, role)
            assert abs(got[0] - ref.energy_top) <= 1e-11 * F and abs(got[1] - ref.energy_tail) <= 1e-11 * F
            assert got[5] == pytest.approx(ref.sigma1_sq, rel=1e-11), (l, role)
            assert got[4] == pytest.approx(ref.g, rel=1e-11), (l, role)
    assert np.allclose(sched.unit_raw, graw, rtol=1e-10, atol=0)
    roles = [[r for r, _ in mats] for mats in units]
    for rule in ru.RULES:
        lam = osp.normalise(ru.raw_scores(rule, gstats, cfg.dh, seed=5, L=L))
        for pct in cfg.budgets:
            n = osch.budget_layer_steps(pct, L, T)
            ref = osch.lifetimes_budget(lam, T, n, smin)
            if rule == "scr_frob" and pct == min(cfg.budgets):
                got = sched
            else:  # the same statistics re-ranked by the library (host arithmetic)
                got = P.schedule_from_stats(roles, [cfg.dh] * L, sched.mat_stats, T, budget_pct=pct, rule=rule,
                                            seed=5)
            if rule not in ("depth", "random"):  # scores from float statistics: far from a tie
                assert ref.cut_margin > 1e-8, (rule, pct, ref.cut_margin)
            assert np.array_equal(got.lifetimes, ref.lifetimes), (rule, pct)
            assert np.array_equal(got.active, osch.active_mask(ref.lifetimes, T))
            assert got.layer_steps == n == int(got.lifetimes.sum())
    # one matrix rule end to end on the GPU (spectra recomputed under that rule)
    got = P.schedule_build(units, [cfg.dh] * L, T, budget_pct=min(cfg.budgets), rule="stable_rank")
    lam = osp.normalise(ru.raw_scores("stable_rank", gstats, cfg.dh))
    ref = osch.lifetimes_budget(lam, T, osch.budget_layer_steps(min(cfg.budgets), L, T), smin)
    assert np.array_equal(got.lifetimes, ref.lifetimes)
    dm.close()
