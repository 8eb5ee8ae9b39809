"""GPU parity of branch-granular scheduling (every residual branch of a block is a scheduled unit
of its own, block-major in execution order) through the C ABI, against the oracle: schedules
bit for bit, per-step and free-running trajectories to the bf16/fp32 bars, all-active equal to
the unscheduled forward bit for bit, long frozen runs crossing blocks, and the drift policy
over branch units."""
import numpy as np
import pytest

import synth
from oracle import drift as od
from oracle import model as om
from oracle import schedule as osch

from helpers import (FREE_RUNNING_CEIL, TOL, chaos_floor, gpu_teacher_forced, gpu_trajectory, oracle_schedule,
                     oracle_trajectory, rel_err)

pytestmark = pytest.mark.gpu

MINIS = ["tiny_ragged", "llada_mini", "dit_mini", "uvit_mini", "sdxl_mini", "sdxl_unet_mini"]


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_29505_amd as P
    P.lib()
    return P


_cache = {}


def workload(name):
    if name not in _cache:
        cfg = synth.get_config(name)
        _cache[name] = (cfg, synth.model_weights(cfg), synth.inputs(cfg))
    return _cache[name]


def branch_schedule(P, dm, cfg, pct):
    U = dm.n_units
    n = osch.budget_layer_steps(pct, U, cfg.T)
    return P.schedule_build(dm.scored_units(), [cfg.dh] * U, cfg.T, budget=n)


@pytest.mark.parametrize("name", MINIS + ["tiny"])
def test_branch_schedule_bit_exact(P, name):
    cfg, w, x = workload(name)
    dm = P.DeviceModel(cfg, w, x, granularity="branch")
    nb = len(om.branches(cfg.arch))
    assert dm.n_units == nb * cfg.L
    for pct in cfg.budgets:
        raw, lam, bs = oracle_schedule(cfg, w, pct, granularity="branch")
        got = branch_schedule(P, dm, cfg, pct)
        assert np.allclose(got.unit_raw, raw, rtol=1e-11, atol=0)
        assert np.allclose(got.unit_score, lam, rtol=1e-11, atol=0)
        assert bs.cut_margin > 1e-9, "near-tie: the comparison below would be fragile"
        assert np.array_equal(got.lifetimes, bs.lifetimes)
        assert np.array_equal(got.active, osch.active_mask(bs.lifetimes, cfg.T))
        assert got.layer_steps == osch.budget_layer_steps(pct, dm.n_units, cfg.T)
    dm.close()


@pytest.mark.parametrize("name", MINIS)
def test_branch_step_parity_teacher_forced(P, name):
    cfg, w, x = workload(name)
    dm = P.DeviceModel(cfg, w, x, granularity="branch")
    pct = cfg.budgets[-1]
    _, _, bs = oracle_schedule(cfg, w, pct, granularity="branch")
    mask = osch.active_mask(bs.lifetimes, cfg.T)
    ref = oracle_trajectory(cfg, w, x, mask, granularity="branch")
    sched = branch_schedule(P, dm, cfg, pct)
    assert np.array_equal(sched.lifetimes, bs.lifetimes)
    got = gpu_teacher_forced(dm, cfg, ref.z, x["z"], sched)
    errs = [rel_err(g, r) for g, r in zip(got, ref.z)]
    print(name, "branch units, teacher-forced per-step error", ["%.2e" % e for e in errs])
    assert max(errs) <= TOL[cfg.dtype], errs
    dm.close()


@pytest.mark.parametrize("name", MINIS)
def test_branch_trajectory_parity(P, name):
    """Free-running, with the bound of the block-unit test (the oracle's own divergence under
    tiny perturbations of z_1, at least 2e-2, capped)."""
    cfg, w, x = workload(name)
    dm = P.DeviceModel(cfg, w, x, granularity="branch")
    _, _, bs = oracle_schedule(cfg, w, cfg.budgets[-1], granularity="branch")
    mask = osch.active_mask(bs.lifetimes, cfg.T)
    got = gpu_trajectory(dm, cfg, x, P.schedule_from_lifetimes(bs.lifetimes, cfg.T))
    if cfg.dtype == "f32":
        ref = oracle_trajectory(cfg, w, x, mask, granularity="branch")
        bounds = [TOL["f32"]] * cfg.T
    else:
        ref, floor = chaos_floor(cfg, w, x, mask, granularity="branch")
        assert max(floor) < FREE_RUNNING_CEIL, floor
        bounds = [min(FREE_RUNNING_CEIL, max(TOL["bf16"], 2 * f)) for f in floor]
    errs = [rel_err(g, r) for g, r in zip(got, ref.z)]
    print(name, "branch units, free-running per-step error", ["%.2e" % e for e in errs])
    assert all(e <= b for e, b in zip(errs, bounds)), (errs, bounds)
    dm.close()


@pytest.mark.parametrize("name", MINIS)
def test_branch_all_active_equals_unscheduled_bitwise(P, name):
    """Every branch active is the unscheduled forward bit for bit, and so is the block model's."""
    cfg, w, x = workload(name)
    dm = P.DeviceModel(cfg, w, x, granularity="branch")
    steps = min(cfg.T, 3)
    a = gpu_trajectory(dm, cfg, x, P.schedule_from_lifetimes([cfg.T] * dm.n_units, cfg.T), steps)
    b = gpu_trajectory(dm, cfg, x, None, steps)
    dm.close()
    dk = P.DeviceModel(cfg, w, x)
    c = gpu_trajectory(dk, cfg, x, None, steps)
    dk.close()
    for za, zb, zc in zip(a, b, c):
        assert np.array_equal(za, zb)
        assert np.array_equal(zb, zc)


@pytest.mark.parametrize("name", ["llada_mini", "dit_mini", "uvit_mini", "sdxl_mini", "sdxl_unet_mini"])
def test_branch_frozen_runs(P, name):
    """Short, mixed lifetimes: frozen runs that start and end inside blocks, cross block
    boundaries, end at U-ViT out-blocks (whose skip linear runs first) and at ResNet branches,
    and are added by the next branch's pre-norm; teacher-forced against the oracle."""
    cfg, w, x = workload(name)
    dm = P.DeviceModel(cfg, w, x, granularity="branch")
    U = dm.n_units
    S = np.array([1 + (7 * j) % 3 if j % 5 else cfg.T for j in range(U)])
    mask = osch.active_mask(S, cfg.T)
    ref = oracle_trajectory(cfg, w, x, mask, granularity="branch")
    got = gpu_teacher_forced(dm, cfg, ref.z, x["z"], P.schedule_from_lifetimes(S, cfg.T))
    errs = [rel_err(g, r) for g, r in zip(got, ref.z)]
    print(name, "branch units, frozen runs, per-step error", ["%.2e" % e for e in errs])
    assert max(errs) <= TOL[cfg.dtype], errs
    dm.close()


@pytest.mark.parametrize("name", ["tiny_ragged", "llada_mini", "uvit_mini"])
def test_branch_drift_policy(P, name):
    """The causal drift policy over branch units: exact selection on the GPU's drift values,
    the reduction against the recorded branch inputs, the masked steps teacher-forced."""
    import torch
    cfg, w, x = workload(name)
    dm = P.DeviceModel(cfg, w, x, granularity="branch")
    U, M, d = dm.n_units, cfg.M, cfg.d
    _, _, bs = oracle_schedule(cfg, w, cfg.budgets[-1], granularity="branch")
    sched = P.schedule_from_lifetimes(bs.lifetimes, cfg.T)
    mask = osch.active_mask(bs.lifetimes, cfg.T)
    z = torch.from_numpy(x["z"].copy()).cuda()
    cache = P.Cache(dm)
    cache.reset()
    buf = dm.drift_buffer()
    slot = (M * d * 4 + 255) // 256 * 256 // 4
    rows, drifts, snaps = [], [], []
    for s in range(1, cfg.T + 1):
        row, dr = dm.drift_step(z, s, sched, cache, buf)
        torch.cuda.synchronize()
        rows.append(row)
        drifts.append(dr)
        f = buf[: U * slot * 4].view(torch.float32).view(U, slot)[:, : M * d]
        snaps.append(f.cpu().numpy().astype(np.float64))
    assert rows[0].tolist() == [1] * U
    for s in range(2, cfg.T + 1):
        m_s = int(mask[s - 1].sum())
        assert np.array_equal(rows[s - 1], od.select(drifts[s - 1], m_s)), s
    for s in range(3, cfg.T + 1):
        want = [od.drift(snaps[s - 2][j], snaps[s - 3][j]) for j in range(U)]
        assert np.allclose(drifts[s - 1], want, rtol=1e-11, atol=0), s
    model = om.Model(cfg, w, x, granularity="branch")
    ref = od.trajectory(model, x["z"], mask, forced_rows=np.array(rows))
    cache = P.Cache(dm)
    cache.reset()
    zt = torch.empty(x["z"].shape, dtype=torch.float32, device="cuda")
    errs = []
    for s in range(1, cfg.T + 1):
        src = x["z"] if s == 1 else ref.z[s - 2]
        zt.copy_(torch.from_numpy(np.ascontiguousarray(src, dtype=np.float32)))
        dm.step_masked(zt, s, rows[s - 1], cache)
        errs.append(rel_err(zt.cpu().numpy().astype(np.float64), ref.z[s - 1]))
    print(name, "branch units, drift teacher-forced errors", ["%.2e" % e for e in errs])
    assert max(errs) <= TOL[cfg.dtype], errs
    dm.close()


@pytest.mark.parametrize("granularity", ["block", "branch"])
@pytest.mark.parametrize("pattern", ["tail_active", "alternating_long"])
def test_runs_longer_than_one_launch(P, granularity, pattern):
    """Frozen runs longer than the 32 updates one launch takes (40 blocks, 80 branch units):
    the launcher splits them, launches the full segments on their own and hands the last one
    to the next active unit's pre-norm; fp32 teacher-forced against the oracle (1e-4)."""
    cfg = synth.get_config("tiny_ragged", L=40)
    w, x = synth.model_weights(cfg), synth.inputs(cfg)
    dm = P.DeviceModel(cfg, w, x, granularity=granularity)
    U = dm.n_units
    if pattern == "tail_active":
        S = np.ones(U, int)
        S[-1] = cfg.T
    else:
        S = np.array([cfg.T if j in (0, 37, 38, U - 1) else 1 for j in range(U)])
    mask = osch.active_mask(S, cfg.T)
    ref = oracle_trajectory(cfg, w, x, mask, granularity=granularity)
    got = gpu_teacher_forced(dm, cfg, ref.z, x["z"], P.schedule_from_lifetimes(S, cfg.T))
    errs = [rel_err(g, r) for g, r in zip(got, ref.z)]
    print(granularity, pattern, "per-step error", ["%.2e" % e for e in errs])
    assert max(errs) <= TOL["f32"], errs
    dm.close()
