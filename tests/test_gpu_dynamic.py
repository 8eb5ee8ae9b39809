"""GPU parity of the input-aware baselines (appendix "Protocol Details", "Dynamic
baselines") through the C ABI: the masked step with non-nested active sets, the causal
activation-drift policy and the oracle-replay search, against the oracle."""
import numpy as np
import pytest

import synth
from oracle import drift as od
from oracle import model as om
from oracle import replay as orp
from oracle import schedule as osch

from helpers import TOL, oracle_schedule, rel_err

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


def workload(name, **kw):
    key = (name, tuple(sorted(kw.items())))
    if key not in _cache:
        cfg = synth.get_config(name, **kw)
        _cache[key] = (cfg, synth.model_weights(cfg), synth.inputs(cfg))
    return _cache[key]


def gpu_drift_run(P, dm, cfg, x, sched):
    """Free-running drift-policy trajectory; per step the row, the lagged drift, z, and the
    recorded unit inputs (the drift buffer's slots) after the step."""
    import torch
    L, M, d = cfg.L, cfg.M, cfg.d
    z = torch.from_numpy(x["z"].copy()).cuda()
    cache = P.Cache(dm)
    cache.reset()
    buf = dm.drift_buffer()
    slot = (M * d * 4 + 255) // 256 * 256 // 4
    rows, drifts, zs, snaps = [], [], [], []
    for s in range(1, cfg.T + 1):
        row, dr = dm.drift_step(z, s, sched, cache, buf)
        torch.cuda.synchronize()
        rows.append(row)
        drifts.append(dr)
        zs.append(z.cpu().numpy().astype(np.float64))
        f = buf[: L * slot * 4].view(torch.float32).view(L, slot)[:, : M * d]
        snaps.append(f.cpu().numpy().astype(np.float64))
    return rows, drifts, zs, snaps


@pytest.mark.parametrize("name", MINIS)
def test_drift_policy(P, name):
    """Selection (exact host logic), the drift reduction (on the GPU's own recorded inputs)
    and the masked steps the policy runs (teacher-forced against the oracle)."""
    import torch
    cfg, w, x = workload(name)
    dm = P.DeviceModel(cfg, w, x)
    pct = cfg.budgets[-1]
    _, _, bs = oracle_schedule(cfg, w, pct)
    sched = P.schedule_from_lifetimes(bs.lifetimes, cfg.T)
    mask = osch.active_mask(bs.lifetimes, cfg.T)
    rows, drifts, zs, snaps = gpu_drift_run(P, dm, cfg, x, sched)
    # selection: step 1 full, m_s units, the oracle's top-m rule on the GPU's drift values
    assert rows[0].tolist() == [1] * cfg.L
    for s in range(2, cfg.T + 1):
        m_s = int(mask[s - 1].sum())
        assert int(rows[s - 1].sum()) == m_s
        assert np.array_equal(rows[s - 1], od.select(drifts[s - 1], m_s)), s
    assert np.all(drifts[1] == 0)
    # the reduction: d_{l,s-1} from the unit inputs recorded at steps s-1 and s-2
    for s in range(3, cfg.T + 1):
        want = [od.drift(snaps[s - 2][l], snaps[s - 3][l]) for l in range(cfg.L)]
        assert np.allclose(drifts[s - 1], want, rtol=1e-11, atol=0), s
    # the steps: oracle trajectory on the GPU's rows, GPU masked steps fed the oracle's states
    ref = od.trajectory(om.Model(cfg, w, x), x["z"], mask, forced_rows=np.array(rows))
    cache = P.Cache(dm)
    cache.reset()
    zt = torch.empty(x["z"].shape, dtype=torch.float32, device="cuda")
    errs = []
    for s in range(1, cfg.T + 1):
        src = x["z"] if s == 1 else ref.z[s - 2]
        zt.copy_(torch.from_numpy(np.ascontiguousarray(src, dtype=np.float32)))
        dm.step_masked(zt, s, rows[s - 1], cache)
        errs.append(rel_err(zt.cpu().numpy().astype(np.float64), ref.z[s - 1]))
    print(name, "drift rows", [r.tolist() for r in rows], "teacher-forced errors", ["%.2e" % e for e in errs])
    assert max(errs) <= TOL[cfg.dtype], errs
    if cfg.dtype == "f32":
        # fp32: the oracle's own policy makes the same choices and the states agree
        own = od.trajectory(om.Model(cfg, w, x), x["z"], mask)
        for s in range(cfg.T):
            assert np.array_equal(own.active[s], rows[s])
            assert rel_err(zs[s], own.z[s]) <= TOL["f32"]
    dm.close()


def test_masked_step_errors(P):
    import torch
    cfg, w, x = workload("llada_mini")
    dm = P.DeviceModel(cfg, w, x)
    z = torch.from_numpy(x["z"].copy()).cuda()
    cache = P.Cache(dm)
    cache.reset()
    row = np.ones(cfg.L, np.uint8)
    row[1] = 0
    with pytest.raises(P.SgdError) as e:
        dm.step_masked(z, 1, row, cache)  # unit 1 frozen before any update exists
    assert e.value.code == -6
    dm.step_masked(z, 1, np.ones(cfg.L, np.uint8), cache)
    with pytest.raises(P.SgdError) as e:
        dm.step_masked(z, 3, row, cache)  # out of order
    assert e.value.code == -5
    dm.step_masked(z, 2, row, cache)
    torch.cuda.synchronize()
    dm.close()


def _margins_ok(log, rel=1e-4):
    """Every round's least deviation is separated from the next and from tau by > rel."""
    by_round = {}
    for (s, r, j), v in log.items():
        by_round.setdefault((s, r), []).append(v)
    for vals in by_round.values():
        v = sorted(vals)
        if len(v) > 1 and v[1] - v[0] <= rel * v[1]:
            return False
    return True


@pytest.mark.parametrize("name,ceiling_pct", [("tiny_ragged", 50), ("tiny", 50), ("tiny", 0)])
def test_replay_search_fp32(P, name, ceiling_pct):
    """fp32 workloads: the GPU search makes the oracle's decisions (lifetimes bit for bit)
    and measures its deviations to 1e-5."""
    import torch
    cfg, w, x = workload(name)
    ceiling = osch.budget_layer_steps(ceiling_pct, cfg.L, cfg.T) if ceiling_pct else 0
    ref = orp.search(om.Model(cfg, w, x), x["z"], tau_agree=5e-3, max_layer_steps=ceiling)
    assert _margins_ok(ref.log), "near-tie: the decisions below would be fragile"
    dm = P.DeviceModel(cfg, w, x)
    z1 = torch.from_numpy(x["z"].copy()).cuda()
    life, evals, dlog = dm.replay_search(z1, tau_agree=5e-3, max_layer_steps=ceiling, log=True)
    print(name, "replay lifetimes", life.tolist(), "oracle", ref.lifetimes.tolist(), "evaluations", evals)
    assert life.tolist() == ref.lifetimes.tolist()
    assert evals == ref.evaluations
    for (s, r, j), v in ref.log.items():
        assert dlog[s - 1, r, j] == pytest.approx(v, rel=1e-5, abs=1e-9), (s, r, j)
    assert int(np.isfinite(dlog).sum()) == len(ref.log)
    assert np.array_equal(z1.cpu().numpy(), x["z"])  # z_1 untouched
    dm.close()


def test_replay_inert_units(P):
    """Units whose branches are identically zero freeze at deviation exactly 0 (tau = 0)."""
    import torch
    cfg, w, x = workload("tiny_ragged")
    w = [dict(u) for u in w]
    for l in (0, 2):
        for key in ("w_o", "w2"):
            w[l][key] = np.zeros_like(w[l][key])
    dm = P.DeviceModel(cfg, w, x)
    life, _, dlog = dm.replay_search(torch.from_numpy(x["z"].copy()).cuda(), tau_agree=0.0, log=True)
    assert life.tolist() == [1, cfg.T, 1]
    assert dlog[1, 0, 0] == 0.0 and dlog[1, 0, 2] == 0.0 and dlog[1, 0, 1] > 0
    dm.close()


@pytest.mark.parametrize("name", ["llada_mini", "sdxl_mini"])
def test_replay_search_bf16(P, name):
    """bf16: the decisions follow from the GPU's own measured deviations (exact host logic),
    the ceiling holds, and the first round's deviations match the oracle's at step 2."""
    import torch
    cfg, w, x = workload(name)
    L, T = cfg.L, cfg.T
    ceiling = osch.budget_layer_steps(cfg.budgets[-1], L, T)
    dm = P.DeviceModel(cfg, w, x)
    life, evals, dlog = dm.replay_search(torch.from_numpy(x["z"].copy()).cuda(), tau_agree=5e-3,
                                         max_layer_steps=ceiling, log=True)
    active = int(sum(np.sum(np.arange(1, T + 1) <= S) for S in life))
    assert active <= ceiling
    frozen = np.zeros(L, bool)
    spent = L
    for s in range(2, T + 1):
        r = 0
        while not frozen.all():
            cand = [j for j in range(L) if not frozen[j]]
            vals = dlog[s - 1, r, cand]
            assert np.all(np.isfinite(vals))
            best = cand[int(np.argmin(vals))]
            planned = spent + (T - s + 1) * (L - frozen.sum())
            if vals.min() > 5e-3 and planned <= ceiling:
                break
            assert life[best] == s - 1
            frozen[best] = True
            r += 1
        spent += L - int(frozen.sum())
    ref = orp.search(om.Model(cfg, w, x), x["z"], tau_agree=5e-3, max_layer_steps=ceiling)
    got = np.array([dlog[1, 0, j] for j in range(L)])
    want = np.array([ref.log[(2, 0, j)] for j in range(L)])
    print(name, "step-2 deviations gpu", got, "oracle", want)
    assert np.allclose(got, want, rtol=0.1, atol=1e-3)
    dm.close()
