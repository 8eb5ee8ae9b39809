"""Shared helpers of the test suite: run the oracle and the HIP path on the same seeded inputs."""
from __future__ import annotations

import numpy as np

import synth
from oracle import model as om
from oracle import schedule as osch
from oracle import spectral as osp

TOL = {"f32": 1e-4, "bf16": 2e-2}
# Ceiling of the free-running bf16 trajectory bound: the bound follows the oracle's own
# divergence under tiny input perturbations (the bf16-quantised trajectory map is chaotic),
# but never exceeds this.
FREE_RUNNING_CEIL = 8e-2


def load_fullsize_golden(name):
    """The oracle's statistics of every scored matrix of a full-size workload and its unit
    raw scores, as written by tests/golden/make_fullsize_scores.py.
    Returns (stats: list over units of {role: MatrixStats}, raw: float64 [L])."""
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", f"fullsize_{name}.txt")
    stats, raw = [], []
    for line in open(path):
        f = line.split()
        if not f or f[0].startswith("#"):
            continue
        if f[0] == "mat":
            u, role, m, n = int(f[1]), f[2], int(f[3]), int(f[4])
            e_top, e_tail, frob, s1, g = map(float, f[5:10])
            while len(stats) <= u:
                stats.append({})
            a, b = e_top + 1e-6 * frob, e_tail + 1e-6 * frob
            stats[u][role] = osp.MatrixStats(m, n, osp.rank_k(m, n), e_top, e_tail, frob,
                                             float(np.log(a / b)) if b > 0 else float("inf"), g, s1)
        elif f[0] == "raw":
            assert int(f[1]) == len(raw)
            raw.append(float(f[2]))
    return stats, np.array(raw, np.float64)


def rel_err(x: np.ndarray, ref: np.ndarray) -> float:
    """max_i |x_i - ref_i| / max_i |ref_i|  (the error metric of the parity gate)."""
    ref = np.asarray(ref, np.float64)
    return float(np.max(np.abs(np.asarray(x, np.float64) - ref)) / max(np.max(np.abs(ref)), 1e-30))


def unit_raw_scores(cfg, weights, granularity="block"):
    """The oracle's raw score q~ of every scheduled unit: per block, or per residual branch."""
    raw = []
    for u in weights:
        mats = osp.unit_matrices(u, cfg.d, cfg.dtype)
        if granularity == "branch":
            raw += [osp.unit_score(osp.branch_matrices(mats, b), cfg.dh).raw for b in om.branches(cfg.arch)]
        else:
            raw.append(osp.unit_score(mats, cfg.dh).raw)
    return np.array(raw)


def oracle_schedule(cfg, weights, pct, granularity="block"):
    raw = unit_raw_scores(cfg, weights, granularity)
    lam = osp.normalise(raw)
    n = osch.budget_layer_steps(pct, len(raw), cfg.T)
    bs = osch.lifetimes_budget(lam, cfg.T, n, osch.s_min_default(cfg.T))
    return raw, lam, bs


def oracle_trajectory(cfg, weights, inputs, mask, steps=None, granularity="block"):
    m = om.Model(cfg, weights, inputs, granularity=granularity)
    return om.trajectory(m, inputs["z"], mask, steps)


def gpu_trajectory(dm, cfg, inputs, sched, steps=None, cache=None):
    """Run steps 1..steps on the GPU; returns the list of z after each step (host float64)."""
    import torch
    z = torch.from_numpy(inputs["z"].copy()).cuda()
    steps = cfg.T if steps is None else steps
    if sched is not None and cache is None:
        from paper_2609_29505_amd import Cache
        cache = Cache(dm)
    if cache is not None:
        cache.reset()
    out = []
    for s in range(1, steps + 1):
        dm.step(z, s, sched, cache)
        out.append(z.cpu().numpy().astype(np.float64))
    torch.cuda.synchronize()
    return out


def gpu_teacher_forced(dm, cfg, oracle_z, z0, sched):
    """Step s of the GPU path fed the oracle's state z_s (its own cache carries over).

    Returns the GPU's z_{s+1} for s = 1..T, each to compare with the oracle's z_{s+1}: the
    per-step implementation error, without the amplification of earlier differences by the
    trajectory map.
    """
    import torch
    from paper_2609_29505_amd import Cache
    cache = Cache(dm)
    cache.reset()
    out = []
    z = torch.empty(z0.shape, dtype=torch.float32, device="cuda")
    for s in range(1, cfg.T + 1):
        src = z0 if s == 1 else oracle_z[s - 2]
        z.copy_(torch.from_numpy(np.ascontiguousarray(src, dtype=np.float32)))
        dm.step(z, s, sched, cache)
        out.append(z.cpu().numpy().astype(np.float64))
    return out


def chaos_floor(cfg, weights, inputs, mask, rels=(1e-7, 1e-5), seeds=(1, 2), granularity="block"):
    """Divergence of the oracle from itself when its initial state is perturbed (relative
    perturbations `rels`, seeded): the sensitivity of the bf16-quantised trajectory map.
    Returns the unperturbed trajectory and, per step, the largest divergence observed."""
    a = oracle_trajectory(cfg, weights, inputs, mask, granularity=granularity)
    floor = [0.0] * len(a.z)
    for rel in rels:
        for seed in seeds:
            x2 = dict(inputs)
            rng = np.random.default_rng(seed)
            x2["z"] = (inputs["z"] * (1 + rel * rng.standard_normal(inputs["z"].shape))).astype(np.float32)
            b = oracle_trajectory(cfg, weights, x2, mask, granularity=granularity)
            floor = [max(f, rel_err(p, q)) for f, p, q in zip(floor, b.z, a.z)]
    return a, floor
