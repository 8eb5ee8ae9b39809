"""bench.py's frozen-path accounting against the launches the library actually makes.

`frozen_launches` predicts, from a schedule's active mask, every frozen-run launch and every
pre-norm that absorbs a frozen run, of a
step (maximal runs of frozen units, at most 32, ended by U-ViT out-blocks); the library's
own profiler counts the frozen-run launches of the same steps.
"""
import os
import sys

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_29505_amd as P
    P.lib()
    return P


@pytest.mark.parametrize("name", ["llada_mini", "uvit_mini", "dit_mini", "sdxl_unet_mini"])
def test_frozen_launch_count(P, name):
    import torch

    import bench

    cfg = synth.get_config(name)
    w, x = synth.model_weights(cfg), synth.inputs(cfg)
    dm = P.DeviceModel(cfg, w, x)
    rng = np.random.default_rng(5)
    # lifetimes with frozen runs of every length, including units frozen from step 2 on
    lifetimes = rng.integers(1, cfg.T + 1, size=cfg.L)
    lifetimes[: cfg.L // 2] = 1
    sched = P.schedule_from_lifetimes(lifetimes, cfg.T)
    z = torch.from_numpy(x["z"].copy()).cuda()
    cache = P.Cache(dm)
    counts = {}
    for kclass in ("frozen", "fold"):
        cache.reset()
        z.copy_(torch.from_numpy(x["z"]))
        dm.profile_begin(kclass, 4096)
        for s in range(1, cfg.T + 1):
            dm.step(z, s, sched, cache)
        torch.cuda.synchronize()
        counts[kclass] = dm.profile_end()[1]
    act = np.asarray(sched.active, bool)
    launches = [bench.frozen_launches(cfg, act[s]) for s in range(cfg.T)]
    assert counts["frozen"] == sum(len(a) for a, _ in launches)
    assert counts["fold"] == sum(len(f) for _, f in launches)
    assert counts["frozen"] + counts["fold"] > 0
    dm.close()
