"""A whole scheduled trajectory captured as one HIP graph (sgd_graph_capture) and replayed:
every replay equals the eager trajectory bit for bit, with eager work of the program itself
and synchronisations between the replays."""
import numpy as np
import pytest

import synth
from oracle import schedule as osch

from helpers import gpu_trajectory, oracle_schedule

pytestmark = pytest.mark.gpu

_cache = {}


def workload(name):
    if name not in _cache:
        cfg = synth.get_config(name)
        _cache[name] = (cfg, synth.model_weights(cfg), synth.inputs(cfg))
    return _cache[name]


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_29505_amd as P
    P.lib()
    return P


@pytest.mark.parametrize("name,granularity", [("tiny_ragged", "block"), ("llada_mini", "block"),
                                              ("dit_mini", "block"), ("uvit_mini", "block"),
                                              ("sdxl_mini", "block"), ("sdxl_unet_mini", "block"),
                                              ("llada_mini", "branch"), ("sdxl_mini", "branch")])
def test_graph_replays_equal_eager(P, name, granularity):
    import torch
    cfg, w, x = workload(name)
    dm = P.DeviceModel(cfg, w, x, granularity=granularity)
    _, _, bs = oracle_schedule(cfg, w, cfg.budgets[-1], granularity=granularity)
    sched = P.schedule_from_lifetimes(bs.lifetimes, cfg.T)
    eager = gpu_trajectory(dm, cfg, x, sched)[-1]  # z after step T
    eager_un = gpu_trajectory(dm, cfg, x, None)[-1]
    stream = torch.cuda.Stream()
    z0 = torch.from_numpy(x["z"].copy()).cuda()
    z = torch.empty_like(z0)
    cache = P.Cache(dm)
    with torch.cuda.stream(stream):
        g = dm.capture(z, sched, cache, stream)
        gu = dm.capture(z, None, None, stream)
    other = torch.from_numpy(x["z"].copy()).cuda()
    for rep in range(3):
        with torch.cuda.stream(stream):
            z.copy_(z0)
            g.launch(stream)
        stream.synchronize()
        assert np.array_equal(z.cpu().numpy().astype(np.float64), eager), rep
        # eager work between replays: a library trajectory on another state, torch ops
        c2 = P.Cache(dm)
        c2.reset()
        for s in range(1, 3):
            dm.step(other, s, sched, c2)
        other.mul_(1.0001)
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            z.copy_(z0)
            gu.launch(stream)
        stream.synchronize()
        assert np.array_equal(z.cpu().numpy().astype(np.float64), eager_un), rep
    g.close()
    gu.close()
    dm.close()


def test_graph_capture_errors(P):
    import torch
    cfg, w, x = workload("llada_mini")
    dm = P.DeviceModel(cfg, w, x)
    z = torch.from_numpy(x["z"].copy()).cuda()
    sched = P.schedule_from_lifetimes([cfg.T] * cfg.L, cfg.T)
    stream = torch.cuda.Stream()
    with pytest.raises(P.SgdError) as e:
        dm.capture(z, sched, None, stream)  # a schedule needs a cache
    assert e.value.code == -1
    bad = P.schedule_from_lifetimes([cfg.T] * (cfg.L + 1), cfg.T)
    with pytest.raises(P.SgdError):
        with torch.cuda.stream(stream):
            dm.capture(z, bad, P.Cache(dm), stream)  # wrong unit count: refused inside capture
    # the stream is usable afterwards: a valid capture and launch still work
    cache = P.Cache(dm)
    with torch.cuda.stream(stream):
        g = dm.capture(z, sched, cache, stream)
        g.launch(stream)
    stream.synchronize()
    assert np.isfinite(z.cpu().numpy()).all()
    g.close()
    dm.close()
