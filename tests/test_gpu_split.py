"""GPU parity of the split MLP output GEMM: where one round of 128 x 128 tiles is the best unsplit
plan of a long-K output GEMM (K >= 8192; the LLaDA-8B shape), the launcher runs it in two K
ranges into fp32 partial products and the next unit's pre-norm adds them to the stream, unless
the next unit is frozen or the step stores the unit's cached update.  A LLaDA-shaped stack with
an 8192-wide MLP takes that path; teacher-forced against the oracle and all-active against the
unscheduled forward bit for bit."""
import numpy as np
import pytest

import synth
from oracle import schedule as osch

from helpers import TOL, gpu_teacher_forced, gpu_trajectory, oracle_trajectory, rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_29505_amd as P
    P.lib()
    return P


@pytest.fixture(scope="module")
def wide():
    # 200 tokens x d = 256: the 256 x 8192 output GEMM's best unsplit plan is one round of
    # 128 x 128 tiles, so it runs as two K ranges of 256 x 128 tiles
    cfg = synth.get_config("llada_mini", F=8192, T=6)
    return cfg, synth.model_weights(cfg), synth.inputs(cfg)


@pytest.mark.parametrize("granularity", ["block", "branch"])
def test_split_output_gemm_teacher_forced(P, wide, granularity):
    """Every fourth unit lives two steps: before that the units ahead of it take the split
    product, afterwards they do not (a frozen unit follows) and the frozen unit folds into the
    next pre-norm; the stores of cached updates at s = S_l take the unsplit epilogue.  Per-step
    error against the oracle."""
    cfg, w, x = wide
    dm = P.DeviceModel(cfg, w, x, granularity=granularity)
    U = dm.n_units
    S = np.array([cfg.T if j % 4 != 1 else 2 for j in range(U)])
    mask = osch.active_mask(S, cfg.T)
    ref = oracle_trajectory(cfg, w, x, mask, granularity=granularity)
    got = gpu_teacher_forced(dm, cfg, ref.z, x["z"], P.schedule_from_lifetimes(S, cfg.T))
    errs = [rel_err(g, r) for g, r in zip(got, ref.z)]
    print(granularity, "split output GEMM, teacher-forced per-step error", ["%.2e" % e for e in errs])
    assert max(errs) <= TOL["bf16"], errs
    dm.close()


def test_split_output_gemm_all_active_is_unscheduled(P, wide):
    cfg, w, x = wide
    dm = P.DeviceModel(cfg, w, x)
    a = gpu_trajectory(dm, cfg, x, P.schedule_from_lifetimes([cfg.T] * cfg.L, cfg.T), 3)
    b = gpu_trajectory(dm, cfg, x, None, 3)
    dm.close()
    for za, zb in zip(a, b):
        assert np.array_equal(za, zb)


def test_split_output_gemm_graph_replays_equal_eager(P, wide):
    """The split product and its partial-adding pre-norm captured in a whole-trajectory HIP
    graph: two replays, with eager work between them, equal the eager trajectory bit for bit."""
    import torch
    cfg, w, x = wide
    dm = P.DeviceModel(cfg, w, x)
    S = np.array([cfg.T, 2, cfg.T, cfg.T])
    sched = P.schedule_from_lifetimes(S, cfg.T)
    eager = gpu_trajectory(dm, cfg, x, sched)[-1]
    stream = torch.cuda.Stream()
    z0 = torch.from_numpy(x["z"].copy()).cuda()
    z = torch.empty_like(z0)
    cache = P.Cache(dm)
    with torch.cuda.stream(stream):
        g = dm.capture(z, sched, cache, stream)
    other = torch.from_numpy(x["z"].copy()).cuda()
    for rep in range(2):
        with torch.cuda.stream(stream):
            z.copy_(z0)
            g.launch(stream)
        stream.synchronize()
        assert np.array_equal(z.cpu().numpy().astype(np.float64), eager), rep
        c2 = P.Cache(dm)
        c2.reset()
        dm.step(other, 1, sched, c2)
        torch.cuda.synchronize()
    g.close()
    dm.close()
