"""The allocation-free step entry point (sgd_denoise_step_noalloc): its output against the
workspace entry point's (sgd_denoise_step), bit for bit, on two calls in a row, the second
on a smaller workload; and its refusal of a workload whose workspace exceeds the scratch."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_29505_amd as P
    P.lib()
    return P


def _trajectory(P, dm, cfg, x, sched, noalloc):
    import torch
    z = torch.from_numpy(x["z"].copy()).cuda()
    cache = P.Cache(dm)
    cache.reset()
    out = []
    for s in range(1, cfg.T + 1):
        (dm.step_noalloc if noalloc else dm.step)(z, s, sched, cache)
        out.append(z.cpu().numpy())
    torch.cuda.synchronize()
    return out


def test_noalloc_matches_workspace_entry_point(P):
    # first call: the reduced LLaDA-shaped workload; second: a smaller (fp32 tiny) one
    for name in ("llada_mini", "tiny_ragged"):
        cfg = synth.get_config(name)
        w, x = synth.model_weights(cfg), synth.inputs(cfg)
        dm = P.DeviceModel(cfg, w, x)
        sched = P.schedule_from_lifetimes([1 + (l * 5) % cfg.T for l in range(cfg.L)], cfg.T)
        a = _trajectory(P, dm, cfg, x, sched, noalloc=False)
        b = _trajectory(P, dm, cfg, x, sched, noalloc=True)
        for s, (za, zb) in enumerate(zip(a, b)):
            assert np.array_equal(za, zb), (name, s + 1)
        dm.close()


def test_noalloc_full_size_llada_first_steps(P):
    """The LLaDA-8B-shaped workload's workspace fits the scratch: its first two steps agree
    bit for bit with the workspace entry point."""
    import torch
    cfg = synth.get_config("llada")
    w, x = synth.model_weights(cfg, workers=16), synth.inputs(cfg)
    dm = P.DeviceModel(cfg, w, x)
    assert dm.workspace_bytes <= 96 * 1024 * 1024
    S = [1 if l % 2 else cfg.T for l in range(cfg.L)]
    sched = P.schedule_from_lifetimes(S, cfg.T)
    outs = []
    for noalloc in (False, True):
        z = torch.from_numpy(x["z"].copy()).cuda()
        cache = P.Cache(dm)
        cache.reset()
        for s in (1, 2):
            (dm.step_noalloc if noalloc else dm.step)(z, s, sched, cache)
        outs.append(z.cpu().numpy())
        del cache
    assert np.array_equal(outs[0], outs[1])
    dm.close()


def test_noalloc_refuses_large_workspace(P):
    import torch
    cfg = synth.get_config("dit_mini", B=100)
    dm = P.DeviceModel(cfg, synth.model_weights(cfg), synth.inputs(cfg))
    assert dm.workspace_bytes > 96 * 1024 * 1024
    z = torch.zeros((cfg.B, cfg.N, cfg.d), dtype=torch.float32, device="cuda")
    with pytest.raises(P.SgdError) as e:
        dm.step_noalloc(z, 1, None, None)
    assert e.value.code == -1 and "scratch" in str(e.value)
    dm.close()
