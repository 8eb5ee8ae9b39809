"""Pins for branch-granular scheduling in the oracle: every pre-norm residual branch of a block
is a scheduled unit of its own (Sec. 3.1's residual units taken at branch level; Alg. 2 walks
them in stack order).  Block l's branches are units l * nb + k in execution order."""
import numpy as np
import pytest

import synth
from oracle import drift as odr
from oracle import model as om
from oracle import schedule as sch
from oracle import spectral as sp


def load(name, **kw):
    cfg = synth.get_config(name, **kw)
    return cfg, synth.model_weights(cfg), synth.inputs(cfg)


def test_branches_per_architecture():
    assert om.branches("tiny") == ("attn", "mlp")
    assert om.branches("llada") == ("attn", "mlp")
    assert om.branches("dit") == ("attn", "mlp")
    assert om.branches("uvit") == ("attn", "mlp")
    assert om.branches("sdxl") == ("attn", "xattn", "mlp")
    assert om.branches("sdxl_unet") == ("resnet", "attn", "xattn", "mlp")
    cfg, w, x = load("sdxl_mini")
    m = om.Model(cfg, w, x, granularity="branch")
    assert m.nb == 3 and m.n_units == 3 * cfg.L
    assert om.Model(cfg, w, x).n_units == cfg.L
    with pytest.raises(ValueError):
        om.Model(cfg, w, x, granularity="layer")


@pytest.mark.parametrize("name", ["tiny_ragged", "dit_mini", "uvit_mini", "sdxl_mini", "sdxl_unet_mini"])
def test_all_active_branch_units_equal_unscheduled(name):
    """Every branch active reproduces the unscheduled forward bit for bit, as block units do."""
    cfg, w, x = load(name)
    m = om.Model(cfg, w, x, granularity="branch")
    ones = np.ones((cfg.T, m.n_units), np.uint8)
    a = om.trajectory(m, x["z"], ones, steps=2)
    b = om.trajectory(om.Model(cfg, w, x), x["z"], None, steps=2)
    for za, zb in zip(a.z, b.z):
        assert np.array_equal(za, zb)


@pytest.mark.parametrize("name", ["llada_mini", "sdxl_unet_mini"])
def test_branch_caches_are_the_branch_outputs(name):
    """After an all-active step the cached update of branch unit (l, k) is that branch's output:
    the stream advances by exactly it, and a block's branch updates summed in execution order
    give the block unit's cached update bit for bit."""
    cfg, w, x = load(name)
    mb = om.Model(cfg, w, x, granularity="branch")
    mk = om.Model(cfg, w, x)
    cross = [mb.cross_kv(u) for u in mb.units] if cfg.arch in om.CROSS_ARCHS else None
    cb, ck, inputs = {}, {}, {}
    eps_b = om.denoise_step(mb, x["z"], 1, [1] * mb.n_units, cb, cross, unit_inputs=inputs)
    eps_k = om.denoise_step(mk, x["z"], 1, [1] * cfg.L, ck, cross)
    assert np.array_equal(eps_b, eps_k)
    nb = mb.nb
    for l in range(cfg.L):
        total = cb[l * nb]
        for k in range(1, nb):
            total = total + cb[l * nb + k]
        assert np.array_equal(total, ck[l])
        for k in range(nb - 1):
            j = l * nb + k
            assert np.array_equal(inputs[j] + cb[j], inputs[j + 1])


def test_frozen_branch_adds_its_cached_update():
    """A frozen branch unit adds its own cached update to the current stream and nothing else:
    with the MLP branches of two blocks frozen, every other branch still runs on the stream."""
    cfg, w, x = load("llada_mini")
    m = om.Model(cfg, w, x, granularity="branch")
    U = m.n_units
    cache, inputs = {}, {}
    om.denoise_step(m, x["z"], 1, [1] * U, cache)
    z2 = np.array(x["z"], np.float64) * 0.5
    row = np.ones(U, np.uint8)
    frozen = [1 * 2 + 1, 2 * 2 + 1]  # the MLP branches of blocks 1 and 2
    row[frozen] = 0
    stale = {j: cache[j].copy() for j in range(U)}
    om.denoise_step(m, z2, 2, row, cache, unit_inputs=inputs)
    for j in frozen:
        assert np.array_equal(cache[j], stale[j])  # read, not refreshed
        assert np.array_equal(inputs[j] + stale[j], inputs[j + 1])
    # every active branch refreshed its slot on the new stream
    for j in range(U):
        if j not in frozen:
            assert not np.array_equal(cache[j], stale[j])


def test_equal_branch_lifetimes_match_block_units():
    """Branch lifetimes equal within each block give the block schedule's trajectory up to the
    order of the additions (h + a + m against h + (a + m) for a frozen block)."""
    cfg, w, x = load("tiny_ragged")
    mk = om.Model(cfg, w, x)
    mb = om.Model(cfg, w, x, granularity="branch")
    S = np.array([cfg.T, 2, 5, 1][:cfg.L])
    mask_k = sch.active_mask(S, cfg.T)
    mask_b = sch.active_mask(np.repeat(S, mb.nb), cfg.T)
    a = om.trajectory(mk, x["z"], mask_k)
    b = om.trajectory(mb, x["z"], mask_b)
    for za, zb in zip(a.z, b.z):
        assert np.allclose(za, zb, rtol=0, atol=1e-12 * np.abs(za).max())


@pytest.mark.parametrize("name", ["llada_mini", "sdxl_mini", "sdxl_unet_mini"])
def test_branch_scores_sum_to_the_block_score(name):
    """Eq. app-block-score sums the block's component scores: the branch units' raw scores
    (one component each; a ResNet branch both of its convolutions) add up to the block's."""
    cfg, w, _ = load(name)
    for u in w:
        mats = sp.unit_matrices(u, cfg.d, cfg.dtype)
        block = sp.unit_score(mats, cfg.dh).raw
        parts = [sp.unit_score(sp.branch_matrices(mats, b), cfg.dh).raw for b in om.branches(cfg.arch)]
        assert all(p > 0 for p in parts)
        assert sum(parts) == pytest.approx(block, rel=1e-14)


def test_drift_policy_over_branch_units():
    """The causal drift policy ranks branch units: m_s of the U = nb L units each step, the
    first step full, and each branch unit's input is the stream arriving at that branch."""
    cfg, w, x = load("tiny_ragged")
    m = om.Model(cfg, w, x, granularity="branch")
    U = m.n_units
    S = np.array([cfg.T, 2, 5, 1, 3, cfg.T, 4, 2][:U])
    static = sch.active_mask(S, cfg.T)
    tr = odr.trajectory(m, x["z"], static, steps=5)
    assert tr.active[0].tolist() == [1] * U
    for s in range(5):
        assert int(tr.active[s].sum()) == int(static[s].sum())
        assert tr.drift[s].shape == (U,)
