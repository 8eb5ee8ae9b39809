"""Pins for the oracle's units, jagged step and sampler (Sec. 3.1, Alg. 2)."""
import math

import numpy as np
import pytest

import synth
from oracle import model as om
from oracle import numerics as nu
from oracle import schedule as sch


def load(name, **kw):
    cfg = synth.get_config(name, **kw)
    w = synth.model_weights(cfg)
    x = synth.inputs(cfg)
    return cfg, w, x


# ---------------------------------------------------------------- numerics

def test_round_bf16_cases():
    # representable values are fixed points
    for v in (0.0, 1.0, -2.5, 0.15625, 3.0e38 * 0 + 65280.0):
        assert nu.round_bf16(np.array([v]))[0] == v
    one = 1.0
    ulp = 2.0 ** -7  # bf16 spacing in [1, 2)
    # exactly half-way: ties to even
    assert nu.round_bf16(np.array([one + ulp / 2]))[0] == one
    assert nu.round_bf16(np.array([one + 3 * ulp / 2]))[0] == one + 2 * ulp
    # just above half-way rounds up
    assert nu.round_bf16(np.array([one + ulp / 2 + 2 ** -20]))[0] == one + ulp
    assert nu.round_bf16(np.array([-(one + ulp / 2 + 2 ** -20)]))[0] == -(one + ulp)
    # decode of raw bits
    assert nu.decode(np.array([0x3F80, 0xC000, 0x3E20], np.uint16), "bf16").tolist() == [1.0, -2.0, 0.15625]


# ---------------------------------------------------------------- elementwise

def test_norms():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((3, 5, 64)) * 4 + 1
    y = om.rmsnorm(x, np.ones(64), eps=0.0)
    assert np.allclose(np.mean(y * y, axis=-1), 1.0)
    y = om.layernorm(x, eps=0.0)
    assert np.allclose(y.mean(axis=-1), 0.0, atol=1e-12)
    assert np.allclose(y.var(axis=-1), 1.0)
    w, b = rng.standard_normal(64), rng.standard_normal(64)
    assert np.allclose(om.layernorm(x, w, b, eps=0.0), y * w + b)


def test_activations():
    xs = np.array([-3.0, -0.5, 0.0, 0.7, 2.0])
    ref = np.array([0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in xs])
    assert np.allclose(om.gelu_erf(xs), ref, rtol=1e-15, atol=1e-16)
    assert np.max(np.abs(om.gelu_tanh(xs) - ref)) < 1e-3  # tanh form approximates the erf form
    assert om.silu(np.array([0.0]))[0] == 0.0
    assert om.silu(np.array([40.0]))[0] == pytest.approx(40.0)
    assert om.silu(np.array([1.0]))[0] == pytest.approx(1.0 / (1.0 + math.exp(-1.0)), rel=1e-15)


def test_timestep_embedding():
    e = om.timestep_embedding(0.0, 8)
    assert e.tolist() == [1, 1, 1, 1, 0, 0, 0, 0]
    e = om.timestep_embedding(2.0, 4)
    assert e == pytest.approx([math.cos(2), math.cos(2 * 0.01), math.sin(2), math.sin(2 * 0.01)])
    assert om.timestep_value(1, 50) == 1000.0 and om.timestep_value(50, 50) == 20.0


def test_rope():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((1, 2, 9, 16))
    r = om.rope(x)
    assert np.allclose(r[..., 0, :], x[..., 0, :])  # position 0 is the identity
    # each (i, i + half) pair is rotated: pair norms are preserved
    n0 = x[..., :8] ** 2 + x[..., 8:] ** 2
    n1 = r[..., :8] ** 2 + r[..., 8:] ** 2
    assert np.allclose(n0, n1)
    # relative position: <rope(q)_m, rope(k)_n> depends only on m - n
    q = np.broadcast_to(rng.standard_normal(16), (1, 1, 9, 16))
    k = np.broadcast_to(rng.standard_normal(16), (1, 1, 9, 16))
    dots = np.einsum("...md,...nd->...mn", om.rope(q), om.rope(k))[0, 0]
    for delta in range(-3, 4):
        diag = np.diagonal(dots, offset=delta)
        assert np.allclose(diag, diag[0])


def test_attention_textbook_and_single_key():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 2, 5, 4))
    k = rng.standard_normal((1, 2, 7, 4))
    v = rng.standard_normal((1, 2, 7, 4))
    out = om.attention(q, k, v)
    for h in range(2):
        for i in range(5):
            logits = [sum(q[0, h, i, t] * k[0, h, j, t] for t in range(4)) / 2.0 for j in range(7)]
            mx = max(logits)
            w = [math.exp(a - mx) for a in logits]
            tot = sum(w)
            ref = [sum(w[j] / tot * v[0, h, j, t] for j in range(7)) for t in range(4)]
            assert np.allclose(out[0, h, i], ref, rtol=1e-13, atol=1e-14)
    one = om.attention(q, k[:, :, :1], v[:, :, :1])
    assert np.allclose(one, np.broadcast_to(v[:, :, :1], one.shape))


# ---------------------------------------------------------------- step semantics

@pytest.mark.parametrize("name", ["tiny_ragged", "llada_mini", "uvit_mini", "sdxl_mini"])
def test_all_active_equals_unscheduled(name):
    cfg, w, x = load(name)
    m = om.Model(cfg, w, x)
    ones = np.ones((cfg.T, cfg.L), np.uint8)
    a = om.trajectory(m, x["z"], ones, steps=3)
    b = om.trajectory(m, x["z"], None, steps=3)
    for za, zb in zip(a.z, b.z):
        assert np.array_equal(za, zb)


def _lifetimes(cfg, w, pct):
    from oracle import spectral as sp
    raw = [sp.unit_score(sp.unit_matrices(u, cfg.d, cfg.dtype), cfg.dh).raw for u in w]
    lam = sp.normalise(raw)
    n = sch.budget_layer_steps(pct, cfg.L, cfg.T)
    return sch.lifetimes_budget(lam, cfg.T, n, sch.s_min_default(cfg.T)).lifetimes


@pytest.mark.parametrize("name", ["tiny_ragged", "llada_mini", "uvit_mini"])
def test_step_one_is_unscheduled_and_cache_is_branch_sum(name):
    cfg, w, x = load(name)
    m = om.Model(cfg, w, x)
    S = _lifetimes(cfg, w, cfg.budgets[-1])
    mask = sch.active_mask(S, cfg.T)
    sched = om.trajectory(m, x["z"], mask)
    full = om.trajectory(m, x["z"], None, steps=1)
    assert np.array_equal(sched.z[0], full.z[0])
    # replay: the cached update of unit l is F_l evaluated at step S_l on the scheduled stream
    z = np.array(x["z"], np.float64)
    cache = {}
    for s in range(1, cfg.T + 1):
        eps = om.denoise_step(m, z, s, mask[s - 1], cache)
        for l in range(cfg.L):
            if s == S[l]:
                snap = cache[l].copy()
                cache[("snap", l)] = snap
        z = om.sampler_update(cfg, z, eps, s)
    for l in range(cfg.L):
        assert np.array_equal(cache[l], cache[("snap", l)])  # never refreshed after S_l


def test_frozen_unit_adds_cached_delta_to_current_stream():
    """A unit whose branch output does not depend on its input (zero weights, nonzero
    biases) reproduces the unscheduled run when frozen: the frozen rule adds the cached
    update to the *current* stream rather than replaying a stale hidden state."""
    cfg, w, x = load("uvit_mini")
    w = [dict(u) for u in w]
    target = 1  # an in-block, so its output also feeds a skip connection
    for key in ("w_o", "w2"):
        w[target][key] = np.zeros_like(w[target][key])
    m = om.Model(cfg, w, x)
    S = np.full(cfg.L, cfg.T)
    S[target] = 1
    mask = sch.active_mask(S, cfg.T)
    a = om.trajectory(m, x["z"], mask, steps=4)
    b = om.trajectory(m, x["z"], None, steps=4)
    for za, zb in zip(a.z, b.z):
        assert np.allclose(za, zb, rtol=0, atol=1e-12 * np.abs(zb).max())
    assert not np.array_equal(a.z[0], a.z[1])  # the state really moves between steps


def test_frozen_cache_missing_raises():
    cfg, w, x = load("tiny_ragged")
    m = om.Model(cfg, w, x)
    with pytest.raises(RuntimeError):
        om.denoise_step(m, x["z"], 2, [1, 0, 1], {})


def test_dit_adaln_zero_makes_identity_block():
    cfg, w, x = load("dit_mini")
    w = [dict(u) for u in w]
    w[0]["w_ada"] = np.zeros_like(w[0]["w_ada"])
    w[0]["b_ada"] = np.zeros_like(w[0]["b_ada"])
    m = om.Model(cfg, w, x)
    h = np.array(x["z"], np.float64)
    out, delta = m.unit_active(0, h, 500.0)
    assert np.array_equal(delta, np.zeros_like(delta))
    assert np.array_equal(out, h)


def test_uvit_skip_linear_identity():
    cfg, w, x = load("uvit_mini")
    d = cfg.d
    m = om.Model(cfg, w, x)
    u = dict(m.units[cfg.L - 1])
    u["w_skip"] = np.concatenate([np.eye(d), np.zeros((d, d))], axis=1)
    u["b_skip"] = np.zeros(d)
    rng = np.random.default_rng(3)
    h, skip = rng.standard_normal((1, 4, d)), rng.standard_normal((1, 4, d))
    assert np.array_equal(m.skip_linear(u, h, skip), nu.round_bf16(h))


def test_sampler_rows():
    cfg = synth.get_config("llada_mini")
    rng = np.random.default_rng(0)
    z = rng.standard_normal((cfg.B, cfg.N, cfg.d))
    eps = rng.standard_normal((cfg.B, cfg.N, cfg.d))
    out = om.sampler_update(cfg, z, eps, 1)
    r0 = cfg.prompt_rows
    assert np.array_equal(out[:, :r0], z[:, :r0])
    assert np.allclose(out[:, r0:], z[:, r0:] - eps[:, r0:] / cfg.T)


def test_uvit_time_token_rewritten_each_step():
    cfg, w, x = load("uvit_mini")
    m = om.Model(cfg, w, x)
    h1 = om.initial_stream(m, x["z"], 1)
    h2 = om.initial_stream(m, x["z"], 2)
    assert np.allclose(h1[:, 0], om.timestep_embedding(1000.0, cfg.d))
    assert not np.allclose(h1[:, 0], h2[:, 0])
    assert np.array_equal(h1[:, 1:], h2[:, 1:])


def test_generator_spectrum_is_planted():
    """The synthetic generator's record of its planted singular values matches an SVD."""
    cfg = synth.get_config("tiny")
    u = synth.unit_weights(cfg, 0, keep_planted=True)
    pl = u["_planted"]["w1"]
    s = np.linalg.svd(np.asarray(u["w1"], np.float64), compute_uv=False)
    assert np.allclose(s, pl.s, rtol=1e-6)
