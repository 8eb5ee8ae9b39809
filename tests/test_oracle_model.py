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


# ---------------------------------------------------------------- cross-attention branch
# Pins of the SDXL cross-attention branch (the component scored by Eq. app-xattn-score):
# the keys and values are projections of the conditioning sequence by W_K^x and W_V^x
# (stored stacked as w_xkv = [W_K^x; W_V^x]), the queries come from the LayerNorm of the
# current stream, and the branch output is the attention output through W_O^x plus b_O^x.

def _sdxl_f32(**kw):
    """The reduced SDXL workload in fp32 storage: no bf16 rounding points, so the branch is
    exact float64 arithmetic and can be compared with an independent computation."""
    return load("sdxl_mini", dtype="f32", **kw)


def test_xattn_one_token_context_is_value_projection():
    """With a single context token the softmax weight is 1 for every query, so every query
    receives that token's value projection: out = (c W_V^x^T) W_O^x^T + b_O^x.  A K/V swap
    in the w_xkv split would give the key projection instead."""
    cfg, w, x = _sdxl_f32(ctx_len=1)
    d = cfg.d
    m = om.Model(cfg, w, x)
    u = m.units[0]
    rng = np.random.default_rng(11)
    h = rng.standard_normal((cfg.B, 7, d))
    out = m.xattn_branch(u, h, *m.cross_kv(u))
    c = np.asarray(x["ctx"], np.float64)  # [B, 1, ctx_dim]
    wv = u["w_xkv"][d:]                   # W_V^x: rows d..2d of the stacked storage
    wk = u["w_xkv"][:d]
    for b in range(cfg.B):
        v = c[b, 0] @ wv.T
        ref = v @ u["w_xo"].T + u["b_xo"]
        assert np.allclose(out[b], np.broadcast_to(ref, out[b].shape), rtol=1e-12, atol=1e-12)
        wrong = (c[b, 0] @ wk.T) @ u["w_xo"].T + u["b_xo"]
        assert not np.allclose(out[b, 0], wrong, rtol=1e-3)


def test_xattn_zero_output_projection_gives_bias():
    cfg, w, x = _sdxl_f32()
    m = om.Model(cfg, w, x)
    u = dict(m.units[0])
    u["w_xo"] = np.zeros_like(u["w_xo"])
    h = np.random.default_rng(12).standard_normal((cfg.B, 5, cfg.d))
    out = m.xattn_branch(u, h, *m.cross_kv(u))
    assert np.array_equal(out, np.broadcast_to(u["b_xo"], out.shape))


def test_xattn_textbook_per_head():
    """Per-head cross-attention written out independently: LayerNorm (biased variance,
    eps 1e-5, gain and shift) of the stream, one query row at a time against the 77
    context keys of each head, softmax, weighted value sum, heads concatenated."""
    cfg, w, x = _sdxl_f32()
    d, H, dh = cfg.d, cfg.H, cfg.dh
    m = om.Model(cfg, w, x)
    u = m.units[1]
    rng = np.random.default_rng(13)
    h = rng.standard_normal((cfg.B, 3, d)) * 2.0 + 0.5
    out = m.xattn_branch(u, h, *m.cross_kv(u))
    c = np.asarray(x["ctx"], np.float64)
    wq, wk, wv = u["w_xq"], u["w_xkv"][:d], u["w_xkv"][d:]
    for b in range(cfg.B):
        keys = [[float(np.dot(c[b, j], wk[r])) for r in range(d)] for j in range(cfg.ctx_len)]
        vals = [[float(np.dot(c[b, j], wv[r])) for r in range(d)] for j in range(cfg.ctx_len)]
        for i in range(h.shape[1]):
            row = h[b, i]
            mu = sum(row) / d
            var = sum((v - mu) ** 2 for v in row) / d
            xn = [(row[t] - mu) / math.sqrt(var + 1e-5) * u["normx_w"][t] + u["normx_b"][t] for t in range(d)]
            qv = [float(np.dot(xn, wq[r])) for r in range(d)]
            o = []
            for hh in range(H):
                sl = slice(hh * dh, (hh + 1) * dh)
                logits = [sum(a * bb for a, bb in zip(qv[sl], keys[j][sl])) / math.sqrt(dh)
                          for j in range(cfg.ctx_len)]
                mx = max(logits)
                e = [math.exp(a - mx) for a in logits]
                tot = sum(e)
                o += [sum(e[j] / tot * vals[j][hh * dh + t] for j in range(cfg.ctx_len)) for t in range(dh)]
            ref = np.array([float(np.dot(o, u["w_xo"][r])) for r in range(d)]) + u["b_xo"]
            assert np.allclose(out[b, i], ref, rtol=1e-10, atol=1e-10 * np.abs(ref).max())


def test_xattn_norm_is_layernorm():
    """LayerNorm removes a per-row constant offset (RMSNorm would not)."""
    cfg, w, x = _sdxl_f32()
    m = om.Model(cfg, w, x)
    u = m.units[0]
    h = np.random.default_rng(14).standard_normal((cfg.B, 4, cfg.d))
    kv = m.cross_kv(u)
    a = m.xattn_branch(u, h, *kv)
    b = m.xattn_branch(u, h + 3.0, *kv)
    assert np.allclose(a, b, rtol=1e-9, atol=1e-9 * np.abs(a).max())
