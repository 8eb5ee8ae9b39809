"""Pins for the SDXL UNet ResNet units of the oracle: the 3 x 3 convolution on the unfolded
kernel, GroupNorm, the unfolded-kernel score (Eq. app-conv-score) and the unit structure."""
import functools

import numpy as np
import pytest
from scipy.signal import correlate2d

import synth
from oracle import model as om
from oracle import spectral as sp


@functools.lru_cache(maxsize=None)
def load(name, **kw):
    cfg = synth.get_config(name, **kw)
    return cfg, synth.model_weights(cfg), synth.inputs(cfg)


def test_conv3x3_against_scipy_correlate():
    rng = np.random.default_rng(0)
    B, side, ci, co = 2, 5, 3, 4
    x = rng.standard_normal((B, side * side, ci))
    k = rng.standard_normal((co, ci, 3, 3))  # the paper's C_out x C_in x k_h x k_w tensor
    w = k.transpose(0, 2, 3, 1).reshape(co, 9 * ci)  # stored: column (3 ky + kx) C_in + c
    out = om.conv3x3(x, w, side)
    for b in range(B):
        img = x[b].reshape(side, side, ci)
        for o in range(co):
            ref = sum(correlate2d(img[:, :, c], k[o, c], mode="same", boundary="fill") for c in range(ci))
            assert np.allclose(out[b, :, o].reshape(side, side), ref, rtol=1e-12, atol=1e-12)


def test_conv3x3_identity_and_shift_taps():
    rng = np.random.default_rng(1)
    side, c = 4, 3
    x = rng.standard_normal((1, side * side, c))
    w = np.zeros((c, 9 * c))
    w[np.arange(c), 4 * c + np.arange(c)] = 1.0  # centre tap
    assert np.array_equal(om.conv3x3(x, w, side), x)
    w = np.zeros((c, 9 * c))
    w[np.arange(c), 1 * c + np.arange(c)] = 1.0  # tap (ky, kx) = (0, 1): the row above
    out = om.conv3x3(x, w, side).reshape(side, side, c)
    img = x.reshape(side, side, c)
    assert np.array_equal(out[1:], img[:-1]) and np.all(out[0] == 0)


def test_group_norm_special_cases():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 9, 8)) * 3 + 1
    one, zero = np.ones(8), np.zeros(8)
    y = om.group_norm(x, 8, one, zero, eps=0.0)  # one channel per group: per-channel statistics
    assert np.allclose(y.mean(axis=1), 0, atol=1e-12) and np.allclose(y.var(axis=1), 1)
    y = om.group_norm(x, 1, one, zero, eps=0.0)  # one group: the whole sample
    flat = x.reshape(2, -1)
    ref = ((flat - flat.mean(1, keepdims=True)) / flat.std(1, keepdims=True)).reshape(x.shape)
    assert np.allclose(y, ref)
    y = om.group_norm(x, 2, one, zero, eps=0.0)
    g = y.reshape(2, 9, 2, 4)
    assert np.allclose(g.mean(axis=(1, 3)), 0, atol=1e-12) and np.allclose(g.var(axis=(1, 3)), 1)
    w, b = rng.standard_normal(8), rng.standard_normal(8)
    assert np.allclose(om.group_norm(x, 2, w, b, eps=0.0), y * w + b)


def test_unfolded_score_is_layout_free():
    """Eq. app-conv-score unfolds C_out x C_in x k_h x k_w to C_out x (C_in k_h k_w); the
    stored tap-major unfolding is a column permutation with the same singular values."""
    rng = np.random.default_rng(3)
    k = rng.standard_normal((16, 6, 3, 3)) * np.linspace(2, 0.1, 16)[:, None, None, None]
    paper = sp.unfold_conv(k)
    stored = k.transpose(0, 2, 3, 1).reshape(16, 54)
    a, b = sp.matrix_stats(paper), sp.matrix_stats(stored)
    assert a.g == pytest.approx(b.g, rel=1e-13) and a.energy_top == pytest.approx(b.energy_top, rel=1e-13)


def test_unit_score_sums_both_convolutions():
    cfg, w, x = load("sdxl_unet_mini")
    mats = sp.unit_matrices(w[0], cfg.d, cfg.dtype)
    assert {"conv1", "conv2"} <= set(mats)
    us = sp.unit_score(mats, cfg.dh)
    g = {r: s.g for r, s in us.stats.items()}
    want = (sp.q_attn(g["q"], g["k"], g["v"], g["o"], cfg.dh) + sp.q_attn(g["xq"], g["xk"], g["xv"], g["xo"], cfg.dh)
            + sp.q_mlp(g["w1"], g["w2"]) + g["conv1"] + g["conv2"])
    assert us.raw == pytest.approx(want, rel=1e-14)


def test_resnet_unit_structure():
    """A zero second convolution (and bias) makes the ResNet block an identity: the unit is
    then the transformer block alone; a zero time projection leaves its bias."""
    cfg, w, x = load("sdxl_unet_mini")
    w = [dict(u) for u in w]
    w[0]["w_conv2"] = np.zeros_like(w[0]["w_conv2"])
    w[0]["b_conv2"] = np.zeros_like(w[0]["b_conv2"])
    m = om.Model(cfg, w, x)
    u = m.units[0]
    h = np.asarray(x["z"], np.float64)
    t = om.timestep_value(3, cfg.T)
    out, delta = m.unit_active(0, h, t, m.cross_kv(u))
    a = m.attn_branch(u, h)
    xa = m.xattn_branch(u, h + a, *m.cross_kv(u))
    mm = m.mlp_branch(u, h + a + xa)
    assert np.array_equal(out, h + a + xa + mm)
    u2 = dict(u)
    u2["w_temb"] = np.zeros_like(u2["w_temb"])
    assert np.array_equal(m.temb(u2, t), np.broadcast_to(u2["b_temb"], (cfg.B, cfg.d)))
