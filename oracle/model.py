"""Residual units, the jagged denoiser step and the sampler (oracle).

Paper passages followed:
* Sec. 3.1 (Setup): the deterministic update z_{t-1} = alpha_t z_t - beta_t eps,
  residual units h_l = h_{l-1} + F_l(h_{l-1}; c_s), the cached update
  Delta_{l,r} = F_l(h_{l-1,r}; c_r) and the frozen rule
  h_{l,s} = h_{l-1,s} + Delta_{l,r_l(s)}.
* Alg. 2 (Jagged-Stream Execution): walk the units in order; an active unit
  (s <= S_l) computes Delta and refreshes its cache; a frozen unit reads
  its cache; both add Delta to the current residual stream.
* Table "Scope and executor semantics": conditioning, skip inputs and the
  current residual stream keep propagating through frozen units.

The architectures themselves (pre-norm attention + MLP blocks shaped like
LLaDA-8B, DiT-XL/2, U-ViT-L and an SDXL spatial transformer) are standard
and not specified by the paper; their constants are readings of this
implementation (norm epsilons, RoPE base, GELU forms, sinusoidal embeddings),
fixed below.

Precision: float64 everywhere.  For bf16 configs the values the GPU stores
in bf16 are rounded with ``Precision.q``: norm outputs, Q/K/V after bias
and RoPE, attention outputs, MLP hidden activations, U-ViT skip-linear
inputs and the SDXL context projections.  The softmax probabilities are
not rounded.

A multi-branch unit's update Delta is the sum of its branch updates in
execution order (ResNet block, attention, cross-attention, MLP), and the
active path adds each branch to the stream as it is produced, exactly as
the unscheduled forward does.

Unit granularity.  The scheduled unit is one block by default (its branches
share a lifetime and one cached update).  With ``granularity="branch"`` every
pre-norm residual branch of a block is a unit of its own (the residual units
of Sec. 3.1 taken at branch level): block l's branches are units
l * nb, ..., l * nb + nb - 1 in execution order, each with its own lifetime
and cached update (its branch output), nb = len(branches(arch)).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np
from scipy.special import erf

from .numerics import Precision, decode

RMS_EPS = 1e-5
LN_EPS_DIT = 1e-6
LN_EPS = 1e-5
GN_EPS = 1e-5
ROPE_THETA = 10000.0
CROSS_ARCHS = ("sdxl", "sdxl_unet")  # architectures with a cross-attention branch
GRANULARITIES = ("block", "branch")


def branches(arch: str):
    """The residual branches of one block, in execution order."""
    out = ("resnet",) if arch == "sdxl_unet" else ()
    out += ("attn",)
    if arch in CROSS_ARCHS:
        out += ("xattn",)
    return out + ("mlp",)


# --------------------------------------------------------------------------
# elementwise pieces
# --------------------------------------------------------------------------

def rmsnorm(x, w, eps=RMS_EPS):
    """x / sqrt(mean(x^2) + eps) * w over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def layernorm(x, w=None, b=None, eps=LN_EPS):
    """(x - mean) / sqrt(biased var + eps) [* w + b] over the last axis."""
    mu = np.mean(x, axis=-1, keepdims=True)
    xc = x - mu
    y = xc / np.sqrt(np.mean(xc * xc, axis=-1, keepdims=True) + eps)
    if w is not None:
        y = y * w
    if b is not None:
        y = y + b
    return y


def group_norm(x, groups, w, b, eps=GN_EPS):
    """GroupNorm of [B, N, C] (N grid positions, C channels): per sample and per group of
    C / groups consecutive channels, (x - mean) / sqrt(biased variance + eps) over the group's
    positions and channels, then the per-channel gain and shift."""
    B, N, C = x.shape
    g = x.reshape(B, N, groups, C // groups)
    mu = np.mean(g, axis=(1, 3), keepdims=True)
    var = np.mean((g - mu) ** 2, axis=(1, 3), keepdims=True)
    y = ((g - mu) / np.sqrt(var + eps)).reshape(B, N, C)
    return y * w + b


def conv3x3(x, w_unf, side):
    """3 x 3 convolution, stride 1, zero padding 1, on [B, side * side, C_in] (row-major grid)
    with the kernel unfolded to W [C_out, 9 C_in], column (3 ky + kx) C_in + c:
    out[b, (y, x), o] = sum_{ky, kx, c} W[o, (3 ky + kx) C_in + c] in[b, (y + ky - 1, x + kx - 1), c],
    positions outside the grid reading 0.  Written as the unfolded (im2col) matrix times W^T."""
    B, N, ci = x.shape
    img = x.reshape(B, side, side, ci)
    pad = np.zeros((B, side + 2, side + 2, ci), dtype=np.float64)
    pad[:, 1:-1, 1:-1] = img
    cols = [pad[:, ky:ky + side, kx:kx + side, :] for ky in range(3) for kx in range(3)]
    unf = np.concatenate(cols, axis=-1).reshape(B, N, 9 * ci)
    return unf @ w_unf.T


def gelu_erf(x):
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def gelu_tanh(x):
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def silu(x):
    return x / (1.0 + np.exp(-x))


def timestep_embedding(t: float, dim: int) -> np.ndarray:
    """Sinusoidal embedding [cos(t f_i), sin(t f_i)], f_i = 10000^(-i/half), i < half."""
    half = dim // 2
    freqs = np.exp(-math.log(10000.0) * np.arange(half, dtype=np.float64) / half)
    args = t * freqs
    return np.concatenate([np.cos(args), np.sin(args)])


def timestep_value(s: int, T: int) -> float:
    """t_s = 1000 (T - s + 1) / T: s = 1 is the noisiest evaluation."""
    return 1000.0 * (T - s + 1) / T


def rope(x: np.ndarray, theta: float = ROPE_THETA) -> np.ndarray:
    """Rotate-half rotary embedding on [B, H, N, dh] with positions 0..N-1."""
    dh = x.shape[-1]
    half = dh // 2
    inv = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / dh)
    pos = np.arange(x.shape[-2], dtype=np.float64)
    ang = pos[:, None] * inv[None, :]
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """softmax(q k^T / sqrt(dh)) v over the key axis; [B, H, Nq, dh] x [B, H, Nk, dh]."""
    dh = q.shape[-1]
    s = np.matmul(q, np.swapaxes(k, -1, -2)) / math.sqrt(dh)
    s = s - np.max(s, axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / np.sum(p, axis=-1, keepdims=True)
    return np.matmul(p, v)


def heads(x: np.ndarray, H: int) -> np.ndarray:
    B, N, D = x.shape
    return x.reshape(B, N, H, D // H).transpose(0, 2, 1, 3)


def merge_heads(x: np.ndarray) -> np.ndarray:
    B, H, N, dh = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B, N, H * dh)


# --------------------------------------------------------------------------
# model
# --------------------------------------------------------------------------

def _decode_unit(w: Dict[str, np.ndarray], dt: str) -> Dict[str, np.ndarray]:
    u = {}
    for name, arr in w.items():
        if name.startswith("_"):
            continue
        u[name] = decode(arr, dt) if name.startswith("w") else np.asarray(arr, np.float64)
    return u


class _LazyUnits:
    def __init__(self, weights, dt):
        self.weights, self.dt = weights, dt

    def __len__(self):
        return len(self.weights)

    def __getitem__(self, l):
        return _decode_unit(self.weights[l], self.dt)

    def __iter__(self):
        return (self[l] for l in range(len(self)))


class Model:
    """One workload's weights decoded to float64, plus its architecture rules."""

    def __init__(self, cfg, weights: List[Dict[str, np.ndarray]], inputs: Dict[str, np.ndarray],
                 lazy: bool = False, granularity: str = "block"):
        """``lazy`` decodes a unit's weights each time the unit runs instead of keeping every
        unit in float64 (for the full-size workloads).  ``granularity``: "block" (one scheduled
        unit per block) or "branch" (one per residual branch)."""
        if granularity not in GRANULARITIES:
            raise ValueError(f"granularity {granularity!r}")
        self.cfg = cfg
        self.arch = cfg.arch
        self.granularity = granularity
        self.branch_names = branches(cfg.arch)
        self.nb = len(self.branch_names) if granularity == "branch" else 1
        self.n_units = cfg.L * self.nb
        self.prec = Precision(cfg.dtype == "bf16")
        self._raw = weights
        self.units = _LazyUnits(weights, cfg.dtype) if lazy else [_decode_unit(w, cfg.dtype) for w in weights]
        self.class_emb = inputs.get("class_emb")
        if self.class_emb is not None:
            self.class_emb = np.asarray(self.class_emb, np.float64)
        self.ctx = inputs.get("ctx")
        if self.ctx is not None:
            self.ctx = decode(self.ctx, cfg.dtype)

    # ---- U-ViT structure ------------------------------------------------
    def skip_source(self, l: int) -> int:
        """U-ViT: out-block l consumes the output of in-block L-1-l (-1: no skip input)."""
        L = self.cfg.L
        if self.arch != "uvit" or l <= L // 2:
            return -1
        return L - 1 - l

    def saves_skip(self, l: int) -> bool:
        return self.arch == "uvit" and l < self.cfg.L // 2

    # ---- conditioning ---------------------------------------------------
    def adaln(self, u: Dict[str, np.ndarray], t: float) -> List[np.ndarray]:
        """DiT: [shift1, scale1, gate1, shift2, scale2, gate2] = SiLU(c) W_ada^T + b, c = emb(t) + y."""
        c = timestep_embedding(t, self.cfg.d)[None, :] + self.class_emb
        mod = silu(c) @ u["w_ada"].T + u["b_ada"]
        return np.split(mod, 6, axis=-1)

    def cross_kv(self, u: Dict[str, np.ndarray]):
        """SDXL: K^x, V^x from the context sequence; independent of the step."""
        d, H, q = self.cfg.d, self.cfg.H, self.prec.q
        kv = self.ctx @ u["w_xkv"].T
        return q(heads(kv[..., :d], H)), q(heads(kv[..., d:], H))

    # ---- branches ---------------------------------------------------------
    def _norm(self, u, h, which: str, mod=None):
        a = self.arch
        if a in ("tiny", "llada"):
            return rmsnorm(h, u[f"{which}_w"])
        if a == "dit":
            shift, scale = mod
            return layernorm(h, eps=LN_EPS_DIT) * (1.0 + scale[:, None, :]) + shift[:, None, :]
        return layernorm(h, u[f"{which}_w"], u[f"{which}_b"], eps=LN_EPS)

    def attn_branch(self, u, h, mod=None):
        cfg, q = self.cfg, self.prec.q
        d, H = cfg.d, cfg.H
        xn = q(self._norm(u, h, "norm1", mod[0:2] if mod else None))
        qkv = xn @ u["w_qkv"].T
        if "b_qkv" in u:
            qkv = qkv + u["b_qkv"]
        Q, K, V = heads(qkv[..., :d], H), heads(qkv[..., d:2 * d], H), heads(qkv[..., 2 * d:], H)
        if self.arch == "llada":
            Q, K = rope(Q), rope(K)
        o = q(merge_heads(attention(q(Q), q(K), q(V))))
        a = o @ u["w_o"].T
        if "b_o" in u:
            a = a + u["b_o"]
        if mod:
            a = mod[2][:, None, :] * a
        return a

    def xattn_branch(self, u, h, kx, vx):
        cfg, q = self.cfg, self.prec.q
        xn = q(layernorm(h, u["normx_w"], u["normx_b"], eps=LN_EPS))
        Q = q(heads(xn @ u["w_xq"].T, cfg.H))
        o = q(merge_heads(attention(Q, kx, vx)))
        return o @ u["w_xo"].T + u["b_xo"]

    def mlp_branch(self, u, h, mod=None):
        cfg, q = self.cfg, self.prec.q
        F = cfg.F
        xn = q(self._norm(u, h, "norm2", mod[3:5] if mod else None))
        z = xn @ u["w1"].T
        if "b1" in u:
            z = z + u["b1"]
        if self.arch == "llada":
            hid = silu(z[..., :F]) * z[..., F:]
        elif self.arch in CROSS_ARCHS:
            hid = z[..., F:] * gelu_erf(z[..., :F])
        elif self.arch == "dit":
            hid = gelu_tanh(z)
        else:
            hid = gelu_erf(z)
        m = q(hid) @ u["w2"].T
        if "b2" in u:
            m = m + u["b2"]
        if mod:
            m = mod[5][:, None, :] * m
        return m

    def skip_linear(self, u, h, skip):
        """U-ViT out-block entry: [h ; skip] W_skip^T + b (always executed)."""
        q = self.prec.q
        return np.concatenate([q(h), q(skip)], axis=-1) @ u["w_skip"].T + u["b_skip"]

    def temb(self, u, t: float) -> np.ndarray:
        """SDXL UNet ResNet block: the time-embedding projection SiLU(c) W_t^T + b_t per sample,
        c = emb(t) + y (the conditioning keeps propagating, Table "Scope and executor
        semantics")."""
        c = timestep_embedding(t, self.cfg.d)[None, :] + self.class_emb
        return silu(c) @ u["w_temb"].T + u["b_temb"]

    def resnet_branch(self, u, h, t: float):
        """SDXL UNet ResNet block (channels in = out, identity shortcut): GroupNorm, SiLU,
        3 x 3 convolution plus the time-embedding projection, GroupNorm, SiLU, 3 x 3
        convolution.  Its update is added to the stream like any residual branch."""
        cfg, q = self.cfg, self.prec.q
        x1 = q(silu(group_norm(h, cfg.groups, u["gn1_w"], u["gn1_b"])))
        u1 = q(conv3x3(x1, u["w_conv1"], cfg.grid) + u["b_conv1"] + self.temb(u, t)[:, None, :])
        x2 = q(silu(group_norm(u1, cfg.groups, u["gn2_w"], u["gn2_b"])))
        return conv3x3(x2, u["w_conv2"], cfg.grid) + u["b_conv2"]

    def branch(self, name: str, u, h: np.ndarray, t: float, mod=None, cross=None) -> np.ndarray:
        """The update of one residual branch of a block on the current stream."""
        if name == "resnet":
            return self.resnet_branch(u, h, t)
        if name == "attn":
            return self.attn_branch(u, h, mod)
        if name == "xattn":
            return self.xattn_branch(u, h, *cross)
        return self.mlp_branch(u, h, mod)

    def unit_active(self, l: int, h: np.ndarray, t: float, cross=None):
        """Run unit l's branches on the current stream.  Returns (h_out, Delta_l)."""
        u = self.units[l]
        mod = self.adaln(u, t) if self.arch == "dit" else None
        delta = None
        if self.arch == "sdxl_unet":
            r = self.resnet_branch(u, h, t)
            h = h + r
            delta = r
        a = self.attn_branch(u, h, mod)
        h = h + a
        delta = a if delta is None else delta + a
        if self.arch in CROSS_ARCHS:
            x = self.xattn_branch(u, h, *cross)
            h = h + x
            delta = delta + x
        m = self.mlp_branch(u, h, mod)
        h = h + m
        delta = delta + m
        return h, delta


# --------------------------------------------------------------------------
# the jagged step and the trajectory
# --------------------------------------------------------------------------

@dataclass
class Trajectory:
    z: List[np.ndarray] = field(default_factory=list)    # z after each step (index s-1)
    eps: List[np.ndarray] = field(default_factory=list)  # h_L of each step


def initial_stream(model: Model, z: np.ndarray, s: int) -> np.ndarray:
    """h_0 = z_s; U-ViT's row 0 is the time token, rewritten from t_s."""
    h = np.array(z, dtype=np.float64)
    if model.arch == "uvit":
        h[:, 0, :] = timestep_embedding(timestep_value(s, model.cfg.T), model.cfg.d)[None, :]
    return h


def denoise_step(model: Model, z: np.ndarray, s: int, active: Optional[Sequence[int]],
                 cache: Dict[int, np.ndarray], cross=None,
                 unit_inputs: Optional[Dict[int, np.ndarray]] = None) -> np.ndarray:
    """One network evaluation at step s (Alg. 2).  Returns eps = h_L.

    ``active=None`` is the unscheduled forward (every unit computes, cache untouched).
    ``cross`` (SDXL) holds each unit's step-invariant context keys and values.
    An active unit refreshes ``cache[l]`` with its update (Alg. 2 refreshes at every
    active step; the entry read later is the one from the last active step, S_l for a
    static schedule).  The active set need not be nested in s (the input-aware baselines).
    ``unit_inputs``, if given, receives each unit's input h_{l-1,s}: the residual stream
    arriving at unit l (for a U-ViT out-block, before its skip linear; with branch units, the
    first branch of an out-block likewise).  Units are blocks or branches as
    ``model.granularity`` says; ``active`` and ``cache`` are indexed by unit.
    """
    cfg = model.cfg
    t = timestep_value(s, cfg.T)
    h = initial_stream(model, z, s)
    skips: Dict[int, np.ndarray] = {}
    nb = model.nb
    for l in range(cfg.L):
        if unit_inputs is not None:
            unit_inputs[l * nb] = h.copy()
        src = model.skip_source(l)
        if src >= 0:
            h = model.skip_linear(model.units[l], h, skips[src])
        if nb == 1:
            if active is None or active[l]:
                h, delta = model.unit_active(l, h, t, None if cross is None else cross[l])
                if active is not None:
                    cache[l] = delta
            else:
                if l not in cache:
                    raise RuntimeError(f"unit {l} frozen before its cache was written")
                h = h + cache[l]
        else:
            # branch units: each branch computes or adds its own cached update; a DiT block's
            # modulation is computed when one of its branches computes
            u, mod = None, None
            for k, name in enumerate(model.branch_names):
                j = l * nb + k
                if unit_inputs is not None and k > 0:
                    unit_inputs[j] = h.copy()
                if active is None or active[j]:
                    if u is None:
                        u = model.units[l]
                        mod = model.adaln(u, t) if model.arch == "dit" else None
                    o = model.branch(name, u, h, t, mod, None if cross is None else cross[l])
                    h = h + o
                    if active is not None:
                        cache[j] = o
                else:
                    if j not in cache:
                        raise RuntimeError(f"unit {j} frozen before its cache was written")
                    h = h + cache[j]
        if model.saves_skip(l):
            skips[l] = h
    return h


def sampler_update(cfg, z: np.ndarray, eps: np.ndarray, s: int) -> np.ndarray:
    """z_{s+1} = alpha_s z_s - beta_s eps on the rows the sampler owns (Sec. 3.1).

    Reading: alpha_s = 1, beta_s = 1 / T; rows outside ``cfg.update_rows``
    (LLaDA's prompt rows, U-ViT's time and class tokens) are left unchanged.
    """
    r0, r1 = cfg.update_rows
    out = np.array(z, dtype=np.float64)
    out[:, r0:r1] = 1.0 * z[:, r0:r1] - (1.0 / cfg.T) * eps[:, r0:r1]
    return out


def trajectory(model: Model, z0: np.ndarray, active_mask: Optional[np.ndarray],
               steps: Optional[int] = None) -> Trajectory:
    """Run steps 1..steps (default T).  ``active_mask[s-1, unit]`` or None for unscheduled."""
    cfg = model.cfg
    steps = cfg.T if steps is None else steps
    cross = None
    if model.arch in CROSS_ARCHS:
        cross = [model.cross_kv(u) for u in model.units]
    cache: Dict[int, np.ndarray] = {}
    z = np.array(z0, dtype=np.float64)
    out = Trajectory()
    for s in range(1, steps + 1):
        act = None if active_mask is None else active_mask[s - 1]
        eps = denoise_step(model, z, s, act, cache, cross)
        z = sampler_update(cfg, z, eps, s)
        out.z.append(z)
        out.eps.append(eps)
    return out
