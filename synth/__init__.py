"""Seeded synthetic weights and inputs for the five denoiser workloads.

This module is the only code shared by the CPU oracle tests and the GPU
path.  It draws random numbers and rounds them to the storage dtype; it
holds none of the method's arithmetic (no norms, no attention, no
spectra, no schedule).

Storage conventions (shared by both consumers):

* ``f32`` arrays are ``numpy.float32``.
* ``bf16`` arrays are ``numpy.uint16`` holding bfloat16 bit patterns,
  produced by round-to-nearest-even from float32.
* Weight matrices use the ``[out, in]`` (row-major, K-contiguous) layout of
  a linear layer ``y = x W^T``.
* Norm gains/shifts and linear biases are float32 arrays whose values are
  representable in the config dtype.

Planted spectra.  Each weight matrix is ``W = U diag(s) V^T`` with
``s_i proportional to i^-a`` (``a ~ U[0.3, 1.5]`` per matrix) and
``||W||_F = c sqrt(min(m, n))`` (``c ~ U[0.5, 2]`` per matrix).  ``U`` and
``V`` have orthonormal columns.  For a side of length ``<= 512`` they are
the leading columns of a Haar orthogonal matrix (QR of a Gaussian with the
sign of ``diag(R)`` folded into ``Q``, Mezzadri 2007).  Longer sides use the
leading columns of a Kronecker product ``Q_a (x) Q_b`` of two such Haar
factors; this keeps the singular values exactly planted while making
generation ``O(m n (a + b))`` instead of ``O(m n d)``.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import Dict, List, Optional, Tuple

import numpy as np

# --------------------------------------------------------------------------
# workload configurations
# --------------------------------------------------------------------------

ARCH_IDS = {"tiny": 0, "llada": 1, "dit": 2, "uvit": 3, "sdxl": 4, "sdxl_unet": 5}


@dataclass(frozen=True)
class Config:
    name: str
    arch: str            # tiny | llada | dit | uvit | sdxl
    dtype: str           # f32 | bf16
    B: int               # batch
    N: int               # tokens per sample
    d: int               # model width
    H: int               # heads
    dh: int              # head dim
    F: int               # MLP hidden width
    L: int               # scheduled units (blocks)
    T: int               # denoising steps
    budgets: Tuple[int, ...] = (50,)
    ctx_len: int = 0     # SDXL cross-attention context length
    ctx_dim: int = 0     # SDXL context width
    prompt_rows: int = 0 # LLaDA: leading rows per sample that the sampler never updates
    cfg_id: int = 0      # seed domain
    grid: int = 0        # SDXL UNet units: side of the square latent grid (N = grid^2)
    groups: int = 32     # SDXL UNet units: GroupNorm groups

    @property
    def M(self) -> int:
        return self.B * self.N

    @property
    def gated(self) -> bool:
        return self.arch in ("llada", "sdxl", "sdxl_unet")

    @property
    def update_rows(self) -> Tuple[int, int]:
        """Half-open row range (within one sample) that the sampler updates."""
        if self.arch == "llada":
            return (self.prompt_rows, self.N)
        if self.arch == "uvit":
            return (2, self.N)
        return (0, self.N)


CONFIGS: Dict[str, Config] = {
    # the five workloads at their full sizes
    "tiny": Config("tiny", "tiny", "f32", 1, 256, 256, 4, 64, 1024, 4, 10, (50,), cfg_id=0),
    "llada": Config("llada", "llada", "bf16", 1, 1024, 4096, 32, 128, 12288, 32, 64,
                    (70, 50, 35), prompt_rows=512, cfg_id=1),
    "dit": Config("dit", "dit", "bf16", 32, 256, 1152, 16, 72, 4608, 28, 50, (50,), cfg_id=2),
    "uvit": Config("uvit", "uvit", "bf16", 32, 258, 1024, 16, 64, 4096, 21, 50, (50,), cfg_id=3),
    "sdxl": Config("sdxl", "sdxl", "bf16", 8, 1024, 1280, 20, 64, 5120, 10, 50, (70, 50),
                   ctx_len=77, ctx_dim=2048, cfg_id=4),
    # SDXL UNet stage units: a ResNet block (two 3x3 convolutions on the 32 x 32 latent grid)
    # followed by the spatial transformer block, scored as one unit
    "sdxl_unet": Config("sdxl_unet", "sdxl_unet", "bf16", 8, 1024, 1280, 20, 64, 5120, 10, 50, (70, 50),
                        ctx_len=77, ctx_dim=2048, cfg_id=5, grid=32, groups=32),
    # reduced shapes of the same architectures: several tiles plus ragged
    # tails, small enough for the CPU oracle to run whole trajectories
    "tiny_ragged": Config("tiny_ragged", "tiny", "f32", 2, 72, 128, 2, 64, 256, 3, 6, (50,), cfg_id=10),
    "llada_mini": Config("llada_mini", "llada", "bf16", 1, 200, 256, 2, 128, 384, 4, 12,
                         (70, 50, 35), prompt_rows=100, cfg_id=11),
    "dit_mini": Config("dit_mini", "dit", "bf16", 2, 80, 1152, 16, 72, 1152, 3, 8, (50,), cfg_id=12),
    "uvit_mini": Config("uvit_mini", "uvit", "bf16", 2, 66, 256, 4, 64, 512, 5, 8, (50,), cfg_id=13),
    "sdxl_mini": Config("sdxl_mini", "sdxl", "bf16", 2, 96, 256, 4, 64, 512, 3, 8, (50,),
                        ctx_len=77, ctx_dim=384, cfg_id=14),
    "sdxl_unet_mini": Config("sdxl_unet_mini", "sdxl_unet", "bf16", 2, 100, 256, 4, 64, 512, 3, 8, (50,),
                             ctx_len=77, ctx_dim=384, cfg_id=15, grid=10, groups=32),
}


def get_config(name: str, **overrides) -> Config:
    cfg = CONFIGS[name]
    return replace(cfg, **overrides) if overrides else cfg


# --------------------------------------------------------------------------
# dtype helpers (storage only)
# --------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even); return uint16 bits."""
    src = np.ascontiguousarray(x, dtype=np.float32).reshape(-1)
    out = np.empty(src.shape, dtype=np.uint16)
    step = 1 << 22
    for i in range(0, src.size, step):
        u = src[i:i + step].view(np.uint32).copy()
        lsb = u >> 16
        lsb &= 1
        u += lsb
        u += np.uint32(0x7FFF)
        u >>= 16
        out[i:i + step] = u
        nan = np.isnan(src[i:i + step])
        if nan.any():
            out[i:i + step][nan] = 0x7FC0
    return out.reshape(np.shape(x))


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round a float64/float32 array to the storage dtype."""
    x32 = np.asarray(x, dtype=np.float32)
    if dtype == "f32":
        return np.ascontiguousarray(x32)
    return f32_to_bf16_bits(x32)


def representable(x: np.ndarray, dtype: str) -> np.ndarray:
    """float32 array whose values are representable in ``dtype`` (for gains and biases)."""
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    return bf16_bits_to_f32(f32_to_bf16_bits(np.asarray(x, dtype=np.float32)))


# --------------------------------------------------------------------------
# random orthonormal columns and planted-spectrum matrices
# --------------------------------------------------------------------------

_DENSE_MAX = 512
ROLE_IDS = {"q": 0, "k": 1, "v": 2, "o": 3, "w1": 4, "w2": 5, "ada": 6, "skip": 7,
            "xq": 8, "xk": 9, "xv": 10, "xo": 11, "conv1": 12, "conv2": 13, "temb": 14}


def _rng(cfg_id: int, stream: int, unit: int, role: int, sub: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([cfg_id, stream, unit, role, sub]))


def haar(rng: np.random.Generator, n: int) -> np.ndarray:
    a = rng.standard_normal((n, n))
    q, r = np.linalg.qr(a)
    return q * np.sign(np.diag(r))[None, :]


def _split(m: int) -> Tuple[int, int]:
    """m = a * b with b <= 512 as close to sqrt(m) as possible (b >= a)."""
    best = None
    for b in range(1, min(m, _DENSE_MAX) + 1):
        if m % b == 0:
            a = m // b
            if a > _DENSE_MAX:
                continue
            score = abs(math.log(b / a))
            if best is None or score < best[0]:
                best = (score, a, b)
    if best is None:
        raise ValueError(f"cannot split {m} into two factors <= {_DENSE_MAX}")
    return best[1], best[2]


class OrthCols:
    """First ``d`` columns of an ``m x m`` orthogonal matrix (dense Haar or Kronecker of two)."""

    def __init__(self, rng: np.random.Generator, m: int, d: int):
        self.m, self.d = m, d
        if m <= _DENSE_MAX:
            self.dense = haar(rng, m)[:, :d]
            self.qa = self.qb = None
        else:
            a, b = _split(m)
            self.dense = None
            self.qa, self.qb = haar(rng, a), haar(rng, b)

    def explicit(self) -> np.ndarray:
        if self.dense is not None:
            return self.dense
        pa = -(-self.d // self.qb.shape[0])
        return np.kron(self.qa[:, :pa], self.qb)[:, : self.d]

    def apply(self, x: np.ndarray) -> np.ndarray:
        """Return ``U @ x`` for ``x`` of shape ``[d, n]`` without forming ``U``."""
        dt = x.dtype
        if self.dense is not None:
            return self.dense.astype(dt, copy=False) @ x
        a, b = self.qa.shape[0], self.qb.shape[0]
        pa = -(-self.d // b)
        n = x.shape[1]
        if pa * b != self.d:
            xp = np.zeros((pa * b, n), dtype=dt)
            xp[: self.d] = x
        else:
            xp = x
        # (Q_a (x) Q_b) acting on rows indexed (p, q): contract q with Q_b, then p with Q_a
        t = np.ascontiguousarray(xp.reshape(pa, b, n).transpose(1, 0, 2)).reshape(b, pa * n)
        y1 = (self.qb.astype(dt) @ t).reshape(b, pa, n).transpose(1, 0, 2)            # [pa, b, n]
        y2 = self.qa[:, :pa].astype(dt) @ np.ascontiguousarray(y1).reshape(pa, b * n)  # [a, b*n]
        return y2.reshape(a * b, n)


@dataclass
class Planted:
    """Planted factors of one weight matrix (the generator's own record, for pins)."""
    m: int
    n: int
    a: float
    c: float
    s: np.ndarray  # singular values, descending, float64


def planted_matrix(rng: np.random.Generator, m: int, n: int,
                   work=np.float64) -> Tuple[np.ndarray, Planted]:
    """Draw one planted-spectrum matrix; ``work`` is the arithmetic precision of the assembly."""
    d = min(m, n)
    a = rng.uniform(0.3, 1.5)
    c = rng.uniform(0.5, 2.0)
    s = np.arange(1, d + 1, dtype=np.float64) ** (-a)
    s *= c * math.sqrt(d) / math.sqrt(float(np.sum(s * s)))
    u = OrthCols(rng, m, d)
    v = OrthCols(rng, n, d)
    x = (s[:, None] * v.explicit().T).astype(work, copy=False)  # [d, n]
    w = u.apply(x)                                               # [m, n]
    return w, Planted(m, n, a, c, s)


# --------------------------------------------------------------------------
# model weights
# --------------------------------------------------------------------------

STREAM_WEIGHTS, STREAM_INPUTS, STREAM_COND = 0, 1, 2


def _gain(rng, n, dtype, center=1.0, scale=0.1):
    return representable(center + scale * rng.standard_normal(n), dtype)


def _bias(rng, n, dtype, scale=0.02):
    return representable(scale * rng.standard_normal(n), dtype)


def unit_weights(cfg: Config, unit: int, keep_planted: bool = False) -> Dict[str, np.ndarray]:
    """All parameters of one scheduled unit (one block), seeded by (config, unit, role)."""
    d, F, dt = cfg.d, cfg.F, cfg.dtype
    out: Dict[str, np.ndarray] = {}
    planted: Dict[str, Planted] = {}

    # bf16 storage keeps 8 significant bits, so large bf16 matrices are assembled in
    # float32; float32-stored matrices are assembled in float64
    work = np.float64 if dt == "f32" else np.float32

    def mat(role: str, m: int, n: int) -> np.ndarray:
        w, p = planted_matrix(_rng(cfg.cfg_id, STREAM_WEIGHTS, unit, ROLE_IDS[role]), m, n, work)
        planted[role] = p
        return store(w, dt)

    prm = _rng(cfg.cfg_id, STREAM_WEIGHTS, unit, 100)
    q, k, v = mat("q", d, d), mat("k", d, d), mat("v", d, d)
    out["w_qkv"] = np.ascontiguousarray(np.concatenate([q, k, v], axis=0))
    out["w_o"] = mat("o", d, d)
    out["w1"] = mat("w1", 2 * F if cfg.gated else F, d)
    out["w2"] = mat("w2", d, F)

    arch = cfg.arch
    out["norm1_w"] = _gain(prm, d, dt)
    out["norm2_w"] = _gain(prm, d, dt)
    if arch in ("uvit", "sdxl", "sdxl_unet"):
        out["norm1_b"] = _bias(prm, d, dt)
        out["norm2_b"] = _bias(prm, d, dt)
    if arch == "dit":
        # LayerNorm without affine parameters; AdaLN supplies shift/scale
        del out["norm1_w"], out["norm2_w"]
        out["b_qkv"] = _bias(prm, 3 * d, dt)
        out["w_ada"] = mat("ada", 6 * d, d)
        out["b_ada"] = _bias(prm, 6 * d, dt)
    if arch in ("dit", "uvit", "sdxl", "sdxl_unet"):
        out["b_o"] = _bias(prm, d, dt)
        out["b1"] = _bias(prm, 2 * F if cfg.gated else F, dt)
        out["b2"] = _bias(prm, d, dt)
    if arch == "uvit" and unit > cfg.L // 2:
        out["w_skip"] = mat("skip", d, 2 * d)
        out["b_skip"] = _bias(prm, d, dt)
    if arch == "sdxl_unet":
        # ResNet block: GroupNorm, SiLU, 3x3 convolution (+ time-embedding projection),
        # GroupNorm, SiLU, 3x3 convolution.  A convolution kernel is stored unfolded as
        # [C_out, 9 C_in] with column (3 ky + kx) C_in + c_in (tap-major, channels contiguous);
        # it is planted as that unfolded matrix.
        rrm = _rng(cfg.cfg_id, STREAM_WEIGHTS, unit, 101)
        out["gn1_w"] = _gain(rrm, d, dt)
        out["gn1_b"] = _bias(rrm, d, dt)
        out["w_conv1"] = mat("conv1", d, 9 * d)
        out["b_conv1"] = _bias(rrm, d, dt)
        out["w_temb"] = mat("temb", d, d)
        out["b_temb"] = _bias(rrm, d, dt)
        out["gn2_w"] = _gain(rrm, d, dt)
        out["gn2_b"] = _bias(rrm, d, dt)
        out["w_conv2"] = mat("conv2", d, 9 * d)
        out["b_conv2"] = _bias(rrm, d, dt)
    if arch in ("sdxl", "sdxl_unet"):
        out["normx_w"] = _gain(prm, d, dt)
        out["normx_b"] = _bias(prm, d, dt)
        out["w_xq"] = mat("xq", d, d)
        xk, xv = mat("xk", d, cfg.ctx_dim), mat("xv", d, cfg.ctx_dim)
        out["w_xkv"] = np.ascontiguousarray(np.concatenate([xk, xv], axis=0))
        out["w_xo"] = mat("xo", d, d)
        out["b_xo"] = _bias(prm, d, dt)
    if keep_planted:
        out["_planted"] = planted  # type: ignore[assignment]
    return out


def model_weights(cfg: Config, workers: int = 0, cache_dir: Optional[str] = None,
                  progress=None) -> List[Dict[str, np.ndarray]]:
    """Weights of every unit.

    ``workers > 1`` generates units in a thread pool.  ``cache_dir`` (or the
    ``SGD_SYNTH_CACHE`` environment variable) names a directory where each
    unit is stored as an uncompressed ``.npz`` after its first generation.
    ``progress(unit)`` is called after each unit is ready.
    """
    import os
    cache_dir = cache_dir or os.environ.get("SGD_SYNTH_CACHE") or None

    def one(u: int) -> Dict[str, np.ndarray]:
        w = _one(u)
        if progress is not None:
            progress(u)
        return w

    def _one(u: int) -> Dict[str, np.ndarray]:
        if cache_dir:
            path = os.path.join(cache_dir, f"{cfg.name}_{cfg.cfg_id}_{cfg.d}_{cfg.F}_u{u}.npz")
            if os.path.exists(path):
                with np.load(path, allow_pickle=False) as z:
                    return {k: z[k] for k in z.files}
            w = unit_weights(cfg, u)
            os.makedirs(cache_dir, exist_ok=True)
            tmp = path + f".tmp{os.getpid()}.npz"
            np.savez(tmp, **w)
            os.replace(tmp, path)
            return w
        return unit_weights(cfg, u)

    if workers and workers > 1 and cfg.L > 1:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(max_workers=workers) as ex:
            return list(ex.map(one, range(cfg.L)))
    return [one(u) for u in range(cfg.L)]


# --------------------------------------------------------------------------
# inputs
# --------------------------------------------------------------------------

def inputs(cfg: Config) -> Dict[str, np.ndarray]:
    """Initial state ``z`` [B, N, d] float32 plus conditioning."""
    rng = _rng(cfg.cfg_id, STREAM_INPUTS, 0, 0)
    B, N, d = cfg.B, cfg.N, cfg.d
    out: Dict[str, np.ndarray] = {}
    if cfg.arch == "llada":
        z = np.empty((B, N, d), dtype=np.float32)
        z[:, : cfg.prompt_rows] = rng.standard_normal((B, cfg.prompt_rows, d))
        mask_vec = rng.standard_normal(d)
        z[:, cfg.prompt_rows:] = mask_vec[None, None, :]
    elif cfg.arch == "uvit":
        z = rng.standard_normal((B, N, d)).astype(np.float32)
        z[:, 0] = 0.0  # time token: rewritten from the timestep at every step
    else:
        z = rng.standard_normal((B, N, d)).astype(np.float32)
    out["z"] = np.ascontiguousarray(z.astype(np.float32))
    crng = _rng(cfg.cfg_id, STREAM_COND, 0, 0)
    if cfg.arch in ("dit", "sdxl_unet"):
        out["class_emb"] = crng.standard_normal((B, d)).astype(np.float32)
    if cfg.arch in ("sdxl", "sdxl_unet"):
        ctx = crng.standard_normal((cfg.ctx_len, cfg.ctx_dim))
        out["ctx"] = np.ascontiguousarray(np.broadcast_to(store(ctx, cfg.dtype)[None],
                                                          (B, cfg.ctx_len, cfg.ctx_dim)))
    return out
