"""Spectral scores of weight matrices and residual units (oracle).

Follows Sec. 3.2 (Definition "Regularized Spectral Concentration Ratio",
Eq. scr-reg) and the appendix "Exact Block-Level Scores" (Eqs.
app-matrix-score, app-attn-score, app-xattn-score, app-mlp-score,
app-conv-score, app-block-score, app-score-normalization).

All arithmetic is float64 on the stored weights upcast exactly.

Readings where the paper is silent:
* the default regulariser is eta = 1e-6 (the paper uses the regularised
  form in implementation but never prints eta);
* a gated MLP's input projection W1 is the stacked [W_gate; W_up] matrix;
* fused QKV storage is scored as the three d x d blocks separately.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np

from .numerics import decode

DEFAULT_ETA = 1e-6
NORMALISATION_EPS = 1e-12  # epsilon of Eq. app-score-normalization


def rank_k(m: int, n: int) -> int:
    """k = min(d, max(1, floor(0.1 d))) with d = min(m, n)  (Definition of SCR_eta)."""
    d = min(m, n)
    return min(d, max(1, d // 10))


def singular_values_sq(w: np.ndarray) -> np.ndarray:
    """Squared singular values of ``w`` (float64), descending.

    Small matrices use LAPACK's SVD; larger ones the eigenvalues of the
    Gram matrix of the short side (clamped at zero), which are the squared
    singular values by definition.
    """
    m, n = w.shape
    d = min(m, n)
    if d <= 1024:
        s = np.linalg.svd(w, compute_uv=False)
        return np.sort(s * s)[::-1]
    g = w.T @ w if n <= m else w @ w.T
    lam = np.linalg.eigvalsh(g)
    return np.sort(np.maximum(lam, 0.0))[::-1]


@dataclass
class MatrixStats:
    m: int
    n: int
    k: int
    energy_top: float   # E_k = sum_{i<=k} sigma_i^2
    energy_tail: float  # sum_{i>k} sigma_i^2
    frob_sq: float      # ||W||_F^2 = sum_ij W_ij^2
    scr: float          # SCR_eta (Eq. scr-reg)
    g: float            # ||W||_F sqrt(rho(SCR_eta))  (Eq. app-matrix-score)
    sigma1_sq: float = 0.0  # largest squared singular value ||W||_2^2 (spectral-norm and
                            # stable-rank rankings of Sec. "Static ranking comparisons")


def matrix_stats(w64: np.ndarray, eta: float = DEFAULT_ETA) -> MatrixStats:
    """SCR_eta and g(W) of one matrix (Eq. scr-reg, Eq. app-matrix-score).

    SCR_eta = log((E_k + eta F) / (tail + eta F)) with F = ||W||_F^2.
    rho(u) = e^u / (1 + e^u); at u = SCR_eta this equals A / (A + B) with
    A = E_k + eta F and B = tail + eta F, which is evaluated directly.
    """
    w64 = np.asarray(w64, dtype=np.float64)
    m, n = w64.shape
    k = rank_k(m, n)
    lam = singular_values_sq(w64)
    e_top = float(np.sum(lam[:k]))
    e_tail = float(np.sum(lam[k:]))
    frob_sq = float(np.sum(w64 * w64))
    a = e_top + eta * frob_sq
    b = e_tail + eta * frob_sq
    scr = math.log(a / b) if b > 0 else math.inf
    rho = a / (a + b) if (a + b) > 0 else 0.0
    g = math.sqrt(frob_sq) * math.sqrt(rho)
    return MatrixStats(m, n, k, e_top, e_tail, frob_sq, scr, g, float(lam[0]))


def rho_of(u: float) -> float:
    """rho(u) = e^u / (1 + e^u) (Lemma "Spectral energy sandwich")."""
    if u == math.inf:
        return 1.0
    return 1.0 / (1.0 + math.exp(-u))


# --------------------------------------------------------------------------
# component and unit scores
# --------------------------------------------------------------------------

def q_attn(g_q: float, g_k: float, g_v: float, g_o: float, head_dim: int) -> float:
    """q_attn = g(W_O) g(W_V) [1 + g(W_Q) g(W_K) / sqrt(d_h)]  (Eq. app-attn-score; also
    Eq. app-xattn-score with the cross-attention projections)."""
    return g_o * g_v * (1.0 + g_q * g_k / math.sqrt(head_dim))


def q_mlp(g_w1: float, g_w2: float) -> float:
    """q_mlp = g(W_2) g(W_1)  (Eq. app-mlp-score)."""
    return g_w2 * g_w1


def q_conv(g_kernel: float) -> float:
    """q_conv = g(W_K) of the unfolded C_out x (C_in k_h k_w) kernel (Eq. app-conv-score)."""
    return g_kernel


def unfold_conv(kernel: np.ndarray) -> np.ndarray:
    """C_out x C_in x k_h x k_w -> C_out x (C_in k_h k_w)."""
    c_out = kernel.shape[0]
    return np.asarray(kernel).reshape(c_out, -1)


def normalise(raw: Sequence[float]) -> np.ndarray:
    """Lambda_hat_l = q~_l / (max_j q~_j + eps), eps = 1e-12  (Eq. app-score-normalization)."""
    raw = np.asarray(raw, dtype=np.float64)
    return raw / (np.max(raw) + NORMALISATION_EPS)


# matrix roles of a scheduled unit
ATTN_ROLES = ("q", "k", "v", "o")
XATTN_ROLES = ("xq", "xk", "xv", "xo")
MLP_ROLES = ("w1", "w2")
CONV_ROLES = ("conv1", "conv2")
BRANCH_ROLES = {"resnet": CONV_ROLES, "attn": ATTN_ROLES, "xattn": XATTN_ROLES, "mlp": MLP_ROLES}


def branch_matrices(mats: Dict[str, np.ndarray], branch: str) -> Dict[str, np.ndarray]:
    """The scored matrices of one residual branch of a block (a unit at branch granularity):
    its score is that branch's component of Eq. app-block-score alone."""
    return {r: mats[r] for r in BRANCH_ROLES[branch]}


def unit_matrices(weights: Dict[str, np.ndarray], d: int, dtype: str) -> Dict[str, np.ndarray]:
    """The scored matrices of one unit, as float64 (fused storage split into its blocks)."""
    out: Dict[str, np.ndarray] = {}
    qkv = decode(weights["w_qkv"], dtype)
    out["q"], out["k"], out["v"] = qkv[:d], qkv[d:2 * d], qkv[2 * d:]
    out["o"] = decode(weights["w_o"], dtype)
    out["w1"] = decode(weights["w1"], dtype)
    out["w2"] = decode(weights["w2"], dtype)
    if "w_conv1" in weights:
        # SDXL UNet ResNet block: the kernels as stored unfolded, [C_out, 9 C_in]; the paper
        # unfolds to C_out x (C_in k_h k_w), a column permutation of this matrix, which has
        # the same singular values (Eq. app-conv-score)
        out["conv1"] = decode(weights["w_conv1"], dtype)
        out["conv2"] = decode(weights["w_conv2"], dtype)
    if "w_xq" in weights:
        out["xq"] = decode(weights["w_xq"], dtype)
        xkv = decode(weights["w_xkv"], dtype)
        out["xk"], out["xv"] = xkv[:d], xkv[d:]
        out["xo"] = decode(weights["w_xo"], dtype)
    return out


@dataclass
class UnitScore:
    stats: Dict[str, MatrixStats]
    raw: float  # q~_l


def unit_score(mats: Dict[str, np.ndarray], head_dim: int, eta: float = DEFAULT_ETA) -> UnitScore:
    """q~_l = sum of the unit's component scores (Eq. app-block-score).

    A transformer block holds a self-attention and an MLP component; an SDXL
    spatial-transformer block adds a cross-attention component; an SDXL UNet unit adds its
    ResNet block's two convolutions, one q_conv component each.
    """
    stats = {role: matrix_stats(w, eta) for role, w in mats.items()}
    g = {role: s.g for role, s in stats.items()}
    raw = 0.0
    if all(r in g for r in ATTN_ROLES):
        raw += q_attn(g["q"], g["k"], g["v"], g["o"], head_dim)
    if all(r in g for r in XATTN_ROLES):
        raw += q_attn(g["xq"], g["xk"], g["xv"], g["xo"], head_dim)
    if all(r in g for r in MLP_ROLES):
        raw += q_mlp(g["w1"], g["w2"])
    for role in sorted(g):
        if role.startswith("conv"):
            raw += q_conv(g[role])
    return UnitScore(stats, raw)
