"""ctypes binding of ``include/sgd.h`` (argument marshalling only).

Every computation runs in ``libsgd.so``.  Torch tensors supply device buffers
(``data_ptr()``) and the current HIP stream.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
lib_path = os.path.join(_PKG, "lib", "libsgd.so")

SGD_F32, SGD_BF16 = 0, 1
SGD_ARCH = {"tiny": 0, "llada": 1, "dit": 2, "uvit": 3, "sdxl": 4, "sdxl_unet": 5}
SGD_UNIT = {"block": 0, "branch": 1}
SGD_RULE = {"scr_frob": 0, "random": 1, "depth": 2, "frob": 3, "spectral": 4, "stable_rank": 5,
            "frob_srank": 6, "raw_scr": 7}
SGD_ROLE = {"q": 0, "k": 1, "v": 2, "o": 3, "xq": 4, "xk": 5, "xv": 6, "xo": 7, "w1": 8, "w2": 9, "conv": 10}
SGD_K = {"norm": 0, "gemm_qkv": 1, "attn": 2, "gemm_o": 3, "gemm_w1": 4, "gemm_w2": 5, "frozen": 6,
         "state": 7, "cond": 8, "gemm_skip": 9, "gemm_x": 10, "attn_x": 11, "drift": 12, "gemm_conv": 13, "gnorm": 14, "fold": 15, "norm_parts": 16}
ERRORS = {-1: "SGD_E_ARG", -2: "SGD_E_SHAPE", -3: "SGD_E_DTYPE", -4: "SGD_E_BUDGET", -5: "SGD_E_STEP",
          -6: "SGD_E_CACHE", -7: "SGD_E_HIP", -8: "SGD_E_NUMERIC"}


class SgdError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


# ------------------------------------------------------------------ structs

class sgd_matrix(C.Structure):
    _fields_ = [("ptr", C.c_void_p), ("rows", C.c_int64), ("cols", C.c_int64),
                ("dtype", C.c_int32), ("role", C.c_int32)]


class sgd_unit(C.Structure):
    _fields_ = [("mats", C.POINTER(sgd_matrix)), ("n_mats", C.c_int32), ("head_dim", C.c_int32)]


class sgd_sched_params(C.Structure):
    _fields_ = [("T", C.c_int32), ("budget_layer_steps", C.c_int32), ("tau", C.c_double),
                ("s_min", C.c_int32), ("eta", C.c_double), ("budget_pct", C.c_int32), ("rule", C.c_int32),
                ("seed", C.c_uint64)]


class sgd_schedule(C.Structure):
    _fields_ = [("L", C.c_int32), ("T", C.c_int32), ("lifetimes", C.POINTER(C.c_int32)),
                ("active", C.POINTER(C.c_uint8)), ("unit_raw", C.POINTER(C.c_double)),
                ("unit_score", C.POINTER(C.c_double)), ("mat_stats", C.POINTER(C.c_double)),
                ("layer_steps", C.c_int64), ("cut_margin", C.c_double), ("s_min", C.c_int32)]


_W_FIELDS = ["norm1_w", "norm1_b", "w_qkv", "b_qkv", "w_o", "b_o", "norm2_w", "norm2_b", "w1", "b1", "w2", "b2",
             "normx_w", "normx_b", "w_xq", "w_xkv", "w_xo", "b_xo", "w_ada", "b_ada", "w_skip", "b_skip",
             "gn1_w", "gn1_b", "w_conv1", "b_conv1", "w_temb", "b_temb", "gn2_w", "gn2_b", "w_conv2", "b_conv2"]


class sgd_unit_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _W_FIELDS]


class sgd_model_desc(C.Structure):
    _fields_ = [("arch", C.c_int32), ("dtype", C.c_int32), ("B", C.c_int32), ("N", C.c_int32), ("d", C.c_int32),
                ("H", C.c_int32), ("head_dim", C.c_int32), ("F", C.c_int32), ("L", C.c_int32), ("T", C.c_int32),
                ("ctx_len", C.c_int32), ("ctx_dim", C.c_int32), ("update_row_begin", C.c_int32),
                ("update_row_end", C.c_int32), ("class_emb", C.c_void_p), ("ctx", C.c_void_p),
                ("units", C.POINTER(sgd_unit_weights)), ("grid", C.c_int32), ("groups", C.c_int32),
                ("granularity", C.c_int32)]


class sgd_replay_params(C.Structure):
    _fields_ = [("tau_agree", C.c_double), ("max_layer_steps", C.c_int64)]


class sgd_step_args(C.Structure):
    _fields_ = [("alpha", C.c_float), ("beta", C.c_float), ("workspace", C.c_void_p),
                ("workspace_bytes", C.c_size_t)]


# ------------------------------------------------------------------ library

_lib = None

EXPORTS = ["sgd_last_error", "sgd_version", "sgd_s_min_default", "sgd_budget_layer_steps",
           "sgd_schedule_workspace_bytes", "sgd_schedule_build", "sgd_matrix_stats", "sgd_schedule_from_scores",
           "sgd_schedule_from_stats",
           "sgd_schedule_from_lifetimes", "sgd_model_create", "sgd_model_destroy", "sgd_model_units", "sgd_workspace_bytes",
           "sgd_cache_bytes", "sgd_cache_bind", "sgd_cache_reset", "sgd_cache_destroy", "sgd_denoise_step",
           "sgd_denoise_step_noalloc", "sgd_graph_capture", "sgd_graph_launch", "sgd_graph_destroy",
           "sgd_denoise_step_masked", "sgd_drift_bytes", "sgd_drift_step", "sgd_replay_bytes", "sgd_replay_search",
           "sgd_profile_begin", "sgd_profile_end", "sgd_op_linear", "sgd_op_linear_split", "sgd_op_attention", "sgd_op_norm", "sgd_op_norm_fold",
           "sgd_op_frozen_run", "sgd_op_heads", "sgd_op_residual", "sgd_op_adaln_mod", "sgd_op_group_norm_silu",
           "sgd_op_group_norm_scratch_bytes", "sgd_op_conv3x3"]


def lib() -> C.CDLL:
    """Load libsgd.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(lib_path):
            raise ImportError(f"{lib_path} is missing: build it with `python -m paper_2609_29505_amd.build`")
        L = C.CDLL(lib_path)
        L.sgd_last_error.restype = C.c_char_p
        vp, i32, i64 = C.c_void_p, C.c_int32, C.c_int64
        sig = {
            "sgd_version": [],
            "sgd_budget_layer_steps": [i32, i32, i32, C.POINTER(i64)],
            "sgd_schedule_workspace_bytes": [C.POINTER(sgd_unit), i32, i32, C.POINTER(C.c_size_t)],
            "sgd_schedule_build": [C.POINTER(sgd_unit), i32, C.POINTER(sgd_sched_params), vp, C.c_size_t, vp,
                                   C.POINTER(sgd_schedule)],
            "sgd_matrix_stats": [C.POINTER(sgd_matrix), C.c_double, vp, C.c_size_t, vp, C.POINTER(C.c_double)],
            "sgd_schedule_from_scores": [C.POINTER(C.c_double), i32, C.POINTER(sgd_sched_params), C.POINTER(sgd_schedule)],
            "sgd_schedule_from_stats": [C.POINTER(sgd_unit), i32, C.POINTER(C.c_double), C.POINTER(sgd_sched_params),
                                        C.POINTER(sgd_schedule)],
            "sgd_schedule_from_lifetimes": [i32, i32, C.POINTER(C.c_int32), C.POINTER(sgd_schedule)],
            "sgd_model_create": [C.POINTER(sgd_model_desc), C.POINTER(vp)],
            "sgd_model_destroy": [vp],
            "sgd_model_units": [vp, C.POINTER(C.c_int32)],
            "sgd_graph_capture": [vp, vp, C.POINTER(sgd_schedule), vp, C.POINTER(C.c_float), C.POINTER(C.c_float),
                                  vp, C.c_size_t, vp, C.POINTER(vp)],
            "sgd_graph_launch": [vp, vp],
            "sgd_graph_destroy": [vp],
            "sgd_workspace_bytes": [vp, C.POINTER(C.c_size_t)],
            "sgd_cache_bytes": [vp, C.POINTER(C.c_size_t)],
            "sgd_cache_bind": [vp, vp, C.c_size_t, C.POINTER(vp)],
            "sgd_cache_reset": [vp],
            "sgd_cache_destroy": [vp],
            "sgd_denoise_step": [vp, vp, i32, C.POINTER(sgd_schedule), vp, C.POINTER(sgd_step_args), vp],
            "sgd_denoise_step_masked": [vp, vp, i32, C.POINTER(C.c_uint8), vp, C.POINTER(sgd_step_args), vp],
            "sgd_denoise_step_noalloc": [vp, vp, i32, C.POINTER(sgd_schedule), vp, C.c_float, C.c_float, vp],
            "sgd_drift_bytes": [vp, C.POINTER(C.c_size_t)],
            "sgd_drift_step": [vp, vp, i32, C.POINTER(sgd_schedule), vp, C.POINTER(sgd_step_args), vp, C.c_size_t,
                               C.POINTER(C.c_uint8), C.POINTER(C.c_double), vp],
            "sgd_replay_bytes": [vp, C.POINTER(C.c_size_t)],
            "sgd_replay_search": [vp, vp, C.POINTER(sgd_replay_params), C.POINTER(sgd_step_args), vp, C.c_size_t,
                                  C.POINTER(C.c_int32), C.POINTER(i64), C.POINTER(C.c_double), vp],
            "sgd_profile_begin": [vp, i32, i32],
            "sgd_profile_end": [vp, C.POINTER(C.c_double), C.POINTER(i64)],
            "sgd_op_linear": [i32, vp, i64, vp, i64, vp, vp, i64, i32, i32, i32, i32, i32, i32, vp],
            "sgd_op_linear_split": [i32, vp, vp, vp, vp, i64, i32, i32, i32, i32, vp],
            "sgd_op_attention": [i32, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, vp],
            "sgd_op_norm": [i32, i32, vp, vp, i32, i32, C.c_float, vp, vp, vp, vp, i64, i32, vp],
            "sgd_op_norm_fold": [i32, i32, vp, vp, i32, i32, C.c_float, vp, vp, vp, vp, i64, i32,
                                 C.POINTER(vp), i32, vp],
            "sgd_op_frozen_run": [vp, C.POINTER(vp), i32, i64, vp],
            "sgd_op_heads": [i32, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, i32, i32, i32, vp],
            "sgd_op_residual": [i32, vp, i64, vp, vp, vp, vp, i32, vp, i64, i32, i32, i32, i32, i32, vp],
            "sgd_op_adaln_mod": [i32, vp, vp, vp, vp, i32, i32, i32, vp],
            "sgd_op_group_norm_scratch_bytes": [i32, i32, i32, C.POINTER(C.c_size_t)],
            "sgd_op_group_norm_silu": [i32, vp, vp, i32, i32, i32, i32, C.c_float, vp, vp, vp, C.c_size_t, vp],
            "sgd_op_conv3x3": [vp, vp, vp, vp, i32, vp, vp, i32, i32, i32, i32, vp],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = C.c_int
        L.sgd_s_min_default.argtypes = [i32]
        L.sgd_s_min_default.restype = C.c_int32
        _lib = L
    return _lib


def _check(rc: int) -> None:
    if rc != 0:
        raise SgdError(rc, lib().sgd_last_error().decode())


def s_min_default(T: int) -> int:
    """The library's default minimum lifetime (sgd_s_min_default)."""
    return int(lib().sgd_s_min_default(T))


def budget_layer_steps(pct: int, L: int, T: int) -> int:
    """The library's layer-step ceiling of a percentage budget (sgd_budget_layer_steps)."""
    n = C.c_int64()
    _check(lib().sgd_budget_layer_steps(pct, L, T, C.byref(n)))
    return int(n.value)


# ------------------------------------------------------------------ schedule

class Schedule:
    """Host arrays of an ``sgd_schedule`` plus the struct that points at them."""

    def __init__(self, L: int, T: int, n_mats: int = 0):
        self.lifetimes = np.zeros(L, np.int32)
        self.active = np.zeros((T, L), np.uint8)
        self.unit_raw = np.zeros(L, np.float64)
        self.unit_score = np.zeros(L, np.float64)
        self.mat_stats = np.zeros((max(n_mats, 1), 6), np.float64)
        self.c = sgd_schedule()
        self.c.L, self.c.T = L, T
        self.c.lifetimes = self.lifetimes.ctypes.data_as(C.POINTER(C.c_int32))
        self.c.active = self.active.ctypes.data_as(C.POINTER(C.c_uint8))
        self.c.unit_raw = self.unit_raw.ctypes.data_as(C.POINTER(C.c_double))
        self.c.unit_score = self.unit_score.ctypes.data_as(C.POINTER(C.c_double))
        self.c.mat_stats = self.mat_stats.ctypes.data_as(C.POINTER(C.c_double)) if n_mats else None

    @property
    def layer_steps(self) -> int:
        return int(self.c.layer_steps)

    @property
    def cut_margin(self) -> float:
        return float(self.c.cut_margin)

    @property
    def s_min(self) -> int:
        return int(self.c.s_min)


def _params(T, budget=None, tau=1.0, s_min=None, eta=1e-6, budget_pct=None, rule="scr_frob", seed=0):
    """budget: N* layer-steps; budget_pct: a percentage the library turns into N*; neither:
    tau mode.  s_min None: the library's default."""
    p = sgd_sched_params()
    p.T = T
    p.budget_layer_steps = -1 if budget is None else int(budget)
    p.budget_pct = 0 if budget_pct is None else int(budget_pct)
    p.tau = tau
    p.s_min = 0 if s_min is None else s_min
    p.eta = eta
    p.rule = SGD_RULE[rule]
    p.seed = seed
    return p


def _stream_ptr(stream=None) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return SGD_BF16
    if t.dtype == torch.float32:
        return SGD_F32
    raise ValueError(f"unsupported dtype {t.dtype}")


def _workspace(nbytes: int):
    import torch
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")


def schedule_build(units: Optional[Sequence[Sequence[tuple]]], head_dims: Optional[Sequence[int]], T: int,
                   budget=None, tau=1.0, s_min=None, eta=1e-6, budget_pct=None, rule="scr_frob", seed=0,
                   workers=16, L=None, stream=None) -> Schedule:
    """``units[l]`` is a list of ``(role, tensor)`` pairs (2-D device tensors, bf16 or fp32).
    ``units`` may be None for the depth and random rules (then ``L`` gives the unit count)."""
    if units is None:
        sch = Schedule(L, T)
        p = _params(T, budget, tau, s_min, eta, budget_pct, rule, seed)
        _check(lib().sgd_schedule_build(None, L, C.byref(p), None, 0, None, C.byref(sch.c)))
        return sch
    L = len(units)
    mats_keep = []
    cunits = (sgd_unit * L)()
    n_total = 0
    for l, mats in enumerate(units):
        arr = (sgd_matrix * len(mats))()
        for i, (role, t) in enumerate(mats):
            assert t.is_cuda and t.dim() == 2 and t.is_contiguous()
            arr[i].ptr = t.data_ptr()
            arr[i].rows, arr[i].cols = t.shape
            arr[i].dtype = _dtype_code(t)
            arr[i].role = SGD_ROLE[role]
        mats_keep.append(arr)
        cunits[l].mats = C.cast(arr, C.POINTER(sgd_matrix))
        cunits[l].n_mats = len(mats)
        cunits[l].head_dim = int(head_dims[l])
        n_total += len(mats)
    sch = Schedule(L, T, n_total)
    p = _params(T, budget, tau, s_min, eta, budget_pct, rule, seed)
    nb = C.c_size_t()
    _check(lib().sgd_schedule_workspace_bytes(cunits, L, workers, C.byref(nb)))
    ws = _workspace(nb.value)
    _check(lib().sgd_schedule_build(cunits, L, C.byref(p), C.c_void_p(ws.data_ptr()), ws.numel(),
                                    C.c_void_p(_stream_ptr(stream)), C.byref(sch.c)))
    del ws
    return sch


def matrix_stats(t, eta=1e-6, role="w1", stream=None) -> np.ndarray:
    """{E_k, tail energy, ||W||_F^2, SCR_eta, g, ||W||_2^2} of one device matrix."""
    m = sgd_matrix()
    m.ptr = t.data_ptr()
    m.rows, m.cols = t.shape
    m.dtype = _dtype_code(t)
    m.role = SGD_ROLE[role]
    u = sgd_unit()
    u.mats = C.pointer(m)
    u.n_mats = 1
    u.head_dim = 1
    nb = C.c_size_t()
    _check(lib().sgd_schedule_workspace_bytes(C.byref(u), 1, 1, C.byref(nb)))
    ws = _workspace(nb.value)
    out = (C.c_double * 6)()
    _check(lib().sgd_matrix_stats(C.byref(m), eta, C.c_void_p(ws.data_ptr()), ws.numel(),
                                  C.c_void_p(_stream_ptr(stream)), out))
    return np.array(list(out))


def schedule_from_scores(scores: Sequence[float], T: int, budget=None, tau=1.0, s_min=None,
                         budget_pct=None) -> Schedule:
    sc = np.ascontiguousarray(scores, dtype=np.float64)
    sch = Schedule(len(sc), T)
    p = _params(T, budget, tau, s_min, budget_pct=budget_pct)
    _check(lib().sgd_schedule_from_scores(sc.ctypes.data_as(C.POINTER(C.c_double)), len(sc), C.byref(p),
                                          C.byref(sch.c)))
    return sch


def schedule_from_stats(roles: Sequence[Sequence[str]], head_dims: Sequence[int], mat_stats, T: int, budget=None,
                        tau=1.0, s_min=None, eta=1e-6, budget_pct=None, rule="scr_frob", seed=0) -> Schedule:
    """A rule's schedule from per-matrix statistics (``mat_stats`` [n, 6], the rows an earlier
    ``schedule_build`` returned); ``roles[l]`` lists unit l's matrix roles in that order."""
    L = len(roles)
    st = np.ascontiguousarray(mat_stats, dtype=np.float64)
    keep = []
    cunits = (sgd_unit * L)()
    for l, rl in enumerate(roles):
        arr = (sgd_matrix * len(rl))()
        for i, r in enumerate(rl):
            arr[i].role = SGD_ROLE[r]
        keep.append(arr)
        cunits[l].mats = C.cast(arr, C.POINTER(sgd_matrix))
        cunits[l].n_mats = len(rl)
        cunits[l].head_dim = int(head_dims[l])
    assert st.shape == (sum(len(r) for r in roles), 6)
    sch = Schedule(L, T)
    p = _params(T, budget, tau, s_min, eta, budget_pct, rule, seed)
    _check(lib().sgd_schedule_from_stats(cunits, L, st.ctypes.data_as(C.POINTER(C.c_double)), C.byref(p),
                                         C.byref(sch.c)))
    return sch


def schedule_from_lifetimes(lifetimes: Sequence[int], T: int) -> Schedule:
    lt = np.ascontiguousarray(lifetimes, dtype=np.int32)
    sch = Schedule(len(lt), T)
    _check(lib().sgd_schedule_from_lifetimes(len(lt), T, lt.ctypes.data_as(C.POINTER(C.c_int32)), C.byref(sch.c)))
    return sch


# ------------------------------------------------------------------ single ops

def _p(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def op_linear(A, W, out, bias=None, act=0, gated=False, tile=0, stream=None) -> None:
    """out = act(A W^T + bias) (or the gated form); 2-D contiguous device tensors."""
    M, K = A.shape
    N = out.shape[1]
    _check(lib().sgd_op_linear(_dtype_code(A), _p(A), A.stride(0), _p(W), W.stride(0), _p(bias), _p(out),
                               out.stride(0), M, N, K, act, int(gated), tile, C.c_void_p(_stream_ptr(stream))))


def op_linear_split(A, W, parts, bias=None, stream=None) -> None:
    """parts[s] = A[:, K_s] W[:, K_s]^T (+ bias for s = 0) over ksplit = parts.shape[0] K ranges;
    A [M, K], W [N, K] bf16, parts [ksplit, M, N] fp32, contiguous device tensors."""
    M, K = A.shape
    ks, _, N = parts.shape
    _check(lib().sgd_op_linear_split(_dtype_code(A), _p(A), _p(W), _p(bias), _p(parts), parts.stride(0), M, N, K,
                                     ks, C.c_void_p(_stream_ptr(stream))))


def op_attention(q, k, vt, o, B, H, dh, nq, nk, stream=None) -> None:
    npq, npk = q.shape[-2], k.shape[-2]
    _check(lib().sgd_op_attention(_dtype_code(q), _p(q), _p(k), _p(vt), _p(o), B, H, dh, nq, npq, nk, npk,
                                  C.c_void_p(_stream_ptr(stream))))


def op_norm(kind, x, y, eps, w=None, b=None, shift=None, scale=None, ntok=1, stream=None) -> None:
    M, d = x.shape
    mod_ld = shift.stride(0) if shift is not None else 0
    _check(lib().sgd_op_norm(_dtype_code(y), kind, _p(x), _p(y), M, d, eps, _p(w), _p(b), _p(shift), _p(scale),
                             mod_ld, ntok, C.c_void_p(_stream_ptr(stream))))


def op_norm_fold(kind, x, y, eps, deltas, w=None, b=None, shift=None, scale=None, ntok=1, stream=None) -> None:
    """x += deltas[0] + ... (in order, written back), then the pre-norm of x into y."""
    M, d = x.shape
    mod_ld = shift.stride(0) if shift is not None else 0
    arr = (C.c_void_p * len(deltas))(*[t.data_ptr() for t in deltas])
    _check(lib().sgd_op_norm_fold(_dtype_code(y), kind, _p(x), _p(y), M, d, eps, _p(w), _p(b), _p(shift), _p(scale),
                                  mod_ld, ntok, arr, len(deltas), C.c_void_p(_stream_ptr(stream))))


def op_heads(A, W, q, k, vt, n_proj, which0, ntok, H, dh, bias=None, rope=False, tile=0, stream=None) -> None:
    M, K = A.shape
    np_ = (q if q is not None else k).shape[-2]
    _check(lib().sgd_op_heads(_dtype_code(A), _p(A), _p(W), _p(bias), _p(q), _p(k), _p(vt), M, K, n_proj, which0,
                              ntok, np_, H, dh, int(rope), tile, C.c_void_p(_stream_ptr(stream))))


def op_residual(A, W, h, bias=None, delta=None, delta_mode=0, gate=None, ntok=1, tile=0, stream=None) -> None:
    M, K = A.shape
    N = h.shape[1]
    gate_ld = gate.stride(0) if gate is not None else 0
    _check(lib().sgd_op_residual(_dtype_code(A), _p(A), A.stride(0), _p(W), _p(bias), _p(h), _p(delta), delta_mode,
                                 _p(gate), gate_ld, ntok, M, N, K, tile, C.c_void_p(_stream_ptr(stream))))


def op_adaln_mod(x, W, mod, bias=None, stream=None) -> None:
    B, d = x.shape
    _check(lib().sgd_op_adaln_mod(_dtype_code(W), _p(x), _p(W), _p(bias), _p(mod), B, d, W.shape[0],
                                  C.c_void_p(_stream_ptr(stream))))


def op_group_norm_silu(x, y, groups, w, b, eps=1e-5, stream=None) -> None:
    """y = SiLU(GroupNorm(x) w + b) for x [B, N, C] (fp32 or bf16), y bf16 [B, N, C]."""
    B, N, Cc = x.shape
    nb = C.c_size_t()
    _check(lib().sgd_op_group_norm_scratch_bytes(B, N, groups, C.byref(nb)))
    scratch = _workspace(nb.value)
    _check(lib().sgd_op_group_norm_silu(_dtype_code(x), _p(x), _p(y), B, N, Cc, groups, eps, _p(w), _p(b),
                                        _p(scratch), scratch.numel(), C.c_void_p(_stream_ptr(stream))))


def op_conv3x3(A, W, side, out=None, h=None, bias=None, rowbias=None, tile=0, stream=None) -> None:
    """3x3 convolution of A [M, Cin] (grids of side x side) with W [N, 9 Cin] (see sgd_ops.h)."""
    M, Cin = A.shape
    N = W.shape[0]
    _check(lib().sgd_op_conv3x3(_p(A), _p(W), _p(bias), _p(rowbias), side, _p(out), _p(h), M, N, Cin, tile,
                                C.c_void_p(_stream_ptr(stream))))


def op_frozen_run(h, deltas, stream=None) -> None:
    arr = (C.c_void_p * len(deltas))(*[t.data_ptr() for t in deltas])
    _check(lib().sgd_op_frozen_run(_p(h), arr, len(deltas), h.numel(), C.c_void_p(_stream_ptr(stream))))


# ------------------------------------------------------------------ model

def _to_device(arr: np.ndarray, dtype: str):
    """numpy storage array -> device tensor (uint16 bit patterns are reinterpreted as bf16).
    The host tensor is only read (copied to the device), so read-only arrays are used as they are."""
    import warnings

    import torch
    with warnings.catch_warnings():
        warnings.filterwarnings("ignore", message="The given NumPy array is not writable")
        if arr.dtype == np.uint16:
            t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16)
        else:
            t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32))
    return t.to("cuda", non_blocking=False)


class DeviceModel:
    """Uploads one workload's weights and inputs and owns the ``sgd_model`` handle."""

    def __init__(self, cfg, weights: List[Dict[str, np.ndarray]], inputs: Dict[str, np.ndarray],
                 granularity: str = "block", share: Optional["DeviceModel"] = None):
        """``granularity``: "block" (one scheduled unit per block) or "branch" (one per residual
        branch; see sgd_granularity).  ``share``: a model of the same workload whose device
        weights and inputs this one uses instead of uploading its own."""
        import torch
        self.cfg = cfg
        self.granularity = granularity
        self.dtype = SGD_BF16 if cfg.dtype == "bf16" else SGD_F32
        self.tensors: List[Dict[str, "torch.Tensor"]] = []
        cw = (sgd_unit_weights * cfg.L)()
        for l in range(cfg.L):
            if share is not None:
                dev = share.tensors[l]
            else:
                dev = {k: _to_device(v, cfg.dtype) for k, v in weights[l].items() if not k.startswith("_")}
            self.tensors.append(dev)
            for name in _W_FIELDS:
                if name in dev:
                    setattr(cw[l], name, dev[name].data_ptr())
        self._cw = cw
        if share is not None:
            self.class_emb, self.ctx = share.class_emb, share.ctx
        else:
            self.class_emb = _to_device(inputs["class_emb"], "f32") if "class_emb" in inputs else None
            self.ctx = _to_device(inputs["ctx"], cfg.dtype) if "ctx" in inputs else None
        d = sgd_model_desc()
        d.arch, d.dtype = SGD_ARCH[cfg.arch], self.dtype
        d.B, d.N, d.d, d.H, d.head_dim, d.F, d.L, d.T = cfg.B, cfg.N, cfg.d, cfg.H, cfg.dh, cfg.F, cfg.L, cfg.T
        d.ctx_len, d.ctx_dim = cfg.ctx_len, cfg.ctx_dim
        d.update_row_begin, d.update_row_end = cfg.update_rows
        d.class_emb = self.class_emb.data_ptr() if self.class_emb is not None else None
        d.ctx = self.ctx.data_ptr() if self.ctx is not None else None
        d.units = C.cast(cw, C.POINTER(sgd_unit_weights))
        d.grid, d.groups = cfg.grid, cfg.groups
        d.granularity = SGD_UNIT[granularity]
        h = C.c_void_p()
        _check(lib().sgd_model_create(C.byref(d), C.byref(h)))
        self.h = h
        nu = C.c_int32()
        _check(lib().sgd_model_units(h, C.byref(nu)))
        self.n_units = int(nu.value)
        ws = C.c_size_t()
        _check(lib().sgd_workspace_bytes(h, C.byref(ws)))
        self.workspace_bytes = int(ws.value)
        cb = C.c_size_t()
        _check(lib().sgd_cache_bytes(h, C.byref(cb)))
        self.cache_bytes = int(cb.value)
        self.workspace = torch.empty(max(self.workspace_bytes, 256), dtype=torch.uint8, device="cuda")

    def scored_units(self):
        """Per scheduled unit, the (role, device tensor) pairs the schedule scores (views of fused
        storage): a block's matrices, or with branch units one branch's, in execution order."""
        cfg, d = self.cfg, self.cfg.d
        out = []
        for dev in self.tensors:
            qkv = dev["w_qkv"]
            parts = []
            if "w_conv1" in dev:
                parts.append([("conv", dev["w_conv1"]), ("conv", dev["w_conv2"])])
            parts.append([("q", qkv[:d]), ("k", qkv[d:2 * d]), ("v", qkv[2 * d:]), ("o", dev["w_o"])])
            if "w_xq" in dev:
                xkv = dev["w_xkv"]
                parts.append([("xq", dev["w_xq"]), ("xk", xkv[:d]), ("xv", xkv[d:]), ("xo", dev["w_xo"])])
            parts.append([("w1", dev["w1"]), ("w2", dev["w2"])])
            if self.granularity == "branch":
                out.extend(parts)
            else:
                # a block lists its attention matrices first (the order of mat_stats)
                order = [1, 0] + list(range(2, len(parts))) if "w_conv1" in dev else range(len(parts))
                out.append([m for i in order for m in parts[i]])
        return out

    def step(self, state, s: int, sched: Optional[Schedule], cache: Optional["Cache"], alpha=1.0, beta=None,
             stream=None) -> None:
        a = self._args(alpha, beta)
        _check(lib().sgd_denoise_step(self.h, C.c_void_p(state.data_ptr()), s,
                                      C.byref(sched.c) if sched is not None else None,
                                      cache.h if cache is not None else None, C.byref(a),
                                      C.c_void_p(_stream_ptr(stream))))

    def _args(self, alpha=1.0, beta=None):
        a = sgd_step_args()
        a.alpha = alpha
        a.beta = (1.0 / self.cfg.T) if beta is None else beta
        a.workspace = self.workspace.data_ptr()
        a.workspace_bytes = self.workspace.numel()
        return a

    def capture(self, state, sched: Optional[Schedule], cache: Optional["Cache"], stream, alpha=1.0, beta=None):
        """The whole T-step trajectory on ``state`` as one HIP graph (sgd_graph_capture), captured
        on ``stream`` (a torch.cuda.Stream, not the null stream)."""
        T = self.cfg.T
        al = np.full(T, alpha, np.float32)
        be = np.full(T, (1.0 / T) if beta is None else beta, np.float32)
        g = C.c_void_p()
        _check(lib().sgd_graph_capture(self.h, C.c_void_p(state.data_ptr()),
                                       C.byref(sched.c) if sched is not None else None,
                                       cache.h if cache is not None else None,
                                       al.ctypes.data_as(C.POINTER(C.c_float)), be.ctypes.data_as(C.POINTER(C.c_float)),
                                       C.c_void_p(self.workspace.data_ptr()), self.workspace.numel(),
                                       C.c_void_p(_stream_ptr(stream)), C.byref(g)))
        return Graph(g, keep=(state, sched, cache, self))

    def step_noalloc(self, state, s: int, sched: Optional[Schedule], cache: Optional["Cache"], alpha=1.0, beta=None,
                     stream=None) -> None:
        """sgd_denoise_step on the library's fixed scratch (no workspace, no allocation)."""
        beta = (1.0 / self.cfg.T) if beta is None else beta
        _check(lib().sgd_denoise_step_noalloc(self.h, C.c_void_p(state.data_ptr()), s,
                                              C.byref(sched.c) if sched is not None else None,
                                              cache.h if cache is not None else None, alpha, beta,
                                              C.c_void_p(_stream_ptr(stream))))

    def step_masked(self, state, s: int, active_row, cache: "Cache", alpha=1.0, beta=None, stream=None) -> None:
        """One step with an arbitrary active set (``active_row``: one flag per scheduled unit)."""
        row = np.ascontiguousarray(active_row, dtype=np.uint8)
        a = self._args(alpha, beta)
        _check(lib().sgd_denoise_step_masked(self.h, C.c_void_p(state.data_ptr()), s,
                                             row.ctypes.data_as(C.POINTER(C.c_uint8)), cache.h, C.byref(a),
                                             C.c_void_p(_stream_ptr(stream))))

    def drift_buffer(self):
        """A device buffer of sgd_drift_bytes for drift_step."""
        nb = C.c_size_t()
        _check(lib().sgd_drift_bytes(self.h, C.byref(nb)))
        return _workspace(nb.value)

    def drift_step(self, state, s: int, sched: Schedule, cache: "Cache", drift_buf, alpha=1.0, beta=None,
                   stream=None):
        """One step of the causal activation-drift policy; returns (active row, lagged drift)."""
        L = self.n_units
        row = np.zeros(L, np.uint8)
        dr = np.zeros(L, np.float64)
        a = self._args(alpha, beta)
        _check(lib().sgd_drift_step(self.h, C.c_void_p(state.data_ptr()), s, C.byref(sched.c), cache.h, C.byref(a),
                                    C.c_void_p(drift_buf.data_ptr()), drift_buf.numel(),
                                    row.ctypes.data_as(C.POINTER(C.c_uint8)),
                                    dr.ctypes.data_as(C.POINTER(C.c_double)), C.c_void_p(_stream_ptr(stream))))
        return row, dr

    def replay_search(self, z1, tau_agree=5e-3, max_layer_steps=0, alpha=1.0, beta=None, log=False, stream=None):
        """Oracle-replay search from z1; returns (lifetimes, evaluations, delta log or None)."""
        L, T = self.n_units, self.cfg.T
        nb = C.c_size_t()
        _check(lib().sgd_replay_bytes(self.h, C.byref(nb)))
        buf = _workspace(nb.value)
        p = sgd_replay_params()
        p.tau_agree = tau_agree
        p.max_layer_steps = max_layer_steps
        life = np.zeros(L, np.int32)
        ev = C.c_int64()
        dlog = np.zeros(T * L * L, np.float64) if log else None
        a = self._args(alpha, beta)
        _check(lib().sgd_replay_search(self.h, C.c_void_p(z1.data_ptr()), C.byref(p), C.byref(a),
                                       C.c_void_p(buf.data_ptr()), buf.numel(),
                                       life.ctypes.data_as(C.POINTER(C.c_int32)), C.byref(ev),
                                       dlog.ctypes.data_as(C.POINTER(C.c_double)) if log else None,
                                       C.c_void_p(_stream_ptr(stream))))
        del buf
        return life, int(ev.value), (dlog.reshape(T, L, L) if log else None)

    def profile_begin(self, kclass: str, max_launches: int = 4096) -> None:
        _check(lib().sgd_profile_begin(self.h, SGD_K[kclass] if kclass else -1, max_launches))

    def profile_end(self):
        ms, n = C.c_double(), C.c_int64()
        _check(lib().sgd_profile_end(self.h, C.byref(ms), C.byref(n)))
        return float(ms.value), int(n.value)

    def close(self) -> None:
        if getattr(self, "h", None):
            lib().sgd_model_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Graph:
    """A captured trajectory (sgd_graph); keeps the buffers whose addresses it recorded alive."""

    def __init__(self, h, keep):
        self.h, self._keep = h, keep

    def launch(self, stream) -> None:
        _check(lib().sgd_graph_launch(self.h, C.c_void_p(_stream_ptr(stream))))

    def close(self) -> None:
        if getattr(self, "h", None):
            lib().sgd_graph_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Cache:
    """Per-trajectory delta cache bound to a device buffer."""

    def __init__(self, model: DeviceModel):
        import torch
        self.buf = torch.empty(max(model.cache_bytes, 256), dtype=torch.uint8, device="cuda")
        h = C.c_void_p()
        _check(lib().sgd_cache_bind(model.h, C.c_void_p(self.buf.data_ptr()), self.buf.numel(), C.byref(h)))
        self.h = h

    def reset(self) -> None:
        _check(lib().sgd_cache_reset(self.h))

    def __del__(self):
        try:
            if getattr(self, "h", None):
                lib().sgd_cache_destroy(self.h)
                self.h = None
        except Exception:
            pass
