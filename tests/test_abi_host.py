"""C-ABI tests that need no GPU: the library loads, exports what include/sgd.h declares,
and its host-side schedule logic matches the oracle bit for bit."""
import os
import re

import numpy as np
import pytest

from oracle import schedule as osch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

P = pytest.importorskip("paper_2609_29505_amd")


def _lib_or_skip():
    if not os.path.exists(P.lib_path):
        pytest.skip("libsgd.so not built")
    return P.lib()


def test_exports_match_header():
    _lib_or_skip()
    import subprocess
    hdr = open(os.path.join(ROOT, "include", "sgd.h")).read() + open(os.path.join(ROOT, "include", "sgd_ops.h")).read()
    declared = set(re.findall(r"\b(sgd_[a-z_]+)\s*\(", hdr))
    out = subprocess.run(["nm", "-D", "--defined-only", P.lib_path], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (sgd_[a-z_]+)\b", out))
    assert declared, "no declarations found"
    assert declared <= exported, f"declared but not exported: {declared - exported}"
    assert set(P.binding.EXPORTS) <= exported


def test_version():
    assert _lib_or_skip().sgd_version() == 1


@pytest.mark.parametrize("seed", range(40))
def test_budget_lifetimes_match_oracle(seed):
    _lib_or_skip()
    rng = np.random.default_rng(seed)
    L, T = int(rng.integers(1, 40)), int(rng.integers(1, 101))
    smin = osch.s_min_default(T)
    lam = rng.random(L)
    if seed % 5 == 0:
        lam[rng.integers(0, L)] = 0.0
    if seed % 7 == 0 and L > 2:
        lam[1] = lam[0]  # a tie
    n = int(rng.integers(L * smin, L * T + 1))
    ref = osch.lifetimes_budget(lam, T, n, smin)
    got = P.schedule_from_scores(lam, T, budget=n, s_min=smin)
    assert np.array_equal(got.lifetimes, ref.lifetimes)
    assert got.layer_steps == ref.layer_steps == n
    assert np.array_equal(got.active, osch.active_mask(ref.lifetimes, T))
    if np.isfinite(ref.cut_margin):
        assert got.cut_margin == ref.cut_margin
    else:
        assert not np.isfinite(got.cut_margin)


@pytest.mark.parametrize("tau", [0.25, 0.5, 1.0, 2.0])
def test_tau_lifetimes_match_oracle(tau):
    _lib_or_skip()
    rng = np.random.default_rng(int(tau * 100))
    lam = rng.random(50)
    lam[3] = tau * 7 / 20  # exactly on a breakpoint
    ref = osch.lifetimes_tau(lam, 20, tau, 2)
    got = P.schedule_from_scores(lam, 20, tau=tau, s_min=2)
    assert np.array_equal(got.lifetimes, ref)


def test_from_lifetimes_and_errors():
    _lib_or_skip()
    s = P.schedule_from_lifetimes([3, 1, 5], 5)
    assert s.layer_steps == 9
    assert np.array_equal(s.active, osch.active_mask([3, 1, 5], 5))
    with pytest.raises(P.SgdError) as e:
        P.schedule_from_lifetimes([0, 1], 5)
    assert e.value.code == -1
    with pytest.raises(P.SgdError) as e:
        P.schedule_from_scores([0.5, 0.2], 10, budget=1)
    assert e.value.code == -4
    with pytest.raises(P.SgdError) as e:
        P.schedule_from_scores([0.5, float("nan")], 10, budget=10)
    assert e.value.code == -8
    with pytest.raises(P.SgdError) as e:
        P.schedule_from_scores([0.5, 0.2], 10, tau=-1.0)
    assert e.value.code == -1
