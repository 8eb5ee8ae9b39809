"""Write fullsize_<workload>.txt: the oracle's statistics of every scored matrix of the
full-size workloads, and each unit's raw score q~_l.

Run from the repository root:  python tests/golden/make_fullsize_scores.py [workload ...]

Calls only the oracle (``oracle.spectral``) on the seeded synthetic weights of ``synth``
(generated one unit at a time, so a workload never sits in memory whole).  Per matrix it
stores E_k, the tail energy, ||W||_F^2 and ||W||_2^2 (Sec. 3.2, Eq. scr-reg; the spectral
norm for the static ranking rules of Sec. "Static ranking comparisons") and g(W) (Eq.
app-matrix-score); per unit the raw score q~_l (Eq. app-block-score) at eta = 1e-6.
Values are written with Python's shortest round-trip repr, so they reload bit for bit.
"""
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import synth  # noqa: E402
from oracle import spectral as sp  # noqa: E402

ETA = 1e-6
WORKLOADS = ["tiny", "dit", "uvit", "sdxl", "llada", "sdxl_unet"]


def write(name: str) -> None:
    cfg = synth.get_config(name)
    out = os.path.join(os.path.dirname(os.path.abspath(__file__)), f"fullsize_{name}.txt")
    lines = [f"# oracle statistics of the scored matrices of workload {name} "
             f"(B={cfg.B} N={cfg.N} d={cfg.d} H={cfg.H} dh={cfg.dh} F={cfg.F} L={cfg.L} T={cfg.T} {cfg.dtype}), "
             f"eta = {ETA!r}",
             "# mat <unit> <role> <rows> <cols> <E_k> <tail> <||W||_F^2> <||W||_2^2> <g>",
             "# raw <unit> <q~_l>"]
    t0 = time.time()
    for u in range(cfg.L):
        w = synth.unit_weights(cfg, u)
        mats = sp.unit_matrices(w, cfg.d, cfg.dtype)
        del w
        us = sp.unit_score(mats, cfg.dh, eta=ETA)
        for role, st in us.stats.items():
            lines.append(f"mat {u} {role} {st.m} {st.n} {st.energy_top!r} {st.energy_tail!r} {st.frob_sq!r} "
                         f"{st.sigma1_sq!r} {st.g!r}")
        lines.append(f"raw {u} {us.raw!r}")
        print(f"[{name}] unit {u + 1}/{cfg.L} scored ({time.time() - t0:.0f}s)", flush=True)
        del mats, us
    open(out, "w").write("\n".join(lines) + "\n")


def main(argv):
    for name in (argv or WORKLOADS):
        write(name)


if __name__ == "__main__":
    main(sys.argv[1:])
