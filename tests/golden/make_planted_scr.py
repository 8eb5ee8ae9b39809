"""Write planted_scr.txt: the oracle's SCR statistics of diag(i^-a) spectra.

Run from the repository root:  python tests/golden/make_planted_scr.py
Calls only the oracle.  The test compares these stored values against the
closed form E_k / F = H_k(2a) / H_d(2a) (harmonic sums), which the oracle
does not use.
"""
import math
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
from oracle import spectral as sp  # noqa: E402


def main():
    out = os.path.join(os.path.dirname(os.path.abspath(__file__)), "planted_scr.txt")
    lines = ["# d k a rho0 scr0 scr_eta(1e-6) -- oracle statistics of W = diag(i^-a), i = 1..d",
             "# rho0 = E_k / ||W||_F^2 at eta = 0; scr0 = SCR_0; scr_eta = SCR_eta (Sec. 3.2, Eq. scr-reg)"]
    for d in (10, 64, 256, 1024, 1152, 1280):
        for a in (0.3, 0.5, 1.0, 1.5):
            s = np.arange(1, d + 1, dtype=np.float64) ** (-a)
            w = np.diag(s)
            st0 = sp.matrix_stats(w, eta=0.0)
            ste = sp.matrix_stats(w, eta=1e-6)
            rho0 = st0.energy_top / st0.frob_sq
            lines.append(f"{d} {st0.k} {a} {rho0:.15e} {st0.scr:.15e} {ste.scr:.15e}")
    open(out, "w").write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
