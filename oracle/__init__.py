"""CPU oracle for Spectral-Guided Diffusion's scheduled denoiser step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
CPU-baseline leg of the benchmark may import this package.  The product
path (the HIP library and its Python binding) never calls it and shares no
code with it.

Plain numpy, float64 arithmetic.  Each function follows one passage of the
paper (cited by section / equation / algorithm) and is written for a
reader to check against that passage by eye: no blocking, fusion or
reordering beyond what the definition states.

Modules
-------
``spectral``  Regularised SCR, matrix score g(W), component and unit
              scores, score normalisation (Sec. 3.2 Eq. scr-reg; appendix
              "Exact Block-Level Scores").
``schedule``  Lifetimes from scores (Sec. 4.1 Eq. schedule, Alg. 1) and the
              budget-matching reading of that equation.
``model``     Per-architecture residual units, the jagged step (Alg. 2) and
              the deterministic sampler update (Sec. 3.1).
``numerics``  bfloat16 decode/rounding used to emulate the GPU's storage
              points.
``rules``     The static ranking baselines at a matched budget (Sec. "Static
              ranking comparisons").

Parity status
-------------
Every function is pinned by ``tests/test_oracle_*.py`` against closed forms,
invariants, brute force or textbook special cases, except the points listed
as "parity unpinned" in the module docstrings.
"""
