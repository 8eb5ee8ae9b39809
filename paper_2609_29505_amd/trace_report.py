"""Summary of a rocprofv3 kernel trace of bench.py, as markdown.

    rocprofv3 --kernel-trace --stats --output-format csv -d <dir> -o <w> -- \\
        python3 bench.py --config <w> --no-cpu-baseline --no-kernel-table --taus "" --rules "" \\
        --no-input-aware --no-graph --lifetimes <lifetimes.json>
    python -m paper_2609_29505_amd.trace_report --workload <w> --trace <dir>/<w>_kernel_trace.csv \\
        --lifetimes <lifetimes.json>

Prints the per-kernel statistics of the traced run and the frozen path's HBM rate from the
trace's own durations: bench.py launches the budgets in increasing order, each as T warm-up
steps and three timed T-step trajectories (then the all-active schedule, and the headline budget twice
with per-launch events), so the frozen-run dispatches appear in a known order and each
one's algorithmic bytes follow from the schedule (maximal runs of frozen units, as the
launcher fuses them).  The traced run must launch nothing else that carries frozen units:
no drift policy or replay (--no-input-aware), no graph replays (--no-graph); with
--lifetimes, bench.py also skips the branch-unit schedule.
"""
from __future__ import annotations

import argparse
import csv
import json
import os
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def _grid(r) -> int:
    """Work-items of a dispatch (rocprofv3 names the column Grid_Size or Grid_Size_X)."""
    for k in ("Grid_Size", "Grid_Size_X"):
        if r.get(k):
            return int(r[k])
    return 0


def kernel_stats(rows):
    """Per (kernel, grid size): one template instance serves GEMMs of different shapes (e.g. the
    LLaDA QKV and MLP input GEMMs both run 256 x 192 tiles), which the grid tells apart."""
    agg = defaultdict(lambda: [0, 0.0])
    for r in rows:
        a = agg[(r["Kernel_Name"], _grid(r))]
        a[0] += 1
        a[1] += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3  # us
    tot = sum(v[1] for v in agg.values())
    return sorted(((k, g, n, t, t / n, 100.0 * t / tot) for (k, g), (n, t) in agg.items()), key=lambda x: -x[3])


def _is_fold(name: str) -> bool:
    """A pre-norm kernel instantiated to absorb a frozen run (norm_kernel<..., true>; rocprofv3
    leaves the bf16 instances mangled, where the flag reads Lb1E)."""
    return "norm_kernel" in name and ("true>" in name or "Lb1E" in name)


def frozen_rates(cfg, rows, lifetimes, folded=False):
    """Timed launches carrying frozen units per budget: standalone frozen-run kernels, or (with
    ``folded``) the pre-norms that absorbed a run, matched to the schedule in dispatch order."""
    import numpy as np

    import bench

    T, L = cfg.T, cfg.L
    W, K = T, 3 * T  # bench.py's defaults: T warm-up steps, three whole trajectories
    match = _is_fold if folded else (lambda name: "frozen_run_kernel" in name)
    fr = sorted((r for r in rows if match(r["Kernel_Name"])), key=lambda r: int(r["Start_Timestamp"]))
    i, out = 0, []
    # the budgets in increasing order, then the headline (smallest) budget twice more: the runs
    # in which bench.py records HIP events around the frozen-run and the folding pre-norm
    # launches (not reported here)
    runs = sorted(cfg.budgets)
    for k, pct in enumerate(runs + [runs[0], runs[0]]):
        life = np.asarray(lifetimes[str(pct)])
        act = np.arange(1, T + 1)[:, None] <= life[None, :]
        nbytes, secs, n = 0, 0.0, 0
        for phase, steps in (("warmup", W), ("timed", K)):
            for j in range(steps):
                for b in bench.frozen_launches(cfg, act[j % T])[1 if folded else 0]:
                    r = fr[i]
                    i += 1
                    if phase == "timed":
                        nbytes += b
                        secs += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
                        n += 1
        if k < len(runs):
            out.append((pct, n, nbytes, secs))
    if i != len(fr):
        raise SystemExit(f"trace has {len(fr)} matching dispatches, the schedules predict {i}")
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", required=True)
    ap.add_argument("--trace", required=True)
    ap.add_argument("--lifetimes", required=True)
    args = ap.parse_args()

    import synth

    cfg = synth.get_config(args.workload)
    rows = list(csv.DictReader(open(args.trace)))
    print("| kernel | grid (work-items) | calls | total ms | avg us | % |\n|---|---:|---:|---:|---:|---:|")
    for name, grid, n, t, avg, pc in kernel_stats(rows)[:14]:
        print(f"| `{name[:110]}` | {grid} | {n} | {t / 1e3:.1f} | {avg:.2f} | {pc:.2f} |")
    lt = json.load(open(args.lifetimes))
    print("\n| budget | launches | kind | GB | ms | GB/s | of 8 TB/s |\n|---:|---:|---|---:|---:|---:|---:|")
    alone = frozen_rates(cfg, rows, lt)
    fold = frozen_rates(cfg, rows, lt, folded=True)
    for (pct, n, nb, sc), (_, n2, nb2, sc2) in zip(alone, fold):
        for kind, cnt, byt, sec in (("standalone frozen runs", n, nb, sc), ("pre-norms absorbing a run", n2, nb2, sc2),
                                    ("all launches with frozen units", n + n2, nb + nb2, sc + sc2)):
            if cnt:
                print(f"| {pct}% | {cnt} | {kind} | {byt / 1e9:.2f} | {sec * 1e3:.2f} | {byt / sec / 1e9:.0f} | "
                      f"{byt / sec / 8e12:.3f} |")
    return 0


if __name__ == "__main__":
    sys.exit(main())
