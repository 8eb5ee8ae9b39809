"""Host-side measurement tools on synthetic inputs (no GPU): the counter-record builder, the
kernel-trace report's frozen-run accounting, and bench.py's one-GPU guard."""
import csv
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def _counter_csv(path, counter, rows):
    """rocprofv3 counter_collection.csv with (dispatch id, kernel name, value) rows."""
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for d, name, v in rows:
            w.writerow([d, name, counter, v])


def test_traffic_record_scales_by_the_copy(tmp_path):
    from paper_2609_29505_amd import traffic_record as tr

    # FETCH_SIZE reads half the copy's bytes, WRITE_SIZE all of them (as measured on gfx950)
    kib = 256 * 1024
    _counter_csv(tmp_path / "f.csv", "FETCH_SIZE",
                 [(1, "void k<1>(A)", 1000.0), (2, "void k<1>(A)", 500.0), (3, "void k<1>(A)", 700.0),
                  (4, "__amd_rocclr_copyBuffer", kib / 2), (5, "other", 9.0)])
    _counter_csv(tmp_path / "w.csv", "WRITE_SIZE",
                 [(1, "void k<1>(A)", 100.0), (2, "void k<1>(A)", 300.0), (3, "void k<1>(A)", 500.0),
                  (4, "__amd_rocclr_copyBuffer", float(kib))])
    out = tmp_path / "rec.json"
    argv = ["traffic_record", "--fetch", str(tmp_path / "f.csv"), "--write", str(tmp_path / "w.csv"),
            "--kernel", "k<1>", "--source", "bench.py", "--algorithmic-bytes", "1000", "--out", str(out)]
    old = sys.argv
    try:
        sys.argv = argv
        assert tr.main() == 0
    finally:
        sys.argv = old
    rec = json.load(open(out))
    assert rec["fetch_scale"] == pytest.approx(2.0) and rec["write_scale"] == pytest.approx(1.0)
    # the first dispatch of each pass is left out of the mean
    assert rec["fetch_bytes"] == round((500 + 700) / 2 * 2.0 * 1024)
    assert rec["write_bytes"] == round((300 + 500) / 2 * 1.0 * 1024)
    assert rec["fetch_size_kib_per_dispatch"] == [1000.0, 500.0, 700.0]
    assert len(rec["sha256"]) == 64


def test_traffic_record_groups_split_launches(tmp_path):
    from paper_2609_29505_amd import traffic_record as tr

    # one call = a main launch and a row-tail launch; the pass ends with the copy
    kib = 256 * 1024
    _counter_csv(tmp_path / "f.csv", "FETCH_SIZE",
                 [(1, "void k<1>(A)", 1000.0), (2, "void k<2>(A)", 100.0), (3, "void k<1>(A)", 800.0),
                  (4, "void k<2>(A)", 60.0), (5, "void k<1>(A)", 820.0), (6, "void k<2>(A)", 40.0),
                  (7, "__amd_rocclr_copyBuffer", kib / 2)])
    _counter_csv(tmp_path / "w.csv", "WRITE_SIZE",
                 [(1, "void k<1>(A)", 10.0), (2, "void k<2>(A)", 1.0), (3, "void k<1>(A)", 10.0),
                  (4, "void k<2>(A)", 1.0), (5, "void k<1>(A)", 10.0), (6, "void k<2>(A)", 1.0),
                  (7, "__amd_rocclr_copyBuffer", float(kib))])
    out = tmp_path / "rec.json"
    argv = ["traffic_record", "--fetch", str(tmp_path / "f.csv"), "--write", str(tmp_path / "w.csv"),
            "--kernel", "void k<", "--group", "2", "--source", "bench.py", "--algorithmic-bytes", "1000",
            "--out", str(out)]
    old = sys.argv
    try:
        sys.argv = argv
        assert tr.main() == 0
    finally:
        sys.argv = old
    rec = json.load(open(out))
    assert rec["dispatches_per_call"] == 2
    assert rec["fetch_size_kib_per_dispatch"] == [1100.0, 860.0, 860.0]
    assert rec["fetch_bytes"] == round(860.0 * 2.0 * 1024)
    assert rec["write_bytes"] == round(11.0 * 1024)
    assert tr.grouped([1, 2, 3, 4, 5], 2) == [3, 7]
    with pytest.raises(ValueError):
        tr.grouped([1.0], 0)


def _trace_rows(cfg, lifetimes, extra=0):
    """Frozen-run dispatches in bench.py's order: every budget (T warm-up + 3T timed steps), then
    the headline budget twice more; launch i lasts 1 + i ns."""
    import bench

    T = cfg.T
    runs = sorted(cfg.budgets)
    rows, t = [], 0
    for pct in runs + [runs[0], runs[0]]:
        act = np.arange(1, T + 1)[:, None] <= np.asarray(lifetimes[str(pct)])[None, :]
        for j in range(4 * T):
            for _ in bench.frozen_launch_bytes(cfg, act[j % T]):
                rows.append({"Kernel_Name": "sgd::frozen_run_kernel(sgd::FrozenRun)",
                             "Start_Timestamp": str(t), "End_Timestamp": str(t + 1 + len(rows))})
                t += 1000
    for _ in range(extra):
        rows.append({"Kernel_Name": "sgd::frozen_run_kernel(sgd::FrozenRun)",
                     "Start_Timestamp": str(t), "End_Timestamp": str(t + 1)})
        t += 1000
    return rows


def test_trace_report_frozen_accounting():
    from paper_2609_29505_amd import trace_report

    import bench

    cfg = synth.get_config("tiny")
    lifetimes = {"50": [3, 10, 1, 6]}
    rows = _trace_rows(cfg, lifetimes)
    out = trace_report.frozen_rates(cfg, rows, lifetimes)
    assert [o[0] for o in out] == [50]
    pct, n, nbytes, secs = out[0]
    act = np.arange(1, cfg.T + 1)[:, None] <= np.asarray(lifetimes["50"])[None, :]
    per_step = [bench.frozen_launch_bytes(cfg, act[j % cfg.T]) for j in range(3 * cfg.T)]
    assert n == sum(len(p) for p in per_step)
    assert nbytes == sum(sum(p) for p in per_step)
    # the timed launches of the first run follow its T warm-up steps' launches
    w = sum(len(bench.frozen_launch_bytes(cfg, act[j])) for j in range(cfg.T))
    assert secs == pytest.approx(sum((1 + i) * 1e-9 for i in range(w, w + n)))
    with pytest.raises(SystemExit):
        trace_report.frozen_rates(cfg, _trace_rows(cfg, lifetimes, extra=1), lifetimes)


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in r.stderr


def test_trace_report_separates_grids():
    from paper_2609_29505_amd import trace_report

    rows = [{"Kernel_Name": "gemm<256, 192>", "Grid_Size": "131072", "Start_Timestamp": "0", "End_Timestamp": "96000"},
            {"Kernel_Name": "gemm<256, 192>", "Grid_Size": "262144", "Start_Timestamp": "0", "End_Timestamp": "178000"},
            {"Kernel_Name": "gemm<256, 192>", "Grid_Size": "262144", "Start_Timestamp": "0", "End_Timestamp": "180000"}]
    st = trace_report.kernel_stats(rows)
    assert [(g, n) for _, g, n, _, _, _ in st] == [(262144, 2), (131072, 1)]
    assert st[0][4] == pytest.approx(179.0) and st[1][4] == pytest.approx(96.0)


def test_trace_report_recognises_folding_pre_norms():
    """rocprofv3 demangles the fp32 pre-norms but leaves the bf16 ones mangled (__bf16 is DF16b):
    the folding instance must be recognised in both spellings, and matched in dispatch order."""
    from paper_2609_29505_amd import trace_report

    import bench

    fold_names = ["_ZN3sgd11norm_kernelIDF16bLi4ELi4ELb1EEEvNS_8NormArgsE",
                  "void sgd::norm_kernel<float, 4, 4, true>(sgd::NormArgs)"]
    plain_names = ["_ZN3sgd11norm_kernelIDF16bLi4ELi4ELb0EEEvNS_8NormArgsE",
                   "void sgd::norm_kernel<float, 4, 4, false>(sgd::NormArgs)"]
    assert all(trace_report._is_fold(n) for n in fold_names)
    assert not any(trace_report._is_fold(n) for n in plain_names)

    cfg = synth.get_config("tiny")
    lifetimes = {"50": [3, 10, 1, 6]}
    runs = sorted(cfg.budgets)
    rows, t = [], 0
    for pct in runs + [runs[0], runs[0]]:
        act = np.arange(1, cfg.T + 1)[:, None] <= np.asarray(lifetimes[str(pct)])[None, :]
        for j in range(4 * cfg.T):
            for _ in bench.frozen_launches(cfg, act[j % cfg.T])[1]:
                rows.append({"Kernel_Name": fold_names[0], "Start_Timestamp": str(t), "End_Timestamp": str(t + 5)})
                rows.append({"Kernel_Name": plain_names[0], "Start_Timestamp": str(t + 10), "End_Timestamp": str(t + 15)})
                t += 1000
    out = trace_report.frozen_rates(cfg, rows, lifetimes, folded=True)
    act = np.arange(1, cfg.T + 1)[:, None] <= np.asarray(lifetimes["50"])[None, :]
    n = sum(len(bench.frozen_launches(cfg, act[j % cfg.T])[1]) for j in range(3 * cfg.T))
    assert n > 0 and out[0][1] == n


def test_build_rejects_register_spills():
    """The build reads hipcc's resource-usage remarks and names every kernel that spills."""
    from paper_2609_29505_amd import build
    remarks = "\n".join([
        "a.hip:1:1: remark: Function Name: _ZN3sgd1kEv [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:1:1: remark:     VGPRs: 256 [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:1:1: remark:     SGPRs Spill: 0 [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:1:1: remark:     VGPRs Spill: 5 [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:9:1: remark: Function Name: _ZN3sgd1jEv [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:9:1: remark:     SGPRs Spill: 0 [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:9:1: remark:     VGPRs Spill: 0 [-Rpass-analysis=kernel-resource-usage]",
    ])
    assert build._spills(remarks) == ["_ZN3sgd1kEv: VGPRs Spill: 5"]
    assert build._spills(remarks.replace("Spill: 5", "Spill: 0")) == []
