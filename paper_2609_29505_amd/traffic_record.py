"""HBM traffic record of one kernel from two rocprofv3 counter passes, calibrated by a copy.

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d <dir>/fetch -o p -- \\
        python3 paper_2609_29505_amd/kernel_bench.py --workload llada --kernel gemm_w1 --reps 5 --cold --copy-mib 256
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d <dir>/write -o p -- <same command>
    python -m paper_2609_29505_amd.traffic_record --fetch <dir>/fetch/p_counter_collection.csv \\
        --write <dir>/write/p_counter_collection.csv --kernel gemm_bf16_kernel --copy-mib 256 \\
        --source paper_2609_29505_amd/csrc/gemm_bf16.hip --algorithmic-bytes <B> --out profiles/<k>_<w>_traffic.json

FETCH_SIZE and WRITE_SIZE (KiB per dispatch) count traffic below the L2.  --group N sums
every N consecutive dispatches of the kernel into one call (a GEMM whose rows are split into a
main launch and a row-tail launch).  The same passes
measure a device-to-device copy of --copy-mib MiB (read and written once), and each counter is
scaled by (copy bytes) / (copy counter): the factor that turns the counter into bytes on this
GPU.  The record keeps the SHA-256 of the kernel's source file, so that a reader (bench.py)
reports it only for the kernel source it was taken on.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def per_dispatch(path: str, counter: str, match: str):
    """Counter value per dispatch (summed over the rows of one dispatch) of kernels whose
    name contains `match`, in dispatch order."""
    vals = defaultdict(float)
    for row in csv.DictReader(open(path)):
        if row["Counter_Name"] == counter and match in row["Kernel_Name"]:
            vals[int(row["Dispatch_Id"])] += float(row["Counter_Value"])
    return [vals[k] for k in sorted(vals)]


def grouped(vals, n: int):
    """Sums of n consecutive values (one call of a kernel dispatched as n launches); a
    trailing incomplete group is dropped."""
    if n < 1:
        raise ValueError("group size must be positive")
    return [sum(vals[i:i + n]) for i in range(0, len(vals) - n + 1, n)]


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--fetch", required=True, help="counter_collection.csv of the FETCH_SIZE pass")
    ap.add_argument("--write", required=True, help="counter_collection.csv of the WRITE_SIZE pass")
    ap.add_argument("--kernel", required=True, help="substring of the measured kernel's name")
    ap.add_argument("--copy-match", default="copyBuffer", help="substring of the copy kernel's name")
    ap.add_argument("--copy-mib", type=int, default=256)
    ap.add_argument("--source", required=True, help="kernel source file (repository-relative)")
    ap.add_argument("--algorithmic-bytes", type=float, required=True)
    ap.add_argument("--describe-kernel", default="")
    ap.add_argument("--describe-workload", default="")
    ap.add_argument("--command", action="append", default=[], help="command lines that produced the passes")
    ap.add_argument("--note", default="")
    ap.add_argument("--group", type=int, default=1, help="consecutive dispatches that form one call")
    ap.add_argument("--out", required=True)
    a = ap.parse_args()

    fk = grouped(per_dispatch(a.fetch, "FETCH_SIZE", a.kernel), a.group)
    wk = grouped(per_dispatch(a.write, "WRITE_SIZE", a.kernel), a.group)
    fc = per_dispatch(a.fetch, "FETCH_SIZE", a.copy_match)
    wc = per_dispatch(a.write, "WRITE_SIZE", a.copy_match)
    if not fk or not wk or not fc or not wc:
        print("missing dispatches: kernel", len(fk), len(wk), "copy", len(fc), len(wc), file=sys.stderr)
        return 1
    copy_kib = a.copy_mib * 1024.0
    fscale, wscale = copy_kib / fc[-1], copy_kib / wc[-1]
    # the first dispatch of a pass may see cold instruction and TLB state: average the rest
    fmean = sum(fk[1:] or fk) / len(fk[1:] or fk)
    wmean = sum(wk[1:] or wk) / len(wk[1:] or wk)
    src = os.path.join(ROOT, a.source)
    rec = {
        "kernel": a.describe_kernel or a.kernel,
        "workload": a.describe_workload,
        "source": a.source,
        "sha256": hashlib.sha256(open(src, "rb").read()).hexdigest(),
        "commands": a.command,
        "dispatches_per_call": a.group,
        "fetch_size_kib_per_dispatch": fk,
        "write_size_kib_per_dispatch": wk,
        f"copy_{a.copy_mib}mib_fetch_size_kib": fc,
        f"copy_{a.copy_mib}mib_write_size_kib": wc,
        "fetch_scale": round(fscale, 5),
        "write_scale": round(wscale, 5),
        "fetch_bytes": int(round(fmean * fscale * 1024)),
        "write_bytes": int(round(wmean * wscale * 1024)),
        "algorithmic_bytes": int(a.algorithmic_bytes),
        "note": a.note,
    }
    json.dump(rec, open(a.out, "w"), indent=1)
    print(json.dumps({k: rec[k] for k in ("fetch_bytes", "write_bytes", "algorithmic_bytes", "fetch_scale", "write_scale")}))
    return 0


if __name__ == "__main__":
    sys.exit(main())
