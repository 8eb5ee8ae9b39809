"""Single-kernel microbenchmark of the scheduled step's kernels at a workload's shapes.

    python -m paper_2609_29505_amd.kernel_bench --workload llada --kernel gemm_w1 [--reps 20]
                                                [--cold] [--copy-mib 256]

Runs one kernel class of the step (through the sgd_ops.h entry points, on seeded random
operands of the workload's shapes) `reps` times and prints its average duration from HIP
events.  --cold cycles through enough distinct weight matrices (>= 1 GiB in all) that every
launch streams its weights from HBM, as the step does (each unit has its own weights); by
default one weight matrix is reused and stays in the 256 MB Infinity Cache.  --copy-mib appends a device-to-device copy of that many MiB, a plain copy of known
size that calibrates the FETCH_SIZE / WRITE_SIZE counters of a rocprofv3 --pmc pass run over
the same command.  Kernels: gemm_qkv, gemm_o, gemm_w1, gemm_w2, gemm_w2_split (two K ranges
of fp32 partials), attn, frozen (a run of --frozen-r cached updates).
"""
from __future__ import annotations

import argparse
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="llada")
    ap.add_argument("--kernel", default="gemm_w1")
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--frozen-r", type=int, default=4)
    ap.add_argument("--copy-mib", type=int, default=0)
    ap.add_argument("--cold", action="store_true")
    args = ap.parse_args()

    import torch

    import synth
    from paper_2609_29505_amd import binding as P

    cfg = synth.get_config(args.workload)
    if cfg.dtype != "bf16":
        raise SystemExit("kernel_bench covers the bf16 workloads")
    torch.manual_seed(0)
    dev = "cuda"
    bf = torch.bfloat16
    M, d, F, H, dh, N, B = cfg.M, cfg.d, cfg.F, cfg.H, cfg.dh, cfg.N, cfg.B
    np_ = (N + 63) // 64 * 64

    def rnd(*shape, scale=1.0, dtype=bf):
        return (torch.randn(*shape, device=dev) * scale).to(dtype)

    def weights(*shape, scale=1.0):
        # one matrix, or (--cold) a cycle of copies that no cache level holds
        n = 1
        if args.cold:
            nbytes = 2 * shape[0] * shape[1]
            n = max(2, -(-(1 << 30) // nbytes))
        ws = [rnd(*shape, scale=scale) for _ in range(n)]
        state = {"i": -1}

        def nxt():
            state["i"] = (state["i"] + 1) % n
            return ws[state["i"]]
        return nxt

    k = args.kernel
    if k == "gemm_w1":
        n1 = 2 * F if cfg.gated else F
        A, W, out = rnd(M, d), weights(n1, d, scale=d ** -0.5), torch.empty(M, F, device=dev, dtype=bf)
        act = {"llada": 3, "dit": 2}.get(cfg.arch, 1)
        fn = lambda: P.op_linear(A, W(), out, act=act, gated=cfg.gated)  # noqa: E731
        flop = 2.0 * M * n1 * d
    elif k == "gemm_qkv":
        A, W = rnd(M, d), weights(3 * d, d, scale=d ** -0.5)
        q = torch.empty(B * H, np_, dh, device=dev, dtype=bf)
        kk = torch.empty_like(q)
        vt = torch.empty(B * H, dh, np_, device=dev, dtype=bf)
        fn = lambda: P.op_heads(A, W(), q, kk, vt, 3, 0, N, H, dh, rope=cfg.arch == "llada")  # noqa: E731
        flop = 2.0 * M * 3 * d * d
    elif k in ("gemm_o", "gemm_w2"):
        kd = d if k == "gemm_o" else F
        A, W, h = rnd(M, kd), weights(d, kd, scale=kd ** -0.5), torch.randn(M, d, device=dev)
        fn = lambda: P.op_residual(A, W(), h)  # noqa: E731
        flop = 2.0 * M * d * kd
    elif k == "gemm_w2_split":
        # the MLP output GEMM in two K ranges of fp32 partial products (the step's split path)
        A, W = rnd(M, F), weights(d, F, scale=F ** -0.5)
        parts = torch.empty(2, M, d, device=dev)
        fn = lambda: P.op_linear_split(A, W(), parts)  # noqa: E731
        flop = 2.0 * M * d * F
    elif k == "attn":
        q = rnd(B * H, np_, dh)
        kk = rnd(B * H, np_, dh)
        vt = rnd(B * H, dh, np_)
        o = torch.empty(B, N, H * dh, device=dev, dtype=bf)
        fn = lambda: P.op_attention(q, kk, vt, o, B, H, dh, N, N)  # noqa: E731
        flop = 4.0 * B * H * N * N * dh
    elif k == "frozen":
        h = torch.randn(M * d, device=dev)
        deltas = [torch.randn(M * d, device=dev) for _ in range(args.frozen_r)]
        fn = lambda: P.op_frozen_run(h, deltas)  # noqa: E731
        flop = 0.0
    else:
        raise SystemExit(f"unknown kernel {k}")

    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / args.reps * 1e3
    line = f"{cfg.name} {k}{' (cold weights)' if args.cold else ''}: {us:.1f} us per launch"
    if flop:
        line += f", {flop / us / 1e6:.1f} TFLOP/s"
    else:
        nbytes = (2 + args.frozen_r) * M * d * 4
        line += f", {nbytes / us / 1e3:.0f} GB/s algorithmic ({nbytes / 2**20:.0f} MiB)"
    print(line, flush=True)
    if args.copy_mib:
        x = torch.ones(args.copy_mib * 2**18, device=dev)
        y = torch.empty_like(x)
        y.copy_(x)
        torch.cuda.synchronize()
        print(f"copy: {args.copy_mib} MiB read, {args.copy_mib} MiB written", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
