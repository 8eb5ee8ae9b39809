"""Throughput of the scheduled denoiser step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config llada] [--budget 35]

A "step" is one network evaluation of the whole unit stack plus the sampler update,
for the full batch of the workload (Alg. 2 + the update of Sec. 3.1).  Timing is done in
whole T-step trajectories (a fresh cache and z_1 each): ceil(K / T) of them, at least one,
so every timed step is part of a complete trajectory and the timed mask rows are the whole
schedule.  `value` = T / median trajectory time.  Inputs and weights are seeded synthetic
data with the workload's shapes (planted power-law spectra), resident in HBM before timing.

Prints one JSON line.  `value` is scheduled denoising steps/s at the headline budget; the
all-active rate (every unit computing at every step, same launcher), the other budgets, the
tau-mode schedules and the static ranking rules (with each one's output deviation from the
all-active trajectory) are reported beside it.  `roofline` times the dominant kernel (the gated MLP input GEMM)
with HIP events on the launch stream inside the timed region.  `cpu_baseline` times the
CPU oracle on a bounded sample (a few units of an all-active step).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15      # dense MFMA bf16, FLOP/s
PEAK_F32 = 157.3e12     # fp32 vector
PEAK_HBM = 8.0e12       # bytes/s
MAX_RUN = 32            # frozen units fused into one launch at most (kMaxRun of the launcher)


def log(msg: str) -> None:
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def unit_flops(cfg) -> dict:
    """Algorithmic FLOP of one active unit, per GEMM / attention (2 M N K; 4 B H S_q S_k d_h)."""
    M, d, F, H, dh, N, B = cfg.M, cfg.d, cfg.F, cfg.H, cfg.dh, cfg.N, cfg.B
    f = {
        "gemm_qkv": 2.0 * M * 3 * d * d,
        "attn": 4.0 * B * H * N * N * dh,
        "gemm_o": 2.0 * M * d * d,
        "gemm_w1": 2.0 * M * (2 * F if cfg.gated else F) * d,
        "gemm_w2": 2.0 * M * d * F,
    }
    if cfg.arch in ("sdxl", "sdxl_unet"):
        f["gemm_x"] = 2.0 * M * d * d * 2
        f["attn_x"] = 4.0 * B * H * N * cfg.ctx_len * dh
    if cfg.arch == "sdxl_unet":
        f["gemm_conv"] = 2.0 * M * d * 9 * d  # per 3x3 convolution (two per ResNet block)
    return f


def frozen_launches(cfg, active_row):
    """Algorithmic HBM bytes of every launch of one step that carries frozen units (Sec. 3.1
    frozen rule), as (standalone frozen-run launches, pre-norms that absorbed a run).

    The launcher fuses a maximal run of consecutive frozen units (at most MAX_RUN; U-ViT
    out-blocks, whose skip linear always runs, end a run) into one pass that reads h and the
    r cached updates and writes h: (2 + r) M d fp32 values, plus, for U-ViT in-blocks, a
    bf16 copy of h after every unit of the run (the long-skip inputs).  A run that ends at an
    active unit starting with its pre-norm (not a U-ViT out-block, not a UNet unit, no copies)
    is added by that norm instead, which also writes the normalised rows: (2 + r) M d 4 +
    M d (element size) bytes."""
    L = cfg.L
    es = 2 if cfg.dtype == "bf16" else 4
    half = L // 2
    uvit = cfg.arch == "uvit"
    alone, folded, l = [], [], 0
    while l < L:
        if active_row[l] or (uvit and l > half):
            l += 1
            continue
        r = 0
        while l < L and not active_row[l] and not (uvit and l > half) and r < MAX_RUN:
            r += 1
            l += 1
        snaps = r if uvit else 0  # U-ViT: every unit up to the mid block copies h out
        fold = (not snaps and l < L and active_row[l] and not (uvit and l > half)
                and cfg.arch != "sdxl_unet")
        if fold:
            folded.append((2 + r) * cfg.M * cfg.d * 4 + cfg.M * cfg.d * es)
        else:
            alone.append((2 + r) * cfg.M * cfg.d * 4 + snaps * cfg.M * cfg.d * es)
    return alone, folded


def frozen_launch_bytes(cfg, active_row) -> list:
    """Bytes of the standalone frozen-run launches of one step (see frozen_launches)."""
    return frozen_launches(cfg, active_row)[0]


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=0,
                    help="steps to time, rounded up to whole trajectories (default 3 T)")
    ap.add_argument("--warmup", type=int, default=0, help="warm-up steps per schedule (default T)")
    ap.add_argument("--config", default="llada")
    ap.add_argument("--budget", type=int, default=0, help="headline budget in percent (default: smallest)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="oracle sample: units of one all-active step, run until this much CPU time")
    ap.add_argument("--profile-kernel", default="gemm_w1")
    ap.add_argument("--no-kernel-table", action="store_true",
                    help="skip the per-kernel-class timing passes of the all-active schedule")
    ap.add_argument("--save-lifetimes", default="", help="write the built lifetimes (JSON) here")
    ap.add_argument("--lifetimes", default="", help="reuse lifetimes saved by --save-lifetimes "
                    "instead of rebuilding the spectra (e.g. under a kernel tracer)")
    ap.add_argument("--taus", default="0.5,1,2",
                    help="tau-mode schedules (Eq. schedule at a fixed tau) timed beside the budgets; '' for none")
    ap.add_argument("--rules", default="random,depth,frob,spectral,stable_rank,frob_srank,raw_scr",
                    help="static ranking rules timed at the headline budget; '' for none")
    ap.add_argument("--no-input-aware", action="store_true",
                    help="skip the activation-drift policy and the oracle-replay search")
    ap.add_argument("--tau-agree", type=float, default=5e-3, help="oracle-replay tolerance")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip timing the headline schedule as a replayed HIP graph (e.g. under a kernel tracer, "
                         "whose dispatch accounting expects eager launches only)")
    ap.add_argument("--no-branch-units", action="store_true",
                    help="skip the branch-granular schedule (every residual branch a unit of its own)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (batches would shard by "
              "sample with no exchange; LLaDA would need tensor parallelism).",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import synth
    import paper_2609_29505_amd as P

    cfg = synth.get_config(args.config)
    T, L = cfg.T, cfg.L
    K = args.steps or 3 * T
    n_traj = max(1, -(-K // T))  # whole trajectories
    W = args.warmup or T
    budgets = sorted(cfg.budgets)
    head = args.budget or budgets[0]
    if head not in budgets:
        budgets.append(head)

    log(f"config {cfg.name}: B={cfg.B} N={cfg.N} d={cfg.d} F={cfg.F} L={L} T={T}; generating weights")
    t0 = time.time()
    cache_dir = os.environ.get("SGD_SYNTH_CACHE") or "/tmp/sgd_synth_cache"
    done = []
    weights = synth.model_weights(cfg, workers=min(16, os.cpu_count() or 1), cache_dir=cache_dir,
                                  progress=lambda u: (done.append(u), log(f"unit {u} ready ({len(done)}/{L})")))
    inputs = synth.inputs(cfg)
    log(f"weights ready in {time.time() - t0:.1f}s; uploading")
    torch.cuda.set_device(0)
    dm = P.DeviceModel(cfg, weights, inputs)
    torch.cuda.synchronize()
    log(f"workspace {dm.workspace_bytes / 2**20:.0f} MiB, cache {dm.cache_bytes / 2**20:.0f} MiB; building schedules")

    t0 = time.time()
    scheds = {}
    units = dm.scored_units()
    roles = [[r for r, _ in u] for u in units]
    rule_names = [r for r in args.rules.split(",") if r]
    if args.lifetimes:
        saved = json.load(open(args.lifetimes))
        for pct in budgets:
            scheds[pct] = P.schedule_from_lifetimes(saved[str(pct)], T)
        scores = saved.get("scores")
        mat_stats = np.array(saved["mat_stats"]) if "mat_stats" in saved else None
    else:
        scheds[head] = P.schedule_build(units, [cfg.dh] * L, T, budget_pct=head)
        scores = scheds[head].unit_score.tolist()
        mat_stats = scheds[head].mat_stats.copy()
    t_build = time.time() - t0
    for pct in budgets:
        if args.lifetimes:
            continue
        if pct != head:  # same spectra, lifetimes at another budget
            scheds[pct] = P.schedule_from_scores(scheds[head].unit_score, T, budget_pct=pct)
        log(f"budget {pct}%: N*={scheds[pct].layer_steps} lifetimes={scheds[pct].lifetimes.tolist()} "
            f"margin={scheds[pct].cut_margin:.3g}")
    log(f"schedule ready in {t_build:.1f}s (spectra of {sum(len(u) for u in units)} matrices; "
        f"offline, not timed)")
    if args.save_lifetimes:
        rec = {str(p): scheds[p].lifetimes.tolist() for p in budgets}
        rec["scores"] = scores
        rec["mat_stats"] = mat_stats.tolist() if mat_stats is not None else None
        json.dump(rec, open(args.save_lifetimes, "w"))
    taus = [float(t) for t in args.taus.split(",") if t] if scores is not None else []
    tau_scheds = {t: P.schedule_from_scores(scores, T, tau=t) for t in taus}
    # the static ranking baselines at the headline budget, re-ranked from the same spectra
    rule_scheds = {}
    for r in rule_names:
        if r in ("depth", "random"):
            rule_scheds[r] = P.schedule_build(None, None, T, budget_pct=head, rule=r, seed=2024, L=L)
        elif mat_stats is not None:
            rule_scheds[r] = P.schedule_from_stats(roles, [cfg.dh] * L, mat_stats, T, budget_pct=head, rule=r)
    all_active = P.schedule_from_lifetimes([T] * L, T)

    z0 = torch.from_numpy(inputs["z"]).cuda()
    z = z0.clone()
    cache = P.Cache(dm)
    stream = torch.cuda.current_stream()

    def trajectory(sched, steps=T):
        """Enqueue steps 1..steps of a fresh trajectory (cache reset, z = z_1)."""
        cache.reset()
        z.copy_(z0)
        for s in range(1, steps + 1):
            dm.step(z, s, sched, cache)

    def timed(sched, profile=None, stepper=None):
        """W warm-up steps, then n_traj whole trajectories, each bracketed by HIP events on
        the step stream.  Returns the per-trajectory times (ms) and the profile record.
        ``stepper(s)`` replaces the scheduled step (the input-aware policies)."""
        step_fn = stepper or (lambda s: dm.step(z, s, sched, cache))
        w = W
        while w > 0:
            cache.reset()
            z.copy_(z0)
            for s in range(1, min(w, T) + 1):
                step_fn(s)
            w -= T
        torch.cuda.synchronize()
        if profile:
            dm.profile_begin(profile, 16384)
        evs = []
        for _ in range(n_traj):
            cache.reset()
            z.copy_(z0)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for s in range(1, T + 1):
                step_fn(s)
            e1.record(stream)
            evs.append((e0, e1))
        torch.cuda.synchronize()
        times = [a.elapsed_time(b) for a, b in evs]
        prof = dm.profile_end() if profile else None
        return times, prof

    def rate(times):
        return T * 1000.0 / float(np.median(times))

    results = {}
    for pct in budgets:
        times, _ = timed(scheds[pct])
        results[pct] = times
        log(f"budget {pct}%: {n_traj} trajectories of {T} steps, median {np.median(times):.2f} ms "
            f"-> {rate(times):.2f} steps/s")
    value_head = rate(results[head])
    act_head = np.asarray(scheds[head].active, np.uint8)
    def graph_timed(sched):
        """The schedule captured as one HIP graph per trajectory (sgd_graph_capture), one
        warm-up replay, then n_traj replays bracketed by HIP events on a stream of its own."""
        gstream = torch.cuda.Stream()
        torch.cuda.synchronize()
        evs = []
        with torch.cuda.stream(gstream):
            graph = dm.capture(z, sched, cache, gstream)
            z.copy_(z0)
            graph.launch(gstream)
            for _ in range(n_traj):
                z.copy_(z0)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(gstream)
                graph.launch(gstream)
                e1.record(gstream)
                evs.append((e0, e1))
        gstream.synchronize()
        graph.close()
        return [a.elapsed_time(b) for a, b in evs]

    t_graph = None
    if not args.no_graph:
        t_graph = graph_timed(scheds[head])
        log(f"budget {head}% as one HIP graph per trajectory: median {np.median(t_graph):.2f} ms -> "
            f"{rate(t_graph):.2f} steps/s (eager launches {value_head:.2f})")
    t_all, _ = timed(all_active)
    z_full = z.clone()  # the all-active trajectory's final state
    log(f"all-active: median {np.median(t_all):.2f} ms per trajectory -> {rate(t_all):.2f} steps/s")
    all_rate = rate(t_all)
    # kernel timings in runs of their own, so that the steps/s figures above carry no
    # per-launch events: the frozen-run kernel in the headline schedule (the all-active
    # schedule has none), the profiled kernel class in the all-active schedule
    ms_fz, prof_fz = timed(scheds[head], "frozen")
    _, prof_fold = timed(scheds[head], "fold")
    ms_pk, prof_all = timed(all_active, args.profile_kernel)
    log(f"profiled runs: headline with frozen-run events {np.median(ms_fz):.2f} ms, all-active with "
        f"{args.profile_kernel} events {np.median(ms_pk):.2f} ms per trajectory")
    kernels = {} if args.no_kernel_table else kernel_table(cfg, n_traj, T, lambda c: timed(all_active, c)[1])

    def deviation():
        """Output deviation of the trajectory just run from the all-active one: the synthetic
        stand-in for the quality metrics (relative L2 and max-abs errors of the final state)."""
        d = (z - z_full).double()
        return {"rel_l2": float(d.norm() / z_full.double().norm()),
                "rel_max": float(d.abs().max() / z_full.double().abs().max())}

    tau_res = {}
    for t, sch in tau_scheds.items():
        times, _ = timed(sch)
        tau_res[t] = (times, deviation())
        log(f"tau {t:g}: {sch.layer_steps} layer-steps -> {rate(times):.2f} steps/s")
    rule_res = {}
    dev_head = None
    if rule_scheds:
        timed(scheds[head])
        dev_head = deviation()
    for r, sch in rule_scheds.items():
        times, _ = timed(sch)
        rule_res[r] = (times, deviation())
        log(f"rule {r}: lifetimes {sch.lifetimes.tolist()} -> {rate(times):.2f} steps/s, "
            f"deviation {rule_res[r][1]['rel_l2']:.3e} (method {dev_head['rel_l2']:.3e})")

    input_aware = None
    if not args.no_input_aware:
        # appendix "Dynamic baselines": the causal activation-drift policy at the headline
        # schedule's per-step active counts, and the oracle-replay pattern under the headline
        # budget as its ceiling (search not timed; one replay of the pattern is)
        drift_buf = dm.drift_buffer()
        d_rows = []

        def drift_step(s):
            row, _ = dm.drift_step(z, s, scheds[head], cache, drift_buf)
            d_rows.append(row)

        times, _ = timed(scheds[head], stepper=drift_step)
        d_dev = deviation()
        last = np.array(d_rows[-T:])
        input_aware = {"drift": {"steps_per_s": round(rate(times), 3), "speedup": round(rate(times) / all_rate, 4),
                                 "layer_steps": int(last.sum()), "deviation": d_dev,
                                 "rows_differ_from_static": int(np.sum(np.any(last != act_head, axis=1)))}}
        log(f"drift policy: {rate(times):.2f} steps/s (static {value_head:.2f}), deviation {d_dev['rel_l2']:.3e}")
        del drift_buf
        t0 = time.time()
        life, evals, _ = dm.replay_search(z0, tau_agree=args.tau_agree, max_layer_steps=scheds[head].layer_steps)
        torch.cuda.synchronize()
        t_search = time.time() - t0
        rsch = P.schedule_from_lifetimes(life, T)
        times, _ = timed(rsch)
        r_dev = deviation()
        input_aware["replay"] = {"steps_per_s": round(rate(times), 3), "speedup": round(rate(times) / all_rate, 4),
                                 "layer_steps": rsch.layer_steps, "ceiling": scheds[head].layer_steps,
                                 "tau_agree": args.tau_agree, "lifetimes": life.tolist(), "deviation": r_dev,
                                 "search_s": round(t_search, 2), "search_evaluations": evals}
        log(f"oracle replay: search {t_search:.1f}s ({evals} evaluations), lifetimes {life.tolist()} -> "
            f"{rate(times):.2f} steps/s, deviation {r_dev['rel_l2']:.3e}")

    branch_units = None
    if not args.no_branch_units and not args.lifetimes:
        # the same budget over branch units (each residual branch its own lifetime and cached
        # update), on the same device weights; spectra rebuilt per branch (offline, not timed)
        dmb = P.DeviceModel(cfg, weights, inputs, granularity="branch", share=dm)
        U = dmb.n_units
        bsch = P.schedule_build(dmb.scored_units(), [cfg.dh] * U, T, budget_pct=head)
        cache_b = P.Cache(dmb)

        def branch_step(s):
            if s == 1:
                cache_b.reset()
            dmb.step(z, s, bsch, cache_b)

        times, _ = timed(None, stepper=branch_step)
        b_dev = deviation()
        branch_units = {"units": U, "steps_per_s": round(rate(times), 3), "speedup": round(rate(times) / all_rate, 4),
                        "unit_steps": bsch.layer_steps, "of": U * T, "deviation": b_dev,
                        "lifetimes": bsch.lifetimes.tolist()}
        log(f"branch units ({U}): {bsch.layer_steps} unit-steps -> {rate(times):.2f} steps/s, "
            f"deviation {b_dev['rel_l2']:.3e}")
        del cache_b
        dmb.close()

    value = rate(results[head])
    head_ms = float(np.median(results[head]))

    # roofline of the dominant kernel, from the all-active run (largest launch count)
    fl = unit_flops(cfg)
    kern = args.profile_kernel
    kms, kn = prof_all
    kavg = kms / max(kn, 1) / 1000.0
    peak = PEAK_BF16 if cfg.dtype == "bf16" else PEAK_F32
    achieved = fl.get(kern, 0.0) / kavg if kavg > 0 else 0.0
    roofline = {"bound": "mfma", "kernel": kern, "achieved": achieved / 1e12, "peak": peak / 1e12,
                "unit": "TFLOP/s", "frac": achieved / peak, "traffic": None,
                "avg_launch_us": kavg * 1e6, "launches": kn,
                "flop_per_launch": fl.get(kern, 0.0)}

    # the mask rows actually timed: n_traj whole trajectories of the headline schedule
    act = np.asarray(scheds[head].active, bool)
    timed_rows = np.concatenate([act] * n_traj)
    active_frac = float(timed_rows.mean())
    mean_active = float(timed_rows.sum(axis=1).mean())
    # frozen path: algorithmic bytes of every launch that carries frozen units in the timed
    # steps (standalone frozen runs and pre-norms that absorbed a run) / their time
    fl = [frozen_launches(cfg, row) for row in timed_rows]
    b_alone = sum(sum(a) for a, _ in fl)
    b_fold = sum(sum(f) for _, f in fl)
    n_alone_want = sum(len(a) for a, _ in fl)
    n_fold_want = sum(len(f) for _, f in fl)
    fms, fn = prof_fz if prof_fz else (0.0, 0)
    fdms, fdn = prof_fold if prof_fold else (0.0, 0)
    frozen = None
    if fn or fdn:
        tot_b, tot_s = b_alone + b_fold, (fms + fdms) / 1000.0
        frozen = {"bound": "hbm", "kernel": "frozen_run + pre-norms that absorb a frozen run",
                  "achieved": tot_b / tot_s / 1e9, "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                  "frac": tot_b / tot_s / PEAK_HBM, "bytes": tot_b,
                  "standalone": {"launches": fn, "expected": n_alone_want, "bytes": b_alone,
                                 "avg_launch_us": fms * 1000.0 / fn if fn else None,
                                 "GB/s": b_alone / (fms / 1000.0) / 1e9 if fn else None},
                  "folded_into_norm": {"launches": fdn, "expected": n_fold_want, "bytes": b_fold,
                                       "avg_launch_us": fdms * 1000.0 / fdn if fdn else None,
                                       "GB/s": b_fold / (fdms / 1000.0) / 1e9 if fdn else None},
                  "note": "h and the cached updates; h may be served from the 256 MB Infinity Cache"}
    tr = committed_traffic(kern, cfg)
    roofline["traffic"] = tr["total_bytes"] if tr else None
    roofline["traffic_detail"] = tr
    if frozen:
        # counter record of one isolated frozen-run launch (a run of r cached updates): measured
        # HBM bytes against its algorithmic bytes, so the ratio applies to every launch
        ftr = committed_traffic("frozen_run", cfg)
        frozen["traffic_detail"] = ftr
        frozen["traffic_over_algorithmic"] = (ftr["total_bytes"] / ftr["algorithmic_bytes"]
                                              if ftr and ftr.get("algorithmic_bytes") else None)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, weights, inputs, mean_active, args.cpu_seconds)

    lay = {pct: scheds[pct].layer_steps for pct in budgets}
    line = {
        "metric": "denoise steps/s scheduled vs all-active; MFMA % peak; LLaDA-8B shape",
        "value": round(value, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": n_traj * T,
        "steps_requested": K,
        "trajectories": n_traj,
        "warmup": W,
        "ms_per_step": round(head_ms / T, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic (seeded planted-spectrum weights and inputs)",
        "config": {"workload": f"{cfg.name}: B={cfg.B} N={cfg.N} d={cfg.d} H={cfg.H} F={cfg.F} L={L} T={T}",
                   "budget_pct": head, "layer_steps": lay[head], "of": L * T,
                   "global_batch": cfg.B, "seq_len": cfg.N, "parallelism": "single GPU"},
        "graph_steps_per_s": round(rate(t_graph), 3) if t_graph else None,
        "all_active_steps_per_s": round(all_rate, 3),
        "speedup_vs_all_active": round(value / all_rate, 4),
        "skipped_layer_step_fraction": round(1 - active_frac, 4),
        "ideal_speedup": round(1 / active_frac, 4),
        "budgets": {str(p): {"steps_per_s": round(rate(results[p]), 3), "layer_steps": lay[p],
                             "speedup": round(rate(results[p]) / all_rate, 4),
                             "traj_ms": [round(t, 3) for t in results[p]]} for p in budgets},
        "all_active_traj_ms": [round(t, 3) for t in t_all],
        "tau": {f"{t:g}": {"steps_per_s": round(rate(tm), 3), "layer_steps": tau_scheds[t].layer_steps,
                           "frac_layer_steps": round(tau_scheds[t].layer_steps / (L * T), 4),
                           "speedup": round(rate(tm) / all_rate, 4), "deviation": dv}
                for t, (tm, dv) in tau_res.items()},
        "rules": {"budget_pct": head, "scr_frob": {"steps_per_s": round(value, 3), "deviation": dev_head},
                  **{r: {"steps_per_s": round(rate(tm), 3), "speedup": round(rate(tm) / all_rate, 4),
                         "layer_steps": rule_scheds[r].layer_steps, "deviation": dv}
                     for r, (tm, dv) in rule_res.items()}},
        "input_aware": input_aware,
        "branch_units": branch_units,
        "roofline": roofline,
        "kernels": kernels,
        "frozen_path": frozen,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    dm.close()
    return 0


def kernel_table(cfg, n_traj, T, profile) -> dict:
    """Average launch duration of every kernel class of the all-active step (HIP events around
    each launch on the step's stream, one timed pass per class) with its algorithmic work:
    FLOP against the MFMA peak of the workload's dtype, bytes against HBM for the norms."""
    M, d, F, H, dh, N, B = cfg.M, cfg.d, cfg.F, cfg.H, cfg.dh, cfg.N, cfg.B
    es = 2 if cfg.dtype == "bf16" else 4
    peak = PEAK_BF16 if cfg.dtype == "bf16" else PEAK_F32
    fl = unit_flops(cfg)
    classes = ["gemm_qkv", "attn", "gemm_o", "gemm_w1", "gemm_w2", "norm", "norm_parts"]
    if cfg.arch in ("sdxl", "sdxl_unet"):
        classes += ["gemm_x", "attn_x"]
    if cfg.arch == "sdxl_unet":
        classes += ["gemm_conv", "gnorm"]
    if cfg.arch == "uvit":
        classes += ["gemm_skip"]
        fl["gemm_skip"] = 2.0 * M * d * 2 * d
    if cfg.arch == "dit":
        classes += ["cond"]
    out = {}
    for c in classes:
        ms, n = profile(c)
        if not n:
            continue
        rec = {"launches": n, "avg_us": round(ms * 1000.0 / n, 2)}
        if c == "gnorm":
            # GroupNorm + SiLU: fp32 stream in (first) or bf16 convolution output in (second),
            # bf16 out; launches alternate
            nbytes = M * d * ((4 + 2) + (2 + 2)) / 2
            rec.update({"GB/s": round(nbytes * n / (ms / 1000.0) / 1e9, 1),
                        "frac_hbm": round(nbytes * n / (ms / 1000.0) / PEAK_HBM, 4)})
        elif c in ("norm", "norm_parts"):
            # fp32 stream in, normalised rows out; adding a split output GEMM's two partial
            # products also reads them and writes the stream back
            nbytes = M * d * (4 + es) if c == "norm" else M * d * (4 * 4 + es)
            rec.update({"GB/s": round(nbytes * n / (ms / 1000.0) / 1e9, 1),
                        "frac_hbm": round(nbytes * n / (ms / 1000.0) / PEAK_HBM, 4)})
        elif c == "gemm_x":
            # cross q / o projections every step, context k / v once per trajectory and unit
            n_ctx = cfg.L * n_traj
            total = (n - n_ctx) * 2.0 * M * d * d + n_ctx * 2.0 * B * cfg.ctx_len * 2 * d * cfg.ctx_dim
            rec.update({"TFLOP/s": round(total / (ms / 1000.0) / 1e12, 1),
                        "frac_peak": round(total / (ms / 1000.0) / peak, 4)})
        elif c in fl:
            rec.update({"TFLOP/s": round(fl[c] * n / (ms / 1000.0) / 1e12, 1),
                        "frac_peak": round(fl[c] * n / (ms / 1000.0) / peak, 4)})
        out[c] = rec
    return out


def cpu_baseline(cfg, weights, inputs, mean_active, seconds):
    """Oracle (numpy float64) on a bounded sample: units of one all-active step, in stack order,
    until `seconds` have passed (at least two units, at most the whole stack).

    Scaled to steps/s of the timed scheduled trajectories: the oracle's time per step is its
    time per active unit times the mean active units per timed step (frozen units cost an
    addition each).
    """
    import dataclasses

    import numpy as np
    from oracle import model as om

    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
    log(f"cpu baseline: oracle on units of an all-active step, about {seconds:.0f}s ({threads} threads)")
    m = om.Model(dataclasses.replace(cfg), weights, inputs, lazy=True)
    h = om.initial_stream(m, inputs["z"], 1)
    t0 = time.time()
    n = 0
    while n < cfg.L and (n < 2 or time.time() - t0 < seconds):
        cross = m.cross_kv(m.units[n]) if cfg.arch in ("sdxl", "sdxl_unet") else None
        if cfg.arch == "uvit" and n > cfg.L // 2:
            break  # out-blocks need the skip inputs of the whole in-stack; in-blocks suffice
        h, _ = m.unit_active(n, h, om.timestep_value(1, cfg.T), cross)
        n += 1
    dt = time.time() - t0
    per_unit = dt / n
    per_step = per_unit * mean_active
    log(f"cpu baseline: {n} units in {dt:.1f}s, {per_unit:.2f}s per active unit -> {per_step:.1f}s per scheduled step")
    return {"value": round(1.0 / per_step, 6), "unit": "steps/s", "cores": threads, "kind": "oracle",
            "sample": f"{n} of {cfg.L} units of one all-active step at full size ({dt:.1f}s), "
                      f"scaled by {mean_active:.2f} mean active units per scheduled step"}


def committed_traffic(kern: str, cfg):
    """HBM bytes per launch of the timed kernel from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE passes (profiles/<kernel>_<workload>_traffic.json), scaled by the copy-kernel
    calibration recorded there; None unless the record was taken on this exact kernel source."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{kern}_{cfg.name}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    src = os.path.join(ROOT, rec.get("source", ""))
    if not os.path.exists(src) or hashlib.sha256(open(src, "rb").read()).hexdigest() != rec.get("sha256"):
        return None
    return {"fetch_bytes": rec["fetch_bytes"], "write_bytes": rec["write_bytes"],
            "total_bytes": rec["fetch_bytes"] + rec["write_bytes"],
            "algorithmic_bytes": rec.get("algorithmic_bytes"), "profile": os.path.relpath(path, ROOT)}


if __name__ == "__main__":
    sys.exit(main())
