#!/usr/bin/env python3
"""Throughput of the VestigeKV decode step on one MI355X.

One step = query prep -> index scan (score) -> exact top-k (select) ->
[certified admission] -> gather-attend, over one batch of synthetic MLA
decode state resident in HBM.  Default workload: 32 sequences x 128 heads x
131072 cached rows (rho = 1/32 budget + 512 recent rows, rope + rank-64
digest index) -- the long-context configuration the metric is quoted on.

Prints ONE JSON line.  ``value`` = archived rows scored per second =
B * (T - W) / t_step, with t_step the median of the timed steps (each step
bracketed by HIP events on the step's stream).  ``roofline`` is for the
dominant kernel (the index scan), timed with HIP events on the stream it runs
on; ``roofline.step`` gives the whole step against the same HBM peak.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "archived KV rows scored+attended/sec per decode step; % of HBM peak BW"
HBM_PEAK_GBS = 8000.0
SCORE_SOURCE = os.path.join(ROOT, "paper_2609_03949_amd", "csrc", "k_score.hip")


def log(msg: str):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_hash(path: str) -> str:
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def traffic_for(kernel: str, workload: str, launches_per_step: int):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary, or
    None when it is missing or was taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("source_sha256_16") != source_hash(SCORE_SOURCE):
        return None
    return rec.get("bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="cfg4")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--no-stages", action="store_true",
                    help="skip the per-stage diagnostic pass (each stage call timed alone)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 1 GiB device copy (counter scale for --pmc runs)")
    ap.add_argument("--path", choices=("index", "kept"), default="index",
                    help="index: top-k of the index scan is the attended tier (vkv_step_run); kept: the "
                         "deployed path -- the sigma tier of the closed blocks is attended, the index scan "
                         "feeds the calibrated trigger (vkv_step_run_kept)")
    ap.add_argument("--sketch", action="store_true",
                    help="(kept path) content queries near a 48-dim subspace and the index basis V_r fitted "
                         "on the GPU to 4096 prefix queries of the same law (vkv_sketch_basis)")
    ap.add_argument("--page", type=int, default=0,
                    help="(index path) also build the page boxes of this many rows and time the page "
                         "bounds; report the share of pages whose bound is below theta (outside the timed "
                         "region, not in the step)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: libvkv has no multi-GPU path "
              "(sequences are independent and would shard across GPUs with no communication).",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_03949_amd as vkv
    from paper_2609_03949_amd import budget, synth

    cfg = synth.CONFIGS[args.config]
    dev = torch.device("cuda:0")
    if args.path == "kept":
        return run_kept_path(args, cfg, dev)
    log(f"workload {synth.describe(cfg)}")
    t0 = time.time()
    wl = synth.make_workload(cfg, dev)
    torch.cuda.synchronize()
    log(f"generated inputs in {time.time() - t0:.1f}s")
    ctx = vkv.Context(0)
    B, H, T, W, A, k = wl["B"], wl["H"], wl["T"], wl["W"], wl["A"], wl["k"]
    mode, r = cfg.mode, cfg.r
    two_tier = cfg.two_tier

    # ---- index build (the compression event; timed separately, not in the step)
    if mode == synth.MODE_ROPE:
        cols, has_rope = 0, True
    elif mode == synth.MODE_DIGEST:
        cols, has_rope = r, False
    else:
        cols, has_rope = 64 + r, True
    index = torch.empty(B, T, cols, dtype=torch.bfloat16, device=dev) if cols else None
    eta = eps = gam = None
    if two_tier:
        eta = torch.empty(B, T, dtype=torch.float32, device=dev)
        eps = torch.empty_like(eta)
        gam = torch.empty_like(eta)
    digest_ms = None
    if index is not None or two_tier:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        vkv.digest_build(ctx, wl["cache"], wl["P"], r if mode != synth.MODE_ROPE else 0,
                         has_rope, index, eta, eps, gam)
        e1.record()
        torch.cuda.synchronize()
        digest_ms = e0.elapsed_time(e1)
        log(f"index build {digest_ms:.2f} ms")
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], W, mode,
                    r if mode != synth.MODE_ROPE else 0, index=index, index_has_rope=has_rope,
                    P=wl["P"], eta=eta, eps=eps, gam=gam)
    bufs = vkv.Buffers(step, k, two_tier=two_tier)
    stream = torch.cuda.current_stream()

    def run_step():
        vkv.step_run(ctx, step, bufs.ws, k, None, bufs.ub, bufs.sel, bufs.theta, bufs.adm,
                     bufs.adm_count, bufs.cap, cfg.scale, bufs.out, bufs.lse, stream, bufs.cert_mult)

    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()
    if args.copy_probe:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("copy probe: 3 x 1 GiB device copies done")
        del src, dst

    # ---- timed region: K steps through vkv_step_run, an event between
    # consecutive steps on the step's stream; the library records HIP events
    # around each score scan on the stream it runs on
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    ctx.set_timing(True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(args.steps):
        run_step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    score_launch_ms = ctx.score_timing()
    ctx.set_timing(False)
    step_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    total_ms = evs[0].elapsed_time(evs[-1])
    ms_per_step = float(np.median(step_ms))
    assert len(score_launch_ms) == args.steps, (len(score_launch_ms), args.steps)
    launch_ms = float(np.median(score_launch_ms))
    adm_total = int(bufs.adm_count.sum().item()) if two_tier else 0
    log(f"step median {ms_per_step:.4f} ms (mean {total_ms / args.steps:.4f}, min {min(step_ms):.4f}, "
        f"max {max(step_ms):.4f}) over {args.steps} steps; score launch median {launch_ms:.4f} ms; "
        f"wall {wall / args.steps * 1e3:.4f} ms")

    # ---- diagnostics outside the timed region: each stage call timed alone
    stages = ["query_prep", "score", "select"] + (["admit"] if two_tier else []) + ["attend"]
    per_stage = None
    if not args.no_stages:
        nev = len(stages) + 1
        reps = max(3, min(args.steps, 10))
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(reps)]
        for s_ in range(reps):
            ev = evs[s_]
            ev[0].record(stream)
            vkv.query_prep(ctx, step, bufs.ws, stream)
            ev[1].record(stream)
            vkv.score(ctx, step, bufs.ws, None, bufs.ub, stream, bufs.cert_mult)
            ev[2].record(stream)
            vkv.select(ctx, step, bufs.ws, k, bufs.sel, bufs.theta, stream)
            ev[3].record(stream)
            j = 3
            if two_tier:
                vkv.admit(ctx, step, bufs.ws, k, bufs.sel, bufs.theta, bufs.ub, bufs.adm,
                          bufs.adm_count, bufs.cap, stream, bufs.cert_mult)
                j += 1
                ev[j].record(stream)
            vkv.attend(ctx, step, bufs.ws, k, bufs.sel, bufs.adm, bufs.adm_count, bufs.cap,
                       cfg.scale, bufs.out, bufs.lse, stream)
            ev[j + 1].record(stream)
        torch.cuda.synchronize()
        per_stage = {name: float(np.mean([evs[s_][i].elapsed_time(evs[s_][i + 1]) for s_ in range(reps)]))
                     for i, name in enumerate(stages)}
        per_stage["step_with_stage_events"] = float(np.mean([evs[s_][0].elapsed_time(evs[s_][-1])
                                                       for s_ in range(reps)]))
        log(f"stages alone (ms): {json.dumps({k_: round(v, 4) for k_, v in per_stage.items()})}")

    # ---- optional: page boxes and their interval bounds (page-bound pruning),
    # outside the timed region; the share of pages below theta is what a scan
    # that skips pages by the bound would save
    page_info = None
    if args.page > 0:
        npg = (A + args.page - 1) // args.page
        n_idx = cols if cols else 64
        box = torch.empty(B, max(npg, 1), 2, n_idx, dtype=torch.bfloat16, device=dev)
        bound = torch.empty(B, max(npg, 1), dtype=torch.float64, device=dev)
        run_step()
        vkv.page_box(ctx, step, args.page, box, stream)   # warm-up (first launches load the kernels)
        vkv.page_bound(ctx, step, bufs.ws, args.page, box, bound, stream)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev[0].record(stream)
        vkv.page_box(ctx, step, args.page, box, stream)
        ev[1].record(stream)
        vkv.page_bound(ctx, step, bufs.ws, args.page, box, bound, stream)
        ev[2].record(stream)
        torch.cuda.synchronize()
        below = int((bound[:, :npg] < bufs.theta[:, None]).sum().item())
        page_info = {"page": args.page, "pages": B * npg, "below_theta": below,
                     "box_ms": ev[0].elapsed_time(ev[1]), "bound_ms": ev[1].elapsed_time(ev[2])}
        log(f"page bound (page {args.page}): {below} of {B * npg} pages below theta "
            f"({100.0 * below / max(1, B * npg):.3f}%); boxes {page_info['box_ms']:.3f} ms, "
            f"bounds {page_info['bound_ms']:.3f} ms")

    rows_per_s = B * A / (ms_per_step * 1e-3)
    sb = budget.step_bytes(B, H, T, W, k, mode, r, two_tier, adm_total)
    step_gbs = sb["total"] / (ms_per_step * 1e-3) / 1e9
    scan_bytes = sb["scan"]
    achieved = scan_bytes / (launch_ms * 1e-3) / 1e9
    workload = args.config
    traffic = traffic_for("score_kernel", workload, 1)
    line = {
        "metric": METRIC,
        "value": rows_per_s,
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ms_per_step_stats": {"median": ms_per_step, "mean": total_ms / args.steps,
                              "min": float(min(step_ms)), "max": float(max(step_ms)),
                              "p90": float(np.percentile(step_ms, 90))},
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": synth.describe(cfg),
            "B": B, "H": H, "T": T, "W": W, "k": k, "r": r,
            "mode": synth.MODE_NAMES[mode], "two_tier": two_tier,
        },
        "hbm_frac_step": step_gbs / HBM_PEAK_GBS,
        "step_gbs": step_gbs,
        "step_bytes": sb,
        "stage_ms": per_stage,
        "attended_rows_per_seq": k + W + (adm_total / B if two_tier else 0),
        "index_build_ms": digest_ms,
        **({"page_bound": page_info} if page_info else {}),
        "roofline": {
            "bound": "hbm",
            "kernel": "score_stream_kernel (index scan)",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "bytes_per_launch": scan_bytes,
            "launch_ms": launch_ms,
            "launch_ms_is": "median of the timed launches",
            "launches_timed": len(score_launch_ms),
            # the whole step (score, select, attend and the rest) against the
            # same peak: algorithmic bytes of the step / median step time
            "step": {
                "bound": "hbm",
                "achieved": step_gbs,
                "peak": HBM_PEAK_GBS,
                "unit": "GB/s",
                "frac": step_gbs / HBM_PEAK_GBS,
                "bytes_per_step": sb["total"],
                "ms": ms_per_step,
            },
        },
    }

    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, cfg, args.cpu_seconds)
    print(json.dumps(line), flush=True)
    ctx.close()


def run_kept_path(args, cfg, dev):
    """The deployed per-step path on the same workload (the deployment
    specification's request lifecycle): the closed 4096-row blocks of every
    sequence get their sigma once (block close), the sigma tier (4 sinks + the
    sigma-top-(k-4) rows) is the attended tier, and each step runs query prep ->
    index scan with the certificate -> the tier's exact maximum logit ->
    calibrated trigger (z from this step's own queries, conformal quantile at
    tau_s = 18/19) -> attention over tier, recent window and fired rows."""
    import math

    import numpy as np
    import torch

    import paper_2609_03949_amd as vkv
    from paper_2609_03949_amd import budget, synth

    if not (cfg.mode & 1):
        raise SystemExit("the kept path needs the branch summand in the index key (a mode with rope)")
    if args.sketch:
        cfg = cfg.with_(queries="lowrank")
    log(f"workload {synth.describe(cfg)} (kept path)")
    wl = synth.make_workload(cfg, dev)
    ctx = vkv.Context(0)
    B, H, T, W, A, k, r = wl["B"], wl["H"], wl["T"], wl["W"], wl["A"], wl["k"], cfg.r
    rr = r if cfg.mode != synth.MODE_ROPE else 0
    sketch_ms = None
    if args.sketch:
        if rr == 0:
            raise SystemExit("--sketch needs a digest (r > 0)")
        qpre = synth.prefix_queries(cfg, 4096, dev)
        kws = torch.empty(vkv.sketch_workspace_size(rr), dtype=torch.uint8, device=dev)
        Pg = torch.empty(rr, 512, dtype=torch.bfloat16, device=dev)
        energy = torch.empty(2, dtype=torch.float64, device=dev)
        t0 = time.perf_counter()
        vkv.sketch_basis(ctx, qpre, rr, 8, kws, Pg, energy)
        sketch_ms = (time.perf_counter() - t0) * 1e3
        en = energy.cpu().numpy()
        log(f"sketch basis from 4096 prefix queries: {sketch_ms:.2f} ms, captures {en[0] / en[1] * 100:.2f}% "
            f"of their second moment")
        wl["P"] = Pg
    cols = 64 + rr
    index = torch.empty(B, T, cols, dtype=torch.bfloat16, device=dev)
    eta = torch.empty(B, T, dtype=torch.float32, device=dev)
    eps, gam = torch.empty_like(eta), torch.empty_like(eta)
    vkv.digest_build(ctx, wl["cache"], wl["P"], rr, True, index, eta, eps, gam)
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], W, cfg.mode, rr, index=index, index_has_rope=True,
                    P=wl["P"], eta=eta, eps=eps, gam=gam)
    # block close: sigma of the closed blocks, then the tier (timed once; not per step)
    nblk = A // vkv.SIGMA_BLOCK
    n_closed = nblk * vkv.SIGMA_BLOCK
    sig = torch.empty(B, max(n_closed, 1), dtype=torch.float64, device=dev)
    sws = torch.empty(max(vkv.sigma_workspace_size(B, nblk), 256), dtype=torch.uint8, device=dev)
    K = vkv.sigma_tier_size(n_closed, k - 4)
    kept = torch.empty(B, max(K, 1), dtype=torch.int32, device=dev)
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    e0.record()
    vkv.sigma_close(ctx, wl["cache"], 0, nblk, 16 if T <= 16384 else 64, sws, sig)
    e1.record()
    vkv.sigma_select(ctx, sig, n_closed, k - 4, 4, kept)
    e2.record()
    torch.cuda.synchronize()
    close_ms, select_ms = e0.elapsed_time(e1), e1.elapsed_time(e2)
    log(f"block close: sigma of {nblk} blocks x {B} sequences {close_ms:.3f} ms, tier select {select_ms:.3f} ms")
    ws = vkv.alloc_workspace(step, K, A)
    # calibration on this step's queries: the causal argmax over the whole
    # context, the tier's maximum, the required inflations of the hard pairs
    vkv.query_prep(ctx, step, ws)
    smax_all = torch.empty(B, H, dtype=torch.float64, device=dev)
    arg_all = torch.empty(B, H, dtype=torch.int32, device=dev)
    smax_t = torch.empty_like(smax_all)
    arg_t = torch.empty_like(arg_all)
    vkv.row_max(ctx, step, None, True, smax_all, arg_all)
    vkv.row_max(ctx, step, kept, True, smax_t, arg_t)
    hard = torch.empty(B, H, dtype=torch.int32, device=dev)
    zq = torch.empty(B, H, dtype=torch.float64, device=dev)
    vkv.required_inflation(ctx, step, ws, K, kept, smax_t, arg_all, hard, zq)
    torch.cuda.synchronize()
    hz = zq[hard != 0].cpu().numpy()
    z, min_hard, krank = vkv.conformal_z(hz, tau=(9, 10), zmax=8.0)
    cm = z / math.sqrt(512 - rr)
    log(f"calibration: {len(hz)} hard (query, head) pairs of {B * H}, z = {z:.4f} (rank {krank}), "
        f"cert_mult = {cm:.5f}")
    f32 = dict(dtype=torch.float32, device=dev)
    ub = torch.empty(B, A, **f32)   # the step reads only the trigger margins (no key buffer)
    smax = torch.empty(B, H, dtype=torch.float64, device=dev)
    arg = torch.empty(B, H, dtype=torch.int32, device=dev)
    fired = torch.empty(B, A, dtype=torch.int32, device=dev)
    cnt = torch.empty(B, dtype=torch.int32, device=dev)
    out = torch.empty(B, H, 512, dtype=torch.bfloat16, device=dev)
    lse = torch.empty(B, H, **f32)
    stream = torch.cuda.current_stream()

    def run_step():
        vkv.step_run_kept(ctx, step, ws, K, kept, None, ub, cm, smax, arg, 0, fired, cnt, A, cfg.scale, out, lse,
                          stream)

    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(stream)
    for i in range(args.steps):
        run_step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    step_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    ms = float(np.median(step_ms))
    fired_total = int(cnt.sum().item())
    frac = fired_total / (B * (A - K))
    sb = budget.step_bytes(B, H, T, W, K, cfg.mode, r, True, fired_total)
    log(f"kept path: step median {ms:.4f} ms; fired {fired_total} rows = {frac * 100:.3f}% of the archived rows "
        f"outside the tier")
    line = {
        "metric": METRIC, "value": B * A / (ms * 1e-3), "unit": "rows/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": synth.describe(cfg), "path": "kept (sigma tier + calibrated trigger)",
                   "B": B, "H": H, "T": T, "W": W, "tier": K, "r": r},
        "tier_rows_per_seq": K, "fired_fraction": frac, "z": z, "cert_mult": cm, "hard_pairs": int(len(hz)),
        "block_close_ms": close_ms, "tier_select_ms": select_ms, "sketch_basis_ms": sketch_ms,
        "step_gbs": sb["total"] / (ms * 1e-3) / 1e9, "hbm_frac_step": sb["total"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
    }
    print(json.dumps(line), flush=True)
    ctx.close()


def cpu_model() -> dict:
    """The host CPU as the kernel reports it (model name, family/model/stepping,
    logical CPUs in this process's affinity set)."""
    info = {}
    try:
        for line in open("/proc/cpuinfo"):
            k, _, v = line.partition(":")
            k, v = k.strip(), v.strip()
            if k in ("model name", "cpu family", "model", "stepping", "vendor_id") and k not in info:
                info[k] = v
    except OSError:
        pass
    try:
        import subprocess
        out = subprocess.run(["lscpu"], capture_output=True, text=True).stdout.splitlines()
        for l in out:
            if l.startswith("Model name") and "lscpu_model" not in info:
                info["lscpu_model"] = l.split(":", 1)[1].strip()
            if l.startswith("Socket(s)"):
                info["sockets"] = l.split(":", 1)[1].strip()
    except Exception:
        pass
    # AMD's family numbers: 25 (19h) is Zen 3 / Zen 4, 26 (1Ah) is Zen 5
    if info.get("vendor_id") == "AuthenticAMD":
        fam = {"25": "Zen 3 / Zen 4 (family 19h)", "26": "Zen 5 (family 1Ah)"}.get(info.get("cpu family", ""))
        if fam:
            info["core_family"] = fam
    info["logical_cpus_affinity"] = len(os.sched_getaffinity(0))
    info["logical_cpus_total"] = os.cpu_count()
    return info


def cpu_baseline(wl, cfg, target_s: float):
    """The fp64 oracle, as it stands, on whole sequences of the same workload:
    index keys -> top-k -> [bound + admission] -> attention.  The oracle's own
    index build for the sample runs first and is not timed (it is the
    compression event, timed separately on both sides).  Two figures: the
    oracle with its OpenMP threads over rows (``value``), and the same step on
    one thread for one sequence (``value_1thread``)."""
    import numpy as np  # noqa: F401

    import oracle
    from paper_2609_03949_amd import synth

    sys.path.insert(0, os.path.join(ROOT, "tests"))
    oracle.build(force=False)
    nthreads = oracle.max_threads()
    mode, r, W, k = cfg.mode, cfg.r, wl["W"], wl["k"]
    rr = r if mode != synth.MODE_ROPE else 0
    if mode == synth.MODE_ROPE:
        has_rope, cols = True, 0
    elif mode == synth.MODE_DIGEST:
        has_rope, cols = False, r
    else:
        has_rope, cols = True, 64 + r

    def host_seq(b):
        import torch
        t = torch.tensor([b], device=wl["cache"].device)
        cache = synth.to_numpy_bits(wl["cache"].index_select(0, t))
        q_lat = synth.to_numpy_bits(wl["q_lat"].index_select(0, t))
        q_rope = synth.to_numpy_bits(wl["q_rope"].index_select(0, t))
        P = synth.to_numpy_bits(wl["P"]) if wl["P"] is not None else None
        index = eta = eps = gam = None
        if cols or cfg.two_tier:
            index, eta, eps, gam = oracle.digest_build(cache, P, rr, with_rope=has_rope,
                                                       scalars=cfg.two_tier, nthreads=nthreads)
            if not cols:
                index = None
        return cache, q_lat, q_rope, P, index, eta, eps, gam

    def one_step(inputs, threads):
        cache, q_lat, q_rope, P, index, eta, eps, gam = inputs
        t0 = time.perf_counter()
        oracle.step(cache, q_lat, q_rope, index, P, rr, mode, W, k, cfg.scale,
                    two_tier=cfg.two_tier, eta=eta, eps=eps, gam=gam, index_has_rope=has_rope,
                    nthreads=threads)
        return time.perf_counter() - t0

    done_rows = 0
    elapsed = 0.0
    seqs_done = 0
    b = 0
    build_s = 0.0
    first = None
    while elapsed < target_s and b < wl["B"]:
        tb = time.perf_counter()
        inputs = host_seq(b)
        build_s += time.perf_counter() - tb
        if first is None:
            first = inputs
        elapsed += one_step(inputs, nthreads)
        done_rows += wl["A"]
        seqs_done += 1
        b += 1
        log(f"cpu oracle: sequence {b - 1} done, {elapsed:.1f}s timed so far")
    one_s = one_step(first, 1)
    log(f"cpu oracle, one thread: one sequence in {one_s:.1f}s")
    return {
        "value": done_rows / elapsed,
        "unit": "rows/s",
        "cores": nthreads,
        "kind": "oracle",
        "sample": f"{seqs_done} whole sequence(s) of the same workload (A={wl['A']} archived rows each), "
                  f"one full step each; fp64 oracle with OpenMP over rows ({nthreads} threads); oracle "
                  f"index build ({build_s:.1f}s) not timed",
        "value_1thread": wl["A"] / one_s,
        "sample_1thread": f"sequence 0 of the same workload, one full step, one thread ({one_s:.2f}s)",
        "cpu": cpu_model(),
        "timed_s": elapsed,
    }


if __name__ == "__main__":
    main()
