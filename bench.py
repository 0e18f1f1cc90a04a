#!/usr/bin/env python3
"""Benchmark of the batched draft step on one MI355X.

One bench step = one whole draft of the pool: the truncated S'-step loop of the 1.3B-shaped DiT over
N = 16 seed-distinct candidates (1560 image tokens, 512 text tokens), every third block skipped and
activation proxies on odd steps -- every row of the hot path (truncation, dispatch, computed blocks,
cache stores, proxies, skips, head + Euler update).  Inputs are resident in HBM and the prompt's
cross-attention K/V is prepared before the timed region (it is timed separately, as is the
refinement of the selected candidate).

Prints one JSON line.  ``value`` = candidates drafted per second.  ``roofline`` reports the dominant
kernel by GPU time -- the residual-epilogue GEMM (``k_linear_dma8<EPI_RESIDUAL>``: the self- and
cross-attention output projections and the MLP down-projection with gate, residual and cache store) --
timed live with HIP events that the library records on its launch stream around every launch of those
sites inside the timed region; ``roofline_secondary`` does the same for the MLP up-projection.
``cpu_baseline`` times the CPU oracle on a bounded sample.  ``c2_full_step`` is one full-quality step
of one candidate (the refinement's steps), and ``secondary_workloads`` drafts the 14B-shaped pool of 4
and the 1.3B-shaped pool of 64 (each with a short timed region of its own).
"""
import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # 256 CUs x 4096 bf16 FLOP/clk (dense MFMA) x 2.4 GHz
PEAK_HBM_GBS = 8000.0


def block_flops(shape, T, text_len):
    D, F = shape.hidden, shape.mlp_hidden
    gemm = 2 * T * D * (3 * D) + 2 * T * D * D + 2 * T * D * D + 2 * T * D * D + 2 * 2 * T * D * F
    attn = 4 * T * T * D + 4 * T * text_len * D
    return gemm + attn


def draft_flops(wl, traces):
    """Algorithmic FLOPs of one draft of the pool: computed blocks only, plus patch embed and head
    (the embed only where it is live)."""
    s = wl.shape
    T = wl.tokens
    per_block = block_flops(s, T, wl.text_len)
    total = 0
    for tr in traces:
        n_comp = sum(1 for e in tr if e[0] == 0)
        first = next((e[0] for e in tr if e[0] != 1), 0)
        embed = 2 * T * s.patch_dim * s.hidden if first == 0 else 0
        total += n_comp * per_block + embed + 2 * T * s.hidden * s.patch_dim
    return total * wl.n


def site_rooflines(wl, traces, breakdown):
    """Per launch site of one draft: algorithmic TFLOP/s against the bf16 MFMA peak (projections,
    attention) or algorithmic HBM GB/s against 8 TB/s (LayerNorms: read 4 + write 2 bytes per element;
    proxies: (order + 1) fp32 reads + 1 write per element), from the site timings of that draft."""
    s = wl.shape
    M, D, F, T, Lt = wl.n * wl.tokens, s.hidden, s.mlp_hidden, wl.tokens, wl.text_len
    flops = {"qkv": 2.0 * M * 3 * D * D, "out": 2.0 * M * D * D, "cross_q": 2.0 * M * D * D,
             "out_cross": 2.0 * M * D * D, "mlp_up": 2.0 * M * F * D, "mlp_down": 2.0 * M * D * F,
             "attn_self": 4.0 * wl.n * T * T * D, "attn_cross": 4.0 * wl.n * T * Lt * D}
    out = {}
    for site, f in flops.items():
        b = breakdown.get(site)
        if b:
            tf = f * b["launches"] / (b["ms"] / 1e3) / 1e12
            out[site] = {"bound": "mfma", "TFLOPs": round(tf, 1), "frac": round(tf / PEAK_BF16_TFLOPS, 4)}
    b = breakdown.get("norm")
    if b:
        gbs = 6.0 * M * D * b["launches"] / (b["ms"] / 1e3) / 1e9
        out["norm"] = {"bound": "hbm", "GBs": round(gbs, 1), "frac": round(gbs / PEAK_HBM_GBS, 4)}
    b = breakdown.get("proxy")
    if b:
        nbytes = sum(4.0 * M * D * (e[1] + 2) for tr in traces for e in tr if e[0] == 2 and e[3])
        gbs = nbytes / (b["ms"] / 1e3) / 1e9
        out["proxy"] = {"bound": "hbm", "GBs": round(gbs, 1), "frac": round(gbs / PEAK_HBM_GBS, 4)}
    return out


def recorded_traffic(profile="linear_residual_traffic.md"):
    """HBM bytes per launch of a kernel from its committed counter summary under profiles/, or None if
    the kernel source has changed since the counters were taken (or there is no summary)."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", profile)
    src = os.path.join(ROOT, "paper_2607_04461_amd", "csrc", "gemm.hip")
    try:
        txt = open(path).read()
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
        rec = re.search(r"gemm_source_sha256 \| ([0-9a-f]{64})", txt).group(1)
        val = float(re.search(r"traffic_bytes_per_launch \| ([0-9.e+]+)", txt).group(1))
    except (OSError, AttributeError, ValueError):
        return None
    return val if rec == sha else None


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, W, z0, text, traces):
    """The oracle, as it stands, on candidate 0 of the pool: its first two steps are timed, and the
    draft's time per candidate is extrapolated from the pool's own dispatch traces -- each step costs
    the timed computing step scaled by its number of computed blocks, or the timed proxy-only step.
    The oracle's BLAS runs with the threads the process may use (``cores``)."""
    from oracle import dit as odit
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        host_cpus = len(os.sched_getaffinity(0))
        limit = min(host_cpus, int(os.environ.get("OMP_NUM_THREADS", host_cpus)))
        threadpool_limits(limit)
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        host_cpus = cores = os.cpu_count()
    sched = wl.schedule()
    t0 = time.time()
    kv = odit.prepare_text(W, wl.shape, text)
    cache = odit.PoolCache(wl.shape.num_blocks)
    t1 = time.time()
    z = z0.astype(np.float64)
    times, ncomp = [], []
    for k in range(2):
        skip, proxy = wl.masks(k)
        ts = time.time()
        z, tr = odit.draft_step(W, wl.shape, z, sched[k], sched[k + 1], kv, wl.cond_index(), skip, proxy,
                                cache, candidates=[0])
        times.append(time.time() - ts)
        ncomp.append(sum(1 for e in tr if e[0] == 0))
    assert ncomp[0] > 0 and ncomp[1] == 0, "the sample expects a computing step followed by a proxy-only step"
    per_block = times[0] / ncomp[0]
    per_cand = 0.0
    for tr in traces:
        n = sum(1 for e in tr if e[0] == 0)
        per_cand += n * per_block if n else times[1]
    n_compute_steps = sum(1 for tr in traces if any(e[0] == 0 for e in tr))
    return {"value": 1.0 / per_cand, "unit": "candidates/s", "cores": int(cores), "kind": "oracle",
            "host_cpus": int(host_cpus), "cpu_model": cpu_model(),
            "sample": (f"candidate 0 of the pool: step 0 ({ncomp[0]} computed blocks) {times[0]:.1f} s and "
                       f"step 1 (proxies only) {times[1]:.2f} s, extrapolated over the draft's traces "
                       f"({n_compute_steps} computing + {len(traces) - n_compute_steps} proxy-only steps); "
                       f"text preparation {t1 - t0:.1f} s excluded; fp64 numpy, BLAS on {cores} threads")}


def describe_workload(wl, traces) -> str:
    """The workload in words, from its shape and the dispatch traces the run produced."""
    s = wl.shape
    skips = [sum(1 for e in tr if e[0] == 1) for tr in traces]
    comp = [sum(1 for e in tr if e[0] == 0) for tr in traces]
    proxy_steps = [k for k, tr in enumerate(traces) if any(e[0] == 2 for e in tr)]
    skip_txt = (f"{skips[0]} of {s.num_blocks} blocks skipped every step" if len(set(skips)) == 1
                else f"{min(skips)}..{max(skips)} of {s.num_blocks} blocks skipped per step")
    prompts = f"{wl.n_cond} prompts" if wl.n_cond > 1 else "1 prompt"
    return (f"{wl.name}: DiT of {s.num_blocks} blocks, D={s.hidden}, {s.heads} heads x {s.head_dim}, "
            f"MLP {s.mlp_hidden}; N={wl.n} candidates over {prompts}, {wl.tokens} image tokens "
            f"({wl.latent_h}x{wl.latent_w} latent, patch {s.patch}), {wl.text_len} text tokens x "
            f"{s.text_dim}; S'={wl.steps_draft} of {wl.steps_total} steps; {skip_txt}; proxies on steps "
            f"{proxy_steps}; {sum(comp)} block evaluations per candidate")


def secondary_draft(name, steps, warmup=1):
    """Draft throughput of another workload (its own short timed region): candidates/s, ms per draft,
    algorithmic TFLOP/s and the fraction of the bf16 peak."""
    import torch
    from paper_2607_04461_amd import synth
    from paper_2607_04461_amd.pool import DraftPool
    wl = synth.WORKLOADS[name]
    flat, _ = synth.make_weights(wl.shape, wl.seed_w, threads=16)
    pool = DraftPool(wl, dtype="bf16", weights=flat)
    del flat
    z0 = torch.from_numpy(synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)).cuda()

    def one_draft():
        pool.latents.copy_(z0)
        ctypes.memset(pool.meta, 0, ctypes.sizeof(pool.meta))
        return [pool.draft_step(k) for k in range(wl.steps_draft)]

    traces = one_draft()
    for _ in range(warmup - 1):
        one_draft()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        one_draft()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    pool.close()
    flops = draft_flops(wl, traces)
    tf = flops / (ms / 1e3) / 1e12
    return {"workload": describe_workload(wl, traces), "value": round(wl.n / (ms / 1e3), 3),
            "unit": "candidates/s", "ms_per_draft": round(ms, 2), "drafts_timed": steps,
            "algorithmic_tflop_per_draft": round(flops / 1e12, 2), "tflops": round(tf, 1),
            "mfma_frac": round(tf / PEAK_BF16_TFLOPS, 4)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="wan1.3b_pool16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-breakdown", action="store_true")
    ap.add_argument("--no-refine", action="store_true", help="skip timing the refinement")
    ap.add_argument("--no-sde", action="store_true", help="skip timing the stochastic-update kernel")
    ap.add_argument("--no-secondary", action="store_true", help="skip the 14B pool and the pool of 64")
    ap.add_argument("--calibration-copy", type=int, default=0, metavar="MIB",
                    help="also run a plain device copy of this many MiB three times (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the draft pool runs on a single MI355X and no multi-GPU path "
              "is built; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_04461_amd import flashbon as fb
    from paper_2607_04461_amd import synth
    from paper_2607_04461_amd.pool import DraftPool

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    fb.load()
    wl = synth.WORKLOADS[args.workload]
    t_gen = time.time()
    flat, W = synth.make_weights(wl.shape, wl.seed_w, threads=16)
    z0 = synth.make_latents(wl.n, wl.shape.latent_channels, wl.latent_h, wl.latent_w)
    text = synth.make_text(wl.n_cond, wl.text_len, wl.shape.text_dim)
    print(f"# inputs generated in {time.time() - t_gen:.1f} s", file=sys.stderr, flush=True)
    pool = DraftPool(wl, dtype="bf16", weights=flat)
    z0_dev = torch.from_numpy(z0).cuda()
    stream = torch.cuda.current_stream()

    def one_draft():
        pool.latents.copy_(z0_dev)
        ctypes.memset(pool.meta, 0, ctypes.sizeof(pool.meta))
        return [pool.draft_step(k) for k in range(wl.steps_draft)]

    # text preparation (once per prompt), timed on its own
    fb.flashbon_set_timing(pool.model, ["text"])
    pool.text_kv_valid.value = 0
    traces = one_draft()
    torch.cuda.synchronize()
    text_ms, _ = fb.flashbon_read_timing(pool.model, "text")
    fb.flashbon_set_timing(pool.model, [])
    for _ in range(max(0, args.warmup - 1)):
        one_draft()
    torch.cuda.synchronize()
    print(f"# warm-up done", file=sys.stderr, flush=True)

    # timed region: K whole drafts; the dominant kernel (the residual-epilogue GEMM at its three sites)
    # and the MLP up-projection are timed in place, per launch, on the library's stream
    res_sites = ["out", "out_cross", "mlp_down"]
    fb.flashbon_set_timing(pool.model, res_sites + ["mlp_up"])
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        one_draft()
    ev1.record(stream)
    torch.cuda.synchronize()
    total_ms = ev0.elapsed_time(ev1)
    site_t = {site: fb.flashbon_read_timing(pool.model, site) for site in res_sites + ["mlp_up"]}
    fb.flashbon_set_timing(pool.model, [])
    ms_per_step = total_ms / args.steps
    value = wl.n / (ms_per_step / 1e3)
    flops = draft_flops(wl, traces)
    tflops = flops / (ms_per_step / 1e3) / 1e12
    M, D, F = wl.n * wl.tokens, wl.shape.hidden, wl.shape.mlp_hidden
    site_flops = {"out": 2.0 * M * D * D, "out_cross": 2.0 * M * D * D, "mlp_down": 2.0 * M * D * F,
                  "mlp_up": 2.0 * M * F * D}
    res_ms = sum(site_t[x][0] for x in res_sites)
    res_n = sum(site_t[x][1] for x in res_sites)
    res_flops = sum(site_flops[x] * site_t[x][1] for x in res_sites)
    res_avg_ms = res_ms / max(res_n, 1)
    res_tflops = res_flops / (res_ms / 1e3) / 1e12
    res_plans = {x: fb.flashbon_op_linear_plan(fb.BF16, M, D, K, fb.EPI_RESIDUAL)
                 for x, K in (("out", D), ("mlp_down", F))}
    up_ms, up_n = site_t["mlp_up"]
    up_avg_ms = up_ms / max(up_n, 1)
    up_tflops = site_flops["mlp_up"] / (up_avg_ms / 1e3) / 1e12
    up_plan = fb.flashbon_op_linear_plan(fb.BF16, M, F, D, fb.EPI_GELU)
    print(f"# {args.steps} drafts in {total_ms:.1f} ms; residual GEMM {res_n} calls avg {res_avg_ms:.3f} ms; "
          f"mlp_up {up_n} calls avg {up_avg_ms:.3f} ms", file=sys.stderr, flush=True)

    breakdown = None
    if not args.no_breakdown:
        fb.flashbon_set_timing(pool.model, fb.SITES)
        one_draft()
        torch.cuda.synchronize()
        breakdown = {}
        for site in fb.SITES:
            ms, n = fb.flashbon_read_timing(pool.model, site)
            if n:
                breakdown[site] = {"ms": round(ms, 3), "launches": n}
        fb.flashbon_set_timing(pool.model, [])

    # selection (multi-stage Elo over a seeded synthetic verifier) and refinement of the winner
    refine_ms = selection = None
    if not args.no_refine:
        verifier = synth.SyntheticVerifier(wl.n, seed=7)
        one_draft()
        torch.cuda.synchronize()
        s0 = time.time()
        sel = pool.select(verifier.scores, verifier.judge)
        sel_ms = (time.time() - s0) * 1e3
        selection = {"winner": sel, "pairwise_calls": pool.last_selection[2],
                     "host_ms_incl_verifier": round(sel_ms, 3)}
        pool.refine(sel)                           # warm-up of the N = 1 shapes
        torch.cuda.synchronize()
        r0 = time.time()
        pool.refine(sel)
        torch.cuda.synchronize()
        refine_ms = round((time.time() - r0) * 1e3, 2)

    # C2: one full-quality step of one candidate at the pool's shape (every block computed), from the
    # refinement's steps, host launch overhead included
    c2 = None
    if refine_ms is not None:
        steps_r = wl.steps_total - wl.steps_draft
        c2_ms = refine_ms / steps_r
        c2_flops = block_flops(wl.shape, wl.tokens, wl.text_len) * wl.shape.num_blocks + \
            4.0 * wl.tokens * wl.shape.patch_dim * wl.shape.hidden
        c2_tf = c2_flops / (c2_ms / 1e3) / 1e12
        c2 = {"workload": f"one candidate of {wl.name}, all {wl.shape.num_blocks} blocks computed (N=1, "
                          f"{wl.tokens} tokens)", "ms_per_step": round(c2_ms, 3),
              "algorithmic_tflop_per_step": round(c2_flops / 1e12, 3), "tflops": round(c2_tf, 1),
              "mfma_frac": round(c2_tf / PEAK_BF16_TFLOPS, 4), "steps_timed": steps_r}

    # the stochastic update (App. A.1, Eq. 20) at the pool's latent shape: one fused unpatchify +
    # update launch; HBM-bound, algorithmic bytes = read z, read v, write z (12 bytes per element)
    sde = None
    if not args.no_sde:
        C, H, Wd, p = wl.shape.latent_channels, wl.latent_h, wl.latent_w, wl.shape.patch
        v_tok = torch.randn(M, C * p * p, device="cuda")
        z_sde = torch.randn(wl.n, C, H, Wd, device="cuda")
        args_sde = (wl.n, C, H, Wd, p, v_tok, z_sde, 0.8, 0.78, 0.3, 1234, 0)
        for _ in range(5):
            fb.flashbon_op_unpatch_sde(*args_sde)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(200):
            fb.flashbon_op_unpatch_sde(*args_sde)
        e1.record()
        torch.cuda.synchronize()
        sde_us = e0.elapsed_time(e1) / 200 * 1e3
        sde_bytes = 12.0 * z_sde.numel()
        sde = {"kernel": "k_head_update (Philox4x32-10 + Box-Muller normals, unpatchify, Eq. 20 update)",
               "elements": z_sde.numel(), "avg_launch_us": round(sde_us, 2), "bound": "hbm",
               "achieved_GBs": round(sde_bytes / sde_us / 1e3, 1), "peak_GBs": PEAK_HBM_GBS,
               "frac": round(sde_bytes / sde_us / 1e3 / PEAK_HBM_GBS, 4)}
        del v_tok, z_sde

    if args.calibration_copy:
        n = args.calibration_copy * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    result = {
        "metric": ("draft candidates/sec (1.3B-shaped DiT, N=16) + % bf16 MFMA peak" if wl.name == "wan1.3b_pool16"
                   else f"draft candidates/sec ({wl.name}) + % bf16 MFMA peak"),
        "value": round(value, 3),
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) latents and text, N(0,0.02^2) random-init weights)",
        "config": {
            "workload": describe_workload(wl, traces),
            "global_batch": wl.n, "seq_len": wl.tokens, "parallelism": "none (1 GPU)",
        },
        "tflops_end_to_end": round(tflops, 2),
        "mfma_frac_end_to_end": round(tflops / PEAK_BF16_TFLOPS, 4),
        "algorithmic_tflop_per_step": round(flops / 1e12, 3),
        "roofline": {
            "kernel": ("residual-epilogue GEMM k_linear_dma8<EPI_RESIDUAL> (gate, residual, cache store) at "
                       "its three sites per computed block: self-attention and cross-attention output "
                       "projections (M=%d N=%d K=%d: %s) and MLP down-projection (K=%d: %s); FLOPs and time "
                       "summed over every launch of those sites, timed per call"
                       % (M, D, D, res_plans["out"][1], F, res_plans["mlp_down"][1])),
            "bound": "mfma", "achieved": round(res_tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": round(res_tflops / PEAK_BF16_TFLOPS, 4), "traffic": recorded_traffic("linear_residual_traffic.md"),
            "traffic_unit": "bytes per launch, averaged over the three sites' launches (FETCH_SIZE + "
                            "WRITE_SIZE, copy-calibrated)",
            "avg_launch_ms": round(res_avg_ms, 4), "launches": res_n,
            "algorithmic_gflop_per_launch": round(res_flops / max(res_n, 1) / 1e9, 2),
            "sites": {x: {"launches": site_t[x][1], "avg_ms": round(site_t[x][0] / max(site_t[x][1], 1), 4),
                          "tflops": round(site_flops[x] * site_t[x][1] / (site_t[x][0] / 1e3) / 1e12, 1)}
                      for x in res_sites},
        },
        "roofline_secondary": {
            "kernel": ("MLP up-projection + GELU (M=%d N=%d K=%d): %s, EPI_GELU; timed per call"
                       % (M, F, D, up_plan[1])),
            "bound": "mfma", "achieved": round(up_tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": round(up_tflops / PEAK_BF16_TFLOPS, 4), "traffic": recorded_traffic("linear_mlp_up_traffic.md"),
            "traffic_unit": "bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
            "avg_launch_ms": round(up_avg_ms, 4), "launches": up_n, "kernels_per_launch": up_plan[0],
        },
        "text_prep_ms": round(text_ms, 3),
        "selection": selection,
        "sde_update": sde,
        "refine_ms": refine_ms,
        "refine_steps": wl.steps_total - wl.steps_draft,
        "c2_full_step": c2,
        "site_breakdown_one_draft": breakdown,
        "site_rooflines_one_draft": site_rooflines(wl, traces, breakdown) if breakdown else None,
    }
    pool.close()
    del pool
    if not args.no_secondary:
        result["secondary_workloads"] = {}
        for name, k in (("wan1.3b_pool64", 3), ("wan14b_pool4", 3)):
            print(f"# secondary workload {name}", file=sys.stderr, flush=True)
            result["secondary_workloads"][name] = secondary_draft(name, k)
            torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle sample", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(wl, W, z0, text, traces)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
