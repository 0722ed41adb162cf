#!/usr/bin/env python3
"""Benchmark of the HSA forward pass on one MI355X.

A step is one pass of the whole path over one chunk of synthetic input with
everything resident in HBM: hsa_state_update over every page of the layer
(cold build of the linear state and page index), hsa_page_select (query
summary, page scores, top-k_h) and hsa_forward_selected (sparse branch,
linear branch, gated merge) -- the two halves of hsa_forward, the same
kernels, called apart so that an event between them times the attention
launch inside every timed step.
Default workload (``--config c3``): one layer, 12 heads x d128, 4680
queries, 120 history pages of 1560 tokens (187,200 keys) plus the 3 current
pages, head-adaptive budgets k_h drawn from {2, 4, 8, 16}. The other
workloads (single layer c2, prompt switch c4, streaming 30 layers c5) are
reported as sub-objects (``--sub``).

Every step and every phase is timed with its own HIP event pair on the
stream the library launches on; ``value`` is the median step time over
``--steps`` steps after ``--warmup`` untimed ones, with p10/p90 beside it.

Prints one JSON line. ``value`` is milliseconds per chunk (lower is better);
the line also carries effective TFLOP/s, per-phase times, the roofline of the
dominant kernel (the attention launch, timed inside the steps) and the fp64
oracle timed on this host's cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def attn_flops(wl, k_eff, n_q):
    d, P = wl.head_dim, wl.page_size
    return sum(4.0 * n_q * (k + wl.n_cur) * P * d for k in k_eff) * wl.batch


def linear_flops(wl, n_q):
    return 2.0 * n_q * wl.head_dim ** 2 * wl.heads * wl.batch


def state_flops_bytes(wl, n_pages):
    keys = n_pages * wl.page_size * wl.heads * wl.batch
    esize = 2 if wl.dtype == "bf16" else 4
    return 2.0 * keys * wl.head_dim ** 2, keys * 2 * wl.head_dim * esize


def time_loop(fn, iters, torch):
    """Mean ms of fn over iters back-to-back calls (one event pair around all
    of them, on torch's current stream, where the library launches)."""
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(iters):
        fn()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / iters


def time_each(fn, iters, torch, keep=False):
    """Per-call ms of fn: one event pair around each call, on torch's current
    stream (the stream the library launches on). Returns the sorted times
    (and, with keep, the event pairs in call order)."""
    import numpy as np
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(iters)]
    torch.cuda.synchronize()
    for a, b in evs:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    t = np.sort(np.array([a.elapsed_time(b) for a, b in evs]))
    return (t, evs) if keep else t


def time_med(fn, iters, torch):
    """Median per-call ms of fn (time_each)."""
    return float(np.median(time_each(fn, iters, torch)))


def stats(t):
    """median / p10 / p90 / mean of per-call times (ms)."""
    import numpy as np
    return {"median": round(float(np.median(t)), 4), "p10": round(float(np.percentile(t, 10)), 4),
            "p90": round(float(np.percentile(t, 90)), 4), "mean": round(float(np.mean(t)), 4),
            "n": int(len(t))}


def kernel_source_hash() -> str:
    """Hash of the attention kernel sources; HBM traffic figures measured with
    rocprofv3 counters apply only to the sources they were measured on."""
    import hashlib
    h = hashlib.sha256()
    for f in ("hsa_attn.hip", "hsa_device.h"):
        with open(os.path.join(ROOT, "paper_2609_34606_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, key: str = "hbm_bytes_per_launch"):
    """HBM bytes per attention launch (page-level kernel; key
    hbm_bytes_per_launch_tile_list: the block-sparse one) from the committed
    counter summary of this workload, if it was taken on the current kernel
    sources, else None."""
    v = profile_value(f"attn_{workload}_hbm_traffic.txt", key)
    return None if v is None else int(v) or None


def measured_mfma_busy(workload: str):
    """Fraction of the SIMD cycles of the page walk's launch in which the MFMA
    pipe is busy (rocprofv3 SQ_VALU_MFMA_BUSY_CYCLES over 1024 SIMDs x the
    launch's shader cycles), from the committed counter summary of this
    workload, if it was taken on the current kernel sources, else None."""
    return profile_value(f"attn_pp_kernel_{workload}_counters.txt", "mfma_busy_fraction")


def measured_shader_clock(workload: str):
    """Shader clock (GHz) of the page walk's launch: its per-shader-engine
    busy cycles (rocprofv3 SQ_BUSY_CYCLES / 32) over each dispatch's duration
    from the kernel trace of the same run, from the committed counter
    summary of this workload, if it was taken on the current kernel sources,
    else None."""
    return profile_value(f"attn_pp_kernel_{workload}_counters.txt", "shader_clock_ghz")


def profile_value(name: str, key: str):
    """A key: value figure of a committed summary under profiles/, if the
    summary was taken on the current kernel sources, else None."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    try:
        return float(kv[key])
    except (KeyError, ValueError):
        return None


def host_cpu():
    """(logical CPUs, CPU model) of this host."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return os.cpu_count(), model


def cpu_baseline(wl, dev, k_h, heads):
    """The fp64 oracle on this host's cores over a bounded sample of heads."""
    from oracle import hsa_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    nproc, model = host_cpu()
    host = dict(q=dev["q"].float().cpu().numpy(), k_pool=dev["k_pool"].float().cpu().numpy(),
                v_pool=dev["v_pool"].float().cpu().numpy(),
                page_table=dev["page_table"].cpu().numpy())
    t0 = time.perf_counter()
    O.hsa_forward(host["q"], host["k_pool"], host["v_pool"], host["page_table"], wl.n_cand,
                  wl.n_cur, list(k_h), heads=heads)
    dt = time.perf_counter() - t0
    scale = wl.heads / len(heads)
    return {"value": round(dt * scale * 1e3, 1), "unit": "ms/chunk", "cores": int(threads),
            "kind": "oracle", "nproc": nproc, "cpu_model": model,
            "threads_note": "cores = BLAS threads the numpy oracle ran with (its matrix products "
                            "are the multi-threaded part; the rest is one Python thread)",
            "sample": f"{len(heads)} of {wl.heads} heads of one {wl.name} chunk (all queries, "
                      f"cold state), {dt:.1f} s, scaled x{scale:g} to the chunk"}


def bench_core(args, wl, dev=None):
    """One workload: the step (cold fold, page selection, attention) timed
    per step and per part, the parts again back to back, and the attention
    launch with its roofline. Returns (result, layer, inputs, selection)."""
    import torch
    from paper_2609_34606_amd import HsaLayer, hsa_page_select
    from synth_inputs import make_case_torch

    if dev is None:
        dev = make_case_torch(wl, "cuda:0")
    torch.cuda.synchronize()
    q, k_h = dev["q"], [int(x) for x in dev["k_h"]]
    k_max = max(1, max(k_h))
    n_q, n_pages = wl.n_q, wl.n_pages
    layer = HsaLayer(wl.batch, wl.heads, wl.head_dim, wl.page_size, q.dtype, q.device,
                     k_pool=dev["k_pool"], v_pool=dev["v_pool"], page_table=dev["page_table"])
    out = torch.empty_like(q)
    sel = torch.empty((wl.batch, wl.heads, k_max), dtype=torch.int32, device=q.device)

    # events between the fold, the page selection and the attention launch of
    # each step, so that the step's parts are timed where they run (the fold
    # right after the previous step's attention launch, the attention right
    # after the selection)
    mids = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(args.steps)]
    k_step = [0]
    ws = layer.workspace("sel", 1 << 24)

    def select():
        hsa_page_select(layer.cfg, q, n_q, layer.page_kmean, layer.max_pages, wl.n_cand, k_h, k_max,
                        sel, ws=ws)

    def attend():
        layer.forward_selected(q, sel, wl.n_cand, wl.n_cur, k_h, k_max=k_max, out=out)

    def step(mark=False):
        layer.fold(0, n_pages)
        if mark:
            mids[k_step[0]][0].record()
        select()
        if mark:
            mids[k_step[0]][1].record()
            k_step[0] += 1
        attend()

    for _ in range(args.warmup):
        step()
    # the timed region: exactly `steps` steps between two synchronisations,
    # each step bracketed by its own event pair
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    t_step, step_evs = time_each(lambda: step(True), args.steps, torch, keep=True)
    wall_ms = (time.perf_counter() - t0) * 1e3
    # warm steps: the state carried, only the current pages folded (as a
    # streaming chunk does), then the same selection and attention
    def warm_step():
        layer.fold(wl.n_cand, wl.n_cur)
        select()
        attend()

    for _ in range(2):
        warm_step()
    t_warm_step = time_each(warm_step, args.steps, torch)
    t_fold_in = np.array([a.elapsed_time(m1) for (a, _), (m1, _) in zip(step_evs, mids)])
    t_sel_in = np.array([m1.elapsed_time(m2) for (m1, m2) in mids])
    t_attn_in = np.array([m2.elapsed_time(b) for (_, b), (_, m2) in zip(step_evs, mids)])
    log(f"{wl.name}: step median {np.median(t_step):.4f} ms")
    n = args.steps
    # each part again, back to back (other cache and clock conditions than in
    # the step: the attention re-reads the pages it has just read)
    t_state = time_each(lambda: layer.fold(0, n_pages), n, torch)
    t_warm = time_each(lambda: layer.fold(wl.n_cand, wl.n_cur), n, torch)
    t_sel = time_each(select, n, torch)
    t_fwd = time_each(lambda: layer.forward(q, wl.n_cand, wl.n_cur, k_h, k_max=k_max, out=out),
                      n, torch)
    t_attn = time_each(attend, n, torch)
    k_eff = [min(k, wl.n_cand) for k in k_h]
    fa = attn_flops(wl, k_eff, n_q)
    fl = linear_flops(wl, n_q)
    fs, bs = state_flops_bytes(wl, n_pages)
    total = fa + fl + fs
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    ms = float(np.median(t_step))
    ms_attn_mean = float(np.mean(t_attn_in))
    achieved = fa / (ms_attn_mean * 1e-3) / 1e12
    ms_state = float(np.median(t_state))
    res = {
        "value": round(ms, 4), "unit": "ms/chunk", "ms_per_step": round(ms, 4),
        "step_ms": stats(t_step), "timed_region_wall_ms": round(wall_ms, 3),
        "effective_tflops": round(total / (ms * 1e-3) / 1e12, 2),
        "mfma_util_attention": round(achieved / peak, 4),
        "config": {"workload": wl.name, "batch": wl.batch, "heads": wl.heads,
                   "head_dim": wl.head_dim, "n_q": n_q, "page_size": wl.page_size,
                   "history_pages": wl.n_cand, "current_pages": wl.n_cur, "k_h": k_h,
                   "state": "cold (all pages folded every step)", "parallelism": "single GPU"},
        "warm_step_ms": dict(stats(t_warm_step), note="state carried: only the current pages "
                                                       "folded, then selection and attention"),
        "step_parts_ms": {"state_update_cold": stats(t_fold_in), "page_select": stats(t_sel_in),
                          "attention_launch": stats(t_attn_in),
                          "note": "the three parts of the timed steps (events between them); "
                                  "phases_ms times each part alone, back to back"},
        "phases_ms": {"state_update_cold": stats(t_state),
                      "state_update_warm_current_pages": stats(t_warm),
                      "page_select": stats(t_sel), "forward": stats(t_fwd),
                      "attention_launch": stats(t_attn)},
        "state_update_hbm_gbs": round(bs / (ms_state * 1e-3) / 1e9, 1),
        "state_update_hbm_frac": round(bs / (ms_state * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "state_update_in_step_hbm_frac": round(bs / (float(np.median(t_fold_in)) * 1e-3) / 1e9
                                               / PEAK_HBM_GBS, 4),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                     "traffic": measured_traffic(wl.name),
                     "kernel": "attention launch (hsa_forward_selected) inside the timed steps "
                               "(mean of per-step HIP event times)",
                     "flops_per_launch": fa,
                     "frac_at_median_launch": round(fa / (float(np.median(t_attn_in)) * 1e-3) / 1e12 / peak, 4),
                     "frac_back_to_back": round(fa / (float(np.mean(t_attn)) * 1e-3) / 1e12 / peak, 4),
                     "mfma_busy_frac_counters": measured_mfma_busy(wl.name),
                     "shader_clock_ghz_counters": measured_shader_clock(wl.name),
                     "mfma_busy_note": "share of SIMD cycles with the MFMA pipe busy (rocprof counters, "
                                       "committed summary); frac above is against the nominal peak, "
                                       "which assumes the 2.4 GHz clock"},
    }
    return res, layer, dev, sel


def bench_single(args, wl):
    import torch
    res, layer, dev, sel = bench_core(args, wl)
    q, k_h = dev["q"], [int(x) for x in dev["k_h"]]
    k_max = max(1, max(k_h))
    line = {
        "metric": "HSA ms/chunk + effective TFLOP/s (MFMA util %) at 12 heads x d128, 4680 queries",
        "value": res["value"], "unit": "ms/chunk", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": res["ms_per_step"], "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
    }
    line.update({k: v for k, v in res.items() if k not in line})
    if not args.no_adaptive:
        line["adaptive"] = bench_adaptive(args, wl, layer, q, k_h, k_max, sel)
        if wl.dtype == "bf16":
            line["linformer"] = bench_linformer(args, wl, layer, q, k_h, k_max, sel)
            line["retrieval"] = bench_retrieval(args, wl, layer, q, k_h, k_max)
            line["tier"] = bench_tier(args, wl, dev, layer, q, k_h, k_max, sel)
    if not args.no_cpu_baseline:
        # every head up to the c3 history (about 10 s of oracle work on 16
        # threads), two heads of longer ones
        heads = list(range(wl.heads)) if wl.heads * wl.n_pages <= 12 * 130 else [0, 1]
        log("timing the oracle on the host ...")
        line["cpu_baseline"] = cpu_baseline(wl, dev, k_h, heads)
    del layer, dev, sel
    torch.cuda.empty_cache()
    return line


def kept_work(wl, sel_row, kept, n_kept, n_q):
    """Algorithmic attention flops of one head's kept blocks, and the 64-key
    tiles its 128-query tiles walk (union of the kept sets of their two query
    blocks) against the tiles all query blocks of the tile keep."""
    import numpy as np
    P, d = wl.page_size, wl.head_dim
    n_sel = int((sel_row >= 0).sum())
    nbh, nbc = -(-P // 128), -(-P // 64)

    def keys_tiles(j):
        if j < n_sel * nbh:
            k0 = (j % nbh) * 128
            nk = min(128, P - k0)
        else:
            k0 = ((j - n_sel * nbh) % nbc) * 64
            nk = min(64, P - k0)
        return nk, -(-nk // 64)

    flops, walked, kept_tiles = 0.0, 0, 0
    n_qb = len(n_kept)
    for i in range(n_qb):
        rows = min(64, n_q - 64 * i)
        for j in kept[i, :n_kept[i]]:
            nk, nt = keys_tiles(int(j))
            flops += 4.0 * rows * nk * d
            kept_tiles += nt
    for t in range(-(-n_qb // 2)):
        u = set(kept[2 * t, :n_kept[2 * t]].tolist())
        if 2 * t + 1 < n_qb:
            u |= set(kept[2 * t + 1, :n_kept[2 * t + 1]].tolist())
        walked += 2 * sum(keys_tiles(j)[1] for j in u)   # two query blocks per walk
    return flops, walked, kept_tiles


def bench_adaptive(args, wl, layer, q, k_h, k_max, sel):
    """The head-adaptive block-sparse path on the same layer and chunk: step
    (cold fold + hsa_forward_adaptive), the block selection alone, and the
    sparse branch alone; its attention launch is the sparse-branch call minus
    the selection it runs first."""
    import numpy as np
    import torch
    from paper_2609_34606_amd import (TAU_MAX, TAU_MIN, hsa_adaptive_workspace_size,
                                      hsa_block_count, hsa_block_select, hsa_sparse_attn_adaptive)
    n_q, n_pages = wl.n_q, wl.n_pages
    out = torch.empty_like(q)

    def step():
        layer.fold(0, n_pages)
        layer.forward_adaptive(q, wl.n_cand, wl.n_cur, k_h, k_max=k_max, out=out)

    for _ in range(args.warmup):
        step()
    ms = time_med(step, args.steps, torch)
    ms_fwd = time_med(lambda: layer.forward_adaptive(q, wl.n_cand, wl.n_cur, k_h, k_max=k_max,
                                                      out=out, sel_out=sel), args.steps, torch)
    ws = layer.workspace("adaptive_parts", hsa_adaptive_workspace_size(layer.cfg, n_q, k_max,
                                                                       wl.n_cur))
    ms_bsel = time_med(lambda: hsa_block_select(layer.cfg, q, n_q, layer.pool, sel, k_max,
                                                 wl.n_cand, wl.n_cur, ws=ws), args.steps, torch)
    o_sp = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    ms_sp = time_med(lambda: hsa_sparse_attn_adaptive(layer.cfg, q, n_q, layer.pool, sel, k_max,
                                                       k_h, wl.n_cand, wl.n_cur, o_sp, ws=ws),
                      args.steps, torch)
    # kept sets of this chunk (untimed) for the algorithmic flops
    n_qb = -(-n_q // 64)
    nb = hsa_block_count(layer.cfg, k_max, wl.n_cur)
    n_kept = torch.zeros((wl.batch, wl.heads, n_qb), dtype=torch.int32, device=q.device)
    kept = torch.zeros((wl.batch, wl.heads, n_qb, nb), dtype=torch.int32, device=q.device)
    gini = torch.zeros((wl.batch, wl.heads), dtype=torch.float64, device=q.device)
    hsa_block_select(layer.cfg, q, n_q, layer.pool, sel, k_max, wl.n_cand, wl.n_cur, gini=gini,
                     n_kept=n_kept, kept=kept, kept_len=nb, ws=ws)
    torch.cuda.synchronize()
    sel_h, nk_h, kp_h = sel.cpu().numpy(), n_kept.cpu().numpy(), kept.cpu().numpy()
    fa, walked, kept_tiles, frac = 0.0, 0, 0, []
    for b in range(wl.batch):
        for h in range(wl.heads):
            f, w_, k_ = kept_work(wl, sel_h[b, h], kp_h[b, h], nk_h[b, h], n_q)
            fa, walked, kept_tiles = fa + f, walked + w_, kept_tiles + k_
            n_blk = hsa_block_count(layer.cfg, int((sel_h[b, h] >= 0).sum()), wl.n_cur)
            frac.append(float(nk_h[b, h].mean()) / n_blk)
    ms_attn = ms_sp - ms_bsel
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    achieved = fa / (ms_attn * 1e-3) / 1e12
    return {
        "tau_min": TAU_MIN, "tau_max": TAU_MAX, "ms_per_step": round(ms, 4),
        "phases_ms": {"forward_adaptive": round(ms_fwd, 4), "block_select": round(ms_bsel, 4),
                      "sparse_attn_adaptive": round(ms_sp, 4),
                      "attention_launch": round(ms_attn, 4)},
        "kept_block_fraction": round(float(np.mean(frac)), 4),
        "gini_mean": round(float(gini.cpu().numpy().mean()), 5),
        "walked_over_kept_tiles": round(walked / max(1, kept_tiles), 3),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4),
                     "traffic": measured_traffic(wl.name, "hbm_bytes_per_launch_tile_list"),
                     "kernel": "attn_bf16_kernel, tile-list mode (sparse-branch launch)",
                     "flops_per_launch": fa,
                     "mfma_busy_frac_counters": profile_value(
                         f"attn_bf16_kernel_tile_list_{wl.name}_counters.txt", "mfma_busy_fraction"),
                     "shader_clock_ghz_counters": profile_value(
                         f"attn_bf16_kernel_tile_list_{wl.name}_counters.txt", "shader_clock_ghz")},
    }


def bench_linformer(args, wl, layer, q, k_h, k_max, sel, rank=64):
    """The paper's two branches on the same layer and chunk: page selection,
    head-adaptive block-sparse sparse branch and the Linformer linear branch
    over the compressed pages (rank 64, seeded projections). The step is the
    cold page index (hsa_state_update) + the compression of every page +
    hsa_forward_linformer; the branch launch is the attention over the
    compressed pool for the step's selection."""
    import torch
    from paper_2609_34606_amd import config as mkcfg
    from paper_2609_34606_amd import hsa_sparse_attn, hsa_sparse_attn_workspace_size, kv_pool
    from synth_inputs import make_projections
    n_q, n_pages = wl.n_q, wl.n_pages
    e_k, e_v = make_projections(wl, rank)
    to = lambda a: torch.from_numpy(a).to(q.device).to(q.dtype)
    layer.set_projections(to(e_k), to(e_v))
    out = torch.empty_like(q)

    def step():
        layer.fold(0, n_pages)
        layer.compress(0, n_pages)
        layer.forward_linformer(q, wl.n_cand, wl.n_cur, k_h, k_max=k_max, out=out)

    for _ in range(args.warmup):
        step()
    ms = time_med(step, args.steps, torch)
    ms_cold = time_med(lambda: layer.compress(0, n_pages), args.steps, torch)
    ms_warm = time_med(lambda: layer.compress(wl.n_cand, wl.n_cur), args.steps, torch)
    ms_fwd = time_med(lambda: layer.forward_linformer(q, wl.n_cand, wl.n_cur, k_h, k_max=k_max,
                                                       out=out, sel_out=sel), args.steps, torch)
    crank = mkcfg(wl.batch, wl.heads, wl.head_dim, rank, q.dtype)
    cpool = kv_pool(layer.ck, layer.cv, layer.page_table, crank)
    o_lin = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    ws = layer.workspace("lin_attn", hsa_sparse_attn_workspace_size(crank, n_q, k_max, wl.n_cur))
    ms_br = time_med(lambda: hsa_sparse_attn(crank, q, n_q, cpool, sel, k_max, k_h, wl.n_cand,
                                              wl.n_cur, o_lin, ws=ws), args.steps, torch)
    k_eff = [min(k, wl.n_cand) for k in k_h]
    fb = sum(4.0 * n_q * (k + wl.n_cur) * rank * wl.head_dim for k in k_eff) * wl.batch
    esz = 2
    cbytes = n_pages * wl.heads * wl.batch * (2 * wl.page_size * wl.head_dim * esz +
                                             2 * rank * wl.head_dim * esz)
    peak = PEAK_BF16_TFLOPS
    return {
        "rank": rank, "projections": "seeded N(0, 1/P)", "ms_per_step": round(ms, 4),
        "phases_ms": {"compress_cold_all_pages": round(ms_cold, 4),
                      "compress_current_pages": round(ms_warm, 4),
                      "forward_linformer": round(ms_fwd, 4),
                      "linformer_branch_launch": round(ms_br, 4)},
        "compress_hbm_gbs": round(cbytes / (ms_cold * 1e-3) / 1e9, 1),
        "compress_hbm_frac": round(cbytes / (ms_cold * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "branch_roofline": {"bound": "mfma", "achieved": round(fb / (ms_br * 1e-3) / 1e12, 2),
                            "peak": peak, "unit": "TFLOP/s",
                            "frac": round(fb / (ms_br * 1e-3) / 1e12 / peak, 4),
                            "flops_per_launch": fb},
    }


def bench_retrieval(args, wl, layer, q, k_h, k_max):
    """Stage-1 prompt-level retrieval (cosine top-1 over the chunks' prompt
    embeddings, 4096-dim) alone and in front of the forward pass."""
    import torch
    from paper_2609_34606_amd import hsa_chunk_select, hsa_forward_retrieval
    from paper_2609_34606_amd import hsa_retrieval_workspace_size
    from synth_inputs import make_prompts
    pe, ce, cf = make_prompts(wl)
    t = lambda a: torch.from_numpy(a).to(q.device)
    pe, ce, cf = t(pe), t(ce), t(cf)
    M, E = ce.shape[1], ce.shape[2]
    rng = torch.empty((wl.batch, 2), dtype=torch.int32, device=q.device)
    ms_s1 = time_med(lambda: hsa_chunk_select(layer.cfg, pe, ce, E, M, cf, wl.n_cand, rng),
                      args.steps, torch)
    out = torch.empty_like(q)
    ws = layer.workspace("retrieval", hsa_retrieval_workspace_size(layer.cfg, wl.n_q, k_max, wl.n_cur))
    ms_fwd = time_med(lambda: hsa_forward_retrieval(
        layer.cfg, q, wl.n_q, layer.pool, pe, ce, E, M, cf, wl.n_cand, wl.n_cur, k_h, k_max,
        layer.kv_state, layer.k_state, layer.page_kmean, None, None, out, ws=ws), args.steps, torch)
    return {"chunks": M, "emb_dim": E, "pages_per_chunk": int(cf[0, 1] - cf[0, 0]),
            "phases_ms": {"stage1_chunk_select": round(ms_s1, 4),
                          "forward_retrieval": round(ms_fwd, 4)}}


def bench_tier(args, wl, dev, main_layer, q, k_h, k_max, sel, n_slots=8, n_set=6):
    """Host-managed tiers on a second pool of n_slots slots over the
    workload's pages (the rest in pinned host memory, or two host slots and a
    file under the system's temporary directory). Each timed fetch brings
    n_set pages back into the pool and moves as many out, alternating two
    disjoint sets. Reports the pages moved per fetch, the time and the
    host<->device rate; and, for the prefetch, the time of a prefetch of
    n_set pages on a side stream alone, of the main layer's attention
    launches alone, and of the two issued together (the overlap of copies
    with compute, as when one layer's pages move while another computes)."""
    import tempfile

    import numpy as np
    import torch
    from paper_2609_34606_amd import HsaLayer, HsaTier
    H, d, P = wl.heads, wl.head_dim, wl.page_size
    npg = min(wl.n_pages, 2 * n_set + n_slots)
    dt = dev["q"].dtype
    cuda = dev["q"].device
    page_bytes = 2 * H * P * d * (2 if wl.dtype == "bf16" else 4)
    pool_k = torch.empty((n_slots, H, P, d), dtype=dt, device=cuda)
    pool_v = torch.empty((n_slots, H, d, P), dtype=dt, device=cuda)
    table = torch.full((wl.batch, npg), -1, dtype=torch.int32, device=cuda)
    layer = HsaLayer(wl.batch, H, d, P, dt, cuda, k_pool=pool_k, v_pool=pool_v, page_table=table)
    sets = [np.arange(0, n_set, dtype=np.int32)[None], np.arange(n_set, 2 * n_set, dtype=np.int32)[None]]
    iters = max(10, args.steps)

    def make(l2, l3, tmp, backup=False):
        host_k = torch.empty((max(l2, 1), H, P, d), dtype=dt, pin_memory=True)
        host_v = torch.empty((max(l2, 1), H, d, P), dtype=dt, pin_memory=True)
        tier = HsaTier(layer.cfg, layer.pool, l2, host_k, host_v, l3_dir=tmp if l3 else None,
                       l3_slots=l3, backup=backup)
        t_commit = 0.0
        for p in range(npg):
            slot = tier.place(0, p)
            pool_k[slot] = dev["k_pool"][int(dev["page_table"][0, p])]
            pool_v[slot] = dev["v_pool"][int(dev["page_table"][0, p])]
            if backup:
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                tier.commit()
                t_commit += time.perf_counter() - t0
        tier.fetch(sets[1])
        torch.cuda.synchronize()
        tier.commit_s = t_commit
        return tier, (host_k, host_v)

    def cycle(tier):
        s0 = tier.stats()
        t0 = time.perf_counter()
        for i in range(iters):
            tier.fetch(sets[i % 2])
            torch.cuda.synchronize()
        dt_s = (time.perf_counter() - t0) / iters
        s1 = tier.stats()
        moved = {k: (s1[k] - s0[k]) / iters for k in s1}
        per = moved["evictions"] + moved["fetches"]
        return {"pages_moved_per_fetch": per, "pages_to_file_per_fetch": moved["spills"],
                "pages_from_file_per_fetch": moved["reloads"],
                "file_writes_per_fetch": moved["backups"], "ms_per_fetch": round(dt_s * 1e3, 3),
                "host_device_gbs": round(per * page_bytes / dt_s / 1e9, 1)}

    res = {"pool_slots": n_slots, "pages": npg, "pages_per_fetch": n_set,
           "page_bytes": page_bytes,
           "note": "a page moved is one key block and one value block of every head; a fetch "
                   "moves pages with one swap kernel per page (pool slot <-> pinned host "
                   "memory, both directions at once), a prefetch with DMA copies"}
    # the link itself: one pinned copy of n_set pages' bytes each way
    hbuf = torch.empty(n_set * page_bytes, dtype=torch.uint8, pin_memory=True)
    dbuf = torch.empty(n_set * page_bytes, dtype=torch.uint8, device=cuda)
    ms_h2d = time_loop(lambda: dbuf.copy_(hbuf, non_blocking=True), iters, torch)
    ms_d2h = time_loop(lambda: hbuf.copy_(dbuf, non_blocking=True), iters, torch)
    # both directions at once, each on its own stream
    hbuf2 = torch.empty(n_set * page_bytes, dtype=torch.uint8, pin_memory=True)
    dbuf2 = torch.empty_like(dbuf)
    s_out = torch.cuda.Stream()

    def both():
        s_out.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s_out):
            hbuf2.copy_(dbuf2, non_blocking=True)
        dbuf.copy_(hbuf, non_blocking=True)
        torch.cuda.current_stream().wait_stream(s_out)

    ms_both = time_loop(both, iters, torch)
    res["link_gbs"] = {"h2d": round(n_set * page_bytes / ms_h2d / 1e6, 1),
                       "d2h": round(n_set * page_bytes / ms_d2h / 1e6, 1),
                       "both_directions": round(2 * n_set * page_bytes / ms_both / 1e6, 1)}
    del hbuf, dbuf, hbuf2, dbuf2
    with tempfile.TemporaryDirectory() as tmp:
        tier, keep = make(npg - n_slots + 1, 0, tmp)
        res["host_tier"] = dict(host_slots=npg - n_slots + 1, **cycle(tier))
        # prefetch beside the attention: forwards on the compute stream, the
        # prefetch of the other set on a side stream (an empty fetch first, so
        # that no page is held)
        side = torch.cuda.Stream()
        n_fwd = 6
        out = torch.empty_like(q)

        def forwards():
            for _ in range(n_fwd):
                main_layer.forward_selected(q, sel, wl.n_cand, wl.n_cur, k_h, k_max=k_max, out=out)

        def timed(fn):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for i in range(iters):
                fn(i)
                torch.cuda.synchronize()
            return (time.perf_counter() - t0) / iters * 1e3

        empty = np.zeros((1, 0), np.int32)
        ms_f = timed(lambda i: forwards())
        ms_p = timed(lambda i: (tier.fetch(empty), tier.prefetch(sets[i % 2], stream=side)))
        ms_b = timed(lambda i: (tier.fetch(empty), forwards(), tier.prefetch(sets[i % 2], stream=side)))
        res["prefetch_overlap"] = {
            "attention_launches": n_fwd, "ms_attention": round(ms_f, 3),
            "ms_prefetch": round(ms_p, 3), "ms_together": round(ms_b, 3),
            "together_over_longer": round(ms_b / max(ms_f, ms_p), 3),
            "together_over_sum": round(ms_b / (ms_f + ms_p), 3)}
        tier.close()
        del keep
        n_l2 = 2
        tier, keep = make(n_l2, npg - n_slots - n_l2 + 1, tmp)
        res["file_tier"] = dict(host_slots=n_l2, file_slots=npg - n_slots - n_l2 + 1,
                                file_dir=tmp.rsplit("/", 1)[0], **cycle(tier))
        tier.close()
        del keep
        # backup mode: every page written to its own file slot by a commit
        # right after it is placed; pages leaving the host tier then cost no
        # file write
        tier, keep = make(n_l2, npg, tmp, backup=True)
        st = tier.stats()
        res["file_backup_tier"] = dict(
            host_slots=n_l2, file_slots=npg, pages_written=st["backups"],
            commit_gbs=round(st["backups"] * page_bytes / tier.commit_s / 1e9, 2),
            **cycle(tier))
        tier.close()
    return res


def bench_streaming(args, wl):
    """30 independent layers x 60 chunks. Per chunk each layer folds its 3 new
    pages into its linear state and page index and runs HSA over its grown
    history. Two launch modes over the same pool and inputs:

    * sequential layers (the reported value): one hsa_state_update and one
      hsa_forward per layer, as a model whose layers run one after another;
    * batched layers: the 30 layers as the 30 batch entries of one
      hsa_state_update and one hsa_forward per chunk (each layer's pages are
      its own page-table row), as when the layers' inputs are all ready.
    """
    import numpy as np
    import torch
    from paper_2609_34606_amd import HsaLayer
    from synth_inputs import make_case_torch
    from synth_inputs.configs import streaming_chunk

    L = args.layers or wl.layers
    T = args.chunks or wl.chunks
    npg = wl.n_cur * T
    H, d, P = wl.heads, wl.head_dim, wl.page_size
    k_pool = torch.empty((L * npg, H, P, d), dtype=torch.bfloat16, device="cuda:0")
    v_pool = torch.empty((L * npg, H, d, P), dtype=torch.bfloat16, device="cuda:0")
    table = torch.full((L, npg), -1, dtype=torch.int32, device="cuda:0")
    q_all = torch.empty((T, L, wl.n_q, H, d), dtype=torch.bfloat16, device="cuda:0")
    # all pages and queries are generated up front (untimed); layer l owns
    # pool slots [l*npg, (l+1)*npg)
    for t in range(1, T + 1):
        wt = streaming_chunk(wl, t).replace(n_cand=0)
        for l in range(L):
            dd = make_case_torch(wt, "cuda:0", layer=l, chunk=t, k_pool=k_pool, v_pool=v_pool,
                                 slot_base=l * npg + wl.n_cur * (t - 1))
            table[l, wl.n_cur * (t - 1):wl.n_cur * t] = dd["page_table"][0]
            q_all[t - 1, l] = dd["q"][0]
    torch.cuda.synchronize()
    log(f"streaming inputs ready: {L} layers x {T} chunks")
    k_h = list(wl.budgets())
    k_max = max(k_h)

    def run(mode):
        if mode == "sequential":
            layers = [HsaLayer(1, H, d, P, torch.bfloat16, "cuda:0", k_pool=k_pool, v_pool=v_pool,
                               page_table=table[l:l + 1]) for l in range(L)]
            outs = [torch.empty((1, wl.n_q, H, d), dtype=torch.bfloat16, device="cuda:0")
                    for _ in range(L)]
        else:
            layer = HsaLayer(L, H, d, P, torch.bfloat16, "cuda:0", k_pool=k_pool, v_pool=v_pool,
                             page_table=table)
            out = torch.empty((L, wl.n_q, H, d), dtype=torch.bfloat16, device="cuda:0")
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        per_chunk = []
        for t in range(1, T + 1):
            n_cand = wl.n_cur * (t - 1)
            s.record()
            if mode == "sequential":
                for l in range(L):
                    layers[l].fold(n_cand, wl.n_cur)
                    layers[l].forward(q_all[t - 1, l:l + 1], n_cand, wl.n_cur, k_h, k_max=k_max,
                                      out=outs[l])
            else:
                layer.fold(n_cand, wl.n_cur)
                layer.forward(q_all[t - 1], n_cand, wl.n_cur, k_h, k_max=k_max, out=out)
            e.record()
            torch.cuda.synchronize()
            per_chunk.append(s.elapsed_time(e))
        return np.array(per_chunk)

    seq = run("sequential")
    bat = run("batched")
    flops = 0.0
    for t in range(1, T + 1):
        n_cand = wl.n_cur * (t - 1)
        k_eff = [min(k, n_cand) for k in k_h]
        flops += L * (attn_flops(wl, k_eff, wl.n_q) + linear_flops(wl, wl.n_q) +
                      state_flops_bytes(wl, wl.n_cur)[0])
    return {
        "metric": "HSA ms/chunk + effective TFLOP/s (MFMA util %) at 12 heads x d128, 4680 queries",
        "value": round(float(seq.mean()), 3), "unit": "ms/chunk (30 layers)", "n_gpus": 1,
        "steps": T, "warmup": 0, "ms_per_step": round(float(seq.mean()), 3),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "effective_tflops": round(flops / (seq.sum() * 1e-3) / 1e12, 2),
        "ms_per_chunk_t_ge_4": round(float(seq[3:].mean()), 3) if T > 3 else None,
        "chunk_ms": stats(np.sort(seq)),
        "batched_layers": {"ms_per_chunk": round(float(bat.mean()), 3),
                           "chunk_ms": stats(np.sort(bat)),
                           "ms_per_chunk_t_ge_4": round(float(bat[3:].mean()), 3) if T > 3 else None,
                           "effective_tflops": round(flops / (bat.sum() * 1e-3) / 1e12, 2)},
        "config": {"workload": wl.name, "layers": L, "chunks": T, "heads": H, "head_dim": d,
                   "n_q": wl.n_q, "page_size": P, "pages_per_chunk": wl.n_cur, "k_h": k_h,
                   "layer_launch": "sequential (one launch pair per layer)",
                   "parallelism": "single GPU"},
    }


def bench_sub(args, name):
    """A further workload as a sub-object of the line: its step and phase
    times and the attention roofline (c2, c4), or the streaming summary (c5)."""
    import torch
    from synth_inputs import WORKLOADS
    wl = WORKLOADS[name]
    if wl.layers > 1:
        r = bench_streaming(args, wl)
        keep = ("value", "unit", "ms_per_step", "effective_tflops", "ms_per_chunk_t_ge_4",
                "chunk_ms", "batched_layers", "config")
        return {k: r[k] for k in keep if k in r}
    r, layer, dev, sel = bench_core(args, wl)
    del layer, dev, sel
    torch.cuda.empty_cache()
    return r


def measured_ceilings():
    """Reference ceilings of this GPU, measured with library kernels beside
    the path's own (none of them is part of the path): the HBM rate of a
    device copy of 1.2 GB (read + written bytes) and of a fill of the same
    size (written bytes), and the bf16 matrix rate of a library GEMM of
    8192 x 8192 x 8192. Medians over 10 runs after 3 warmups. (A library
    reduction reads far below the copy's rate, so it is no read ceiling.)"""
    import torch
    n = 1200 << 20
    a = torch.ones(n // 2, dtype=torch.bfloat16, device="cuda:0")
    b = torch.empty_like(a)
    copy_ms = time_after_warmup(lambda: b.copy_(a), torch)
    fill_ms = time_after_warmup(lambda: b.fill_(1.0), torch)
    del a, b
    m = 8192
    x = torch.randn((m, m), dtype=torch.bfloat16, device="cuda:0")
    y = torch.randn((m, m), dtype=torch.bfloat16, device="cuda:0")
    z = torch.empty((m, m), dtype=torch.bfloat16, device="cuda:0")
    gemm_ms = time_after_warmup(lambda: torch.matmul(x, y, out=z), torch)
    del x, y, z
    torch.cuda.empty_cache()
    return {"device_copy_tb_s": round(2 * n / (copy_ms * 1e-3) / 1e12, 3),
            "device_fill_tb_s": round(n / (fill_ms * 1e-3) / 1e12, 3),
            "gemm_bf16_8192_tflop_s": round(2 * m ** 3 / (gemm_ms * 1e-3) / 1e12, 1),
            "peaks": {"hbm_tb_s": PEAK_HBM_GBS / 1e3, "bf16_tflop_s": PEAK_BF16_TFLOPS},
            "note": "library kernels (torch copy and fill, hipBLASLt GEMM), not the path's own"}


def time_after_warmup(fn, torch, warmup=3, iters=10):
    for _ in range(warmup):
        fn()
    return time_med(fn, iters, torch)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="c3", help="main workload, c1..c5")
    ap.add_argument("--sub", default="c2,c4,c5",
                    help="comma-separated further workloads reported as sub-objects ('' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-adaptive", action="store_true",
                    help="skip the head-adaptive block-sparse, Linformer, retrieval and tier "
                         "measurements")
    ap.add_argument("--layers", type=int, default=0, help="c5 only: override the layer count")
    ap.add_argument("--chunks", type=int, default=0, help="c5 only: override the chunk count")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the reference ceilings (a device copy, a fill and a library "
                         "bf16 GEMM) measured after the workloads")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the run, copy a MIB-sized device buffer 3 times (a plain copy of "
                         "known size, to scale HBM byte counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the HSA path here is a single-GPU build "
              "(sharding over heads or pages is described in the design notes, not implemented); "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if args.steps < 1:
        print("--steps must be >= 1", file=sys.stderr)
        sys.exit(2)
    from synth_inputs import WORKLOADS
    wl = WORKLOADS[args.config]
    res = bench_streaming(args, wl) if wl.layers > 1 else bench_single(args, wl)
    subs = [x for x in args.sub.split(",") if x and x != args.config]
    if subs:
        res["sub_configs"] = {}
        for name in subs:
            log(f"sub-workload {name} ...")
            res["sub_configs"][name] = bench_sub(args, name)
    if not args.no_ceilings:
        log("measured ceilings ...")
        res["ceilings_measured"] = measured_ceilings()
    if args.copy_calibration:
        import torch
        n = args.copy_calibration << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        res["copy_calibration_bytes"] = n
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
