#!/usr/bin/env python3
"""Benchmark of MemDecay's per-decode-step retention path on one MI355X.

A step is the whole path over one batch: md_observe_step (append, attention
mass, EWMA, refresh, and on the fused kernel also the token and page scores),
md_score_pages (here with no outputs requested, so it adds no work),
md_select_evict (budgeted page selection) and md_compact (page-table
compaction).  All inputs (the paged key cache, every step's queries and
appended keys) are resident in HBM before timing starts.

The default workload is the ragged batch: 64 agent sessions of U[2,048,
65,536] cached tokens with Qwen2.5-3B's attention shape (36 layers, 16 query
/ 2 KV heads, d = 128), 16-token pages and a 20 % budget, 64 decode steps.
The same run also measures the ragged batch with 64-token pages, the
long-horizon batch (16 sessions x 32,768 tokens, 1.5B shape, 25 % budget,
128 steps) and the batch of short sessions (32 x 1,700 tokens, 3B shape,
30 % budget, 256 steps, on the fused kernel with row groups) as
sub-records.

For every workload, step 1 runs three times on a copy of the state first
(so the code objects are loaded), then one trajectory from the fresh cache:
step 1 (the bulk eviction down to the budget) and the warm-up steps, then
the timed steps, then the rest of the workload's steps.  Every step outside
the timed region is bracketed by an event pair on the library's stream, and
the timed region by one pair around all of its steps (an event between two
steps costs the stream a few microseconds), so the record holds the first
step, the timed steps' mean, the median of the untimed steady steps and the
mean over the workload's whole run.

Printed on stdout: one JSON line.  value = tokens scored per second over the
timed steps (the sum over sessions and timed steps of the cached tokens
scored, divided by the wall time of the timed steps, bracketed by
synchronisations); roofline = the dominant kernel's (the fused
attention-mass kernel, or the attention-logits kernel of the multi-kernel
path) algorithmic bytes per launch over its event-timed average duration,
against MI355X's 8 TB/s; cpu_baseline = the CPU oracle, session-parallel on
the host's cores, on a sample of the same workload.
"""
from __future__ import annotations

import argparse
import gc
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "cached tokens scored+evicted per second per decode step; achieved HBM GB/s vs peak"
PEAK_HBM_GBS = 8000.0
DEFAULT_WORKLOAD = "ragged_p16"
DEFAULT_ALSO = "ragged_p64,long32k,qwen3_32x1700"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash(kernel: str) -> str:
    from paper_2607_10582_amd.rocprof_summary import source_hash
    return source_hash("k_" + kernel)


def describe(w, n0s) -> str:
    n = f"{int(n0s[0])}" if len(set(n0s.tolist())) == 1 else f"U[{w.n0_range[0]},{w.n0_range[1]}]"
    return (f"{w.name}: {w.S} sessions x {n} cached tokens, {w.L} layers, {w.Hq}/{w.Hkv} heads, "
            f"d {w.d}, pages of {w.P}{' (region-aligned)' if w.region_aligned else ''}, "
            f"budget {int(w.budget_frac * 100)}%, {w.steps} decode steps")


def setup(w, steps_total, dev, fused=None, offload_pages=0, drop_threshold=0.0, row_groups=True):
    import torch
    from paper_2607_10582_amd.cache import MemDecay, PagedCache
    from synth import configs as C
    from synth import generator as g

    n0s = g.prefix_lengths(w)
    B = g.budgets(w, n0s)
    b, lam = g.region_priors(w)
    ws = C.with_overrides(w, steps=max(steps_total, 1))
    n_phys = g.pages_needed(ws, n0s)
    spans = [g.region_spans(w, s, int(n0s[s])) for s in range(w.S)]
    pages = [PagedCache.pages_for(spans[s], w.P, w.region_aligned) for s in range(w.S)]
    # every decode step may open a page with region-aligned pages
    grow = steps_total if w.region_aligned else (steps_total + w.P - 1) // w.P
    max_pages = max(pages) + grow + 1
    cache = PagedCache(L=w.L, Hq=w.Hq, Hkv=w.Hkv, d=w.d, P=w.P, S=w.S, max_pages=max_pages,
                       n_phys=n_phys, device=dev, offload_pages=offload_pages)
    perm = g.page_permutation(w, n_phys)
    pos = 0
    for s in range(w.S):
        n0 = int(n0s[s])
        m = pages[s]
        keys = g.torch_keys(w, s, n0, dev)
        cache.load_session(s, keys, spans[s], perm[pos:pos + m], budget=int(B[s]), clock=n0,
                           region_aligned=w.region_aligned)
        pos += m
        del keys
    cache.set_free_pages(perm[pos:][::-1])

    def make_md():
        return MemDecay(cache, torch.from_numpy(b), torch.from_numpy(lam), rho=w.rho, alpha=w.alpha,
                        tau_scale=w.tau_scale, pinned_mask=w.pinned_mask, fused=fused,
                        region_aligned=w.region_aligned, quant_threshold=w.quant_threshold,
                        attention_norm=w.attention_norm, window=w.window, drop_threshold=drop_threshold,
                        row_groups=row_groups)

    inputs = []
    for k in range(1, steps_total + 1):
        q = g.torch_window_queries(w, k, dev)
        nk = g.torch_append_keys(w, k, dev)
        reg = torch.full((w.S,), g.append_region(w, k), dtype=torch.uint8, device=dev)
        inputs.append((q, nk, reg))
    torch.cuda.synchronize(dev)
    # Timing protocol: the first observation runs three times on a copy of
    # the caller-side state (restored after each run; the key pool too when
    # the quantised tier may rewrite it), so that the measured trajectory
    # starts with the code objects loaded; then a fresh handle.
    first = next(k for k in range(1, steps_total + 1) if inputs[k - 1][0] is not None)
    names = ["region", "t_ins", "t_ref", "importance", "page_table", "page_serial", "n_pages", "n_tokens",
             "n_live", "page_format", "clock", "next_serial", "budget", "free_list", "free_count"]
    if w.quant_threshold > 0:
        names.append("k_pool")
    if offload_pages > 0:
        names += list(PagedCache.OFFLOAD_BUFFERS)
    snap = {n: getattr(cache, n).clone() for n in names}
    for r in range(3):
        md = make_md()
        for k in range(1, first + 1):
            q, nk, reg = inputs[k - 1]
            md.step(k, q, nk, reg, page_scores=False)
        md.close()
        for n in names:
            getattr(cache, n).copy_(snap[n])
    del snap
    torch.cuda.synchronize(dev)
    return n0s, B, cache, make_md(), inputs


def cpu_baseline(w, n0s, B, budget_s: float):
    """The CPU oracle, as it stands, session-parallel on the host's cores:
    one worker process per core (one BLAS thread each), one session per
    worker (the workload's first sessions).  Step 1 (the bulk eviction) runs
    untimed; then whole steps of all sampled sessions are timed until
    ``budget_s``.  The keys and queries are the device-drawn ones the GPU
    run uses, copied to the host."""
    import torch
    from oracle.pool import SessionPool, host_cores
    from synth import generator as g

    cores = host_cores()
    n_s = min(cores, w.S)
    sample = list(range(n_s))
    b, lam = g.region_priors(w)
    dev = torch.device("cuda:0")
    t_setup = time.perf_counter()
    pool = SessionPool(cores)
    try:
        for s in sample:
            n0 = int(n0s[s])
            kb = g.torch_keys(w, s, n0, dev).view(torch.int16).cpu().numpy().view(np.uint16)
            kw = dict(L=w.L, Hq=w.Hq, Hkv=w.Hkv, d=w.d, P=w.P, b=b[s], lam=lam[s], alpha=w.alpha, rho=w.rho,
                      tau_scale=w.tau_scale, pinned_mask=w.pinned_mask, budget=int(B[s]), clock=n0,
                      region=g.region_spans(w, s, n0), capacity=n0 + w.steps,
                      attention_norm=w.attention_norm, region_aligned=w.region_aligned,
                      quant_threshold=w.quant_threshold)
            pool.add(s, kw, kb, n0)
            del kb

        def inputs(k):
            qt = g.torch_window_queries(w, k, dev)
            q = None if qt is None else qt.cpu().numpy()
            nk = g.torch_append_keys(w, k, dev).view(torch.int16).cpu().numpy().view(np.uint16)
            r = g.append_region(w, k)
            return {s: (None if q is None else q[s], nk[s], r) for s in sample}

        log(f"cpu baseline: {n_s} sessions on {pool.workers} workers, set up in "
            f"{time.perf_counter() - t_setup:.1f} s")
        k = 1
        while True:                     # untimed up to the first observation (the bulk eviction)
            inp = inputs(k)
            pool.step(inp)
            k += 1
            if next(iter(inp.values()))[0] is not None:
                break
        k0 = k
        scored = steps = 0
        elapsed = 0.0
        while elapsed < budget_s and k <= w.steps:
            inp = inputs(k)
            t0 = time.perf_counter()
            recs = pool.step(inp)
            elapsed += time.perf_counter() - t0
            if next(iter(inp.values()))[0] is not None:     # only observation steps score tokens
                scored += sum(r.n for r in recs.values())
            steps += 1
            k += 1
    finally:
        pool.close()
    return {"value": scored / elapsed, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"sessions 0-{n_s - 1} of {w.S} ({w.name}), one per worker process "
                      f"({pool.workers} workers x 1 BLAS thread on {cores} cores), {steps} steady decode steps "
                      f"(steps {k0}-{k - 1}, after the untimed bulk eviction), {scored} token-steps in "
                      f"{elapsed:.1f} s of wall time, numpy float64",
            "seconds_per_step": elapsed / max(steps, 1)}


def load_traffic(kernel: str, workload: str):
    """Counter-measured HBM bytes per launch of ``kernel``, if a profile of
    the current kernel source exists."""
    path = os.path.join(ROOT, "profiles", f"k_{kernel}_{workload}_pmc.json")
    if not os.path.exists(path):
        return None, None
    with open(path) as f:
        d = json.load(f)
    if d.get("kernel_source_sha256_16") != kernel_source_hash(kernel):
        return None, "stale"
    return d.get("hbm_bytes_per_launch"), path


def quantised_tokens(cache) -> int:
    """Tokens held in quantised pages now (such pages are never a session's
    last page, so each holds P slots)."""
    npg = cache.n_pages.cpu().numpy()
    fmt = cache.page_format.cpu().numpy()
    tot = 0
    for s in range(cache.S):
        ids = cache.page_table[s, :int(npg[s])].cpu().numpy()
        tot += int(fmt[ids].sum()) * cache.P
    return tot


def calibrate_copy(mib: int):
    """A plain device copy of known size, for scaling the FETCH_SIZE /
    WRITE_SIZE counters."""
    import torch
    n = mib * (1 << 20)
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copied {n} bytes 5 times")


def measure(w, W: int, K: int, dev, *, multi_kernel=False, calibrate=0, offload_pages=0, drop_threshold=0.0,
            row_groups=True):
    """One trajectory of workload w from a fresh cache: steps 1..W (warm-up;
    step 1 the bulk eviction), W+1..W+K timed, then on to the workload's
    last step.  Returns the record (value, roofline, step times)."""
    import torch
    from synth import configs as C
    from synth import generator as g

    total = max(w.steps, W + K)
    t_setup = time.perf_counter()
    n0s, B, cache, md, inputs = setup(w, total, dev, fused=False if multi_kernel else None, row_groups=row_groups,
                                      offload_pages=offload_pages, drop_threshold=drop_threshold)
    log(f"setup {time.perf_counter() - t_setup:.1f} s: {describe(w, n0s)}")
    stream = md.stream
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(total + 1)]

    def run(k):
        q, nk, reg = inputs[k - 1]
        md.step(k, q, nk, reg, page_scores=False)

    # warm-up, every step event-timed; the tokens of step 1 (the bulk
    # eviction) are counted on their own
    c_start = md.counters()
    first_end = torch.cuda.Event(enable_timing=True)
    for k in range(1, W + 1):
        ev[k - 1].record(stream)
        run(k)
        if k == 1:
            first_end.record(stream)
            c_first = md.counters()
    ev[W].record(stream)
    torch.cuda.synchronize(dev)
    c0 = md.counters()
    kcfg = md.kernel_config()
    hot = "attend" if kcfg["steady_fused"] and not kcfg["spill"] else "logits"
    log(f"kernel config {kcfg}; timing k_{hot}")
    md.profile((hot,))
    q_tok0 = quantised_tokens(cache) if w.quant_threshold > 0 else 0
    if calibrate:
        n_buckets = 64
        abar = torch.zeros(cache.n_phys * w.P, dtype=torch.float32, device=dev)
        stats = [torch.zeros((w.S, 7, n_buckets), dtype=torch.int64, device=dev) for _ in range(3)]
        cal_ev = []
    timed_ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    timed_ev[0].record(stream)
    for k in range(W + 1, W + K + 1):
        q, nk, reg = inputs[k - 1]
        if calibrate and q is not None:
            # a calibration pass: the step's masses go to the lifetime bins
            md.observe(k, q, nk, reg, abar_out=abar)
            ce = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            ce[0].record(stream)
            md.calib_accumulate(abar, calibrate, stats)
            ce[1].record(stream)
            cal_ev.append(ce)
            md.score(page_score=False)
            md.select()
            md.compact()
        else:
            run(k)
    timed_ev[1].record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - t0
    hot_ms, launches = md.profile_read(hot)
    md.profile(())
    c1 = md.counters()
    q_tok1 = quantised_tokens(cache) if w.quant_threshold > 0 else 0
    # the rest of the workload's run
    for k in range(W + K + 1, total + 1):
        ev[k - 1].record(stream)
        run(k)
    ev[total].record(stream)
    torch.cuda.synchronize(dev)
    warm_ms = [ev[0].elapsed_time(first_end)] + [ev[i].elapsed_time(ev[i + 1]) for i in range(1, W)]
    timed_ms = timed_ev[0].elapsed_time(timed_ev[1])
    rest_ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(W + K, total)]
    untimed_steady = warm_ms[1:] + rest_ms
    status = md.device_status()
    if status != 0:
        log(f"device status {status:#x}")
        sys.exit(1)

    scored = c1[0] - c0[0]
    # quantised tier: tokens in quantised pages per step, the mean of the
    # counts before and after the timed steps (the set changes slowly); their
    # keys take d + 1 bytes per (layer, KV head) row instead of 2 d (codes,
    # and a 16-byte scale line per 16 tokens)
    q_tok = (q_tok0 + q_tok1) / 2 if w.quant_threshold > 0 else 0
    q_saved = K * q_tok * (w.k_bytes_per_token - w.L * w.Hkv * (w.d + 1))
    kb = w.k_bytes_per_token
    # the queries of the observation steps: W per session and step
    n_obs = sum(1 for k in range(W + 1, W + K + 1) if g.observes(w, k))
    q_bytes = w.S * w.L * w.Hq * w.d * 4 * w.window * n_obs / K
    # algorithmic bytes over the timed launches: every cached key once and the
    # queries once; the fused kernel also reads and writes each token's
    # importance (Eq. 2), reads its refresh clock and region (Eq. 3, Eq. 4),
    # and reads each page's table entry and writes its score (Eq. 5)
    if hot == "attend":
        hot_bytes = scored * (kb + 13) + (scored // w.P) * 8 + K * q_bytes - q_saved
    else:
        hot_bytes = scored * kb + K * q_bytes - q_saved
    avg_launch_s = hot_ms / 1e3 / max(launches, 1)
    per_launch_bytes = hot_bytes / max(launches, 1)
    achieved = per_launch_bytes / avg_launch_s / 1e9
    # the counters were taken on the workload as named: a quantised tier
    # switched on from the command line reads other bytes (its own profile
    # name carries the threshold)
    prof_name = w.name if w.quant_threshold == C.get(w.name).quant_threshold else f"{w.name}_quant{w.quant_threshold:g}"
    traffic, traffic_src = load_traffic(hot, prof_name)
    # whole step: K + per-token state (region 1, a 4+4, t_ref 4+4) + per-page
    # score and page-table entry + the queries
    step_bytes = scored * (kb + 17) + scored // w.P * 8 + K * q_bytes - q_saved
    # the first observation (step 1) on the same terms
    scored1 = c_first[0] - c_start[0]
    first_bytes = scored1 * (kb + 17) + scored1 // w.P * 8 + (w.S * w.L * w.Hq * w.d * 4 * w.window
                                                              if g.observes(w, 1) else 0)
    rec = {
        "value": scored / wall,
        "unit": "tokens/s",
        "ms_per_step": wall * 1e3 / K,
        "workload": describe(w, n0s),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": traffic,
                     "traffic_source": None if traffic is None else os.path.relpath(traffic_src, ROOT),
                     "kernel": f"k_{hot}", "launches": launches,
                     "avg_launch_us": avg_launch_s * 1e6,
                     "algorithmic_bytes_per_launch": per_launch_bytes},
        "tokens_scored_per_step": scored / K,
        "tokens_evicted_per_step": (c1[3] - c0[3]) / K,
        "quantised_tokens_per_step": q_tok,
        "pages_evicted": c1[2] - c0[2],
        "first_step_ms": warm_ms[0],
        "first_step_tokens": scored1,
        "first_step_algorithmic_bytes": first_bytes,
        "first_step_frac_of_peak": first_bytes / (warm_ms[0] / 1e3) / 1e9 / PEAK_HBM_GBS,
        "steady_step_ms_mean": timed_ms / K,
        "step_ms_median": float(np.median(untimed_steady)) if untimed_steady else timed_ms / K,
        "run_mean_ms": (sum(warm_ms) + timed_ms + sum(rest_ms)) / total,
        "run_steps": total,
        "calib_us_per_observation": (sum(a.elapsed_time(b) for a, b in cal_ev) * 1e3 / len(cal_ev)
                                     if calibrate and cal_ev else None),
        "step_algorithmic_gbs": step_bytes / wall / 1e9,
        "step_frac_of_peak": step_bytes / wall / 1e9 / PEAK_HBM_GBS,
        "observe_path": {"first": "fused" if kcfg["first_fused"] else "multi-kernel",
                         "first_row_groups": kcfg["first_row_groups"],
                         "steady": "fused" if kcfg["steady_fused"] else "multi-kernel",
                         "steady_row_groups": kcfg["steady_row_groups"]},
    }
    if offload_pages > 0:
        # offload tier: pages moved over the host link in the timed steps,
        # each a page of keys (L Hkv P d bf16 values): to host memory,
        # back from it, and read by the observation of host-memory pages
        page_bytes = w.L * w.Hkv * w.P * w.d * 2
        moved = (c1[4] - c0[4]) + (c1[5] - c0[5]) + (c1[7] - c0[7])
        rec["offload"] = {"host_pages_per_session": offload_pages, "drop_threshold": drop_threshold,
                          "pages_offloaded_per_step": (c1[4] - c0[4]) / K,
                          "pages_recalled_per_step": (c1[5] - c0[5]) / K,
                          "pages_dropped_per_step": (c1[6] - c0[6]) / K,
                          "host_pages_observed_per_step": (c1[7] - c0[7]) / K,
                          "host_link_bytes_per_step": moved * page_bytes / K,
                          "host_link_gbs": moved * page_bytes / wall / 1e9}
    md.close()
    del cache, inputs, md
    torch.cuda.synchronize(dev)
    torch.cuda.empty_cache()
    return rec, n0s, B


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--also", default=None,
                    help=f"comma-separated workloads measured as sub-records in the same run "
                         f"(default with the default workload: {DEFAULT_ALSO}; '' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--multi-kernel", action="store_true",
                    help="observe on the multi-kernel path (logits in HBM) at every step instead of "
                         "letting the library pick")
    ap.add_argument("--no-row-groups", action="store_true",
                    help="keep every fused unit on all (layer, KV head) rows: without row groups, "
                         "batches whose units fill less than half of the fused grid take the "
                         "multi-kernel path")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB")
    ap.add_argument("--calibrate", type=int, default=0, metavar="BUCKET_STEPS",
                    help="also accumulate the region-lifetime statistics (Sec. IV-B) at every "
                         "observation, in age buckets of this many steps, and time it")
    ap.add_argument("--quant-threshold", type=float, default=None,
                    help="quantised tier: override the workload's threshold (0: off)")
    ap.add_argument("--offload-pages", type=int, default=0,
                    help="offload tier: host-memory pages per session (0: off)")
    ap.add_argument("--drop-threshold", type=float, default=0.0,
                    help="offload tier: pages scoring below it are dropped, not kept in host memory")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the retention path shards over sessions with no "
              f"exchange, and the benchmark measures one GPU's share (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return

    import torch
    # The HIP runtime starts before the library is loaded (see
    # binding.load_library): its exit handlers then run after the library's.
    dev = torch.device("cuda:0")
    torch.cuda.init()
    torch.cuda.set_device(dev)
    torch.cuda.synchronize(dev)
    from paper_2607_10582_amd import binding
    from synth import configs as C

    binding.load_library()
    w = C.get(args.workload)
    if args.quant_threshold is not None:
        w = C.with_overrides(w, quant_threshold=args.quant_threshold)
    also = args.also if args.also is not None else (DEFAULT_ALSO if args.workload == DEFAULT_WORKLOAD else "")
    also = [a for a in also.split(",") if a and a != w.name]
    W, K = args.warmup, args.steps
    if W < 1:
        log("note: the warm-up includes step 1, the bulk eviction; --warmup raised to 1")
        W = 1

    main_rec, n0s, B = measure(w, W, K, dev, multi_kernel=args.multi_kernel, calibrate=args.calibrate,
                               offload_pages=args.offload_pages, drop_threshold=args.drop_threshold,
                               row_groups=not args.no_row_groups)
    subs = {}
    for name in also:
        # each workload starts from device memory as a fresh process has it:
        # the previous workload's buffers go back to the driver first
        gc.collect()
        torch.cuda.empty_cache()
        rec, _, _ = measure(C.get(name), W, K, dev, multi_kernel=args.multi_kernel,
                            row_groups=not args.no_row_groups)
        subs[name] = rec
        log(f"{name}: {rec['value']:.4g} tokens/s, k_{rec['roofline']['kernel'][2:]} "
            f"{rec['roofline']['frac']:.3f} of peak")

    line = {
        "metric": METRIC,
        "value": main_rec["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": main_rec["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": main_rec["workload"], "sessions": w.S,
                   "cached_tokens_per_session": int(n0s[0]) if w.n0 else f"U[{w.n0_range[0]},{w.n0_range[1]}]",
                   "layers": w.L, "q_heads": w.Hq, "kv_heads": w.Hkv, "head_dim": w.d,
                   "page_size": w.P, "budget_frac": w.budget_frac, "decode_steps": w.steps,
                   "parallelism": "none"},
        "roofline": main_rec["roofline"],
    }
    for key in ("tokens_scored_per_step", "tokens_evicted_per_step", "quantised_tokens_per_step",
                "pages_evicted", "first_step_ms", "first_step_tokens", "first_step_algorithmic_bytes",
                "first_step_frac_of_peak", "steady_step_ms_mean", "step_ms_median", "run_mean_ms",
                "run_steps", "calib_us_per_observation", "step_algorithmic_gbs", "step_frac_of_peak",
                "observe_path"):
        line[key] = main_rec[key]
    if "offload" in main_rec:
        line["offload"] = main_rec["offload"]
    line["workloads"] = subs
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, n0s, B, args.cpu_seconds)
    else:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
