#!/usr/bin/env python3
"""Benchmark of MemDecay's per-decode-step retention path on one MI355X.

A step is the whole path over one batch: md_observe_step (append, attention
mass, EWMA, refresh, and on the fused kernel also the token and page scores),
md_score_pages (here with no outputs requested, so it adds no work),
md_select_evict (budgeted page selection) and md_compact (page-table
compaction).  All inputs
(the paged key cache, every step's queries and appended keys) are resident in
HBM before timing starts.  The default workload is 16 sessions of 32,768
cached tokens with Qwen2.5-1.5B's attention shape (28 layers, 12 query / 2 KV
heads, d = 128), 16-token pages and a 25 % budget.  The warm-up steps include
the first step's bulk eviction (32,768 -> 8,192 tokens per session); the
timed steps are the steady state that follows.

Printed on stdout: one JSON line.  value = tokens scored per second (the
sum over sessions and timed steps of the cached tokens scored, divided by
the wall time of the timed steps); roofline = the dominant kernel's (the
fused attention-mass kernel, or the attention-logits kernel of the
multi-kernel path) algorithmic bytes per launch over its event-timed average
duration, against MI355X's 8 TB/s; cpu_baseline = the CPU oracle on one session of the same
workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "cached tokens scored+evicted per second per decode step; achieved HBM GB/s vs peak"
PEAK_HBM_GBS = 8000.0
CSRC = os.path.join(ROOT, "paper_2607_10582_amd", "csrc")
KERNEL_SRC = {"logits": os.path.join(CSRC, "md_kernels.hip"), "attend": os.path.join(CSRC, "md_attend.hip")}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash(kernel: str) -> str:
    with open(KERNEL_SRC[kernel], "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def describe(w, n0s) -> str:
    n = f"{int(n0s[0])}" if len(set(n0s.tolist())) == 1 else f"U[{w.n0_range[0]},{w.n0_range[1]}]"
    return (f"{w.name}: {w.S} sessions x {n} cached tokens, {w.L} layers, {w.Hq}/{w.Hkv} heads, "
            f"d {w.d}, pages of {w.P}{' (region-aligned)' if w.region_aligned else ''}, "
            f"budget {int(w.budget_frac * 100)}%")


def setup(w, steps_total, dev, fused=None):
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
                       n_phys=n_phys, device=dev)
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
    md = MemDecay(cache, torch.from_numpy(b), torch.from_numpy(lam), rho=w.rho, alpha=w.alpha,
                  tau_scale=w.tau_scale, pinned_mask=w.pinned_mask, fused=fused,
                  region_aligned=w.region_aligned, quant_threshold=w.quant_threshold,
                  attention_norm=w.attention_norm, window=w.window)
    inputs = []
    for k in range(1, steps_total + 1):
        q = g.torch_window_queries(w, k, dev)
        nk = g.torch_append_keys(w, k, dev)
        reg = torch.full((w.S,), g.append_region(w, k), dtype=torch.uint8, device=dev)
        inputs.append((q, nk, reg))
    torch.cuda.synchronize(dev)
    return n0s, B, cache, md, inputs


def cpu_baseline(w, n0s, B, budget_s: float, max_steps: int):
    """The CPU oracle, as it stands, on session 0 of the workload: step 1 (the
    bulk eviction) untimed, then steady steps timed until ``budget_s``."""
    import torch
    import oracle
    from synth import generator as g

    try:
        from threadpoolctl import threadpool_info
        threads = max([1] + [int(i.get("num_threads", 1)) for i in threadpool_info()])
    except Exception:
        threads = 1
    b, lam = g.region_priors(w)
    n0 = int(n0s[0])
    dev = torch.device("cuda:0")
    kb = g.torch_keys(w, 0, n0, dev).view(torch.int16).cpu().numpy().view(np.uint16)
    sess = oracle.session_from_workload(w, 0, region=g.region_spans(w, 0, n0), keys_bits=kb,
                                        b=b[0], lam=lam[0], budget=int(B[0]),
                                        capacity=n0 + max_steps)
    del kb

    def inputs(k):
        qt = g.torch_window_queries(w, k, dev)
        q = None if qt is None else qt[0].cpu().numpy()
        nk = g.torch_append_keys(w, k, dev)[0].view(torch.int16).cpu().numpy().view(np.uint16)
        return q, nk, g.append_region(w, k)

    # untimed up to the first observation (the bulk eviction)
    k = 1
    while True:
        q, nk, r = inputs(k)
        sess.step(q, nk, r)
        k += 1
        if q is not None:
            break
    k0 = k
    scored = 0
    steps = 0
    elapsed = 0.0
    while elapsed < budget_s and k <= max_steps:
        q, nk, r = inputs(k)
        t0 = time.perf_counter()
        rec = sess.step(q, nk, r)
        elapsed += time.perf_counter() - t0
        if q is not None:     # only observation steps score tokens
            scored += rec.n
        steps += 1
        k += 1
    return {"value": scored / elapsed, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"session 0 of {w.S} ({w.name}), {steps} steady decode steps (steps {k0}-{k - 1}, "
                      f"after the bulk eviction), {scored} token-steps in {elapsed:.1f} s, numpy float64",
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
    import torch
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


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="long32k")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--multi-kernel", action="store_true",
                    help="observe on the multi-kernel path (logits in HBM) at every step instead of "
                         "letting the library pick")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB")
    ap.add_argument("--calibrate", type=int, default=0, metavar="BUCKET_STEPS",
                    help="also accumulate the region-lifetime statistics (Sec. IV-B) at every "
                         "observation, in age buckets of this many steps, and time it")
    ap.add_argument("--quant-threshold", type=float, default=None,
                    help="quantised tier: override the workload's threshold (0: off)")
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
    from paper_2607_10582_amd import binding
    from synth import configs as C
    from synth import generator as g

    binding.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = C.get(args.workload)
    if args.quant_threshold is not None:
        w = C.with_overrides(w, quant_threshold=args.quant_threshold)
    W, K = args.warmup, args.steps
    if W + K > w.steps:
        log(f"note: {W + K} steps asked, the workload defines {w.steps} decode steps")
    t_setup = time.perf_counter()
    n0s, B, cache, md, inputs = setup(w, W + K, dev, fused=False if args.multi_kernel else None)
    log(f"setup {time.perf_counter() - t_setup:.1f} s: {describe(w, n0s)}")

    # warm-up; the first step (the bulk eviction down to the budget) is
    # timed on its own with an event pair on the library's stream
    first_ms = None
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    first_obs = None
    for k in range(1, W + 1):
        q, nk, reg = inputs[k - 1]
        timed = first_obs is None and q is not None
        if timed:
            first_obs = k
            e0.record(md.stream)
        md.step(k, q, nk, reg, page_scores=False)
        if timed:
            e1.record(md.stream)
    torch.cuda.synchronize(dev)
    if first_obs is not None:
        first_ms = e0.elapsed_time(e1)
    c0 = md.counters()
    kcfg = md.kernel_config()
    hot = "attend" if kcfg["steady_fused"] and not kcfg["spill"] else "logits"
    log(f"kernel config {kcfg}; timing k_{hot}")
    md.profile((hot,))
    stream = md.stream
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    step_ev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    q_tok0 = quantised_tokens(cache) if w.quant_threshold > 0 else 0
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    ev0.record(stream)
    if args.calibrate:
        n_buckets = 64
        abar = torch.zeros(cache.n_phys * w.P, dtype=torch.float32, device=dev)
        stats = [torch.zeros((w.S, 7, n_buckets), dtype=torch.int64, device=dev) for _ in range(3)]
        cal_ev = []
    for i, k in enumerate(range(W + 1, W + K + 1)):
        q, nk, reg = inputs[k - 1]
        step_ev[i].record(stream)
        if args.calibrate and q is not None:
            # a calibration pass: the step's masses go to the lifetime bins
            md.observe(k, q, nk, reg, abar_out=abar)
            ce = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            ce[0].record(stream)
            md.calib_accumulate(abar, args.calibrate, stats)
            ce[1].record(stream)
            cal_ev.append(ce)
            md.score(page_score=False)
            md.select()
            md.compact()
        else:
            md.step(k, q, nk, reg, page_scores=False)
    step_ev[K].record(stream)
    ev1.record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - t0
    per_step = sorted(step_ev[i].elapsed_time(step_ev[i + 1]) for i in range(K))
    gpu_ms = ev0.elapsed_time(ev1)
    hot_ms, launches = md.profile_read(hot)
    md.profile(())
    c1 = md.counters()
    status = md.device_status()
    if status != 0:
        log(f"device status {status:#x}")
        sys.exit(1)

    scored = c1[0] - c0[0]
    # quantised tier: tokens in quantised pages per step, the mean of the
    # counts before and after the timed steps (the set changes slowly); their
    # keys take d + 1 bytes per (layer, KV head) row instead of 2 d (codes,
    # and a 16-byte scale line per 16 tokens)
    q_tok = (q_tok0 + quantised_tokens(cache)) / 2 if w.quant_threshold > 0 else 0
    q_saved = K * q_tok * (w.k_bytes_per_token - w.L * w.Hkv * (w.d + 1))
    evicted_tokens = c1[3] - c0[3]
    evicted_pages = c1[2] - c0[2]
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

    line = {
        "metric": METRIC,
        "value": scored / wall,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": wall * 1e3 / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": describe(w, n0s), "sessions": w.S,
                   "cached_tokens_per_session": int(n0s[0]) if w.n0 else "ragged",
                   "layers": w.L, "q_heads": w.Hq, "kv_heads": w.Hkv, "head_dim": w.d,
                   "page_size": w.P, "budget_frac": w.budget_frac, "parallelism": "none"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": traffic,
                     "kernel": f"k_{hot}", "launches": launches,
                     "avg_launch_us": avg_launch_s * 1e6,
                     "algorithmic_bytes_per_launch": per_launch_bytes},
        "tokens_scored_per_step": scored / K,
        "quantised_tokens_per_step": q_tok,
        "tokens_evicted_per_step": evicted_tokens / K,
        "pages_evicted": evicted_pages,
        "gpu_event_ms_per_step": gpu_ms / K,
        "step_ms_median": per_step[K // 2],
        "first_step_ms": first_ms,
        "calib_us_per_observation": (sum(a.elapsed_time(b) for a, b in cal_ev) * 1e3 / len(cal_ev)
                                     if args.calibrate and cal_ev else None),
        "step_algorithmic_gbs": step_bytes / wall / 1e9,
        "step_frac_of_peak": step_bytes / wall / 1e9 / PEAK_HBM_GBS,
    }
    md.close()
    del cache, inputs
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, n0s, B, args.cpu_seconds, w.steps)
    else:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
