"""Summaries of rocprofv3 CSV output for the retention path's kernels.

Two uses:

* ``trace``: per-kernel launch counts and durations from a
  ``rocprofv3 --kernel-trace --stats --output-format csv`` run, as a short
  markdown table.  The fused kernel's launches fall into three kinds, told
  apart by size against the median launch: md_init's residency checks
  (under a third of it), first observations of whole prompts, the bulk
  eviction (over twice it), and steady steps; the table gives the steady
  and the first-observation averages apart.
* ``hits``: L2 (TCC) hit rate of one kernel's steady launches from a
  ``--pmc TCC_HIT_sum TCC_MISS_sum`` run.
* ``pmc``: HBM bytes per launch of one kernel from two counter runs
  (``--pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE``), each scaled by what the
  same counter reads for a plain device copy of known size.  Writes the JSON
  file bench.py reads as ``roofline.traffic`` (tied to a hash of the kernel
  source it was taken on) and prints a markdown summary.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import statistics
from collections import defaultdict

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
KERNEL_SOURCES = {"k_attend": "md_attend.hip", "k_logits": "md_kernels.hip"}
HEADERS = ("md_internal.h", "md_device.h")   # included by both sources


def source_hash(kernel: str) -> str:
    """Hash of the kernel's source file and the headers it includes: a
    counter profile holds for the code it was taken on."""
    h = hashlib.sha256()
    for name in (KERNEL_SOURCES[kernel],) + HEADERS:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def short_name(name: str) -> str:
    n = name.replace("(anonymous namespace)::", "")
    for p in ("void ", "md::"):
        if n.startswith(p):
            n = n[len(p):]
    return n.split("(")[0].strip()


def _one(pattern: str) -> str:
    hits = sorted(glob.glob(pattern))
    if not hits:
        raise FileNotFoundError(pattern)
    return hits[0]


def kinds(values):
    """Indices of (steady, first-observation, residency-check) launches of the
    fused kernel, by size against the median launch (steady launches are
    most of any run)."""
    med = statistics.median(values)
    steady = [i for i, v in enumerate(values) if med / 3 <= v <= 2 * med]
    bulk = [i for i, v in enumerate(values) if v > 2 * med]
    check = [i for i, v in enumerate(values) if v < med / 3]
    return steady, bulk, check


def trace_table(trace_dir: str, skip: int):
    """Rows (kernel, launches, avg us, total us, steady avg us, launches, first-observation avg
    us, launches) from a kernel trace."""
    rows = list(csv.DictReader(open(_one(os.path.join(trace_dir, "*kernel_trace.csv")))))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    durs = defaultdict(list)
    for r in rows:
        durs[r["Kernel_Name"]].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    out = []
    for name, d in durs.items():
        bulk = []
        if "k_attend" in name:
            st, bk, _ = kinds(d)
            steady, bulk = [d[i] for i in st], [d[i] for i in bk]
        else:
            steady = d[skip:] if ("md::" in name and len(d) > skip) else d
        out.append((short_name(name)[:60], len(d), sum(d) / len(d), sum(d), sum(steady) / len(steady),
                    len(steady), (sum(bulk) / len(bulk)) if bulk else None, len(bulk)))
    out.sort(key=lambda x: -x[3])
    return out


def counter_values(pmc_dir: str, counter: str):
    """{kernel name: [value per dispatch in dispatch order]} for one counter."""
    rows = list(csv.DictReader(open(_one(os.path.join(pmc_dir, "*counter_collection.csv")))))
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    vals = defaultdict(list)
    for r in rows:
        if r["Counter_Name"] == counter:
            vals[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return vals


def copy_factor(pmc_dir: str, counter: str, copy_bytes: int) -> float:
    """Bytes per counter unit, from the device copies of ``copy_bytes``."""
    vals = counter_values(pmc_dir, counter)
    cand = [v for k, v in vals.items() if "copyBuffer" in k]
    if not cand:
        raise RuntimeError(f"no copy kernel in {pmc_dir}")
    med = statistics.median(cand[0])
    return copy_bytes / med


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="mode", required=True)
    t = sub.add_parser("trace")
    t.add_argument("trace_dir")
    t.add_argument("--skip", type=int, default=3)
    t.add_argument("--top", type=int, default=14)
    h = sub.add_parser("hits")
    h.add_argument("pmc_dir")
    h.add_argument("--kernel", default="k_attend")
    h.add_argument("--skip", type=int, default=3)
    p = sub.add_parser("pmc")
    p.add_argument("fetch_dir")
    p.add_argument("write_dir")
    p.add_argument("cal_fetch_dir")
    p.add_argument("cal_write_dir")
    p.add_argument("--kernel", default="k_attend")
    p.add_argument("--workload", required=True)
    p.add_argument("--skip", type=int, default=3)
    p.add_argument("--copy-mib", type=int, default=256)
    p.add_argument("--algorithmic-bytes", type=float, default=None,
                   help="algorithmic bytes per launch, for the ratio")
    p.add_argument("--first-algorithmic-bytes", type=float, default=None,
                   help="algorithmic bytes of a first-observation launch, for its ratio")
    p.add_argument("--json", required=True)
    a = ap.parse_args()

    if a.mode == "trace":
        print("| kernel | launches | avg us | total us | steady avg us (launches) | first observation avg us "
              "(launches) |")
        print("|---|---:|---:|---:|---:|---:|")
        for name, n, avg, tot, st, ns, bk, nb in trace_table(a.trace_dir, a.skip)[:a.top]:
            b = f"{bk:.2f} ({nb})" if bk is not None else ""
            print(f"| `{name}` | {n} | {avg:.2f} | {tot:.1f} | {st:.2f} ({ns}) | {b} |")
        return

    if a.mode == "hits":
        hit = counter_values(a.pmc_dir, "TCC_HIT_sum")
        miss = counter_values(a.pmc_dir, "TCC_MISS_sum")
        names = [n for n in hit if short_name(n).startswith(a.kernel)]
        if not names:
            raise RuntimeError(f"{a.kernel} not in {a.pmc_dir}")
        # every instantiation of the kernel, by dispatch order; the fused
        # kernel's launch kinds are told apart by their accesses
        hs_all = [v for n in names for v in hit[n]]
        ms_all = [v for n in names for v in miss[n]]
        groups = [("steady", list(range(a.skip, len(hs_all))))]
        if a.kernel == "k_attend":
            st, bk, _ = kinds([h + m for h, m in zip(hs_all, ms_all)])
            groups = [("steady", st), ("first observation", bk)]
        print(f"| {a.kernel} launches | count | L2 (TCC) hits per launch | misses per launch | hit rate |")
        print("|---|---:|---:|---:|---:|")
        for label, idx in groups:
            if not idx:
                continue
            hs, ms = [hs_all[i] for i in idx], [ms_all[i] for i in idx]
            rate = sum(hs) / max(sum(hs) + sum(ms), 1.0)
            print(f"| {label} | {len(idx)} | {statistics.mean(hs):.4g} | {statistics.mean(ms):.4g} | {100 * rate:.1f} % |")
        return

    nbytes = a.copy_mib << 20
    ff = copy_factor(a.cal_fetch_dir, "FETCH_SIZE", nbytes)
    fw = copy_factor(a.cal_write_dir, "WRITE_SIZE", nbytes)
    fetch = counter_values(a.fetch_dir, "FETCH_SIZE")
    write = counter_values(a.write_dir, "WRITE_SIZE")
    # the kernel's instantiation that moved the most bytes (another one may
    # have run only md_init's residency checks)
    key = [k for k in fetch if short_name(k).startswith(a.kernel)]
    if not key:
        raise RuntimeError(f"{a.kernel} not in {a.fetch_dir}")
    name = max(key, key=lambda k: sum(fetch[k]))
    allf = fetch[name]
    allw = write[name]
    # the two runs launch the same sequence; kinds are read off the reads
    st, bk, _ = kinds(allf)
    kf, kw = [allf[i] for i in st], [allw[i] for i in st]
    rd = statistics.mean(kf) * ff
    wr = statistics.mean(kw) * fw
    rec = {"kernel": a.kernel, "workload": a.workload, "kernel_source_sha256_16": source_hash(a.kernel),
           "launches": len(kf), "fetch_bytes_per_launch": rd, "write_bytes_per_launch": wr,
           "hbm_bytes_per_launch": rd + wr, "fetch_bytes_per_counter_unit": ff,
           "write_bytes_per_counter_unit": fw, "copy_bytes": nbytes}
    if bk:
        brd = statistics.mean([allf[i] for i in bk]) * ff
        bwr = statistics.mean([allw[i] for i in bk]) * fw
        rec.update({"first_observation_launches": len(bk), "first_observation_fetch_bytes": brd,
                    "first_observation_write_bytes": bwr, "first_observation_hbm_bytes": brd + bwr})
    if a.algorithmic_bytes:
        rec["algorithmic_bytes_per_launch"] = a.algorithmic_bytes
        rec["traffic_over_algorithmic"] = (rd + wr) / a.algorithmic_bytes
    if bk and a.first_algorithmic_bytes:
        rec["first_observation_algorithmic_bytes"] = a.first_algorithmic_bytes
        rec["first_observation_traffic_over_algorithmic"] = (brd + bwr) / a.first_algorithmic_bytes
    with open(a.json, "w") as f:
        json.dump(rec, f, indent=1)
    print(f"| {a.kernel} on {a.workload} | per launch (mean of {len(kf)} steady launches) |")
    print("|---|---:|")
    print(f"| HBM read (FETCH_SIZE x {ff:.4g} B) | {rd / 1e9:.4f} GB |")
    print(f"| HBM write (WRITE_SIZE x {fw:.4g} B) | {wr / 1e9:.4f} GB |")
    if a.algorithmic_bytes:
        print(f"| algorithmic bytes | {a.algorithmic_bytes / 1e9:.4f} GB |")
        print(f"| traffic / algorithmic | {(rd + wr) / a.algorithmic_bytes:.3f} |")
    if bk:
        print()
        print(f"| {a.kernel} on {a.workload}, first observation (bulk eviction) | per launch (mean of {len(bk)}) |")
        print("|---|---:|")
        print(f"| HBM read | {brd / 1e9:.4f} GB |")
        print(f"| HBM write | {bwr / 1e9:.4f} GB |")
        if a.first_algorithmic_bytes:
            print(f"| algorithmic bytes | {a.first_algorithmic_bytes / 1e9:.4f} GB |")
            print(f"| traffic / algorithmic | {(brd + bwr) / a.first_algorithmic_bytes:.3f} |")


if __name__ == "__main__":
    main()
