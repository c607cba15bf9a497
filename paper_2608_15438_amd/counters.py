"""Summaries of rocprofv3 output for the refinement kernels.

    python -m paper_2608_15438_amd.counters stats TRACE_STATS.csv
        markdown table of the search kernels from a --kernel-trace --stats run

    python -m paper_2608_15438_amd.counters bench BENCH.json
        markdown summary of a headline `bench.py` line

    python -m paper_2608_15438_amd.counters grid GRID.jsonl
        markdown table of a `bench.py --grid` run (one JSON object per line)

    python -m paper_2608_15438_amd.counters traffic --kernel NAME --workload W \\
        --fetch F.csv --write W.csv --copy-fetch CF.csv --copy-write CW.csv \\
        --copy-bytes N --probe-budget P [--command TEXT]
        HBM traffic record (JSON) of one kernel from two --pmc passes
        (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch), each scaled by what the
        same counter reads for a device copy of N bytes per launch.

The record carries the sha256 of the kernel's sources, so a reader can tell
when the kernel changed after the counters were taken.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))

KERNEL_SOURCES = {"k_refine": ["k_refine.hip", "nr_internal.h"],
                  "k_scan": ["k_shared.hip", "nr_internal.h"]}


def source_digest(kernel: str) -> str:
    """sha256 over the sources a refinement kernel is built from."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(HERE, "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _rows(path):
    with open(path, newline="") as fh:
        return list(csv.DictReader(fh))


def per_dispatch(path: str, name_part: str, counter: str) -> list[float]:
    """Counter value of every dispatch whose kernel name contains name_part."""
    out = {}
    for r in _rows(path):
        if r.get("Counter_Name") != counter or name_part not in r.get("Kernel_Name", ""):
            continue
        key = r.get("Dispatch_Id") or r.get("Correlation_Id")
        out[key] = out.get(key, 0.0) + float(r["Counter_Value"])
    return list(out.values())


def _mean(v):
    return sum(v) / len(v) if v else float("nan")


def working(v: list[float]) -> list[float]:
    """Dispatches that did work: the shared schedule also launches the
    per-query kernel for queries whose survivors overflowed, usually with
    none, and such empty launches read next to nothing."""
    top = max(v) if v else 0.0
    return [x for x in v if x >= 0.01 * top]


def traffic(a) -> dict:
    fetch_all = per_dispatch(a.fetch, a.kernel, "FETCH_SIZE")
    fetch = working(fetch_all)
    # the write pass is a second run of the same program: keep the same launches
    write_all = per_dispatch(a.write, a.kernel, "WRITE_SIZE")
    keep = [i for i, x in enumerate(fetch_all) if x >= 0.01 * max(fetch_all)] if fetch_all else []
    write = [write_all[i] for i in keep if i < len(write_all)]
    cf = per_dispatch(a.copy_fetch, a.copy_kernel, "FETCH_SIZE")
    cw = per_dispatch(a.copy_write, a.copy_kernel, "WRITE_SIZE")
    if not (fetch and write and cf and cw):
        raise SystemExit("a counter pass has no dispatch of the named kernel")
    kib = 1024.0
    f_scale = a.copy_bytes / (max(cf) * kib)
    w_scale = a.copy_bytes / (max(cw) * kib)
    fb = _mean(fetch) * kib * f_scale
    wb = _mean(write) * kib * w_scale
    return {"kernel": a.kernel, "workload": a.workload,
            "source_sha256": source_digest(a.kernel),
            "dispatches": {"fetch": len(fetch), "write": len(write)},
            "fetch_kib_per_launch": round(_mean(fetch), 1),
            "write_kib_per_launch": round(_mean(write), 1),
            "copy_bytes_per_launch": a.copy_bytes,
            "copy_fetch_kib": round(max(cf), 1), "copy_write_kib": round(max(cw), 1),
            "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
            "hbm_fetch_bytes_per_launch": int(fb), "hbm_write_bytes_per_launch": int(wb),
            "hbm_bytes_per_launch": int(fb + wb),
            "probe_budget": a.probe_budget,
            "command": a.command}


def stats(path: str) -> str:
    keep = ("nr::", "synth")
    lines = ["| kernel | calls | avg us | min us | max us | total ms |",
             "|---|---:|---:|---:|---:|---:|"]
    for r in _rows(path):
        name = r["Name"]
        if not any(k in name for k in keep):
            continue
        short = name.split("(")[0].replace("void ", "")[:60]
        lines.append(f"| `{short}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.2f} |")
    return "\n".join(lines)


def grid_table(path: str) -> str:
    pts = [json.loads(x) for x in open(path) if x.strip().startswith("{")]
    lines = ["| P | gate | early stop | batch | QPS | Recall@10 | cand/q | read/q | clusters/q | "
             "centroids/q | stopped | refine GB/s | refine ms/call |",
             "|---:|---|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for p in pts:
        st = p["stage_ms_per_call"]
        t5 = sum(st.get(x, 0.0) for x in ("plan", "refine", "merge", "shared_prep", "shared_scan",
                                          "shared_merge"))
        lines.append(f"| {p['probe_budget']} | {p['gate']} | {'on' if p['early_stop'] else 'off'} | "
                     f"{p['batch']} | {p['qps']:.0f} | {p['recall_at_10']:.4f} | "
                     f"{p['cand_per_query']:.0f} | {p['rows_read_per_query']:.0f} | "
                     f"{p['clusters_per_query']:.1f} | {p['centroids_scored_per_query']:.1f} | "
                     f"{p['stopped_frac']:.2f} | {p['refine_gbs']} | {t5:.3f} |")
    return "\n".join(lines)


def bench_summary(path: str) -> str:
    d = json.loads(open(path).read().strip().splitlines()[-1])
    c = d["config"]
    out = [f"Workload `{c['workload']}`: n = {c['n']}, d = {d['config']['d']}, b = {c['b']}, "
           f"{c['queries']} queries, k = {c['k']}, dtype {d['dtype']}.", "",
           "| P | Recall@10 | QPS | candidates/query |", "|---:|---:|---:|---:|"]
    for p in sorted(d["sweep"], key=lambda p: p["probe_budget"]):
        out.append(f"| {p['probe_budget']} | {p['recall']:.4f} | {p['qps']:.0f} | "
                   f"{p['cand_per_query']:.0f} |")
    out += ["", f"Timed point P = {c['probe_budget']}: {d['value']:.0f} QPS ({d['ms_per_step']:.3f} ms "
            f"per search of {c['queries']} queries), Recall@10 = {d['recall_at_10']:.4f} on "
            f"{d['recall_queries']} queries.", ""]
    out.append("| kernel | avg launch ms (HIP events) | algorithmic GB / launch | GB/s | % of 8 TB/s |")
    out.append("|---|---:|---:|---:|---:|")
    for k, v in d.get("kernels", {}).items():
        out.append(f"| `{k}` | {v['avg_launch_ms']:.3f} | {v['alg_bytes_per_launch'] / 1e9:.2f} | "
                   f"{v['achieved_gbs']:.0f} | {100 * v['achieved_gbs'] / 8000:.1f} |")
    r = d["roofline"]
    out += ["", f"Roofline object: kernel `{r['kernel']}`, {r['achieved']:.0f} {r['unit']} of "
            f"{r['peak']:.0f} ({100 * r['frac']:.1f} %), traffic {r['traffic']} bytes per launch.",
            f"Whole refinement stage: {json.dumps(d.get('refine_stage'))}.",
            f"Stage ms per search: {json.dumps(d['stage_ms_per_step'])}.",
            f"Work of one search: {json.dumps(d.get('work'))}.",
            f"Streaming-read self-check: {d.get('hbm_stream_read_gbs')} GB/s.",
            f"CPU baseline (oracle): {json.dumps(d.get('cpu_baseline'))}.", "",
            "JSON line:", "", "```", json.dumps(d), "```"]
    return "\n".join(out)


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    g = sub.add_parser("grid")
    g.add_argument("jsonl")
    b = sub.add_parser("bench")
    b.add_argument("json")
    t = sub.add_parser("traffic")
    t.add_argument("--kernel", required=True, choices=sorted(KERNEL_SOURCES))
    t.add_argument("--workload", required=True)
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--copy-fetch", required=True)
    t.add_argument("--copy-write", required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--copy-kernel", default="copy")
    t.add_argument("--command", default="")
    t.add_argument("--probe-budget", type=int, required=True,
                   help="probe budget of the profiled search (a record holds for that budget only)")
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        print(stats(a.csv))
    elif a.cmd == "grid":
        print(grid_table(a.jsonl))
    elif a.cmd == "bench":
        print(bench_summary(a.json))
    else:
        print(json.dumps(traffic(a), indent=1))


if __name__ == "__main__":
    sys.exit(main())
