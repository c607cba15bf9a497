#!/usr/bin/env python3
"""Benchmark of the batched NeuRoute search on one MI355X.

One step = one nr_search call over the whole query batch (encoder, probe
enumeration, bucket lookup, centroid stage, exact refinement) with queries
and index resident in HBM.  Untimed set-up: the synthetic workload and its
index are built on the GPU (seeded generators, index construction, gate
calibration), ground truth comes from a plain PyTorch brute force, and a
probe-budget sweep picks the fastest point with Recall@10 >= 0.90.  Then W
warm-up and K timed steps run at that point; HIP events around the
refinement kernel (on its launch stream) give its average duration for the
roofline.  The CPU oracle is timed on a bounded query sample.

Prints one JSON line.
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

METRIC = "QPS at Recall@10 ≥ 0.90 (10k-query batch); refine-stage HBM GB/s"
HBM_PEAK_GBS = 8000.0


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=4, help="workload 1..4 (4 = 1B x 128 uint8)")
    ap.add_argument("--no-clustering", action="store_true",
                    help="index without bucket-local clustering (every bucket one cluster)")
    ap.add_argument("--n", type=int, default=0, help="override the base size (smaller instance)")
    ap.add_argument("--k-c", type=int, default=0,
                    help="override the centroid heap size K_c (the workload name gets a -kc suffix)")
    ap.add_argument("--probes", type=str, default="", help="comma list of probe budgets to sweep")
    ap.add_argument("--target-recall", type=float, default=0.90)
    ap.add_argument("--refine-steps", type=int, default=4,
                    help="bisection steps on the probe budget around the recall target")
    ap.add_argument("--gt-queries", type=int, default=1000)
    ap.add_argument("--calib-queries", type=int, default=300)
    ap.add_argument("--oracle-seconds", type=float, default=10.0)
    ap.add_argument("--oracle-stage-gb", type=float, default=8.0)
    ap.add_argument("--oracle-threads", type=int, default=0)
    ap.add_argument("--no-oracle", action="store_true")
    ap.add_argument("--margin-quantile", type=float, default=0.95)
    ap.add_argument("--train-steps", type=int, default=2000,
                    help="train the seeded encoder with L_sim for this many Adam steps before "
                         "the index is built (0: keep the seeded encoder)")
    ap.add_argument("--train-batch", type=int, default=4096)
    ap.add_argument("--train-lr", type=float, default=2e-4)
    ap.add_argument("--calib", choices=("gt", "bootstrap"), default="gt",
                    help="calibration targets: brute-force top-k, or the search's own "
                         "top-k at the largest budget with gate and early stop off")
    ap.add_argument("--s-max-coverage", type=float, default=0.0,
                    help="apply the bucket-score cutoff S_max fitted at this pair coverage "
                         "(0: S_max = +inf, the enumeration bounded by the probe budget alone)")
    ap.add_argument("--n-bins", type=int, default=32,
                    help="score bins of Algorithm 1 when S_max is applied")
    ap.add_argument("--refine-mode", choices=("auto", "per_query", "shared"), default="auto",
                    help="refinement schedule (the same results either way)")
    ap.add_argument("--seed-rows", type=int, default=0,
                    help="shared schedule: rows of each query's own (seed) pass; 0 = the library's")
    ap.add_argument("--gt-cache", type=str, default="",
                    help="directory for the exact top-k of the query and calibration sets "
                         "(reused by later runs on the same workload)")
    ap.add_argument("--quick", action="store_true",
                    help="no recall ground truth and no oracle (for counter passes)")
    ap.add_argument("--copy-calib", action="store_true",
                    help="only run a plain 4 GiB device copy (counter calibration) and exit")
    ap.add_argument("--head-bytes", type=int, default=-1,
                    help="payload layout: 0 row-major, else a head plane of this many bytes "
                         "(default: the first 16 dimensions)")
    ap.add_argument("--head-split", action="store_true",
                    help="store tails after the head plane instead of whole rows (less memory)")
    ap.add_argument("--grid", action="store_true",
                    help="parameter grid instead of the headline: probe budget x gate margin "
                         "quantile x early stop x batch size, one JSON line per point")
    ap.add_argument("--grid-probes", type=str, default="", help="default: the workload's budgets")
    ap.add_argument("--grid-gates", type=str, default="0.99,0.95,0.80")
    ap.add_argument("--grid-batches", type=str, default="1,256,10000")
    return ap.parse_args()


# ----------------------------------------------------------------------------
# ground truth: exact k-NN by plain PyTorch on the device
# ----------------------------------------------------------------------------

def ground_truth(torch, rows_range, n, is_u8, row_ids, Q, k, chunk=1 << 19):
    """Exact top-k by (squared distance, original id) for every query in Q;
    rows_range(s0, s1) returns payload rows [s0, s1) row-major."""
    nq = Q.shape[0]
    if is_u8:
        # integer distances: every fp32 step below is exact (all partial sums
        # of byte products stay below 2^24), then (distance, id) is packed in
        # one int64 key so ties resolve by the lower original id
        Qf = Q.float()
        qq = (Qf * Qf).sum(1)
        m2q = (-2.0 * Qf).T.contiguous()
        best = None
        for s0 in range(0, n, chunk):
            if s0 and s0 % (chunk * 256) == 0:
                log(f"  ground truth: {s0 / n:.0%} of the base")
            X = rows_range(s0, min(n, s0 + chunk)).float()
            d = X @ m2q
            d += (X * X).sum(1)[:, None]
            d += qq[None, :]
            key = d.to(torch.int64)
            del d
            key <<= 32
            key |= row_ids[s0:s0 + chunk][:, None]
            top = torch.topk(key, min(k, key.shape[0]), dim=0, largest=False).values
            del key
            best = top if best is None else torch.topk(torch.cat([best, top]), k, dim=0,
                                                       largest=False).values
        best = best.T.contiguous()
        return (best & 0xFFFFFFFF).cpu().numpy(), (best >> 32).cpu().numpy().astype(np.float32)
    Qd = Q.double()
    qq = (Qd * Qd).sum(1)
    bd, bi = None, None
    for s0 in range(0, n, chunk):
        if s0 and s0 % (chunk * 256) == 0:
            log(f"  ground truth: {s0 / n:.0%} of the base")
        X = rows_range(s0, min(n, s0 + chunk)).double()
        d = (X * X).sum(1)[:, None] - 2 * (X @ Qd.T) + qq[None, :]
        kk = min(k + 8, d.shape[0])
        v, i = torch.topk(d, kk, dim=0, largest=False)
        ids = row_ids[s0:s0 + chunk][i]
        if bd is None:
            bd, bi = v, ids
        else:
            v2, j = torch.topk(torch.cat([bd, v]), k + 8, dim=0, largest=False)
            bi = torch.gather(torch.cat([bi, ids]), 0, j)
            bd = v2
    bd, bi = bd.T.cpu().numpy(), bi.T.cpu().numpy()
    out_i = np.empty((nq, k), np.int64)
    out_d = np.empty((nq, k), np.float32)
    for q in range(nq):
        o = np.lexsort((bi[q], bd[q]))[:k]
        out_i[q], out_d[q] = bi[q][o], bd[q][o]
    return out_i, out_d


def stream_read_ceiling(torch, NR, dev, gib=16, reps=5):
    """Achievable read rate: the library's streaming-read self-check (8 KB
    runs per wave, eight 16-byte non-temporal loads in flight per lane) over a
    16 GiB buffer."""
    x = torch.ones(gib << 28, dtype=torch.float32, device=dev)
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    NR.nr_stream_read(x, sink)
    torch.cuda.synchronize()
    t0 = time.time()
    for _ in range(reps):
        NR.nr_stream_read(x, sink)
    torch.cuda.synchronize()
    gbs = reps * x.numel() * 4 / (time.time() - t0) / 1e9
    del x
    torch.cuda.empty_cache()
    log(f"streaming read of {gib} GiB: {gbs:.0f} GB/s")
    return gbs


def copy_calibration(torch, dev, gib=4, reps=5):
    """A plain device copy of known size (reads and writes gib GiB per
    launch) to scale the FETCH_SIZE / WRITE_SIZE counters."""
    src = torch.ones(gib << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_launch": src.numel(), "launches": reps}), flush=True)


def measured_traffic(kernel, workload, probe_budget):
    """HBM bytes per launch of `kernel` from the committed counter record
    (FETCH_SIZE + WRITE_SIZE, each scaled by a copy of known size), or None
    when there is none, the kernel's sources changed since it was taken, or
    it was taken at another probe budget."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.txt")
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    from paper_2608_15438_amd.counters import source_digest
    if rec.get("source_sha256") != source_digest(kernel):
        log(f"traffic record {os.path.basename(path)} is stale (kernel sources changed)")
        return None
    if rec.get("probe_budget") != probe_budget:
        log(f"traffic record {os.path.basename(path)} was taken at P = {rec.get('probe_budget')}, "
            f"not {probe_budget}")
        return None
    return int(rec["hbm_bytes_per_launch"])


def recall_at_k(res, gt, k):
    r = 0.0
    for a, b in zip(res, gt):
        r += len(set(a[:k].tolist()) & set(b[:k].tolist())) / k
    return r / len(res)


# ----------------------------------------------------------------------------

def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the search shards by query batch or database, see the design notes)", file=sys.stderr)
        sys.exit(2)
    import torch
    from synth import configs as CF
    from synth.gpu import GpuRows
    from paper_2608_15438_amd import index_build as IB
    from paper_2608_15438_amd import calibrate as CAL
    from paper_2608_15438_amd import neuroute as NR

    torch.backends.cuda.matmul.allow_tf32 = False
    torch.set_float32_matmul_precision("highest")
    dev = torch.device("cuda:0")
    if args.copy_calib:
        copy_calibration(torch, dev)
        return
    stream_gbs = stream_read_ceiling(torch, NR, dev)
    w = CF.WORKLOADS[args.config]
    if args.n:
        w = CF.scaled(w, args.n)
    if args.no_clustering:
        import dataclasses
        w = dataclasses.replace(w, cluster_rule="none", name=w.name + "-noclust")
    if args.k_c and args.k_c != w.k_c:
        import dataclasses
        w = dataclasses.replace(w, k_c=args.k_c, name=f"{w.name}-kc{args.k_c}")
    k = w.k
    t_all = time.time()

    # ---- workload and index (untimed)
    log(f"building {w.name}: n={w.n} d={w.d} b={w.b}")
    data = GpuRows(w, "data", dev)
    t0 = time.time()
    hb = args.head_bytes if args.head_bytes >= 0 else 16 * (1 if w.dtype == "u8" else 4)
    enc = None
    if args.train_steps:
        # L_sim training of the seeded encoder on batches of the base rows
        from paper_2608_15438_amd import train as TR
        t1 = time.time()
        enc = TR.train_encoder(IB.seeded_encoder(w), data, w.n, args.train_steps,
                               batch=args.train_batch, lr=args.train_lr, gamma=0.6,
                               seed=w.seed("sample"), device=dev, log=lambda s: log("  ", s))
        torch.cuda.synchronize()
        log(f"encoder trained in {time.time() - t1:.1f}s")
    ix = IB.build_index(w, data, device=dev, chunk=1 << 20, keep_codes=False, encoder=enc,
                        payload_fn=lambda perm: data(perm), log=lambda s: log("  index:", s),
                        head_bytes=hb, head_copy=not args.head_split)
    torch.cuda.synchronize()
    t_build = time.time() - t0
    log(f"index built in {t_build:.1f}s: {ix.n_clusters} clusters")
    Q = GpuRows(w, "query", dev).range(0, w.n_queries)
    gix = NR.Index.from_built(ix, dev)

    # ---- ground truth and gate calibration (untimed)
    t0 = time.time()
    ng = 0 if args.quick else min(args.gt_queries, w.n_queries)
    nc = args.calib_queries
    Qc = GpuRows(w, "calib", dev).range(0, nc)
    # exact top-k of the query and calibration sets: they depend on the base
    # rows and the query sets only, so --gt-cache keeps them across runs
    cache = {}
    if args.gt_cache:
        os.makedirs(args.gt_cache, exist_ok=True)
        for what, m in (("query", ng), ("calib", nc)):
            path = os.path.join(args.gt_cache, f"{w.name}-n{w.n}-k{k}-{what}{m}.npy")
            cache[what] = (path, np.load(path) if m and os.path.exists(path) else None)
    need_q = ng > 0 and cache.get("query", (None, None))[1] is None
    need_c = nc > 0 and cache.get("calib", (None, None))[1] is None
    if need_q or need_c:
        parts = ([Q[:ng]] if need_q else []) + ([Qc] if need_c else [])
        gt_new, _ = ground_truth(torch, lambda a, b: IB.payload_range(ix, a, b), w.n,
                                 w.dtype == "u8", ix.row_ids, torch.cat(parts), k)
        if need_q:
            cache["query"] = (cache.get("query", (None, None))[0], gt_new[:ng])
        if need_c:
            cache["calib"] = (cache.get("calib", (None, None))[0], gt_new[ng if need_q else 0:])
        for path, arr in cache.values():
            if path and arr is not None and not os.path.exists(path):
                np.save(path, arr)
    gt_ids = cache["query"][1] if ng else np.zeros((0, k), np.int64)
    gtc = cache["calib"][1] if nc else np.zeros((0, k), np.int64)
    log(f"ground truth for {ng}+{nc} queries in {time.time() - t0:.1f}s")
    targets = torch.from_numpy(gtc).to(dev)
    if args.calib == "bootstrap":
        # the paper's supervision: the search itself in a higher-recall
        # setting (the largest budget, gate and early stop off)
        loose = NR.Params(l_sel=min(w.l_sel, w.b), r_max=w.r_max, k_c=w.k_c, gate_on=False,
                          early_stop_on=False)
        targets = CAL.bootstrap_targets(gix, Qc, k, NR.NR_MAX_PROBES, loose)
        agree = float((targets.cpu() == torch.from_numpy(gtc)).double().mean())
        log(f"bootstrapped calibration targets: {agree:.3f} of them equal the brute-force ones")
    # bucket scores of the targets and margin points: the library's calibration kernel
    sc, xs, ys = CAL.gpu_calibration(gix, gix.nr_encode(Qc), targets, min(w.l_sel, w.b), w.r_max)
    s95, pcov, qcov = CAL.fit_s_max(sc, 0.95)
    calib = {"targets": "bootstrap" if args.calib == "bootstrap" else "brute-force",
             "queries": nc, "s_max_95": round(s95, 4), "pair_coverage": round(pcov, 4),
             "query_coverage": round(qcov, 4)}
    s_max, n_bins = float("inf"), 1
    if args.s_max_coverage > 0:
        s_max, pc, qc = CAL.fit_s_max(sc, args.s_max_coverage)
        n_bins = args.n_bins
        calib.update({"applied_s_max": round(s_max, 5), "applied_coverage": args.s_max_coverage,
                      "applied_pair_coverage": round(pc, 4), "n_bins": n_bins})
    log("calibration", calib)
    m_x, m_y = CAL.fit_margin(xs, ys, args.margin_quantile)
    params = NR.Params(l_sel=min(w.l_sel, w.b), r_max=w.r_max, k_c=w.k_c, s_max=s_max,
                       n_bins=n_bins, m_x=m_x.tolist(), m_y=m_y.tolist(),
                       shared_seed_rows=args.seed_rows,
                       refine_mode={"auto": NR.NR_REFINE_AUTO, "per_query": NR.NR_REFINE_PER_QUERY,
                                    "shared": NR.NR_REFINE_SHARED}[args.refine_mode])
    if args.grid:
        grid(args, w, gix, Q, gt_ids, ng, xs, ys, CAL, NR, torch, ix.head_copy)
        return

    # ---- probe-budget sweep: recall and QPS per point
    budgets = [int(x) for x in args.probes.split(",")] if args.probes else list(w.probe_budgets)
    sweep = []

    def measure(P):
        ids, _ = gix.nr_search(Q, k, P, params)
        torch.cuda.synchronize()
        t0 = time.time()
        reps = 2
        for _ in range(reps):
            ids, _ = gix.nr_search(Q, k, P, params)
        torch.cuda.synchronize()
        dt = (time.time() - t0) / reps
        rec = recall_at_k(ids[:ng].cpu().numpy(), gt_ids, k) if ng else float("nan")
        rows = gix.nr_last_work()["rows"]
        pt = dict(probe_budget=P, recall=round(rec, 5), qps=round(w.n_queries / dt, 1),
                  cand_per_query=round(rows / w.n_queries, 1))
        sweep.append(pt)
        log("  sweep", pt)
        return pt

    for P in budgets:
        measure(P)
    # bisect between the last budget below the recall target and the first above it
    if ng and len(budgets) > 1:
        for _ in range(args.refine_steps):
            ok_p = sorted(p["probe_budget"] for p in sweep if p["recall"] >= args.target_recall)
            bad_p = sorted(p["probe_budget"] for p in sweep if p["recall"] < args.target_recall)
            if not ok_p or not bad_p:
                break
            hi = ok_p[0]
            lo = max([b for b in bad_p if b < hi], default=None)
            if lo is None or hi - lo <= 8:
                break
            measure((lo + hi) // 2)
    ok = [p for p in sweep if p["recall"] >= args.target_recall]
    head = max(ok, key=lambda p: p["qps"]) if ok else max(sweep, key=lambda p: p["recall"])
    P = head["probe_budget"]

    # ---- timed region: W warm-up + K steps at the chosen point
    for _ in range(args.warmup):
        gix.nr_search(Q, k, P, params)
    torch.cuda.synchronize()
    gix.nr_profile_enable(True)
    gix.nr_profile_read(reset=True)
    torch.cuda.synchronize()
    t0 = time.time()
    for _ in range(args.steps):
        ids, dists = gix.nr_search(Q, k, P, params)
    torch.cuda.synchronize()
    wall = time.time() - t0
    stage_ms, n_timed = gix.nr_profile_read(reset=True)
    gix.nr_profile_enable(False)
    work = gix.nr_last_work()
    rows = work["rows"]
    recall = recall_at_k(ids[:ng].cpu().numpy(), gt_ids, k) if ng else float("nan")
    qps = w.n_queries * args.steps / wall
    _, _, qs = gix.nr_search(Q, k, P, params, qstats=True)
    qs = qs.double().mean(0).cpu().numpy()
    per_query = {name: round(float(qs[i]), 2) for name, i in NR.QS.items()}
    log("per-query means", per_query, "work", work)
    # the refinement kernels.  Algorithmic bytes: k_refine reads whole rows (of
    # fp32 rows past 1 KB, the slabs it reached before the row's sum passed the
    # list's k-th key: refine_bytes);
    # k_scan reads the head of every scanned row, then what it reads of the
    # rows its heads left open (whole rows, or the 1 KB slabs of long rows up
    # to the last one some query needed; without whole rows after the heads,
    # minus the head already read) -- one launch of each per search: the
    # batch fits one chunk
    nt = max(n_timed, 1)
    kernels = {}
    hb = work["head_bytes"]
    scan_body = work["body_bytes"] - (0 if ix.head_copy else work["full_rows"] * hb)
    # the open-pair pass (fp32 rows past 1 KB): the row bytes of the slabs it
    # read; it reads the same amount of query bytes, mostly from cache
    # candidate bytes (every (query, row) pair the kernel settles, at the whole
    # row's size: what a per-query refinement of the same pairs reads)
    for kname, stage, nrows, ab, cand in (
            ("k_refine", "refine", work["own_rows"], work["refine_bytes"],
             work["own_rows"] * w.row_bytes),
            ("k_scan", "shared_scan", work["shared_rows"], work["shared_rows"] * hb + scan_body,
             work["shared_pair_rows"] * w.row_bytes),
            ("k_scan_open", "shared_open", work["open_bytes"] // max(1, w.row_bytes - 1024),
             work["open_bytes"], 0)):
        ms = stage_ms[stage] / nt
        if ms <= 0 or nrows <= 0:
            continue
        kernels[kname] = {"avg_launch_ms": round(ms, 4), "alg_bytes_per_launch": int(ab),
                          "rows_per_launch": int(nrows),
                          "achieved_gbs": round(ab / (ms * 1e-3) / 1e9, 1),
                          "candidate_bytes_per_launch": int(cand),
                          "candidate_gbs": round(cand / (ms * 1e-3) / 1e9, 1),
                          "candidate_frac": round(cand / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    dom = max(kernels, key=lambda n: kernels[n]["avg_launch_ms"])
    refine_ms = kernels[dom]["avg_launch_ms"]
    alg_bytes = kernels[dom]["alg_bytes_per_launch"]
    achieved = kernels[dom]["achieved_gbs"]
    traffic = measured_traffic(dom, w.name, P)
    # the whole refinement stage (step 5): every launch from the plan to the merge
    st5 = sum(stage_ms[x] for x in ("plan", "refine", "merge", "shared_prep", "shared_scan",
                                    "shared_open", "shared_merge")) / nt
    b5 = work["refine_bytes"] + work["shared_rows"] * hb + scan_body + work["open_bytes"]
    cand_bytes = rows * w.row_bytes
    refine_stage = {"ms": round(st5, 4), "bytes_read": int(b5), "candidate_bytes": int(cand_bytes),
                    "candidate_gbs": round(cand_bytes / (st5 * 1e-3) / 1e9, 1),
                    "gbs": round(b5 / (st5 * 1e-3) / 1e9, 1),
                    "frac_of_peak": round(b5 / (st5 * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    log(f"timed: {args.steps} steps, {wall * 1e3 / args.steps:.2f} ms/step, recall {recall:.4f}, "
        f"kernels {kernels}, dominant {dom}")

    # ---- CPU baseline: the oracle on a bounded sample (rows staged in host memory)
    cpu = parity = None
    if not args.no_oracle and not args.quick:
        cpu, parity = oracle_baseline(args, w, ix, gix, Q, P, params, torch, dev)

    out = {
        "metric": METRIC,
        "value": round(qps, 1),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "n": w.n, "d": w.d, "b": w.b, "queries": w.n_queries,
                   "encoder": (f"L_sim-trained, {args.train_steps} steps of {args.train_batch}"
                               if args.train_steps else "seeded"),
                   "layout": (f"head{ix.head_bytes}+" + ("rows" if ix.head_copy else "tail"))
                   if ix.head_bytes else "row-major",
                   "k": k, "probe_budget": P, "l_sel": params.l_sel, "r_max": params.r_max,
                   "k_c": params.k_c, "gate": f"q{int(round(args.margin_quantile * 100))}",
                   "low_quality": "or" if params.lowq_or else "and",
                   "s_max": params.s_max if np.isfinite(params.s_max) else "inf",
                   "early_stop": True, "parallelism": "single-gpu"},
        "recall_at_10": round(recall, 5),
        "recall_queries": ng,
        "cand_per_query": round(rows / w.n_queries, 1),
        "per_query": per_query,
        "rows_read_per_query": round(work["rows_read"] / w.n_queries, 1),
        "work": work,
        "stage_ms_per_step": {s: round(v / max(n_timed, 1), 4) for s, v in stage_ms.items()},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "alg_bytes_per_launch": int(alg_bytes),
                     "avg_launch_ms": round(refine_ms, 4),
                     "bytes": "gathered: the bytes the kernel reads (heads of the rows it scans, "
                              "rows it reads whole)",
                     "candidate_frac": kernels[dom]["candidate_frac"],
                     "stage_frac": refine_stage["frac_of_peak"]},
        "kernels": kernels,
        "refine_stage": refine_stage,
        "cpu_baseline": cpu,
        "parity": parity,
        "calibration": calib,
        "sweep": sweep,
        "hbm_stream_read_gbs": round(stream_gbs, 1),
        "setup_s": {"index_build": round(t_build, 1), "total": round(time.time() - t_all, 1)},
    }
    print(json.dumps(out), flush=True)


def grid(args, w, gix, Q, gt_ids, ng, xs, ys, CAL, NR, torch, head_copy):
    """Probe budget x gate (margin quantile of M) x early stop x batch size.
    Batch 1 runs the first 1,000 queries one call each; larger batches run the
    whole query set in consecutive calls of that size.  Per point: QPS of an
    unprofiled pass, Recall@10 on the ground-truth queries it covers, stage
    milliseconds of a second (profiled) pass, per-query counters of a third."""
    k = w.k
    probes = [int(x) for x in args.grid_probes.split(",")] if args.grid_probes \
        else list(w.probe_budgets)
    gates = [float(x) for x in args.grid_gates.split(",")]
    batches = [int(x) for x in args.grid_batches.split(",")]
    step5 = ("plan", "refine", "merge", "shared_prep", "shared_scan", "shared_open", "shared_merge")

    def run_all(Qr, B, P, params, qstats=False):
        outs = []
        for s0 in range(0, len(Qr), B):
            outs.append(gix.nr_search(Qr[s0:s0 + B], k, P, params, qstats=qstats))
        return outs

    for gq in gates:
        m_x, m_y = CAL.fit_margin(xs, ys, gq)
        for es in (True, False):
            params = NR.Params(l_sel=min(w.l_sel, w.b), r_max=w.r_max, k_c=w.k_c,
                               m_x=m_x.tolist(), m_y=m_y.tolist(), early_stop_on=es)
            for P in probes:
                for B in batches:
                    nq = min(1000, w.n_queries) if B == 1 else w.n_queries
                    Qr = Q[:nq]
                    run_all(Qr[:min(nq, 2 * B)], B, P, params)          # warm-up
                    torch.cuda.synchronize()
                    t0 = time.time()
                    outs = run_all(Qr, B, P, params)
                    torch.cuda.synchronize()
                    wall = time.time() - t0
                    ids = torch.cat([o[0] for o in outs])
                    nr = min(ng, nq)
                    rec = recall_at_k(ids[:nr].cpu().numpy(), gt_ids[:nr], k) if nr else float("nan")
                    # profiled pass: stage times, and rows read by the last call
                    gix.nr_profile_enable(True)
                    gix.nr_profile_read(reset=True)
                    run_all(Qr, B, P, params)
                    torch.cuda.synchronize()
                    st, ncalls = gix.nr_profile_read(reset=True)
                    gix.nr_profile_enable(False)
                    work = gix.nr_last_work()
                    qs = torch.cat([o[2] for o in run_all(Qr, B, P, params, qstats=True)])
                    qm = qs.double().mean(0).cpu().numpy()
                    rows = float(qs[:, NR.QS["rows"]].double().sum())
                    # rows and bytes read: the shared schedule (one call) reports
                    # them; the per-query schedule reads every candidate row
                    shared = B >= nq and work["shared_pairs"]
                    read = work["rows_read"] if shared else rows
                    hb = work["head_bytes"]
                    nbytes = (work["refine_bytes"] + work["shared_rows"] * hb + work["body_bytes"]
                              - (0 if head_copy else work["full_rows"] * hb) + work["open_bytes"]
                              ) if shared else rows * w.row_bytes
                    t5 = sum(st[x] for x in step5)
                    pt = {"workload": w.name, "probe_budget": P, "gate": f"q{int(round(gq * 100))}",
                          "early_stop": es, "batch": B, "queries": nq,
                          "qps": round(nq / wall, 1), "recall_at_10": round(rec, 5),
                          "recall_queries": nr,
                          "cand_per_query": round(rows / nq, 1),
                          "rows_read_per_query": round(read / nq, 1),
                          "clusters_per_query": round(float(qm[NR.QS["clusters"]]), 1),
                          "centroids_scored_per_query": round(float(qm[NR.QS["scored"]]), 2),
                          "centroid_batches_per_query": round(float(qm[NR.QS["batches"]]), 2),
                          "stopped_frac": round(float(qm[NR.QS["stopped"]]), 3),
                          "refine_gbs": round(nbytes / (t5 * 1e-3) / 1e9, 1) if t5 else None,
                          "stage_ms_per_call": {x: round(v / max(ncalls, 1), 4) for x, v in st.items()},
                          "calls": ncalls}
                    print(json.dumps(pt), flush=True)
                    log("grid", {x: pt[x] for x in ("probe_budget", "gate", "early_stop", "batch",
                                                     "qps", "recall_at_10", "refine_gbs")})


def host_cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_threads(args) -> int:
    """One thread per core this process may use: the affinity mask, bounded
    by the CPU share the host grants the job (OMP_NUM_THREADS, when set)."""
    if args.oracle_threads:
        return args.oracle_threads
    aff = len(os.sched_getaffinity(0))
    share = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    return min(aff, share) if share > 0 else aff


def oracle_baseline(args, w, ix, gix, Q, P, params, torch, dev):
    """Time the oracle on a bounded sample: a 32-query pilot sizes the sample
    to about `--oracle-seconds` of wall time on the host threads, capped by
    `--oracle-stage-gb` of staged rows; then one thread on the first 100
    queries (per-core rate).  The oracle's top-k lists of the sample are
    compared with the GPU's for the same queries, searched in the timed
    launch configuration (the whole batch) with the oracle's logits."""
    import oracle as O
    from paper_2608_15438_amd import index_build as IB
    threads = oracle_threads(args)
    e = ix.encoder
    enc = O.Encoder(e.weights, e.biases, e.bn_scale or (), e.bn_shift or (), e.input_scale)
    bc = ix.bc_off.cpu().numpy().astype(np.uint32)
    cl = ix.cl_off.cpu().numpy().astype(np.uint64)
    cent = ix.centroids.cpu().numpy()
    prm = O.RouteParams(n_bins=params.n_bins, s_max=params.s_max, k_c=params.k_c,
                        b_batch=params.b_batch, b_min=params.b_min, t_low=params.t_low,
                        u_heap=params.u_heap, u_front=params.u_front,
                        alpha_front=params.alpha_front, gate_on=params.gate_on,
                        early_stop_on=params.early_stop_on, lowq_or=params.lowq_or,
                        m_x=np.array(params.m_x, np.float32), m_y=np.array(params.m_y, np.float32))

    def stage(nqs):
        Qh = Q[:nqs].cpu().numpy()
        # discovery (untimed): the clusters this sample needs
        lg = O.encode(enc, Qh)
        codes, costs, bins, cnt = O.probes(lg, ix.tau, params.l_sel, params.r_max, P,
                                           params.s_max, params.n_bins)
        lists = O.route(lg, codes, bins, cnt, bc, cent, prm)
        need = np.unique(np.concatenate(lists)).astype(np.int64)
        sizes = (cl[need + 1] - cl[need]).astype(np.int64)
        # stage their rows in host memory behind a cl_off in which every
        # other cluster is empty
        starts = torch.from_numpy(cl[need].astype(np.int64)).to(dev)
        sz_t = torch.from_numpy(sizes).to(dev)
        idx = torch.repeat_interleave(starts, sz_t) + (
            torch.arange(int(sizes.sum()), device=dev) -
            torch.repeat_interleave(torch.cumsum(sz_t, 0) - sz_t, sz_t))
        rows_h = IB.payload_rows(ix, idx).cpu().numpy()
        ids_h = ix.row_ids[idx].cpu().numpy()
        del idx
        cnt_all = np.zeros(ix.n_clusters, np.int64)
        cnt_all[need] = sizes
        cl2 = np.zeros(ix.n_clusters + 1, np.uint64)
        cl2[1:] = np.cumsum(cnt_all)
        return Qh, rows_h, ids_h, cl2

    def run(staged, nqs, min_seconds, n_threads):
        Qh, rows_h, ids_h, cl2 = staged
        # timed: whole passes over the staged sample until min_seconds have
        # elapsed (at least one pass)
        passes, t0 = 0, time.time()
        while True:
            oi, od, ncand, secs = O.search(enc, ix.tau, rows_h, ids_h, bc, cl2, cent, Qh[:nqs],
                                           w.k, params.l_sel, params.r_max, P, prm,
                                           n_threads=n_threads)
            passes += 1
            if time.time() - t0 >= min_seconds:
                break
        return (time.time() - t0) / passes, passes, secs, oi, od

    pilot = min(32, w.n_queries)
    st = stage(pilot)
    dt, _, secs, _, _ = run(st, pilot, 0.0, threads)
    per_q = dt / pilot
    nbytes_pilot = st[1].nbytes
    nqs = int(min(w.n_queries, max(pilot, args.oracle_seconds / max(per_q, 1e-9)),
                  max(pilot, args.oracle_stage_gb * 1e9 / max(nbytes_pilot / pilot, 1.0))))
    nqs = max(nqs, min(w.n_queries, 100))
    st = stage(nqs)
    nbytes = st[1].nbytes
    dt, passes, secs, oi, od = run(st, nqs, args.oracle_seconds, threads)
    cpu_qps = nqs / dt
    # one thread, 100 queries: the per-core rate
    n1 = min(100, nqs)
    dt1, passes1, _, _, _ = run(st, n1, 0.0, 1)
    log(f"oracle: {nqs} queries x {passes} passes on {threads} threads, {dt:.2f}s per pass "
        f"({cpu_qps:.1f} QPS), {nbytes / 1e9:.2f} GB staged; one thread: {n1 / dt1:.1f} QPS")
    # parity of the sample: the GPU in the timed configuration, given the
    # oracle's logits for the whole batch
    lg_all = torch.from_numpy(O.encode(enc, Q.cpu().numpy())).to(dev)
    gi, gd = gix.nr_search(Q, w.k, P, params, logits=lg_all)
    gi, gd = gi[:nqs].cpu().numpy(), gd[:nqs].cpu().numpy()
    id_mis = int((gi != oi).any(1).sum())
    if w.dtype == "u8":
        d_mis = int((gd != od).any(1).sum())
    else:
        d_mis = int((~np.isclose(gd, od, rtol=1e-5, atol=1e-6)).any(1).sum())
    parity = {"queries": nqs, "id_mismatches": id_mis, "dist_mismatches": d_mis,
              "rule": "bit-exact ids and distances" if w.dtype == "u8"
              else "ids exact except fp32 near-ties; distances within 1e-5"}
    log("parity", parity)
    cpu = {"value": round(cpu_qps, 2), "unit": "queries/s", "cores": threads, "kind": "oracle",
           "cpu_model": host_cpu_model(), "affinity_cores": len(os.sched_getaffinity(0)),
           "sample": f"first {nqs} queries of the batch, same index and probe budget, timed over "
                     f"{passes} whole passes; rows of their candidate clusters "
                     f"({nbytes / 1e9:.2f} GB) staged in host memory before timing",
           "seconds": round(dt * passes, 3),
           "per_core": {"value": round(n1 / dt1, 2), "unit": "queries/s", "threads": 1,
                        "queries": n1},
           "stage_seconds_last_pass": dict(zip(("encode", "probe", "route", "refine"),
                                               [round(float(x), 3) for x in secs]))}
    return cpu, parity


if __name__ == "__main__":
    main()
