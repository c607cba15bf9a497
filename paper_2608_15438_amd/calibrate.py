"""Calibration of the centroid-stage gate margin M(x) (Sec. 3.4, "Centroid
gating margin") and of the bucket-score cutoff S_max ("Bucket-score
cutoff"), untimed and shared by both search paths.  The per-query inputs
come from the library's calibration kernel (gpu_calibration); the PyTorch
versions below define the same quantities and serve the CPU checks.

For each calibration query with known top-K targets: x = the best centroid
distance among all centroids of the buckets that hold its targets, y = the
extra margin the farthest target's cluster needs to pass the gate x + y.
Queries are grouped into equal-frequency bins of x; a high quantile of y per
bin gives one knot (at the bin's median x); a running maximum makes the curve
monotone.  Distances are squared L2 in logit space.
"""
from __future__ import annotations

import numpy as np
import torch


def margin_points(logits: torch.Tensor, gt_ids: torch.Tensor, row_of_id: torch.Tensor,
                  cl_off: torch.Tensor, bc_off: torch.Tensor, centroids: torch.Tensor):
    """Per calibration query (x, y); all tensors on one device.

    logits [nq, b] fp32, gt_ids [nq, K] original ids, row_of_id [n] permuted
    row of each original id, cl_off/bc_off int64 offsets, centroids [C, b]."""
    nq, K = gt_ids.shape
    rows = row_of_id[gt_ids.reshape(-1)]
    clus = torch.searchsorted(cl_off, rows, right=True) - 1            # cluster of each target
    buck = torch.searchsorted(bc_off, clus, right=True) - 1            # bucket of each cluster
    xs, ys = [], []
    clus = clus.view(nq, K)
    buck = buck.view(nq, K)
    for q in range(nq):
        bks = torch.unique(buck[q])
        c0, c1 = bc_off[bks], bc_off[bks + 1]
        all_c = torch.cat([torch.arange(int(a), int(b), device=logits.device) for a, b in zip(c0, c1)])
        d_all = ((centroids[all_c].double() - logits[q].double()) ** 2).sum(1)
        d_tgt = ((centroids[clus[q]].double() - logits[q].double()) ** 2).sum(1)
        x = float(d_all.min())
        xs.append(x)
        ys.append(float(d_tgt.max()) - x)
    return np.array(xs), np.array(ys)


def fit_margin(xs: np.ndarray, ys: np.ndarray, quantile: float = 0.95, n_bins: int = 10):
    """Knots (m_x, m_y) of the monotone piecewise-linear M(x)."""
    order = np.argsort(xs, kind="stable")
    xs, ys = xs[order], ys[order]
    groups = np.array_split(np.arange(len(xs)), min(n_bins, max(1, len(xs))))
    mx, my = [], []
    for g in groups:
        if len(g) == 0:
            continue
        mx.append(float(np.float32(np.median(xs[g]))))
        my.append(float(np.float32(np.quantile(ys[g], quantile))))
    my = list(np.maximum.accumulate(np.maximum(np.array(my), 0.0)))
    # knots need strictly increasing x
    kx, ky = [], []
    for x, y in zip(mx, my):
        if kx and x <= kx[-1]:
            ky[-1] = max(ky[-1], y)
            continue
        kx.append(x)
        ky.append(y)
    return np.array(kx, np.float32), np.array(ky, np.float32)


# --------------------------------------------------------------------------
# bootstrapped supervision and the bucket-score cutoff S_max (Sec. 3.4,
# "Calibration"): the calibration top-K lists come from the search itself run
# with a larger budget, and S_max from the enumeration scores of the buckets
# that hold those targets
# --------------------------------------------------------------------------

def bootstrap_targets(gix, queries: torch.Tensor, k: int, probe_budget: int, params):
    """Top-k original ids of the calibration queries from the search run in a
    higher-recall setting (the caller passes the enlarged budget and loose
    parameters, e.g. gate and early stop off); [nq, k] int64 on the device."""
    ids, _ = gix.nr_search(queries, k, probe_budget, params)
    return ids


def target_codes(gt_ids: torch.Tensor, row_of_id: torch.Tensor, cl_off: torch.Tensor,
                 bc_off: torch.Tensor) -> torch.Tensor:
    """Bucket (= code) of every target: original id -> permuted row ->
    cluster -> bucket; ids < 0 (short lists) give -1."""
    ok = gt_ids >= 0
    rows = row_of_id[gt_ids.clamp(min=0).reshape(-1)]
    clus = torch.searchsorted(cl_off, rows, right=True) - 1
    buck = torch.searchsorted(bc_off, clus, right=True) - 1
    return torch.where(ok, buck.view(gt_ids.shape), torch.full_like(gt_ids, -1))


def bucket_scores(logits: torch.Tensor, tau: torch.Tensor, codes: torch.Tensor, l_sel: int,
                  r_max: int) -> torch.Tensor:
    """Enumeration score of each target bucket, fp32 [nq, K]: the query's
    code is its logits' signs against tau; a bucket differs from it in a set
    of dimensions, reachable when all of them are among the l_sel with the
    smallest deviation |l - tau| (ties by dimension) and there are at most
    r_max; its score is then the fp32 sum of those deviations added in rank
    order, as the enumeration adds them.  Unreachable buckets score +inf."""
    nq, b = logits.shape
    lg = logits.float()
    t = tau.float().view(1, b)
    qcode = ((lg >= t).long() << torch.arange(b, device=lg.device)).sum(1)     # [nq]
    dev = (lg - t).abs()                                                        # [nq, b]
    # rank order: (deviation, dimension); argsort of a stable sort on deviation
    order = torch.sort(dev, dim=1, stable=True).indices                        # dim of rank r
    d_rank = torch.gather(dev, 1, order)                                       # deviation of rank r
    diff = codes ^ qcode.view(nq, 1)                                            # [nq, K] flipped bits
    flipped = ((diff.unsqueeze(2) >> order.unsqueeze(1)) & 1).bool()          # [nq, K, b] by rank
    n_flip = flipped.sum(2)
    outside = (flipped[:, :, l_sel:]).any(2) if l_sel < b else torch.zeros_like(n_flip, dtype=torch.bool)
    s = torch.zeros(codes.shape, dtype=torch.float32, device=lg.device)
    for r in range(b):                       # fp32, rank order; adding +0.0 changes nothing
        s = s + torch.where(flipped[:, :, r], d_rank[:, r:r + 1].expand_as(s), torch.zeros_like(s))
    bad = outside | (n_flip > r_max) | (codes < 0)
    return torch.where(bad, torch.full_like(s, float("inf")), s)


def gpu_calibration(gix, logits: torch.Tensor, targets: torch.Tensor, l_sel: int, r_max: int):
    """Bucket scores [nq, K] and margin points (xs, ys) of the calibration
    queries from the library's calibration kernel (nr_calibrate): the
    enumeration's own score of each target bucket, and x / y in the search's
    own squared latent distance.  Queries without targets are dropped."""
    scores, xy = gix.nr_calibrate(logits.float().contiguous(), targets.contiguous(), l_sel, r_max)
    ok = torch.isfinite(xy[:, 0])
    return scores, xy[ok, 0].double().cpu().numpy(), xy[ok, 1].double().cpu().numpy()


def fit_s_max(scores: torch.Tensor, coverage: float = 0.95):
    """S_max: the smallest score that covers the given fraction of all
    (query, target) pairs; also returns the pair coverage and the fraction of
    queries whose whole top-K it covers (the two coverage curves of the
    calibration, read at that threshold)."""
    flat = scores.reshape(-1).double()
    srt = torch.sort(flat).values
    i = min(len(srt) - 1, max(0, int(np.ceil(coverage * len(srt))) - 1))
    s_max = float(srt[i])
    pair_cov = float((flat <= s_max).double().mean())
    query_cov = float((scores <= s_max).all(1).double().mean())
    return s_max, pair_cov, query_cov
