"""Calibration of the centroid-stage gate margin M(x) (Sec. 3.4, "Centroid
gating margin"), untimed and shared by both search paths.

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
