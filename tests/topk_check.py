"""Validity of a GPU top-k list against the oracle's (Sec. 3.1: the k rows of
the candidate set nearest to the query, ties by lower original id).

uint8 distances are exact integers on both sides, so ids and distances must
be equal.  fp32 rows are summed in fp64 by the oracle and in fp32 on the GPU,
so a list may differ from the oracle's only at a near-tie (R27): the rows in
which the two lists differ must all lie within 2e-5 (relative) of the
oracle's k-th distance.  Whatever the ids, every GPU list must be a valid
top-k list: ids distinct, drawn from the rows of C(q), sorted by (distance,
id), each distance equal to a recomputation from its id within 1e-5, and the
padding (-1, +inf) where the oracle pads.
"""
from __future__ import annotations

import numpy as np

DIST_RTOL = 1e-5
TIE_RTOL = 2e-5

# near-tie count over the session, reported by conftest's terminal summary
NEAR_TIES = {"queries": 0, "near_ties": 0}


def allowed_ids(cl_off, row_ids, clusters) -> np.ndarray:
    """Original ids of every row of the given clusters (sorted)."""
    cl = np.asarray(cl_off, np.int64)
    c = np.asarray(clusters, np.int64)
    if len(c) == 0:
        return np.zeros(0, np.int64)
    s, e = cl[c], cl[c + 1]
    idx = np.concatenate([np.arange(a, b) for a, b in zip(s, e)]) if len(c) else np.zeros(0)
    return np.sort(np.asarray(row_ids)[idx.astype(np.int64)])


def exact_dists(X_by_id, q_row, ids) -> np.ndarray:
    """fp64 squared distances of the rows with these original ids."""
    x = np.asarray(X_by_id(ids)).astype(np.float64)
    return ((x - np.asarray(q_row).astype(np.float64)) ** 2).sum(1)


def check_topk(gi, gd, oi, od, *, is_u8, X_by_id=None, Q=None, allowed=None) -> int:
    """Assert that GPU lists (gi, gd) agree with the oracle's (oi, od);
    returns the number of fp32 near-tie queries.  X_by_id(ids) returns the
    rows of the given original ids; allowed(q) the sorted original ids of the
    rows of C(q) (None: not checked)."""
    gi, gd, oi, od = map(np.asarray, (gi, gd, oi, od))
    assert gi.shape == oi.shape and gd.shape == od.shape
    if is_u8:
        assert np.array_equal(gi, oi), np.nonzero((gi != oi).any(1))[0][:10]
        assert np.array_equal(gd, od)
        NEAR_TIES["queries"] += len(gi)
        return 0
    ties = 0
    for q in range(len(oi)):
        ok = oi[q] >= 0
        assert np.array_equal(gi[q] >= 0, ok), q
        n = int(ok.sum())
        assert np.all(np.isinf(gd[q, n:])) and np.all(gi[q, n:] == -1), q
        ids, ds = gi[q, :n], gd[q, :n]
        # distinct ids, sorted by (distance, id)
        assert len(np.unique(ids)) == n, q
        for j in range(n - 1):
            assert ds[j] < ds[j + 1] or (ds[j] == ds[j + 1] and ids[j] < ids[j + 1]), (q, j)
        if allowed is not None:
            a = allowed(q)
            pos = np.searchsorted(a, ids)
            assert np.all(pos < len(a)) and np.array_equal(a[np.minimum(pos, len(a) - 1)], ids), q
        if X_by_id is not None and n:
            true = exact_dists(X_by_id, Q[q], ids)
            assert np.all(np.abs(ds - true) <= DIST_RTOL * true + 1e-6), q
        if np.array_equal(ids, oi[q, :n]):
            assert np.allclose(ds, od[q, :n], rtol=DIST_RTOL, atol=1e-6), q
            continue
        # a near-tie: the rows only one side lists straddle the oracle's k-th
        # distance within the tolerance
        ties += 1
        kth = float(od[q, n - 1])
        g_only = np.setdiff1d(ids, oi[q, :n])
        o_only = np.setdiff1d(oi[q, :n], ids)
        assert len(g_only) == len(o_only), q
        if X_by_id is not None:
            tg = exact_dists(X_by_id, Q[q], g_only)
            to = exact_dists(X_by_id, Q[q], o_only)
            assert np.all(tg <= kth * (1 + TIE_RTOL) + 1e-6), q
            assert np.all(to >= kth * (1 - TIE_RTOL) - 1e-6), q
        else:
            gpos = np.isin(ids, g_only)
            assert np.all(ds[gpos] <= kth * (1 + TIE_RTOL) + 1e-6), q
    NEAR_TIES["queries"] += len(oi)
    NEAR_TIES["near_ties"] += ties
    return ties
