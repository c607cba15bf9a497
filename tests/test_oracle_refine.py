"""Oracle refinement and whole search (Sec. 3.1 problem statement, Sec. 3.4
exact refinement): at full budget the method must return the exact k-NN, which
brute force (itself pinned against NumPy's sort on exact distances) fixes."""
import numpy as np
import pytest

import oracle as O
from tests.instances import instance, oracle_encoder

FULL = dict(gate_on=False, early_stop_on=False)


def _np_knn(X, Q, k):
    """Exact k-NN by NumPy: exact squared distances, lexicographic (dist, id)."""
    Xd = X.astype(np.int64 if X.dtype == np.uint8 else np.float64)
    Qd = Q.astype(Xd.dtype)
    ids = np.empty((len(Q), k), np.int64)
    for q in range(len(Q)):
        d = ((Xd - Qd[q]) ** 2).sum(1)
        o = np.lexsort((np.arange(len(X)), d))[:k]
        ids[q] = o
    return ids


@pytest.mark.parametrize("dtype", ["u8", "f32"])
def test_bruteforce_matches_numpy_sort(oracle_lib, dtype):
    rng = np.random.default_rng(5)
    if dtype == "u8":
        X = rng.integers(0, 4, size=(3000, 16)).astype(np.uint8)   # many exact ties
        Q = rng.integers(0, 4, size=(20, 16)).astype(np.uint8)
    else:
        X = rng.standard_normal((3000, 12)).astype(np.float32)
        Q = rng.standard_normal((20, 12)).astype(np.float32)
    ids, dists = O.bruteforce(X, Q, 10, n_threads=3)
    assert np.array_equal(ids, _np_knn(X, Q, 10))
    ref = ((X[ids].astype(np.float64) - Q[:, None].astype(np.float64)) ** 2).sum(-1)
    assert np.array_equal(dists, ref.astype(np.float32))


def test_bruteforce_pads_short_base(oracle_lib):
    X = np.arange(12, dtype=np.float32).reshape(3, 4)
    ids, dists = O.bruteforce(X, X[:1], 5)
    assert ids[0].tolist() == [0, 1, 2, -1, -1]
    assert np.isinf(dists[0, 3:]).all()


@pytest.mark.parametrize("cfg,n,nq,b_over", [
    (1, 0, 0, None),                      # the tiny case: 20k f32, b=8
    (2, 30_000, 40, (128, 256, 10)),      # SIFT-like u8, b=10
])
def test_full_budget_equals_bruteforce(oracle_lib, cfg, n, nq, b_over):
    ov = {} if b_over is None else {"widths": b_over}
    w, ix, X, Q = instance(cfg, n, nq, **ov)
    b = w.b
    enc = oracle_encoder(ix)
    prm = O.RouteParams(k_c=10 ** 9, **FULL)
    ids, dists, ncand, _ = O.search(enc, ix.tau, ix.rows, ix.row_ids, ix.bc_off, ix.cl_off,
                                    ix.centroids, Q, 10, b, b, 1 << b, prm, n_threads=4)
    gi, gd = O.bruteforce(X, Q, 10)
    assert np.array_equal(ids, gi)
    assert np.array_equal(dists, gd)
    assert np.all(ncand == w.n)


def test_refine_distances_recompute_from_ids(oracle_lib):
    w, ix, X, Q = instance(2, 30_000, 40, widths=(128, 256, 10))
    enc = oracle_encoder(ix)
    prm = O.RouteParams(k_c=64)
    ids, dists, ncand, _ = O.search(enc, ix.tau, ix.rows, ix.row_ids, ix.bc_off, ix.cl_off,
                                    ix.centroids, Q, 10, 10, 7, 16, prm)
    ok = ids >= 0
    rec = ((X[ids[ok]].astype(np.int64) - np.repeat(Q, 10, 0).reshape(-1, 10, 128)[ok].astype(np.int64)) ** 2).sum(-1)
    assert np.array_equal(dists[ok], rec.astype(np.float32))
    # sorted by (distance, id)
    for q in range(len(Q)):
        n = int(ok[q].sum())
        pairs = list(zip(dists[q, :n].tolist(), ids[q, :n].tolist()))
        assert pairs == sorted(pairs)


def test_recall_monotone_in_budget_without_gate(oracle_lib):
    """Gate and early stop off: larger budgets probe a superset of buckets, so
    the candidate set grows and Recall@10 cannot drop."""
    w, ix, X, Q = instance(2, 30_000, 40, widths=(128, 256, 10))
    enc = oracle_encoder(ix)
    gi, _ = O.bruteforce(X, Q, 10)
    prev_r, prev_c = -1.0, None
    for P in (1, 4, 16, 64, 256):
        prm = O.RouteParams(k_c=10 ** 9, **FULL)
        ids, _, nc, _ = O.search(enc, ix.tau, ix.rows, ix.row_ids, ix.bc_off, ix.cl_off,
                                 ix.centroids, Q, 10, 10, 7, P, prm)
        r = O.recall_at_k(ids, gi, 10)
        assert r >= prev_r
        if prev_c is not None:
            assert np.all(nc >= prev_c)
        prev_r, prev_c = r, nc


def test_recall_formula():
    g = np.array([[1, 2, 3, 4]])
    assert O.recall_at_k(np.array([[1, 2, 3, 4]]), g, 4) == 1.0
    assert O.recall_at_k(np.array([[4, 3, 9, 8]]), g, 4) == 0.5
    assert O.recall_at_k(np.array([[7, 8, 9, -1]]), g, 4) == 0.0
    # |G| < k: divide by |G|
    assert O.recall_at_k(np.array([[5, 6, -1, -1]]), np.array([[5, 6, -1, -1]]), 4) == 1.0
    assert O.recall_at_k(np.array([[1, 9, 9, 9], [1, 2, 3, 4]]), g.repeat(2, 0), 4) == (0.25 + 1) / 2
