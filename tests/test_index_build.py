"""Index construction (Sec. 3.3, Sec. 3.2.3): every base vector lands in
exactly one bucket, buckets follow the oracle's own encoder + Eq. 10, the
CSR directory tiles the permuted payload, centroids are cluster means."""
import numpy as np
import pytest

import oracle as O
from synth import configs as CF
from paper_2608_15438_amd import index_build as IB
from tests.instances import instance, oracle_encoder

CASES = [(1, 0, 0, {}), (2, 30_000, 10, {"widths": (128, 256, 10)}),
         (3, 20_000, 10, {"widths": (96, 256, 9), "capacity": 40}),
         (2, 30_000, 10, {"widths": (128, 256, 10), "cluster_rule": "none"})]


@pytest.mark.parametrize("cfg,n,nq,ov", CASES)
def test_index_structure(oracle_lib, cfg, n, nq, ov):
    w, ix, X, Q = instance(cfg, n, nq, **ov)
    b = w.b
    nb = 1 << b
    bc = ix.bc_off.astype(np.int64)
    cl = ix.cl_off.astype(np.int64)
    assert bc.shape == (nb + 1,) and bc[0] == 0 and np.all(np.diff(bc) >= 0)
    assert bc[-1] == ix.n_clusters
    assert cl.shape == (ix.n_clusters + 1,) and cl[0] == 0 and cl[-1] == w.n
    assert np.all(np.diff(cl) > 0)                          # no empty cluster
    assert np.array_equal(np.sort(ix.row_ids), np.arange(w.n))   # a permutation
    assert np.array_equal(ix.rows, X[ix.row_ids])             # payload = permuted base
    # each permuted row's bucket is the binarised oracle logit of that row
    lg = O.encode(oracle_encoder(ix), X)
    codes = ((lg >= ix.tau) * (1 << np.arange(b))).sum(1)
    cl_of_row = np.repeat(np.arange(ix.n_clusters), np.diff(cl))
    bucket_of_cl = np.repeat(np.arange(nb), np.diff(bc))
    assert np.array_equal(bucket_of_cl[cl_of_row], codes[ix.row_ids])
    # rows of a cluster are in original-id order, clusters of a bucket contiguous
    for c in range(0, ix.n_clusters, max(1, ix.n_clusters // 200)):
        r = ix.row_ids[cl[c]:cl[c + 1]]
        assert np.all(np.diff(r) > 0)
        mean = lg[r].astype(np.float64).mean(0)
        assert np.allclose(ix.centroids[c], mean, rtol=1e-5, atol=1e-6)


def test_tau_is_lower_median(oracle_lib):
    w, ix, X, Q = instance(2, 30_000, 10, widths=(128, 256, 10))
    lg = O.encode(oracle_encoder(ix), X)          # n <= 2^20: the sample is the whole base
    s = np.sort(lg, axis=0)
    assert np.array_equal(ix.tau, s[(len(lg) - 1) // 2])


def test_cluster_count_rules(oracle_lib):
    w, ix, X, Q = instance(1)
    k_b = np.diff(ix.bc_off.astype(np.int64))
    sizes = np.bincount(np.repeat(np.arange(1 << w.b), k_b),
                        weights=np.diff(ix.cl_off.astype(np.int64)), minlength=1 << w.b)
    # tiny case: min(4, |B|) clusters per non-empty bucket (k-means may drop empties)
    assert np.all(k_b <= np.minimum(4, sizes))
    assert np.all((k_b >= 1) == (sizes >= 1))
    w3, ix3, _, _ = instance(3, 20_000, 10, widths=(96, 256, 9), capacity=40)
    kb3 = np.diff(ix3.bc_off.astype(np.int64))
    sz3 = np.bincount(np.repeat(np.arange(1 << w3.b), kb3),
                      weights=np.diff(ix3.cl_off.astype(np.int64)), minlength=1 << w3.b)
    assert np.all(kb3 <= np.ceil(sz3 / 40))
    assert np.all(kb3[sz3 <= 40] == (sz3[sz3 <= 40] > 0))   # small buckets: one cluster


def test_no_clustering_rule(oracle_lib):
    # the ablation without bucket-local clustering: a bucket is one cluster,
    # whose centroid is the mean logit of the whole bucket
    w, ix, X, Q = instance(2, 30_000, 10, widths=(128, 256, 10), cluster_rule="none")
    k_b = np.diff(ix.bc_off.astype(np.int64))
    assert np.all(k_b <= 1)
    lg = O.encode(oracle_encoder(ix), X)
    codes = ((lg >= ix.tau) * (1 << np.arange(w.b))).sum(1)
    sizes = np.bincount(codes, minlength=1 << w.b)
    assert np.array_equal(k_b, (sizes > 0).astype(np.int64))
    cl = ix.cl_off.astype(np.int64)
    assert np.array_equal(np.diff(cl), sizes[sizes > 0])


def test_build_is_deterministic(oracle_lib):
    w = CF.scaled(CF.TINY, 3000, 5)
    X = IB.cpu_row_source(w)(np.arange(w.n))
    a = IB.to_numpy(IB.build_index(w, IB.array_row_source(X)))
    b = IB.to_numpy(IB.build_index(w, IB.array_row_source(X)))
    for f in ("rows", "row_ids", "bc_off", "cl_off", "centroids"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
