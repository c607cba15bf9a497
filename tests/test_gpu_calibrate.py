"""The calibration stage on the GPU (nr_calibrate; Sec. 3.4 "Calibration"):
the score of every target's bucket equals, bit for bit, the cost the
oracle's probe sequence gives that bucket (+inf where the enumeration cannot
reach it), and the margin points match the definition recomputed on the host
(x = best centroid distance among the targets' buckets, y = the farthest
target cluster's extra distance)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_15438_amd import neuroute as NR
from tests.instances import instance, oracle_encoder

pytestmark = pytest.mark.gpu

CASES = {
    "sift": (2, 60_000, 300, (("widths", (128, 256, 12)),)),
    "deep": (3, 40_000, 200, (("widths", (96, 256, 12)), ("capacity", 30))),
    "tiny": (1, 0, 0, ()),
}


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda")


def _host_targets(ix, ids):
    """Cluster and bucket (code) of every target id (-1: none)."""
    row_of_id = np.empty(len(ix.row_ids), np.int64)
    row_of_id[ix.row_ids] = np.arange(len(ix.row_ids))
    ok = ids >= 0
    rows = row_of_id[np.where(ok, ids, 0)]
    clus = np.searchsorted(ix.cl_off.astype(np.int64), rows, side="right") - 1
    code = np.searchsorted(ix.bc_off.astype(np.int64), clus, side="right") - 1
    return np.where(ok, clus, -1), np.where(ok, code, -1)


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("l_sel,r_max", [(8, 3), (12, 7)])
def test_bucket_scores_and_margin_points(dev, name, l_sel, r_max):
    cfg, n, nq, ov = CASES[name]
    w, ix, X, Q = instance(cfg, n, nq, **dict(ov))
    l_sel = min(l_sel, w.b)
    gix = NR.Index.from_built(ix, dev)
    lg = O.encode(oracle_encoder(ix), Q)
    K = 10
    tid, _ = O.bruteforce(X, Q, K)
    tid[::7, -3:] = -1                     # some short target lists
    scores, xy = gix.nr_calibrate(torch.from_numpy(lg).to(dev), torch.from_numpy(tid).to(dev),
                                  l_sel, r_max)
    scores, xy = scores.cpu().numpy(), xy.cpu().numpy()
    clus, code = _host_targets(ix, tid)
    # the whole enumeration of every query: cost of each reachable code
    from math import comb
    full = sum(comb(l_sel, r) for r in range(min(r_max, l_sel) + 1))
    oc, ocost, _, on = O.probes(lg, ix.tau, l_sel, r_max, full)
    assert np.all(on == full)
    for q in range(len(Q)):
        cost_of = dict(zip(oc[q].tolist(), ocost[q].tolist()))
        for j in range(K):
            if tid[q, j] < 0:
                assert np.isinf(scores[q, j])
                continue
            exp = np.float32(cost_of.get(int(code[q, j]), np.inf))
            assert scores[q, j].view(np.uint32) == exp.view(np.uint32), (q, j)
    # margin points against the definition in fp64
    cent = ix.centroids.astype(np.float64)
    bc = ix.bc_off.astype(np.int64)
    for q in range(len(Q)):
        ok = tid[q] >= 0
        cands = np.concatenate([np.arange(bc[c], bc[c + 1]) for c in np.unique(code[q][ok])])
        d = ((cent[cands] - lg[q].astype(np.float64)) ** 2).sum(1)
        x = d.min()
        dt = ((cent[clus[q][ok]] - lg[q].astype(np.float64)) ** 2).sum(1).max()
        assert abs(xy[q, 0] - x) <= 1e-5 * max(x, 1e-3), q
        assert abs(xy[q, 1] - (dt - x)) <= 1e-5 * max(dt, 1e-3), q
    gix.close()
