"""Calibration helpers (Sec. 3.4, "Calibration"): the bucket score of a
target equals the cost the enumeration gives that bucket (checked against
the oracle's probe sequence), unreachable buckets score +inf, and the S_max
fit reads the pair-coverage curve at the requested fraction."""
import numpy as np
import torch

import oracle as O
from paper_2608_15438_amd import calibrate as CAL


def _logits(nq, b, seed):
    rng = np.random.default_rng(seed)
    lg = rng.standard_normal((nq, b)).astype(np.float32)
    tau = (0.2 * rng.standard_normal(b)).astype(np.float32)
    return lg, tau


def test_bucket_scores_equal_enumeration_costs():
    b, l_sel, r_max, P = 12, 8, 4, 200
    lg, tau = _logits(40, b, 3)
    codes, costs, _, counts = O.probes(lg, tau, l_sel, r_max, P)
    sc = CAL.bucket_scores(torch.from_numpy(lg), torch.from_numpy(tau),
                           torch.from_numpy(codes.astype(np.int64)), l_sel, r_max).numpy()
    for q in range(len(lg)):
        n = counts[q]
        assert n > 0
        # the same fp32 value, bit for bit: same deviations, same rank order
        assert np.array_equal(sc[q, :n].view(np.uint32), costs[q, :n].view(np.uint32)), q


def test_unreachable_buckets_score_inf():
    b, l_sel, r_max = 10, 4, 2
    lg, tau = _logits(5, b, 7)
    dev = np.abs(lg - tau)
    qcode = ((lg >= tau).astype(np.int64) << np.arange(b)).sum(1)
    rank = np.argsort(dev, axis=1, kind="stable")
    tgt = np.zeros((5, 3), np.int64)
    for q in range(5):
        tgt[q, 0] = qcode[q] ^ (1 << int(rank[q, l_sel]))          # a dimension outside L_sel
        tgt[q, 1] = qcode[q] ^ sum(1 << int(rank[q, r]) for r in range(3))   # 3 > R_max flips
        tgt[q, 2] = qcode[q] ^ (1 << int(rank[q, 0])) ^ (1 << int(rank[q, 1]))
    sc = CAL.bucket_scores(torch.from_numpy(lg), torch.from_numpy(tau), torch.from_numpy(tgt),
                           l_sel, r_max).numpy()
    assert np.all(np.isinf(sc[:, 0])) and np.all(np.isinf(sc[:, 1]))
    exp = (np.take_along_axis(dev, rank[:, :1], 1)[:, 0] + np.take_along_axis(dev, rank[:, 1:2], 1)[:, 0])
    assert np.array_equal(sc[:, 2], exp.astype(np.float32))
    # a short list's missing target (-1) is never covered
    sc2 = CAL.bucket_scores(torch.from_numpy(lg), torch.from_numpy(tau),
                            torch.full((5, 1), -1, dtype=torch.int64), l_sel, r_max)
    assert torch.isinf(sc2).all()


def test_fit_s_max_reads_the_coverage_curve():
    scores = torch.tensor([[0.1, 0.2, 0.3, 0.4], [0.5, 0.6, 0.7, float("inf")]])
    s, pair, query = CAL.fit_s_max(scores, coverage=0.75)
    # 6 of 8 pairs at or below the 6th smallest score
    assert s == np.float32(0.6).item() or abs(s - 0.6) < 1e-7
    assert pair == 0.75 and query == 0.5
    s, pair, query = CAL.fit_s_max(scores, coverage=0.5)
    assert abs(s - 0.4) < 1e-7 and pair == 0.5 and query == 0.5
