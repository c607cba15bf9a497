"""The top-k validity check used by the parity tests catches the mistakes a
GPU list could make: a repeated row, a wrong order, a row outside C(q), a
distance that does not match its id, a clearly better row left out."""
import numpy as np
import pytest

import oracle as O
from tests.topk_check import allowed_ids, check_topk

rng = np.random.default_rng(11)
X = rng.normal(size=(400, 8)).astype(np.float32)
Q = rng.normal(size=(3, 8)).astype(np.float32)
CL_OFF = np.array([0, 100, 250, 400], np.uint64)
ROW_IDS = np.arange(400, dtype=np.int64)
LISTS = [np.array([0, 1], np.uint32), np.array([2], np.uint32), np.array([0, 2], np.uint32)]


def _oracle():
    return O.refine(X, ROW_IDS, CL_OFF, Q, LISTS, 5)[:2]


def _check(gi, gd, oi, od):
    return check_topk(gi, gd, oi, od, is_u8=False, X_by_id=lambda ids: X[ids], Q=Q,
                      allowed=lambda q: allowed_ids(CL_OFF, ROW_IDS, LISTS[q]))


def test_oracle_list_passes():
    oi, od = _oracle()
    assert _check(oi.copy(), od.copy(), oi, od) == 0


@pytest.mark.parametrize("mistake", ["repeat", "order", "outside", "distance", "missed"])
def test_planted_mistakes_fail(mistake):
    oi, od = _oracle()
    gi, gd = oi.copy(), od.copy()
    if mistake == "repeat":          # one near row listed twice
        gi[0, 4], gd[0, 4] = gi[0, 3], gd[0, 3]
    elif mistake == "order":
        gi[1, [1, 2]], gd[1, [1, 2]] = gi[1, [2, 1]], gd[1, [2, 1]]
    elif mistake == "outside":       # a row of cluster 1, which query 1 does not list
        gi[1, 4] = 150
        gd[1, 4] = ((X[150].astype(np.float64) - Q[1]) ** 2).sum()
    elif mistake == "distance":
        gd[2, 0] *= 1.001
    else:                            # the best row replaced by the oracle's 6th
        o6, d6 = O.refine(X, ROW_IDS, CL_OFF, Q, LISTS, 6)[:2]
        gi[0] = np.concatenate([o6[0, 1:6]])
        gd[0] = d6[0, 1:6]
    with pytest.raises(AssertionError):
        _check(gi, gd, oi, od)


def test_near_tie_is_counted():
    """Two rows at the same distance from the query: the oracle keeps the
    lower id; a list holding the other one is still valid (a near-tie)."""
    Xt = np.zeros((4, 2), np.float32)
    Xt[:, 0] = [1.0, 2.0, 2.0, 3.0]
    q = np.zeros((1, 2), np.float32)
    oi = np.array([[0, 1]])
    od = np.array([[1.0, 4.0]], np.float32)
    gi = np.array([[0, 2]])
    gd = od.copy()
    assert check_topk(gi, gd, oi, od, is_u8=False, X_by_id=lambda ids: Xt[ids], Q=q) == 1
    with pytest.raises(AssertionError):   # uint8 lists must be equal
        check_topk(gi, gd, oi, od, is_u8=True)
