"""Oracle centroid stage (Algorithm 2, Sec. 3.4.2) and gate margin curve
(Sec. 3.4, "Centroid gating margin"): a hand-worked example, closed forms of
the gate-off / no-early-stop cases, and invariants."""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
from tests.instances import instance, oracle_encoder

GOLD = os.path.join(os.path.dirname(__file__), "golden")
INF = float("inf")


def fma32(a, b, c):
    """fmaf(a, b, c): the exact a*b+c rounded once to fp32 (ties to even)."""
    exact = Fraction(float(a)) * Fraction(float(b)) + Fraction(float(c))
    f = np.float32(float(exact))
    cands = [np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))]
    best = min(cands, key=lambda v: (abs(Fraction(float(v)) - exact),
                                     int(np.frombuffer(v.tobytes(), np.uint32)[0]) & 1))
    return np.float32(best)


def _micro():
    bc_off = np.array([0, 3, 4, 6, 8, 9, 11, 12], np.uint32)
    mu = np.array([1, 2, 3, 100, 0.5, 4, 5, 6, 100, 7, 8, 100], np.float32)[:, None]
    codes = np.arange(7, dtype=np.uint32)[None]
    bins = np.arange(7, dtype=np.int32)[None]
    return bc_off, mu, codes, bins


def _golden():
    rows = []
    for line in open(os.path.join(GOLD, "alg2_worked_example.txt")):
        if line.strip() and not line.startswith("#"):
            f = [c.strip() for c in line.split("|")]
            rows.append(dict(name=f[0], k_c=int(f[1]), t_low=int(f[2]), es=int(f[3]),
                             lowq_or=int(f[4]), exp=[int(x) for x in f[5].split()],
                             stopped=int(f[6]), alpha=float(f[7])))
    return rows


@pytest.mark.parametrize("case", _golden(), ids=lambda c: c["name"])
def test_worked_example(oracle_lib, case):
    bc_off, mu, codes, bins = _micro()
    prm = O.RouteParams(k_c=case["k_c"], b_batch=2, b_min=1, t_low=case["t_low"], u_heap=1,
                        u_front=1, alpha_front=case["alpha"], gate_on=True,
                        early_stop_on=bool(case["es"]),
                        lowq_or=bool(case["lowq_or"]), m_x=np.array([0.0]), m_y=np.array([10.0]))
    lists, st = O.route(np.zeros((1, 1), np.float32), codes, bins, np.array([7], np.int32),
                        bc_off, mu, prm, with_stats=True)
    assert lists[0].tolist() == case["exp"]
    assert st[0].stopped == case["stopped"]


def test_margin_curve(oracle_lib):
    mx = np.array([1.0, 2.0, 4.0], np.float32)
    my = np.array([0.5, 1.0, 1.0], np.float32)
    prm = O.RouteParams(m_x=mx, m_y=my)
    assert O.margin(prm, -3.0) == 0.5 and O.margin(prm, 1.0) == 0.5
    assert O.margin(prm, 9.0) == 1.0 and O.margin(prm, 4.0) == 1.0
    assert O.margin(prm, 1.5) == 0.75            # linear between knots (exact here)
    assert O.margin(prm, 3.0) == 1.0
    xs = np.linspace(-1, 6, 2001).astype(np.float32)
    ys = [O.margin(prm, float(x)) for x in xs]
    assert np.all(np.diff(ys) >= 0)               # monotone non-decreasing
    assert O.margin(O.RouteParams(), 5.0) == 0.0  # no knots: M == 0


@pytest.mark.parametrize("seed", range(6))
def test_gate_never_rises(oracle_lib, seed):
    """With knots of increasing x and non-decreasing y (the library rejects
    others), M is non-decreasing, and so is the fp32 gate x + M(x): as d_min
    falls the gate never rises, which is what lets the search prune the heap
    once by the last gate while no key is cut."""
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 9))
    mx = np.sort(rng.uniform(0.0, 20.0, m)).astype(np.float32)
    mx = np.unique(mx)
    my = np.sort(rng.uniform(0.0, 5.0, len(mx))).astype(np.float32)
    prm = O.RouteParams(m_x=mx, m_y=my)
    xs = np.sort(np.concatenate([rng.uniform(-2.0, 25.0, 3000), mx.astype(np.float64)])).astype(np.float32)
    ms = np.array([O.margin(prm, float(x)) for x in xs], np.float32)
    assert np.all(np.diff(ms) >= 0)
    theta = xs + ms  # fp32 additions, as the centroid stage forms the gate
    assert theta.dtype == np.float32 and np.all(np.diff(theta) >= 0)


def _probe_lists(cfg, n, nq, P, **ov):
    w, ix, X, Q = instance(cfg, n, nq, **ov)
    enc = oracle_encoder(ix)
    lg = O.encode(enc, Q)
    codes, costs, bins, cnt = O.probes(lg, ix.tau, w.l_sel, w.r_max, P)
    return w, ix, lg, codes, bins, cnt


def test_gate_off_no_stop_takes_every_probed_cluster(oracle_lib):
    w, ix, lg, codes, bins, cnt = _probe_lists(1, 0, 0, 32)
    prm = O.RouteParams(k_c=10 ** 9, gate_on=False, early_stop_on=False, b_batch=5)
    lists = O.route(lg, codes, bins, cnt, ix.bc_off, ix.centroids, prm)
    for q in range(len(lists)):
        exp = set()
        for c in codes[q, :cnt[q]]:
            exp |= set(range(int(ix.bc_off[c]), int(ix.bc_off[c + 1])))
        assert set(lists[q].tolist()) == exp
        assert len(lists[q]) == len(exp)


@pytest.mark.parametrize("k_c,b_batch", [(3, 2), (8, 5), (16, 64)])
def test_closed_form_without_early_stop(oracle_lib, k_c, b_batch):
    """H = the K_c smallest (d, id) among all scored centroids with d <= the
    final gate (the gate only tightens, so pruning H each batch equals one
    final cut); C_dir = every single-cluster probed bucket."""
    w, ix, lg, codes, bins, cnt = _probe_lists(1, 0, 0, 64)
    mx = np.array([0.0, 2.0, 8.0], np.float32)
    my = np.array([1.0, 3.0, 6.0], np.float32)
    prm = O.RouteParams(k_c=k_c, b_batch=b_batch, gate_on=True, early_stop_on=False, m_x=mx, m_y=my)
    lists, st = O.route(lg, codes, bins, cnt, ix.bc_off, ix.centroids, prm, with_stats=True)
    for q in range(len(lists)):
        single, scored = [], []
        for c in codes[q, :cnt[q]]:
            c0, c1 = int(ix.bc_off[c]), int(ix.bc_off[c + 1])
            if c1 - c0 == 1:
                single.append(c0)
            elif c1 - c0 >= 2:
                scored += list(range(c0, c1))
        dist = {}
        for c in scored:
            acc = np.float32(0)
            for j in range(lg.shape[1]):
                t = np.float32(lg[q, j] - ix.centroids[c, j])
                acc = fma32(t, t, acc)
            dist[c] = acc
        if scored:
            dmin = min(dist.values())
            theta = np.float32(dmin + np.float32(O.margin(prm, float(dmin))))
            keep = sorted((dist[c], c) for c in scored if dist[c] <= theta)[:k_c]
        else:
            keep = []
        assert lists[q].tolist() == single + [c for _, c in keep]
        assert st[q].h_size == len(keep) <= k_c


def test_early_stop_only_shrinks(oracle_lib):
    """Stopping early visits a prefix of the bins, so C(q) with early stop is
    never larger than without it and its C_dir is a prefix."""
    w, ix, lg, codes, bins, cnt = _probe_lists(1, 0, 0, 128)
    base = dict(k_c=4, b_batch=2, b_min=1, t_low=1, gate_on=True,
                m_x=np.array([0.0], np.float32), m_y=np.array([0.5], np.float32))
    on, st_on = O.route(lg, codes, bins, cnt, ix.bc_off, ix.centroids,
                        O.RouteParams(early_stop_on=True, **base), with_stats=True)
    off, st_off = O.route(lg, codes, bins, cnt, ix.bc_off, ix.centroids,
                          O.RouteParams(early_stop_on=False, **base), with_stats=True)
    n_stopped = 0
    for q in range(len(on)):
        assert st_on[q].n_dir <= st_off[q].n_dir
        assert on[q][:st_on[q].n_dir].tolist() == off[q][:st_on[q].n_dir].tolist()
        assert len(on[q]) <= len(off[q]) + 4
        n_stopped += st_on[q].stopped
        if st_on[q].stopped:
            assert st_on[q].h_size == 4          # stopping needs a full heap
    assert n_stopped > 0
