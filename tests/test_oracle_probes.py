"""Oracle bucket enumeration (Algorithm 1, Sec. 3.4.1; Eq. 10; deviation
scores) pinned by hand-worked examples and by invariants of the method."""
import math
import os
from itertools import combinations

import numpy as np
import pytest

import oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _golden_rows():
    out = []
    for line in open(os.path.join(GOLD, "alg1_worked_examples.txt")):
        if not line.strip() or line.startswith("#"):
            continue
        f = [c.strip() for c in line.split("|")]
        out.append(dict(name=f[0], b=int(f[1]), tau=np.array(f[2].split(), np.float32),
                        logits=np.array(f[3].split(), np.float32), l_sel=int(f[4]),
                        r_max=int(f[5]), s_max=float(f[6]), n_bins=int(f[7]), P=int(f[8]),
                        codes=[int(x) for x in f[9].split()],
                        costs=[float(x) for x in f[10].split()],
                        bins=[int(x) for x in f[11].split()]))
    return out


@pytest.mark.parametrize("ex", _golden_rows(), ids=lambda e: e["name"])
def test_worked_examples(oracle_lib, ex):
    codes, costs, bins, cnt = O.probes(ex["logits"][None], ex["tau"], ex["l_sel"], ex["r_max"],
                                       ex["P"], ex["s_max"], ex["n_bins"])
    n = cnt[0]
    assert n == len(ex["codes"])
    assert codes[0, :n].tolist() == ex["codes"]
    assert costs[0, :n].tolist() == ex["costs"]
    assert bins[0, :n].tolist() == ex["bins"]


def _random_case(rng, b, ties=False):
    tau = rng.standard_normal(b).astype(np.float32)
    if ties:
        # many exact ties in delta and exact zeros
        lv = rng.integers(-3, 4, size=b).astype(np.float32) * 0.25
        return tau, tau + lv
    return tau, (tau + rng.standard_normal(b) * rng.uniform(0.01, 2.0)).astype(np.float32)


@pytest.mark.parametrize("seed", range(12))
def test_invariants(oracle_lib, seed):
    rng = np.random.default_rng(seed)
    b = int(rng.integers(3, 13))
    l_sel = int(rng.integers(1, b + 1))
    r_max = int(rng.integers(1, l_sel + 1))
    tau, lg = _random_case(rng, b, ties=seed % 2 == 0)
    full = sum(math.comb(l_sel, r) for r in range(r_max + 1))
    P = int(rng.integers(1, full + 3))
    codes, costs, bins, cnt = O.probes(lg[None], tau, l_sel, r_max, P)
    n = int(cnt[0])
    c, s = codes[0, :n], costs[0, :n]
    a = (lg >= tau)
    b0 = int(sum(int(a[j]) << j for j in range(b)))
    assert n == min(P, full)                       # count of flip sets within the radius
    assert c[0] == b0 and s[0] == 0.0               # the base address comes first
    assert np.all(np.diff(s) >= 0)                  # scores never decrease
    assert len(set(c.tolist())) == n                # distinct buckets
    delta = np.abs(lg - tau)
    order = sorted(range(b), key=lambda j: (delta[j], j))
    S = set(order[:l_sel])
    for code, cost in zip(c, s):
        flips = [j for j in range(b) if ((int(code) ^ b0) >> j) & 1]
        assert len(flips) <= r_max                  # radius
        assert set(flips) <= S                      # only the least stable dims flip
        # the score is the sum of the flipped deltas, added in rank order
        acc = np.float32(0)
        for j in sorted(flips, key=lambda j: order.index(j)):
            acc = np.float32(acc + delta[j])
        assert acc == cost
    assert bins[0, :n].tolist() == list(range(n))    # S_max = inf: one bin per probe


@pytest.mark.parametrize("seed", range(6))
def test_prefix_property(oracle_lib, seed):
    rng = np.random.default_rng(100 + seed)
    b = 10
    tau, lg = _random_case(rng, b, ties=True)
    big = O.probes(lg[None], tau, 10, 5, 400)
    for P in (1, 7, 64, 200):
        small = O.probes(lg[None], tau, 10, 5, P)
        n = small[3][0]
        assert np.array_equal(small[0][0, :n], big[0][0, :n])
        assert np.array_equal(small[1][0, :n], big[1][0, :n])


@pytest.mark.parametrize("b", [1, 5, 8, 11])
def test_full_budget_covers_every_code(oracle_lib, b):
    rng = np.random.default_rng(b)
    tau, lg = _random_case(rng, b)
    codes, costs, bins, cnt = O.probes(lg[None], tau, b, b, 1 << b)
    assert cnt[0] == 1 << b
    assert sorted(codes[0].tolist()) == list(range(1 << b))


def test_order_matches_exhaustive_sort(oracle_lib):
    """All flip sets by brute force over itertools.combinations, sorted by
    (score, rank mask): the oracle's sequence is that sort, cut to P."""
    rng = np.random.default_rng(7)
    for trial in range(20):
        b = 9
        tau, lg = _random_case(rng, b, ties=trial % 2 == 0)
        l_sel, r_max = 7, 4
        delta = np.abs(lg - tau)
        order = sorted(range(b), key=lambda j: (delta[j], j))[:l_sel]
        items = []
        for r in range(r_max + 1):
            for comb in combinations(range(l_sel), r):
                acc = np.float32(0)
                for rr in comb:
                    acc = np.float32(acc + delta[order[rr]])
                items.append((float(acc), sum(1 << rr for rr in comb)))
        items.sort()
        codes, costs, bins, cnt = O.probes(lg[None], tau, l_sel, r_max, 50)
        b0 = int(sum(int(lg[j] >= tau[j]) << j for j in range(b)))
        exp_codes = []
        for cost, m in items[:50]:
            c = b0
            for rr in range(l_sel):
                if m >> rr & 1:
                    c ^= 1 << order[rr]
            exp_codes.append(c)
        assert codes[0, :cnt[0]].tolist() == exp_codes
        assert costs[0, :cnt[0]].tolist() == [it[0] for it in items[:50]]


def test_finite_smax_bins(oracle_lib):
    rng = np.random.default_rng(3)
    tau, lg = _random_case(rng, 12)
    s_max, nb = 1.5, 7
    codes, costs, bins, cnt = O.probes(lg[None], tau, 12, 4, 3000, s_max, nb)
    n = cnt[0]
    s = costs[0, :n]
    assert np.all(s[1:] <= np.float32(s_max))
    scale = np.float32(nb) / np.float32(s_max)
    exp = np.minimum(nb - 1, np.floor((s * scale).astype(np.float32)).astype(np.int64))
    assert bins[0, :n].tolist() == exp.tolist()
    assert np.all(np.diff(bins[0, :n]) >= 0)
