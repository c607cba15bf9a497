"""Seeded input generators: Philox known answers, determinism, shapes."""
import os

import numpy as np

from synth import generators as G
from synth.philox import philox4x32_10

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_philox_known_answers():
    rows = [l.split() for l in open(os.path.join(GOLD, "philox4x32_10_kat.txt"))
            if l.strip() and not l.startswith("#")]
    assert len(rows) == 3
    for r in rows:
        v = [int(x, 16) for x in r]
        out = philox4x32_10(*v[:4], v[4], v[5])
        assert [int(o) for o in out] == v[6:10]


def test_irwin_hall_moments():
    z = G.irwin_hall_normals(11, np.arange(4000), 64)
    assert abs(z.mean()) < 0.01
    assert abs(z.std() - 1.0) < 0.01
    assert z.min() >= -6.0 and z.max() <= 6.0


def test_rows_are_addressable_and_deterministic():
    c = G.sift_centers(5, 20, 128)
    a = G.sift_rows(7, c, np.arange(100))
    b = G.sift_rows(7, c, np.array([42, 3, 99]))
    assert np.array_equal(a[[42, 3, 99]], b)
    assert np.array_equal(a, G.sift_rows(7, c, np.arange(100)))
    assert not np.array_equal(a, G.sift_rows(8, c, np.arange(100)))
    assert a.dtype == np.uint8


def test_deep_rows_unit_norm():
    c = G.unit_centers(3, 10, 96)
    x = G.deep_rows(3, c, np.arange(200))
    assert x.dtype == np.float32
    assert np.allclose(np.linalg.norm(x.astype(np.float64), axis=1), 1.0, atol=1e-6)


def test_component_draw_uniform():
    comp = G.component_of(9, np.arange(100000), 10)
    cnt = np.bincount(comp, minlength=10)
    assert cnt.min() > 9500 and cnt.max() < 10500


def test_xavier_bounds():
    w = G.xavier_uniform(1, 0, 256, 128)
    a = np.sqrt(6.0 / 384)
    assert w.shape == (256, 128)
    assert np.abs(w).max() <= a
    assert abs(w.std() - a / np.sqrt(3)) < 0.01 * a
