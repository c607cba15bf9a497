"""Small seeded search instances shared by the tests (built on the CPU with
the index builder; every input comes from the seeded generators)."""
from __future__ import annotations

import functools
from dataclasses import replace

import numpy as np

from synth import configs as CF
from paper_2608_15438_amd import index_build as IB


@functools.lru_cache(maxsize=None)
def instance(cfg: int, n: int = 0, n_queries: int = 0, **overrides):
    """(workload, host index, base rows in original order, queries)."""
    w = CF.WORKLOADS[cfg]
    if n or n_queries or overrides:
        w = CF.scaled(w, n or w.n, n_queries or w.n_queries, **overrides)
    X = IB.cpu_row_source(w)(np.arange(w.n))
    Q = IB.cpu_row_source(w, "query")(np.arange(w.n_queries))
    ix = IB.to_numpy(IB.build_index(w, IB.array_row_source(X)))
    return w, ix, X, Q


def oracle_encoder(ix):
    import oracle as O
    e = ix.encoder
    return O.Encoder(e.weights, e.biases, e.bn_scale or (), e.bn_shift or (), e.input_scale)
