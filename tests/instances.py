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


def head_bytes_for(w) -> int:
    """Head size of the split layout used by the tests and the benchmark:
    the first 16 dimensions of a row."""
    return 16 * (1 if w.dtype == "u8" else 4)


def split_index(ix, dev, copy=False):
    """A device copy of a row-major host index with a head plane, followed by
    the tails or (copy) by the whole rows."""
    import torch
    from dataclasses import replace as dc_replace
    w = ix.workload
    H = head_bytes_for(w)
    rows = torch.from_numpy(np.ascontiguousarray(ix.rows)).to(dev)
    return dc_replace(ix, rows=IB.split_payload([rows], w.n, w.row_bytes, H, dev, copy=copy),
                      head_bytes=H, head_copy=int(copy))


def oracle_encoder(ix):
    import oracle as O
    e = ix.encoder
    return O.Encoder(e.weights, e.biases, e.bn_scale or (), e.bn_shift or (), e.input_scale)


def stage_rows(ix, lists):
    """Host copies of only the rows the given cluster lists touch, behind a
    cl_off in which every other cluster is empty (index arrays may live on
    the GPU).  Returns (rows, row_ids, cl_off) for the oracle."""
    import torch
    cl = ix.cl_off.cpu().numpy().astype(np.int64) if hasattr(ix.cl_off, "cpu") else \
        np.asarray(ix.cl_off).astype(np.int64)
    need = np.unique(np.concatenate([np.asarray(x, np.int64) for x in lists]))
    sizes = cl[need + 1] - cl[need]
    idx = np.repeat(cl[need], sizes) + (np.arange(int(sizes.sum())) -
                                         np.repeat(np.cumsum(sizes) - sizes, sizes))
    if isinstance(ix.rows, torch.Tensor):
        it = torch.from_numpy(idx).to(ix.rows.device)
        rows = IB.payload_rows(ix, it).cpu().numpy()
        ids = ix.row_ids[it].cpu().numpy()
    else:
        rows, ids = ix.rows[idx], ix.row_ids[idx]
    n_cl = len(cl) - 1
    cnt = np.zeros(n_cl, np.int64)
    cnt[need] = sizes
    cl2 = np.zeros(n_cl + 1, np.uint64)
    cl2[1:] = np.cumsum(cnt)
    return rows, ids, cl2
