"""NeuRoute search oracle -- TEST INFRASTRUCTURE ONLY.

A plain, slow CPU implementation (``oracle.c``) of the batched query-time
search of NeuRoute (arXiv 2608.15438) plus NumPy helpers.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it; the product package never imports it.  It shares no code with the GPU
path.

Readings of the paper that the oracle takes are listed next to each C
function; "parity unpinned" marks the ones no test can tie to the paper.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")

OR_U8, OR_F32 = 0, 1


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc (plain C11, no FP contraction)."""
    src = os.path.join(_HERE, "oracle.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                               "-fPIC", "-shared", "-pthread", "-Wall", "-Wno-unused-function",
                               "-o", tmp, src, "-lm"])
        os.replace(tmp, _SO)
    return _SO


class _Encoder(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("widths", C.POINTER(C.c_int32)),
                ("params", C.POINTER(C.c_float)), ("input_scale", C.c_double),
                ("in_dtype", C.c_int32)]


class _RouteParams(C.Structure):
    _fields_ = [("n_bins", C.c_int32), ("s_max", C.c_float),
                ("k_c", C.c_int32), ("b_batch", C.c_int32), ("b_min", C.c_int32),
                ("t_low", C.c_int32), ("u_heap", C.c_int32), ("u_front", C.c_int32),
                ("alpha_front", C.c_float), ("gate_on", C.c_int32), ("early_stop_on", C.c_int32),
                ("lowq_or", C.c_int32), ("m_knots", C.c_int32),
                ("m_x", C.POINTER(C.c_float)), ("m_y", C.POINTER(C.c_float))]


class RouteStats(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("n_probes", "n_nonempty", "n_singleton", "n_scored",
                                         "n_batches", "bins_done", "stopped", "h_size", "n_dir")]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build(force=False)
        L = C.CDLL(_SO)
        P = C.c_void_p
        L.or_encode.argtypes = [C.POINTER(_Encoder), P, C.c_int64, P, P]
        L.or_probes.argtypes = [P, C.c_int64, C.c_int32, P, C.c_int32, C.c_int32, C.c_float,
                                C.c_int32, C.c_int32, P, P, P, P]
        L.or_margin.argtypes = [C.POINTER(_RouteParams), C.c_float]
        L.or_margin.restype = C.c_float
        L.or_route.argtypes = [P, C.c_int64, C.c_int32, P, P, P, C.c_int32, P, P, C.c_int64,
                               C.POINTER(_RouteParams), P, C.c_int64, P, P]
        L.or_refine.argtypes = [P, C.c_int32, C.c_int32, P, P, P, C.c_int64, P, C.c_int64, P,
                                C.c_int32, P, P, P]
        L.or_search.argtypes = [C.POINTER(_Encoder), P, C.c_int32, P, C.c_int32, C.c_int32, P, P,
                                P, P, C.c_int64, P, C.c_int64, C.c_int32, C.c_int32, C.c_int32,
                                C.c_int32, C.POINTER(_RouteParams), C.c_int32, P, P, P, P]
        L.or_bruteforce.argtypes = [P, C.c_int64, C.c_int32, C.c_int32, P, P, C.c_int64,
                                    C.c_int32, C.c_int32, P, P]
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _check(rc: int, what: str):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with code {rc}")


# --------------------------------------------------------------------------
# encoder
# --------------------------------------------------------------------------

@dataclass
class Encoder:
    """Linear layers; hidden ones have an (eval) BatchNorm affine and ReLU."""
    weights: Sequence[np.ndarray]             # layer l: [out, in] fp32
    biases: Sequence[Optional[np.ndarray]]
    bn_scale: Sequence[Optional[np.ndarray]] = ()
    bn_shift: Sequence[Optional[np.ndarray]] = ()
    input_scale: float = 1.0

    def _pack(self, in_dtype: int):
        L = len(self.weights)
        widths = [self.weights[0].shape[1]] + [w.shape[0] for w in self.weights]
        parts = []
        for l, w in enumerate(self.weights):
            out = w.shape[0]
            parts.append(np.ascontiguousarray(w, dtype=np.float32).ravel())
            b = self.biases[l] if l < len(self.biases) and self.biases[l] is not None else np.zeros(out)
            parts.append(np.asarray(b, dtype=np.float32))
            if l + 1 < L:
                sc = self.bn_scale[l] if l < len(self.bn_scale) and self.bn_scale[l] is not None else np.ones(out)
                sh = self.bn_shift[l] if l < len(self.bn_shift) and self.bn_shift[l] is not None else np.zeros(out)
                parts.append(np.asarray(sc, dtype=np.float32))
                parts.append(np.asarray(sh, dtype=np.float32))
        wa = np.asarray(widths, dtype=np.int32)
        pa = np.concatenate(parts).astype(np.float32)
        st = _Encoder(L, wa.ctypes.data_as(C.POINTER(C.c_int32)),
                      pa.ctypes.data_as(C.POINTER(C.c_float)), float(self.input_scale), in_dtype)
        return st, (wa, pa)


def encode(enc: Encoder, x: np.ndarray, with_mag: bool = False):
    """Logits [nq, L_dim] fp32 (fp64 accumulation); optionally the per-logit
    magnitude sum |w*h| + |bias| of the last layer (the tolerance scale)."""
    x = np.ascontiguousarray(x)
    in_dtype = OR_U8 if x.dtype == np.uint8 else OR_F32
    if in_dtype == OR_F32:
        x = x.astype(np.float32, copy=False)
    st, keep = enc._pack(in_dtype)
    nq = x.shape[0]
    b = enc.weights[-1].shape[0]
    out = np.empty((nq, b), dtype=np.float32)
    mag = np.empty((nq, b), dtype=np.float64) if with_mag else None
    _check(lib().or_encode(C.byref(st), _p(x), nq, _p(out), _p(mag)), "encode")
    return (out, mag) if with_mag else out


# --------------------------------------------------------------------------
# probes (Algorithm 1)
# --------------------------------------------------------------------------

def probes(logits: np.ndarray, tau: np.ndarray, l_sel: int, r_max: int, P: int,
           s_max: float = float("inf"), n_bins: int = 1):
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    tau = np.ascontiguousarray(tau, dtype=np.float32)
    nq, b = logits.shape
    codes = np.zeros((nq, P), dtype=np.uint32)
    costs = np.zeros((nq, P), dtype=np.float32)
    bins = np.zeros((nq, P), dtype=np.int32)
    counts = np.zeros(nq, dtype=np.int32)
    _check(lib().or_probes(_p(logits), nq, b, _p(tau), l_sel, r_max, s_max, n_bins, P,
                           _p(codes), _p(costs), _p(bins), _p(counts)), "probes")
    return codes, costs, bins, counts


# --------------------------------------------------------------------------
# centroid stage (Algorithm 2)
# --------------------------------------------------------------------------

@dataclass
class RouteParams:
    n_bins: int = 1
    s_max: float = float("inf")
    k_c: int = 512
    b_batch: int = 64
    b_min: int = 2
    t_low: int = 3
    u_heap: int = 1
    u_front: int = 1
    alpha_front: float = 0.6
    gate_on: bool = True
    early_stop_on: bool = True
    lowq_or: bool = True
    m_x: np.ndarray = field(default_factory=lambda: np.zeros(0, np.float32))
    m_y: np.ndarray = field(default_factory=lambda: np.zeros(0, np.float32))

    def _c(self):
        mx = np.ascontiguousarray(self.m_x, dtype=np.float32)
        my = np.ascontiguousarray(self.m_y, dtype=np.float32)
        st = _RouteParams(self.n_bins, self.s_max, self.k_c, self.b_batch, self.b_min, self.t_low,
                          self.u_heap, self.u_front, self.alpha_front, int(self.gate_on),
                          int(self.early_stop_on), int(self.lowq_or), len(mx),
                          mx.ctypes.data_as(C.POINTER(C.c_float)),
                          my.ctypes.data_as(C.POINTER(C.c_float)))
        return st, (mx, my)


def margin(prm: RouteParams, x: float) -> float:
    st, keep = prm._c()
    return lib().or_margin(C.byref(st), x)


def route(logits, codes, bins, counts, bc_off, centroids, prm: RouteParams, with_stats=False):
    """Per-query candidate clusters C(q) = C_dir followed by H; returns
    (lists, stats) with lists[q] a uint32 array."""
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    codes = np.ascontiguousarray(codes, dtype=np.uint32)
    bins = np.ascontiguousarray(bins, dtype=np.int32)
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    bc_off = np.ascontiguousarray(bc_off, dtype=np.uint32)
    centroids = np.ascontiguousarray(centroids, dtype=np.float32)
    nq, b = logits.shape
    P = codes.shape[1]
    n_clusters = centroids.shape[0]
    k_c = min(prm.k_c, max(n_clusters, 1))
    cap = P + k_c
    clus = np.zeros((nq, cap), dtype=np.uint32)
    n = np.zeros(nq, dtype=np.int32)
    stats = (RouteStats * max(nq, 1))()
    st, keep = prm._c()
    _check(lib().or_route(_p(logits), nq, b, _p(codes), _p(bins), _p(counts), P, _p(bc_off),
                          _p(centroids), n_clusters, C.byref(st), _p(clus), cap, _p(n),
                          C.cast(stats, C.c_void_p)), "route")
    lists = [clus[q, :n[q]].copy() for q in range(nq)]
    if with_stats:
        return lists, [stats[q] for q in range(nq)]
    return lists


# --------------------------------------------------------------------------
# refinement and brute force
# --------------------------------------------------------------------------

def refine(rows, row_ids, cl_off, queries, lists, k: int):
    rows = np.ascontiguousarray(rows)
    queries = np.ascontiguousarray(queries)
    dtype = OR_U8 if rows.dtype == np.uint8 else OR_F32
    nq = queries.shape[0]
    d = rows.shape[1]
    cap = max([len(x) for x in lists] + [1])
    clus = np.zeros((nq, cap), dtype=np.uint32)
    n = np.zeros(nq, dtype=np.int32)
    for q, x in enumerate(lists):
        clus[q, :len(x)] = x
        n[q] = len(x)
    ids = np.empty((nq, k), dtype=np.int64)
    dists = np.empty((nq, k), dtype=np.float32)
    ncand = np.empty(nq, dtype=np.int64)
    rid = None if row_ids is None else np.ascontiguousarray(row_ids, dtype=np.int64)
    _check(lib().or_refine(_p(rows), d, dtype, _p(rid), _p(np.ascontiguousarray(cl_off, dtype=np.uint64)),
                           _p(queries), nq, _p(clus), cap, _p(n), k, _p(ids), _p(dists), _p(ncand)),
           "refine")
    return ids, dists, ncand


def bruteforce(rows, queries, k: int, row_ids=None, n_threads: int = 0):
    """Exact k-NN by (squared distance, id) over every row (Sec. 3.1)."""
    rows = np.ascontiguousarray(rows)
    queries = np.ascontiguousarray(queries)
    dtype = OR_U8 if rows.dtype == np.uint8 else OR_F32
    nq = queries.shape[0]
    ids = np.empty((nq, k), dtype=np.int64)
    dists = np.empty((nq, k), dtype=np.float32)
    rid = None if row_ids is None else np.ascontiguousarray(row_ids, dtype=np.int64)
    nt = n_threads or len(os.sched_getaffinity(0))
    _check(lib().or_bruteforce(_p(rows), rows.shape[0], rows.shape[1], dtype, _p(rid), _p(queries),
                               nq, k, nt, _p(ids), _p(dists)), "bruteforce")
    return ids, dists


def search(enc: Encoder, tau, rows, row_ids, bc_off, cl_off, centroids, queries, k: int,
           l_sel: int, r_max: int, P: int, prm: RouteParams, n_threads: int = 1):
    """The whole path: encode, Algorithm 1, Algorithm 2, refine."""
    rows = np.ascontiguousarray(rows)
    queries = np.ascontiguousarray(queries)
    dtype = OR_U8 if rows.dtype == np.uint8 else OR_F32
    st_e, keep_e = enc._pack(dtype)
    st_r, keep_r = prm._c()
    tau = np.ascontiguousarray(tau, dtype=np.float32)
    centroids = np.ascontiguousarray(centroids, dtype=np.float32)
    nq = queries.shape[0]
    ids = np.empty((nq, k), dtype=np.int64)
    dists = np.empty((nq, k), dtype=np.float32)
    ncand = np.empty(nq, dtype=np.int64)
    secs = np.zeros(4, dtype=np.float64)
    rid = None if row_ids is None else np.ascontiguousarray(row_ids, dtype=np.int64)
    _check(lib().or_search(C.byref(st_e), _p(tau), len(tau), _p(rows), rows.shape[1], dtype,
                           _p(rid), _p(np.ascontiguousarray(bc_off, dtype=np.uint32)),
                           _p(np.ascontiguousarray(cl_off, dtype=np.uint64)), _p(centroids),
                           centroids.shape[0], _p(queries), nq, k, l_sel, r_max, P, C.byref(st_r),
                           n_threads, _p(ids), _p(dists), _p(ncand), _p(secs)), "search")
    return ids, dists, ncand, secs


def recall_at_k(result_ids: np.ndarray, gt_ids: np.ndarray, k: int) -> float:
    """Recall@k (Sec. 4.4): mean over queries of |R_k ∩ G_k| / min(k, |G_k|),
    by unique ids; padding ids (-1) never count."""
    total = 0.0
    for r, g in zip(result_ids, gt_ids):
        G = set(int(x) for x in g[:k] if x >= 0)
        R = set(int(x) for x in r[:k] if x >= 0)
        if not G:
            continue
        total += len(R & G) / min(k, len(G))
    return total / len(result_ids)


def lsim(x: np.ndarray, lat: np.ndarray, gamma: float, tau_emb: float) -> float:
    """The selective similarity loss L_sim of one batch (Sec. 3.2.2, Eq.
    similarityconfig with the mask of Eq. 8), written out in fp64 loops over
    the pairs: rho = sqrt(L_dim / E_dim); a pair i != j counts when its input
    distance is at most tau_emb or its latent distance at most
    gamma * rho * tau_emb; the loss is the mean over counted pairs of
    (latent distance - gamma * rho * input distance)^2."""
    x = np.asarray(x, dtype=np.float64)
    lat = np.asarray(lat, dtype=np.float64)
    B, E = x.shape
    rho = np.sqrt(lat.shape[1] / E)
    num, den = 0.0, 0
    for i in range(B):
        se = np.sqrt(((x - x[i]) ** 2).sum(1))
        sl = np.sqrt(((lat - lat[i]) ** 2).sum(1))
        for j in range(B):
            if j == i:
                continue
            if se[j] <= tau_emb or sl[j] <= gamma * rho * tau_emb:
                num += (sl[j] - gamma * rho * se[j]) ** 2
                den += 1
    return num / den if den else 0.0
