"""Python binding of libneuroute.so (include/neuroute.h) -- argument
marshalling only.  Device buffers are PyTorch CUDA(HIP) tensors, streams are
torch streams; every step of the search runs in the library's HIP kernels.

The library must have been built (``python -m paper_2608_15438_amd.build_lib``
or ``__graft_entry__.build()``); importing the binding without it raises.
"""
from __future__ import annotations

import ctypes as C
import math
import os
from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
SO_PATH = os.path.join(_HERE, "libneuroute.so")

NR_OK, NR_EINVAL, NR_ENOMEM, NR_EDEVICE, NR_EUNSUPPORTED, NR_ECORRUPT = range(6)
NR_U8, NR_F32 = 0, 1
NR_MAX_LAYERS = 8
NR_MAX_KNOTS = 32
NR_MAX_K = 64
NR_MAX_PROBES = 4096
NR_QSTATS = 8
NR_REFINE_AUTO, NR_REFINE_PER_QUERY, NR_REFINE_SHARED = 0, 1, 2
NR_NOALLOC_SCRATCH_BYTES = 64 << 20
NR_STAGES = 10
QS = dict(probes=0, clusters=1, direct=2, scored=3, stopped=4, rows=5, tiles=6, batches=7)
STAGES = ("encode", "probe", "route", "plan", "refine", "merge", "shared_prep", "shared_scan",
          "shared_open", "shared_merge")
WORK = ("tiles", "rows", "rows_read", "own_rows", "shared_rows", "shared_pairs", "survivors",
        "flagged", "fallback_rows", "shared_pair_rows", "full_rows", "head_bytes", "body_bytes",
        "open_bytes", "refine_bytes")

# every symbol include/neuroute.h declares
EXPORTS = ("nr_index_upload", "nr_index_free", "nr_search", "nr_search_ex", "nr_search_noalloc",
           "nr_encode", "nr_calibrate", "nr_pair_sqdist_ws", "nr_pair_sqdist", "nr_lsim_grad",
           "nr_build_tau", "nr_build_codes", "nr_build_plan", "nr_build_index",
           "nr_probe", "nr_route", "nr_route_capacity", "nr_refine", "nr_profile_enable",
           "nr_profile_read", "nr_last_work", "nr_stream_read", "nr_status_string",
           "nr_last_error")


class NRError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: status {status} ({_status_name(status)}): {_last_error()}")
        self.status = status


class nr_index_desc(C.Structure):
    _fields_ = [("n", C.c_int64), ("d", C.c_int32), ("dtype", C.c_int32), ("b", C.c_int32),
                ("n_layers", C.c_int32), ("widths", C.POINTER(C.c_int32)),
                ("weights", C.POINTER(C.POINTER(C.c_float))),
                ("biases", C.POINTER(C.POINTER(C.c_float))),
                ("bn_scale", C.POINTER(C.POINTER(C.c_float))),
                ("bn_shift", C.POINTER(C.POINTER(C.c_float))),
                ("input_scale", C.c_float), ("tau", C.POINTER(C.c_float)),
                ("rows", C.c_void_p), ("row_ids", C.c_void_p), ("bc_off", C.c_void_p),
                ("cl_off", C.c_void_p), ("centroids", C.c_void_p), ("n_clusters", C.c_int64),
                ("head_bytes", C.c_int32), ("head_copy", C.c_int32)]


class nr_build_plan_info(C.Structure):
    _fields_ = [("max_clusters", C.c_int64), ("n_multi", C.c_int64), ("kmax", C.c_int32),
                ("t", C.c_uint32)]


class nr_build_desc(C.Structure):
    _fields_ = [("n", C.c_int64), ("b", C.c_int32), ("logits", C.c_void_p), ("codes", C.c_void_p),
                ("sizes", C.c_void_p), ("kb", C.c_void_p), ("mlist", C.c_void_p),
                ("max_clusters", C.c_int64), ("n_multi", C.c_int64), ("kmax", C.c_int32),
                ("uniforms", C.c_void_p), ("seed", C.c_uint32), ("lloyd", C.c_int32),
                ("sample_per_cluster", C.c_int32)]


NR_CLUSTER_NONE, NR_CLUSTER_CAPACITY, NR_CLUSTER_FIXED, NR_CLUSTER_PER_BUCKET = 0, 1, 2, 3


class nr_params(C.Structure):
    _fields_ = [("l_sel", C.c_int32), ("r_max", C.c_int32), ("s_max", C.c_float),
                ("n_bins", C.c_int32), ("k_c", C.c_int32), ("b_batch", C.c_int32),
                ("b_min", C.c_int32), ("t_low", C.c_int32), ("u_heap", C.c_int32),
                ("u_front", C.c_int32), ("alpha_front", C.c_float), ("gate_on", C.c_int32),
                ("early_stop_on", C.c_int32), ("lowq_or", C.c_int32), ("refine_mode", C.c_int32),
                ("shared_seed_rows", C.c_int32),
                ("m_knots", C.c_int32),
                ("m_x", C.c_float * NR_MAX_KNOTS), ("m_y", C.c_float * NR_MAX_KNOTS)]


_lib = None


def lib():
    """The loaded library; raises if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(SO_PATH):
            raise RuntimeError(f"{SO_PATH} is missing: build it with "
                               "`python -m paper_2608_15438_amd.build_lib`")
        L = C.CDLL(SO_PATH)
        P = C.c_void_p
        L.nr_status_string.restype = C.c_char_p
        L.nr_status_string.argtypes = [C.c_int]
        L.nr_last_error.restype = C.c_char_p
        L.nr_last_error.argtypes = []
        L.nr_index_upload.argtypes = [C.POINTER(nr_index_desc), C.POINTER(P), P]
        L.nr_index_free.argtypes = [P]
        L.nr_search.argtypes = [P, P, C.c_int64, C.c_int32, C.c_int32, C.POINTER(nr_params), P, P, P]
        L.nr_search_ex.argtypes = [P, P, P, C.c_int64, C.c_int32, C.c_int32, C.POINTER(nr_params),
                                   P, P, P, P]
        L.nr_search_noalloc.argtypes = [P, P, P, C.c_int64, C.c_int32, C.c_int32,
                                        C.POINTER(nr_params), P, P, P]
        L.nr_encode.argtypes = [P, P, C.c_int64, P, P]
        L.nr_pair_sqdist_ws.argtypes = [C.c_int64, C.c_int32]
        L.nr_pair_sqdist_ws.restype = C.c_size_t
        L.nr_pair_sqdist.argtypes = [P, C.c_int64, C.c_int32, P, P, P]
        L.nr_lsim_grad.argtypes = [P, P, C.c_int64, C.c_int32, C.c_float, C.c_float, P, P, P]
        L.nr_build_tau.argtypes = [P, C.c_int64, C.c_int32, P, P]
        L.nr_build_codes.argtypes = [P, C.c_int64, C.c_int32, P, P, P, P]
        L.nr_build_plan.argtypes = [P, C.c_int64, C.c_int32, C.c_int32, C.c_uint32, P, P,
                                    C.POINTER(nr_build_plan_info), P]
        L.nr_build_index.argtypes = [C.POINTER(nr_build_desc), P, P, P, P,
                                     C.POINTER(C.c_int64), P]
        L.nr_calibrate.argtypes = [P, P, C.c_int64, P, C.c_int32, C.c_int32, C.c_int32, P, P, P]
        L.nr_probe.argtypes = [P, P, C.c_int64, C.c_int32, C.POINTER(nr_params), P, P, P, P, P]
        L.nr_route.argtypes = [P, P, C.c_int64, C.c_int32, C.POINTER(nr_params), P, P, C.c_int64, P]
        L.nr_route_capacity.argtypes = [P, C.c_int32, C.POINTER(nr_params)]
        L.nr_route_capacity.restype = C.c_int64
        L.nr_refine.argtypes = [P, P, C.c_int64, C.c_int32, P, P, C.c_int64, P, P, P]
        L.nr_profile_enable.argtypes = [P, C.c_int32]
        L.nr_profile_read.argtypes = [P, C.POINTER(C.c_double), C.POINTER(C.c_int64), C.c_int32]
        L.nr_last_work.argtypes = [P, P, C.POINTER(C.c_int64), C.c_int32]
        L.nr_stream_read.argtypes = [P, C.c_int64, P, P]
        for name in EXPORTS:
            getattr(L, name).restype = getattr(L, name).restype or C.c_int
        L.nr_route_capacity.restype = C.c_int64
        L.nr_pair_sqdist_ws.restype = C.c_size_t
        L.nr_status_string.restype = C.c_char_p
        L.nr_last_error.restype = C.c_char_p
        _lib = L
    return _lib


def _status_name(s: int) -> str:
    try:
        return lib().nr_status_string(s).decode()
    except Exception:
        return "?"


def _last_error() -> str:
    try:
        return lib().nr_last_error().decode()
    except Exception:
        return ""


def _check(status: int, what: str):
    if status != NR_OK:
        raise NRError(status, what)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _dev(t: torch.Tensor, name: str):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def nr_stream_read(buf: torch.Tensor, sink: torch.Tensor, stream=None):
    """One streaming pass of 16-byte loads over a device tensor."""
    _dev(buf, "buf")
    _check(lib().nr_stream_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink),
                                _stream(stream)), "nr_stream_read")


def nr_pair_sqdist(x: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
    """Squared distances [B, B] of the rows of x (fp32 [B, D], device)."""
    _dev(x, "x")
    B, D = x.shape
    ws = torch.empty(int(lib().nr_pair_sqdist_ws(B, D)), dtype=torch.float32, device=x.device)
    if out is None:
        out = torch.empty((B, B), dtype=torch.float32, device=x.device)
    _check(lib().nr_pair_sqdist(_ptr(x), B, D, _ptr(ws), _ptr(out), _stream(stream)),
           "nr_pair_sqdist")
    return out


def nr_lsim_grad(d2_emb: torch.Tensor, lat: torch.Tensor, gamma_rho: float, tau_emb: float,
                 stream=None):
    """(num_cnt fp64 [2], grad_lat fp32 [B, L]) of L_sim for one batch."""
    _dev(d2_emb, "d2_emb")
    _dev(lat, "lat")
    B, L = lat.shape
    num_cnt = torch.empty(2, dtype=torch.float64, device=lat.device)
    grad = torch.empty((B, L), dtype=torch.float32, device=lat.device)
    _check(lib().nr_lsim_grad(_ptr(d2_emb), _ptr(lat), B, L, float(gamma_rho), float(tau_emb),
                              _ptr(num_cnt), _ptr(grad), _stream(stream)), "nr_lsim_grad")
    return num_cnt, grad


def nr_build_tau(logits: torch.Tensor, stream=None):
    _dev(logits, "logits")
    ns, b = logits.shape
    tau = torch.empty(b, dtype=torch.float32, device=logits.device)
    _check(lib().nr_build_tau(_ptr(logits), ns, b, _ptr(tau), _stream(stream)), "nr_build_tau")
    return tau


def nr_build_codes(logits: torch.Tensor, tau: torch.Tensor, codes: torch.Tensor,
                   sizes: torch.Tensor, stream=None):
    _dev(logits, "logits")
    m, b = logits.shape
    _check(lib().nr_build_codes(_ptr(logits), m, b, _ptr(tau), _ptr(codes), _ptr(sizes),
                                _stream(stream)), "nr_build_codes")


def nr_build_plan(sizes: torch.Tensor, n: int, b: int, rule: int, param: int, stream=None):
    """(kb, mlist, info) of the cluster rule."""
    kb = torch.empty(1 << b, dtype=torch.int32, device=sizes.device)
    mlist = torch.empty(1 << b, dtype=torch.int32, device=sizes.device)
    info = nr_build_plan_info()
    _check(lib().nr_build_plan(_ptr(sizes), n, b, rule, param, _ptr(kb), _ptr(mlist),
                               C.byref(info), _stream(stream)), "nr_build_plan")
    return kb, mlist, info


def nr_build_index(desc: nr_build_desc, row_ids, bc_off, cl_off, centroids, stream=None):
    nc = C.c_int64()
    _check(lib().nr_build_index(C.byref(desc), _ptr(row_ids), _ptr(bc_off), _ptr(cl_off),
                                _ptr(centroids), C.byref(nc), _stream(stream)), "nr_build_index")
    return nc.value


# --------------------------------------------------------------------------
# search parameters
# --------------------------------------------------------------------------

@dataclass
class Params:
    l_sel: int = 16
    r_max: int = 7
    s_max: float = float("inf")
    n_bins: int = 1
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
    refine_mode: int = NR_REFINE_AUTO
    shared_seed_rows: int = 0
    m_x: Sequence[float] = field(default_factory=list)
    m_y: Sequence[float] = field(default_factory=list)

    def c(self) -> nr_params:
        if len(self.m_x) != len(self.m_y) or len(self.m_x) > NR_MAX_KNOTS:
            raise ValueError("margin knots: m_x and m_y must have equal length <= 32")
        p = nr_params()
        p.l_sel, p.r_max, p.s_max, p.n_bins = self.l_sel, self.r_max, self.s_max, self.n_bins
        p.k_c, p.b_batch, p.b_min, p.t_low = self.k_c, self.b_batch, self.b_min, self.t_low
        p.u_heap, p.u_front, p.alpha_front = self.u_heap, self.u_front, self.alpha_front
        p.gate_on, p.early_stop_on, p.lowq_or = int(self.gate_on), int(self.early_stop_on), int(self.lowq_or)
        p.refine_mode = int(self.refine_mode)
        p.shared_seed_rows = int(self.shared_seed_rows)
        p.m_knots = len(self.m_x)
        for i, (x, y) in enumerate(zip(self.m_x, self.m_y)):
            p.m_x[i] = x
            p.m_y[i] = y
        return p


# --------------------------------------------------------------------------
# index
# --------------------------------------------------------------------------

class Index:
    """An uploaded index.  Device arrays are kept referenced here because the
    library borrows them."""

    def __init__(self, *, n, d, dtype, b, weights, biases, input_scale, tau, rows, row_ids,
                 bc_off, cl_off, centroids, bn_scale=None, bn_shift=None, head_bytes=0,
                 head_copy=0, stream=None):
        L = len(weights)
        self._keep = []
        widths = np.array([weights[0].shape[1]] + [w.shape[0] for w in weights], np.int32)
        wp = (C.POINTER(C.c_float) * L)()
        bp = (C.POINTER(C.c_float) * L)()
        sp = (C.POINTER(C.c_float) * L)()
        hp = (C.POINTER(C.c_float) * L)()
        for l in range(L):
            w = np.ascontiguousarray(weights[l], np.float32)
            self._keep.append(w)
            wp[l] = w.ctypes.data_as(C.POINTER(C.c_float))
            for src, dst in ((biases, bp), (bn_scale, sp), (bn_shift, hp)):
                if src is not None and l < len(src) and src[l] is not None:
                    a = np.ascontiguousarray(src[l], np.float32)
                    self._keep.append(a)
                    dst[l] = a.ctypes.data_as(C.POINTER(C.c_float))
        tau = np.ascontiguousarray(tau, np.float32)
        self._keep += [widths, tau, wp, bp, sp, hp]
        enc_only = rows is None
        self.dev = [] if enc_only else [_dev(rows, "rows"), _dev(row_ids, "row_ids"),
                                        _dev(bc_off, "bc_off"), _dev(cl_off, "cl_off"),
                                        _dev(centroids, "centroids")]
        desc = nr_index_desc()
        desc.n, desc.d, desc.dtype, desc.b, desc.n_layers = n, d, dtype, b, L
        desc.widths = widths.ctypes.data_as(C.POINTER(C.c_int32))
        desc.weights = wp
        desc.biases = bp
        desc.bn_scale = sp
        desc.bn_shift = hp
        desc.input_scale = input_scale
        desc.tau = tau.ctypes.data_as(C.POINTER(C.c_float))
        if not enc_only:
            desc.rows, desc.row_ids, desc.bc_off, desc.cl_off, desc.centroids = [
                t.data_ptr() for t in self.dev]
        desc.n_clusters = 0 if enc_only else centroids.shape[0]
        desc.head_bytes = int(head_bytes)
        desc.head_copy = int(head_copy)
        self.n, self.d, self.dtype, self.b = n, d, dtype, b
        self.n_clusters = 0 if enc_only else int(centroids.shape[0])
        h = C.c_void_p()
        _check(lib().nr_index_upload(C.byref(desc), C.byref(h), _stream(stream)), "nr_index_upload")
        self.handle = h

    @classmethod
    def encoder_only(cls, enc, dtype, tau=None, stream=None):
        """An index holding only the encoder (and tau): for nr_encode, e.g.
        to encode a base before its index exists."""
        b = enc.weights[-1].shape[0]
        d = enc.weights[0].shape[1]
        t = np.zeros(b, np.float32) if tau is None else tau
        return cls(n=0, d=d, dtype=dtype, b=b, weights=enc.weights, biases=enc.biases,
                   bn_scale=enc.bn_scale, bn_shift=enc.bn_shift, input_scale=enc.input_scale,
                   tau=t, rows=None, row_ids=None, bc_off=None, cl_off=None, centroids=None,
                   stream=stream)

    @classmethod
    def from_built(cls, ix, device="cuda", stream=None):
        """Upload an index_build.Index (host or device arrays, either layout)."""
        def dt(a, dtype):
            t = torch.as_tensor(a) if not isinstance(a, torch.Tensor) else a
            return t.to(device=device, dtype=dtype).contiguous()
        rows = ix.rows if isinstance(ix.rows, torch.Tensor) else torch.from_numpy(np.ascontiguousarray(ix.rows))
        rows = rows.to(device).contiguous()
        w = ix.workload
        hb = int(getattr(ix, "head_bytes", 0) or 0)
        if hb:
            n, d, dtype = int(w.n), int(w.d), NR_U8 if w.dtype == "u8" else NR_F32
        else:
            n, d = int(rows.shape[0]), int(rows.shape[1])
            dtype = NR_U8 if rows.dtype == torch.uint8 else NR_F32
        bc = ix.bc_off
        bc = torch.from_numpy(np.asarray(bc).astype(np.int64)) if not isinstance(bc, torch.Tensor) else bc
        cl = ix.cl_off
        cl = torch.from_numpy(np.asarray(cl).astype(np.int64)) if not isinstance(cl, torch.Tensor) else cl
        e = ix.encoder
        return cls(n=n, d=d, dtype=dtype, b=len(ix.tau),
                   weights=e.weights, biases=e.biases, bn_scale=e.bn_scale, bn_shift=e.bn_shift,
                   input_scale=e.input_scale, tau=ix.tau, rows=rows,
                   row_ids=dt(ix.row_ids, torch.int64), bc_off=dt(bc, torch.int32),
                   cl_off=dt(cl, torch.int64), centroids=dt(ix.centroids, torch.float32),
                   head_bytes=hb, head_copy=int(getattr(ix, "head_copy", 0) or 0), stream=stream)

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            lib().nr_index_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---- entry points (same names as the C ABI) ----
    def nr_search(self, queries, k, probe_budget, params: Params, logits=None, qstats=False,
                  stream=None):
        _dev(queries, "queries")
        nq = queries.shape[0]
        ids = torch.empty((nq, k), dtype=torch.int64, device=queries.device)
        dists = torch.empty((nq, k), dtype=torch.float32, device=queries.device)
        qs = torch.zeros((nq, NR_QSTATS), dtype=torch.int32, device=queries.device) if qstats else None
        p = params.c()
        if logits is None and not qstats:
            _check(lib().nr_search(self.handle, _ptr(queries), nq, k, probe_budget, C.byref(p),
                                   _ptr(ids), _ptr(dists), _stream(stream)), "nr_search")
        else:
            if logits is not None:
                _dev(logits, "logits")
            _check(lib().nr_search_ex(self.handle, _ptr(queries), _ptr(logits), nq, k, probe_budget,
                                      C.byref(p), _ptr(ids), _ptr(dists), _ptr(qs), _stream(stream)),
                   "nr_search_ex")
        return (ids, dists, qs) if qstats else (ids, dists)

    def nr_search_noalloc(self, queries, k, probe_budget, params: Params, out_ids, out_dists,
                          logits=None, stream=None):
        """The search that allocates nothing: the caller passes the outputs
        (DEVICE int64 / fp32 [nq, k])."""
        _dev(queries, "queries")
        _dev(out_ids, "out_ids")
        _dev(out_dists, "out_dists")
        nq = queries.shape[0]
        if tuple(out_ids.shape) != (nq, k) or tuple(out_dists.shape) != (nq, k):
            raise ValueError("out_ids and out_dists must be [nq, k]")
        if logits is not None:
            _dev(logits, "logits")
        p = params.c()
        _check(lib().nr_search_noalloc(self.handle, _ptr(queries), _ptr(logits), nq, k,
                                       probe_budget, C.byref(p), _ptr(out_ids), _ptr(out_dists),
                                       _stream(stream)), "nr_search_noalloc")
        return out_ids, out_dists

    def nr_encode(self, queries, stream=None):
        _dev(queries, "queries")
        out = torch.empty((queries.shape[0], self.b), dtype=torch.float32, device=queries.device)
        _check(lib().nr_encode(self.handle, _ptr(queries), queries.shape[0], _ptr(out),
                               _stream(stream)), "nr_encode")
        return out

    def nr_calibrate(self, logits, target_ids, l_sel, r_max, stream=None):
        """Bucket scores [nq, K] of the targets and margin points [nq, 2]."""
        _dev(logits, "logits")
        _dev(target_ids, "target_ids")
        nq, K = target_ids.shape
        scores = torch.empty((nq, K), dtype=torch.float32, device=logits.device)
        xy = torch.empty((nq, 2), dtype=torch.float32, device=logits.device)
        _check(lib().nr_calibrate(self.handle, _ptr(logits), nq, _ptr(target_ids), K, l_sel,
                                  r_max, _ptr(scores), _ptr(xy), _stream(stream)),
               "nr_calibrate")
        return scores, xy

    def nr_probe(self, logits, probe_budget, params: Params, stream=None):
        _dev(logits, "logits")
        nq = logits.shape[0]
        dev = logits.device
        codes = torch.zeros((nq, probe_budget), dtype=torch.int32, device=dev)
        costs = torch.zeros((nq, probe_budget), dtype=torch.float32, device=dev)
        bins = torch.zeros((nq, probe_budget), dtype=torch.int32, device=dev)
        counts = torch.zeros(nq, dtype=torch.int32, device=dev)
        p = params.c()
        _check(lib().nr_probe(self.handle, _ptr(logits), nq, probe_budget, C.byref(p), _ptr(codes),
                              _ptr(costs), _ptr(bins), _ptr(counts), _stream(stream)), "nr_probe")
        return codes, costs, bins, counts

    def nr_route_capacity(self, probe_budget, params: Params):
        p = params.c()
        return int(lib().nr_route_capacity(self.handle, probe_budget, C.byref(p)))

    def nr_route(self, logits, probe_budget, params: Params, stream=None):
        _dev(logits, "logits")
        nq = logits.shape[0]
        cap = self.nr_route_capacity(probe_budget, params)
        clus = torch.zeros((nq, cap), dtype=torch.int32, device=logits.device)
        n = torch.zeros(nq, dtype=torch.int32, device=logits.device)
        p = params.c()
        _check(lib().nr_route(self.handle, _ptr(logits), nq, probe_budget, C.byref(p), _ptr(clus),
                              _ptr(n), cap, _stream(stream)), "nr_route")
        return clus, n

    def nr_refine(self, queries, k, clusters, n_clusters, stream=None):
        _dev(queries, "queries")
        _dev(clusters, "clusters")
        nq = queries.shape[0]
        ids = torch.empty((nq, k), dtype=torch.int64, device=queries.device)
        dists = torch.empty((nq, k), dtype=torch.float32, device=queries.device)
        _check(lib().nr_refine(self.handle, _ptr(queries), nq, k, _ptr(clusters), _ptr(n_clusters),
                               clusters.shape[1], _ptr(ids), _ptr(dists), _stream(stream)),
               "nr_refine")
        return ids, dists

    def nr_profile_enable(self, on=True):
        _check(lib().nr_profile_enable(self.handle, int(on)), "nr_profile_enable")

    def nr_profile_read(self, reset=True):
        ms = (C.c_double * NR_STAGES)()
        n = C.c_int64()
        _check(lib().nr_profile_read(self.handle, ms, C.byref(n), int(reset)), "nr_profile_read")
        return dict(zip(STAGES, list(ms))), n.value

    def nr_last_work(self, stream=None):
        """Work counters of the last search's last chunk, keyed by WORK."""
        v = (C.c_int64 * len(WORK))()
        _check(lib().nr_last_work(self.handle, _stream(stream), v, len(WORK)), "nr_last_work")
        return dict(zip(WORK, list(v)))
