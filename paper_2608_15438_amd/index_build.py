"""Index construction for the NeuRoute search path (untimed, built once).

Follows the paper's index construction (Sec. 3.3) and binarisation (Sec. 3.2.3):

1. logits l = E(x) of every base row (encoder forward pass, fp64 here);
2. tau_j = median of l[:, j] over a subsample ("median") or 0 ("zero", the
   sign code of the tiny case); bit j of a row's code is [l_j >= tau_j] (Eq. 10);
3. bucket allocation: each row joins the bucket of its code;
4. bucket-local clustering in latent space: K_B = ceil(|B| / t) clusters per
   bucket; small buckets are one cluster; larger ones run k-means++ on a
   sample then a few Lloyd passes over the whole bucket (rule "none": every
   bucket is one cluster, the paper's ablation without clustering);
5. the layout the search reads: rows permuted so each cluster is one
   contiguous span (sorted by code, local cluster, original id), a dense
   directory ``bc_off`` (code -> cluster range), ``cl_off`` (cluster -> row
   range) and the centroids (cluster means of the logits, fp32).

Readings where the paper leaves a choice (sample size, pass count, lower
median, cluster-count rules of the synthetic cases) are documented in the
design notes.  Runs on CPU or GPU torch tensors; uses no kernel of the search
library.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Callable, List, Optional, Sequence

import numpy as np
import torch

from synth import generators as G
from synth.configs import Workload

N_LLOYD = 5
SAMPLE_PER_CLUSTER = 64
TAU_SAMPLE = 1 << 20


@dataclass
class Encoder:
    weights: List[np.ndarray]                 # layer l: [out, in] fp32
    biases: List[np.ndarray]                  # layer l: [out] fp32
    input_scale: float
    bn_scale: Optional[List[Optional[np.ndarray]]] = None   # hidden layers only
    bn_shift: Optional[List[Optional[np.ndarray]]] = None

    @property
    def widths(self):
        return [self.weights[0].shape[1]] + [w.shape[0] for w in self.weights]


@dataclass
class Index:
    """Host (numpy) or device (torch) arrays of a built index."""
    workload: Workload
    encoder: Encoder
    tau: np.ndarray            # fp32 [b]
    rows: object               # permuted payload [n, d] (uint8 / fp32), numpy or torch
    row_ids: object            # int64 [n]: original id of permuted row
    bc_off: object             # uint32 [2^b + 1]
    cl_off: object             # uint64 [n_clusters + 1]
    centroids: object          # fp32 [n_clusters, b]
    codes: Optional[object] = None   # uint32 code of each permuted row (diagnostics)
    head_bytes: int = 0        # 0: rows is [n, d]; else a head plane first (see split_payload)
    head_copy: int = 0         # with head_bytes: 1 = whole rows follow the heads, 0 = tails

    @property
    def n_clusters(self) -> int:
        return int(self.centroids.shape[0])

    @property
    def row_bytes(self) -> int:
        return self.workload.row_bytes


def _row_dtype(w: Workload):
    return torch.uint8 if w.dtype == "u8" else torch.float32


def payload_rows(ix: Index, idx) -> torch.Tensor:
    """Row-major payload rows at permuted positions ``idx`` (a torch index
    tensor on the payload's device), whatever the layout."""
    if not ix.head_bytes:
        return ix.rows[idx]
    n, R, H = ix.workload.n, ix.row_bytes, ix.head_bytes
    if ix.head_copy:
        full = ix.rows[n * H:n * H + n * R].view(n, R)
        return full[idx].contiguous().view(_row_dtype(ix.workload)).view(-1, ix.workload.d)
    head = ix.rows[:n * H].view(n, H)
    tail = ix.rows[n * H:n * R].view(n, R - H)
    by = torch.cat([head[idx], tail[idx]], dim=1).contiguous()
    return by.view(_row_dtype(ix.workload)).view(-1, ix.workload.d)


def payload_range(ix: Index, s0: int, s1: int) -> torch.Tensor:
    """Row-major payload rows [s0, s1), whatever the layout."""
    if not ix.head_bytes:
        return ix.rows[s0:s1]
    n, R, H = ix.workload.n, ix.row_bytes, ix.head_bytes
    if ix.head_copy:
        full = ix.rows[n * H:n * H + n * R].view(n, R)[s0:s1]
        return full.contiguous().view(_row_dtype(ix.workload)).view(-1, ix.workload.d)
    head = ix.rows[:n * H].view(n, H)[s0:s1]
    tail = ix.rows[n * H:n * R].view(n, R - H)[s0:s1]
    by = torch.cat([head, tail], dim=1).contiguous()
    return by.view(_row_dtype(ix.workload)).view(-1, ix.workload.d)


def split_payload(rows_chunks, n: int, row_bytes: int, head_bytes: int, device,
                  copy: bool = False) -> torch.Tensor:
    """Head-plane layout of a payload given as consecutive row-major chunks:
    one uint8 buffer holding the head plane [n x head_bytes] (the first
    head_bytes of every row) followed by the tail plane [n x (row_bytes -
    head_bytes)], or with ``copy`` by the whole row-major payload."""
    H, R = head_bytes, row_bytes
    rest = R if copy else R - H
    out = torch.empty(n * (H + rest), dtype=torch.uint8, device=device)
    head = out[:n * H].view(n, H)
    tail = out[n * H:].view(n, rest)
    s0 = 0
    for r in rows_chunks:
        by = r.contiguous().view(torch.uint8).view(r.shape[0], R)
        m = by.shape[0]
        head[s0:s0 + m] = by[:, :H]
        tail[s0:s0 + m] = by if copy else by[:, H:]
        s0 += m
    assert s0 == n
    return out


def seeded_encoder(w: Workload) -> Encoder:
    """Xavier-uniform weights, zero biases, no BatchNorm (identity in eval)."""
    ws, bs = [], []
    for l in range(len(w.widths) - 1):
        ws.append(G.xavier_uniform(w.seed("encoder"), l, w.widths[l + 1], w.widths[l]))
        bs.append(np.zeros(w.widths[l + 1], dtype=np.float32))
    scale = 1.0 / 255.0 if w.kind == "sift" else 1.0
    return Encoder(ws, bs, scale)


# --------------------------------------------------------------------------
# row sources
# --------------------------------------------------------------------------

def cpu_row_source(w: Workload, which: str = "data") -> Callable[[np.ndarray], np.ndarray]:
    """Rows by id from the NumPy generators (seed of the data or query set)."""
    seed_c = w.seed("data")
    seed = w.seed(which)
    if w.kind == "sift":
        centers = G.sift_centers(seed_c, w.n_centers, w.d)
        return lambda ids: G.sift_rows(seed, centers, ids)
    if w.kind == "deep":
        centers = G.unit_centers(seed_c, w.n_centers, w.d)
        return lambda ids: G.deep_rows(seed, centers, ids, kappa=w.kappa, spectrum=w.spectrum)
    centers = G.gauss_centers(seed_c, w.n_centers, w.d)
    return lambda ids: G.gauss_rows(seed, centers, ids)


def array_row_source(x: np.ndarray):
    return lambda ids: x[np.asarray(ids)]


# --------------------------------------------------------------------------
# encoder forward (fp64)
# --------------------------------------------------------------------------

class _TorchEncoder:
    def __init__(self, enc: Encoder, device):
        f = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.float64, device=device)
        self.W = [f(w) for w in enc.weights]
        self.b = [f(b) for b in enc.biases]
        L = len(enc.weights)
        self.sc = [f(enc.bn_scale[l]) if enc.bn_scale and enc.bn_scale[l] is not None else None
                   for l in range(L - 1)]
        self.sh = [f(enc.bn_shift[l]) if enc.bn_shift and enc.bn_shift[l] is not None else None
                   for l in range(L - 1)]
        self.s = enc.input_scale

    def __call__(self, x: torch.Tensor) -> torch.Tensor:
        h = x.to(torch.float64)
        L = len(self.W)
        for l in range(L):
            z = h @ self.W[l].T
            if l == 0:
                z = z * self.s
            z = z + self.b[l]
            if l + 1 < L:
                if self.sc[l] is not None:
                    z = z * self.sc[l]
                if self.sh[l] is not None:
                    z = z + self.sh[l]
                z = torch.clamp_min(z, 0.0)
            h = z
        return h.to(torch.float32)


def _codes(logits: torch.Tensor, tau: torch.Tensor) -> torch.Tensor:
    b = logits.shape[1]
    bits = (logits >= tau).to(torch.int64)
    w = (torch.ones(b, dtype=torch.int64, device=logits.device) << torch.arange(b, device=logits.device))
    return (bits * w).sum(dim=1)


# --------------------------------------------------------------------------
# batched bucket-local k-means (many small independent problems at once)
# --------------------------------------------------------------------------

def _segment_ids(sizes: torch.Tensor) -> torch.Tensor:
    return torch.repeat_interleave(torch.arange(len(sizes), device=sizes.device), sizes)


def sqdist_rows(A: torch.Tensor, Bm: torch.Tensor) -> torch.Tensor:
    """fp64 squared distances of matching rows, the dimensions added in
    order (a fixed order: the HIP builder adds them the same way)."""
    acc = torch.zeros(A.shape[0], dtype=torch.float64, device=A.device)
    for j in range(A.shape[1]):
        t = A[:, j] - Bm[:, j]
        acc = acc + t * t
    return acc


def _pair_argmin(X, seg_of_pt, cent, cent_start, K, chunk=1 << 22):
    """For each point p: argmin_j ||X[p] - cent[cent_start[g] + j]||^2 over its
    group's K[g] centroids (lowest j on ties)."""
    n = X.shape[0]
    out = torch.empty(n, dtype=torch.int64, device=X.device)
    Kp = K[seg_of_pt]
    # process points in blocks whose pair count stays bounded
    cum = torch.cumsum(Kp, 0)
    start = 0
    while start < n:
        base = int(cum[start - 1]) if start > 0 else 0
        end = int(torch.searchsorted(cum, torch.tensor(base + chunk, device=X.device), right=True))
        end = max(end, start + 1)
        end = min(end, n)
        kp = Kp[start:end]
        pid = torch.repeat_interleave(torch.arange(start, end, device=X.device), kp)
        first = torch.cumsum(kp, 0) - kp
        j = torch.arange(len(pid), device=X.device) - torch.repeat_interleave(first, kp)
        cid = cent_start[seg_of_pt[pid]] + j
        d = sqdist_rows(X[pid], cent[cid])
        # segment argmin: min distance then lowest j
        best = torch.full((end - start,), float("inf"), dtype=d.dtype, device=X.device)
        best.scatter_reduce_(0, pid - start, d, reduce="amin", include_self=True)
        hit = d == best[pid - start]
        big = torch.iinfo(torch.int64).max
        jj = torch.where(hit, j, torch.full_like(j, big))
        arg = torch.full((end - start,), big, dtype=torch.int64, device=X.device)
        arg.scatter_reduce_(0, pid - start, jj, reduce="amin", include_self=True)
        out[start:end] = arg
        start = end
    return out


def mix32(x: torch.Tensor, seed: int) -> torch.Tensor:
    """A 32-bit integer hash of int64 values (products stay below 2^63, so it
    is exact and identical on CPU and GPU)."""
    m = 0xFFFFFFFF
    h = (x ^ (seed & m)) & m
    h = ((h >> 16) ^ h) * 0x45D9F3B & m
    h = ((h >> 16) ^ h) * 0x45D9F3B & m
    return (h >> 16) ^ h


# D^2 weights of the k-means++ draws are integers: floor(D^2 * 2^WEIGHT_BITS),
# capped at 2^WEIGHT_CAP_BITS, so that their sums are exact and a group's
# total (at most SAMPLE_CAP members) stays below 2^53
WEIGHT_BITS = 20
WEIGHT_CAP_BITS = 30
SAMPLE_CAP = 1 << 21


def d2_weights(D2: torch.Tensor) -> torch.Tensor:
    w = torch.floor(D2 * float(1 << WEIGHT_BITS))
    return torch.clamp(w, max=float(1 << WEIGHT_CAP_BITS)).to(torch.int64)


def bucket_kmeans(X: torch.Tensor, sizes: torch.Tensor, K: torch.Tensor, seed: int,
                  group_keys: torch.Tensor, ids: torch.Tensor):
    """k-means++ on a sample then N_LLOYD Lloyd passes, independently per group.

    X: fp64 points sorted by (group, original id), ids their original ids;
    sizes[g], K[g] >= 2.  The sample of a group is its first
    min(|g|, 64 K[g]) members ordered by (mix32(id, seed), id); k-means++
    starts from the first of them and draws each further centre with
    probability proportional to its integer D^2 weight, using the group's
    pre-drawn uniform U (cumulative weights in sample order, the first member
    whose running sum exceeds floor(U * total)).  Every sum here is either
    exact (integers) or taken in a fixed order, so the HIP builder, which
    follows the same steps, gets the same clusters.
    Returns (labels per point in [0, K[g]), centroids fp64 [sum K, dim],
    kept mask per centroid: clusters left empty after the last pass are dropped).
    """
    dev = X.device
    seg = _segment_ids(sizes)
    starts = torch.cumsum(sizes, 0) - sizes
    cstart = torch.cumsum(K, 0) - K
    dim = X.shape[1]
    # seeded shuffle inside each group: the sample is the first S_g members
    h = mix32(ids.to(torch.int64), seed)
    order = torch.sort(seg * (1 << 32) + h, stable=True).indices
    S = torch.minimum(torch.minimum(sizes, K * SAMPLE_PER_CLUSTER),
                      torch.full_like(sizes, SAMPLE_CAP))
    pos_in_group = torch.arange(X.shape[0], device=dev) - starts[seg]
    in_sample = pos_in_group < S[seg]
    samp = order[in_sample]                    # point indices, grouped, shuffled
    sseg = seg[samp]
    sstart = torch.cumsum(S, 0) - S
    Xs = X[samp]
    # uniforms for the D^2 draws: one per (group, step)
    kmax = int(K.max())
    U = torch.as_tensor(G.uniform01(seed, group_keys.cpu().numpy(), kmax, G.TAG_SAMPLE + 16),
                        dtype=torch.float64, device=dev)
    cent = torch.zeros((int(K.sum()), dim), dtype=torch.float64, device=dev)
    cent[cstart] = Xs[sstart]                  # first centre: first sampled member
    D2 = sqdist_rows(Xs, cent[cstart][sseg])
    for r in range(1, kmax):
        act_g = K > r
        act_p = act_g[sseg]
        w2 = torch.where(act_p, d2_weights(D2), torch.zeros_like(D2, dtype=torch.int64))
        cs = torch.cumsum(w2, 0)
        tot_before = torch.where(sstart > 0, cs[(sstart - 1).clamp_min(0)],
                                 torch.zeros_like(sstart, dtype=cs.dtype))
        tot = cs[sstart + S - 1] - tot_before
        target = tot_before + torch.floor(U[:, r] * tot.to(torch.float64)).to(torch.int64)
        pick = torch.searchsorted(cs, target, right=True)
        pick = torch.minimum(torch.maximum(pick, sstart), sstart + S - 1)
        # all-zero weights (duplicate points): take the first sampled member
        pick = torch.where(tot > 0, pick, sstart)
        g_act = torch.nonzero(act_g).squeeze(1)
        cent[cstart[g_act] + r] = Xs[pick[g_act]]
        newc = cent[cstart[sseg] + torch.clamp(K[sseg] - 1, max=r)]
        D2 = torch.where(act_p, torch.minimum(D2, sqdist_rows(Xs, newc)), D2)
    labels = None
    for _ in range(N_LLOYD):
        labels = _pair_argmin(X, seg, cent, cstart, K)
        gid = cstart[seg] + labels
        cnt = torch.zeros(cent.shape[0], dtype=torch.float64, device=dev)
        cnt.index_add_(0, gid, torch.ones_like(gid, dtype=torch.float64))
        sums = torch.zeros_like(cent)
        sums.index_add_(0, gid, X)
        nz = cnt > 0
        cent[nz] = sums[nz] / cnt[nz].unsqueeze(1)
    # final: the last assignment defines the clusters; centroids are its means
    gid = cstart[seg] + labels
    cnt = torch.zeros(cent.shape[0], dtype=torch.int64, device=dev)
    cnt.index_add_(0, gid, torch.ones_like(gid))
    return labels, cent, cnt > 0


def tau_sample_ids(seed: int, n: int, ns: int) -> np.ndarray:
    """ns distinct row ids: a seeded permutation prefix for small n, else the
    first distinct values of seeded multiply-shift draws."""
    if n <= ns:
        return np.arange(n)
    if n < 4 * ns:
        return G.seeded_permutation(seed, n)[:ns]
    draws = ((G._u32_words(seed, np.arange(2 * ns), 1, G.TAG_SAMPLE)[:, 0].astype(np.uint64)
              * np.uint64(n)) >> np.uint64(32)).astype(np.int64)
    _, first = np.unique(draws, return_index=True)
    return draws[np.sort(first)][:ns]


def _clusters_per_bucket(w: Workload, sizes: torch.Tensor) -> torch.Tensor:
    if w.cluster_rule == "none":  # no bucket-local clustering: a bucket is one cluster
        return torch.minimum(sizes, torch.ones_like(sizes))
    if w.cluster_rule == "fixed4":
        return torch.minimum(sizes, torch.full_like(sizes, 4))
    if w.cluster_rule == "per_bucket8":
        nz = sizes[sizes > 0]
        t = max(1, int(round(float(nz.double().mean()) / 8.0)))
    else:
        t = w.capacity
    return (sizes + t - 1) // t


# --------------------------------------------------------------------------
# the builder
# --------------------------------------------------------------------------

def build_index(w: Workload, rows_fn: Callable, device="cpu", chunk: int = 1 << 20,
                encoder: Optional[Encoder] = None, keep_codes: bool = True,
                payload_fn: Optional[Callable] = None, log=None,
                head_bytes: int = 0, head_copy: bool = False,
                logits_fn: Optional[Callable] = None) -> Index:
    """Build the index of workload ``w`` from ``rows_fn(ids) -> rows``.

    ``rows_fn`` returns numpy or torch rows for an int64 id array.  With
    ``payload_fn(perm) -> rows`` the permuted payload is produced directly
    (e.g. regenerated on the GPU) instead of gathered from ``rows_fn``.
    With ``head_bytes`` > 0 the payload starts with a head plane, followed by
    the tails or (``head_copy``) by the whole rows.  ``logits_fn(ids)``, when
    given, supplies the fp32 logits of rows (e.g. the search library's
    encoder) in place of this module's fp64 forward pass.
    """
    dev = torch.device(device)
    enc = encoder or seeded_encoder(w)
    fwd = _TorchEncoder(enc, dev)
    b = enc.widths[-1]
    n = w.n

    def rows_t(ids):
        r = rows_fn(ids)
        if isinstance(r, np.ndarray):
            r = torch.from_numpy(r)
        return r.to(dev)

    def logits_of(ids):
        if logits_fn is not None:
            return torch.as_tensor(logits_fn(ids)).to(dev).to(torch.float32)
        return fwd(rows_t(ids))

    say = log or (lambda *a: None)
    # (2) thresholds
    if w.tau_mode == "zero":
        tau = torch.zeros(b, dtype=torch.float32, device=dev)
    else:
        ns = min(n, TAU_SAMPLE)
        perm = tau_sample_ids(w.seed("sample"), n, ns)
        ls = []
        for s0 in range(0, len(perm), chunk):
            ls.append(logits_of(perm[s0:s0 + chunk]))
        L = torch.cat(ls)
        tau = torch.sort(L, dim=0).values[(L.shape[0] - 1) // 2].contiguous()
    say("tau done")
    # (1)+(3) codes and per-code logit sums (for single-cluster buckets)
    codes = torch.empty(n, dtype=torch.int64, device=dev)
    nb = 1 << b
    sums = torch.zeros((nb, b), dtype=torch.float64, device=dev)
    for s0 in range(0, n, chunk):
        ids = np.arange(s0, min(n, s0 + chunk))
        lg = logits_of(ids)
        c = _codes(lg, tau)
        codes[s0:s0 + len(ids)] = c
        sums.index_add_(0, c, lg.double())
    sizes = torch.bincount(codes, minlength=nb)
    say("codes done")
    KB = _clusters_per_bucket(w, sizes)
    multi = torch.nonzero(KB >= 2).squeeze(1)
    # labels of rows in multi-cluster buckets; default 0
    label = torch.zeros(n, dtype=torch.int64, device=dev)
    n_cl_bucket = KB.clone()
    cent_parts = {}
    if len(multi) > 0:
        is_multi = torch.zeros(nb, dtype=torch.bool, device=dev)
        is_multi[multi] = True
        member = torch.nonzero(is_multi[codes]).squeeze(1)
        # group members by bucket (stable by id)
        mc = codes[member]
        o = torch.sort(mc, stable=True).indices
        member = member[o]
        mcodes = mc[o]
        # their logits (second pass over the base)
        Xm = torch.empty((len(member), b), dtype=torch.float64, device=dev)
        mem_np = member.cpu().numpy()
        for s0 in range(0, len(mem_np), chunk):
            ids = mem_np[s0:s0 + chunk]
            Xm[s0:s0 + len(ids)] = logits_of(ids).double()
        gsizes = sizes[multi]
        gK = KB[multi]
        lab, cent, kept = bucket_kmeans(Xm, gsizes, gK, w.seed("sample"), multi, member)
        # renumber kept clusters densely inside each bucket
        cstart = torch.cumsum(gK, 0) - gK
        gseg = _segment_ids(gK)
        kept_i = kept.to(torch.int64)
        rank_in_bucket = torch.cumsum(kept_i, 0) - kept_i
        rank_in_bucket = rank_in_bucket - (torch.cumsum(kept_i, 0) - kept_i)[cstart][gseg]
        gid = cstart[_segment_ids(gsizes)] + lab
        label[member] = rank_in_bucket[gid]
        n_kept = torch.zeros(len(multi), dtype=torch.int64, device=dev)
        n_kept.index_add_(0, gseg, kept_i)
        n_cl_bucket[multi] = n_kept
        cent_parts["multi"] = (multi, n_kept, cent[kept])
    say("clustering done")
    # (5) permutation: by (code, local cluster, original id)
    key = codes * (1 << 20) + label if b <= 40 else None
    perm = torch.sort(key, stable=True).indices
    # cluster directory
    n_clusters = int(n_cl_bucket.sum())
    bc_off = torch.zeros(nb + 1, dtype=torch.int64, device=dev)
    bc_off[1:] = torch.cumsum(n_cl_bucket, 0)
    # cluster sizes (independent of the row order)
    cl_sizes = torch.bincount(bc_off[codes] + label, minlength=n_clusters)
    cl_off = torch.zeros(n_clusters + 1, dtype=torch.int64, device=dev)
    cl_off[1:] = torch.cumsum(cl_sizes, 0)
    # centroids: single-cluster buckets use the bucket mean, others k-means means
    centroids = torch.zeros((n_clusters, b), dtype=torch.float64, device=dev)
    single = torch.nonzero(n_cl_bucket == 1).squeeze(1)
    single = single[KB[single] == 1]
    centroids[bc_off[single]] = sums[single] / sizes[single].unsqueeze(1).double()
    if "multi" in cent_parts:
        mb, nk, cm = cent_parts["multi"]
        first = bc_off[mb]
        seg = _segment_ids(nk)
        within = torch.arange(int(nk.sum()), device=dev) - (torch.cumsum(nk, 0) - nk)[seg]
        centroids[first[seg] + within] = cm
    say("directory done")
    # payload
    if head_bytes:
        big = max(chunk, 1 << 24)
        if payload_fn is not None:
            gen = (payload_fn(perm[s0:s0 + big]) for s0 in range(0, n, big))
        else:
            pn = perm.cpu().numpy()
            gen = (rows_t(pn[s0:s0 + big]) for s0 in range(0, n, big))
        rows = split_payload(gen, n, w.row_bytes, head_bytes, dev, copy=head_copy)
    elif payload_fn is not None:
        rows = payload_fn(perm)
    else:
        pn = perm.cpu().numpy()
        parts = [rows_t(pn[s0:s0 + chunk]) for s0 in range(0, n, chunk)]
        rows = torch.cat(parts) if parts else rows_t(pn[:0])
    say("payload done")
    return Index(
        workload=w, encoder=enc, tau=tau.cpu().numpy().astype(np.float32),
        rows=rows, row_ids=perm,
        bc_off=bc_off.to(torch.int64), cl_off=cl_off, centroids=centroids.to(torch.float32),
        codes=codes[perm] if keep_codes else None, head_bytes=head_bytes,
        head_copy=int(bool(head_copy and head_bytes)),
    )


def to_numpy(ix: Index) -> Index:
    """Host copies with the exact dtypes the search consumes."""
    f = lambda t: t.cpu().numpy() if isinstance(t, torch.Tensor) else t
    return Index(
        workload=ix.workload, encoder=ix.encoder, tau=ix.tau,
        rows=np.ascontiguousarray(f(ix.rows)),
        row_ids=np.ascontiguousarray(f(ix.row_ids)).astype(np.int64),
        bc_off=np.ascontiguousarray(f(ix.bc_off)).astype(np.uint32),
        cl_off=np.ascontiguousarray(f(ix.cl_off)).astype(np.uint64),
        centroids=np.ascontiguousarray(f(ix.centroids)).astype(np.float32),
        codes=None if ix.codes is None else np.ascontiguousarray(f(ix.codes)).astype(np.uint32),
        head_bytes=ix.head_bytes, head_copy=ix.head_copy,
    )
