"""Index construction through the library's kernels (Sec. 3.3 "Bucket
allocation" and "In-bucket clustering", thresholds per Sec. 3.2.3), untimed:

1. latents of every base row: the encoder kernel (nr_encode) on an
   encoder-only index, in chunks;
2. tau: the lower median per dimension over the same seeded sample of rows
   the reference builder uses (nr_build_tau; "zero" workloads use tau = 0);
3. codes (Eq. 10) and bucket sizes (nr_build_codes);
4. clusters per bucket from the workload's rule (nr_build_plan);
5. the k-means++ draws of the multi-cluster buckets from the seeded
   generator (the same Philox uniforms as the reference builder), then
   bucket order, bucket-local k-means, directory and centroids
   (nr_build_index);
6. the payload laid out in the returned row order (a gather, as in the
   reference builder).

Python here only allocates device buffers and moves the seeded draws in; every
step of the construction runs in the library's kernels.
"""
from __future__ import annotations

from typing import Callable, Optional

import numpy as np
import torch

from synth import generators as G
from synth.configs import Workload
from . import index_build as IB
from . import neuroute as NR

_RULES = {"none": (NR.NR_CLUSTER_NONE, 1), "fixed4": (NR.NR_CLUSTER_FIXED, 4),
          "per_bucket8": (NR.NR_CLUSTER_PER_BUCKET, 8)}


def encode_base(eix: NR.Index, rows_fn: Callable, n: int, b: int, device, chunk: int = 1 << 20):
    """Latents [n, b] fp32 of rows 0..n-1 through the encoder kernel."""
    lg = torch.empty((n, b), dtype=torch.float32, device=device)
    for s0 in range(0, n, chunk):
        ids = np.arange(s0, min(n, s0 + chunk))
        x = rows_fn(ids)
        x = torch.as_tensor(x).to(device).contiguous()
        lg[s0:s0 + len(ids)] = eix.nr_encode(x)
    return lg


def build_index_gpu(w: Workload, rows_fn: Callable, device="cuda", encoder=None,
                    chunk: int = 1 << 20, payload_fn: Optional[Callable] = None,
                    head_bytes: int = 0, head_copy: bool = False, log=None,
                    return_logits: bool = False):
    """The index of workload ``w`` built by the library's construction kernels;
    the arguments follow index_build.build_index."""
    dev = torch.device(device)
    say = log or (lambda *a: None)
    enc = encoder or IB.seeded_encoder(w)
    b, n = w.b, w.n
    eix = NR.Index.encoder_only(enc, NR.NR_U8 if w.dtype == "u8" else NR.NR_F32)
    lg = encode_base(eix, rows_fn, n, b, dev, chunk)
    eix.close()
    say("latents done")
    if w.tau_mode == "zero":
        tau = torch.zeros(b, dtype=torch.float32, device=dev)
    else:
        ids = torch.from_numpy(IB.tau_sample_ids(w.seed("sample"), n, min(n, IB.TAU_SAMPLE)))
        tau = NR.nr_build_tau(lg[ids.to(dev)].contiguous())
    codes = torch.empty(n, dtype=torch.int32, device=dev)
    sizes = torch.zeros(1 << b, dtype=torch.int32, device=dev)
    NR.nr_build_codes(lg, tau, codes, sizes)
    rule, param = _RULES.get(w.cluster_rule, (NR.NR_CLUSTER_CAPACITY, w.capacity))
    kb, mlist, info = NR.nr_build_plan(sizes, n, b, rule, param)
    say(f"plan: {info.max_clusters} cluster slots, {info.n_multi} multi-cluster buckets")
    nm, kmax = int(info.n_multi), int(max(info.kmax, 2))
    if nm:
        mcodes = mlist[:nm].cpu().numpy().astype(np.int64)
        U = torch.from_numpy(G.uniform01(w.seed("sample"), mcodes, kmax, G.TAG_SAMPLE + 16)).to(dev)
    else:
        U = torch.zeros((1, kmax), dtype=torch.float64, device=dev)
    mc = int(info.max_clusters)
    row_ids = torch.empty(n, dtype=torch.int64, device=dev)
    bc_off = torch.empty((1 << b) + 1, dtype=torch.int32, device=dev)
    cl_off = torch.empty(mc + 1, dtype=torch.int64, device=dev)
    cent = torch.empty((mc, b), dtype=torch.float32, device=dev)
    desc = NR.nr_build_desc(n=n, b=b, logits=lg.data_ptr(), codes=codes.data_ptr(),
                            sizes=sizes.data_ptr(), kb=kb.data_ptr(), mlist=mlist.data_ptr(),
                            max_clusters=mc, n_multi=nm, kmax=kmax, uniforms=U.data_ptr(),
                            seed=w.seed("sample"), lloyd=IB.N_LLOYD,
                            sample_per_cluster=IB.SAMPLE_PER_CLUSTER)
    nc = NR.nr_build_index(desc, row_ids, bc_off, cl_off, cent)
    say(f"index done: {nc} clusters")
    del U, kb, mlist, sizes
    # payload in the built row order
    if head_bytes:
        big = max(chunk, 1 << 24)
        if payload_fn is not None:
            gen = (payload_fn(row_ids[s0:s0 + big]) for s0 in range(0, n, big))
        else:
            pn = row_ids.cpu().numpy()
            gen = (torch.as_tensor(rows_fn(pn[s0:s0 + big])).to(dev) for s0 in range(0, n, big))
        rows = IB.split_payload(gen, n, w.row_bytes, head_bytes, dev, copy=head_copy)
    elif payload_fn is not None:
        rows = payload_fn(row_ids)
    else:
        rows = torch.as_tensor(rows_fn(row_ids.cpu().numpy())).to(dev)
    ix = IB.Index(workload=w, encoder=enc, tau=tau.cpu().numpy().astype(np.float32), rows=rows,
                  row_ids=row_ids, bc_off=bc_off.to(torch.int64), cl_off=cl_off[:nc + 1],
                  centroids=cent[:nc], codes=None, head_bytes=head_bytes,
                  head_copy=int(bool(head_copy and head_bytes)))
    return (ix, lg, codes) if return_logits else ix
