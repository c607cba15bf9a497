"""Parity at the benchmark's full sizes and launch configuration: the whole
10,000-query batch goes through nr_search on indexes built on the GPU from
the seeded generators:
  * 1M x 128 uint8 (b = 16, ~8 clusters per bucket, the batch-shared
    schedule): every one of the 10,000 lists against the oracle;
  * 1B x 128 uint8 as the benchmark times it (L_sim-trained encoder, gate
    margin calibrated at the 95th percentile from bootstrapped targets,
    P = 304, head plane + whole rows) and with the seeded encoder in three
    layouts and both schedules;
  * 100M x 96 fp32 and 10M x 1536 fp32;
the large ones on a seeded sample of queries that the oracle recomputes one
by one, with the rows of their candidate clusters staged in host memory.
The oracle's logits are passed to the search (nr_search_ex), so that lists
must agree exactly (Sec. 3.1 ties by lower id; fp32 near-ties per R27);
the GPU encoder's own logits are checked against the oracle's separately."""
import gc
import os

import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_15438_amd import calibrate as CAL
from paper_2608_15438_amd import index_build as IB
from paper_2608_15438_amd import neuroute as NR
from synth import configs as CF
from synth import generators as G
from synth.gpu import GpuRows
from tests.instances import head_bytes_for, stage_rows
from tests.topk_check import allowed_ids, check_topk

pytestmark = pytest.mark.gpu

GATE = dict(m_x=[0.0, 1.0], m_y=[0.5, 2.0])


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda")


def _build(w, dev, layout, encoder=None):
    data = GpuRows(w, "data", dev)
    return IB.build_index(w, data, device=dev, keep_codes=False, payload_fn=lambda p: data(p),
                          head_bytes=0 if layout == "rows" else head_bytes_for(w),
                          head_copy=layout == "copy", encoder=encoder)


def _oracle_encoder(ix):
    e = ix.encoder
    return O.Encoder(e.weights, e.biases, e.bn_scale or (), e.bn_shift or (), e.input_scale)


def _route_params(p: NR.Params) -> O.RouteParams:
    return O.RouteParams(n_bins=p.n_bins, s_max=p.s_max, k_c=p.k_c, b_batch=p.b_batch,
                         b_min=p.b_min, t_low=p.t_low, u_heap=p.u_heap, u_front=p.u_front,
                         alpha_front=p.alpha_front, gate_on=p.gate_on,
                         early_stop_on=p.early_stop_on, lowq_or=p.lowq_or,
                         m_x=np.array(p.m_x, np.float32), m_y=np.array(p.m_y, np.float32))


def _check_sample(w, ix, gix, Q, lg, mag, P, params, samp):
    """Search the whole batch with the oracle's logits; recompute the sampled
    queries with the oracle over staged rows; check the GPU encoder too."""
    dev = Q.device
    Qh = Q.cpu().numpy()
    ids, dists = gix.nr_search(Q, w.k, P, params, logits=torch.from_numpy(lg).to(dev))
    ids, dists = ids.cpu().numpy(), dists.cpu().numpy()
    glg = gix.nr_encode(Q).cpu().numpy()
    assert np.all(np.abs(glg.astype(np.float64) - lg) <= 1e-4 * mag)
    bc = ix.bc_off.cpu().numpy().astype(np.uint32)
    cent = ix.centroids.cpu().numpy()
    codes, costs, bins, cnt = O.probes(lg[samp], ix.tau, params.l_sel, params.r_max, P,
                                       params.s_max, params.n_bins)
    lists = O.route(lg[samp], codes, bins, cnt, bc, cent, _route_params(params))
    rows, rid, cl2 = stage_rows(ix, lists)
    oi, od, _ = O.refine(rows, rid, cl2, Qh[samp], lists, w.k)
    # staged rows by original id, for recomputing the GPU's distances
    order = np.argsort(rid)
    rid_sorted = rid[order]

    def x_by_id(q_ids):
        pos = np.searchsorted(rid_sorted, q_ids)
        assert np.array_equal(rid_sorted[np.minimum(pos, len(rid_sorted) - 1)], q_ids)
        return rows[order[pos]]

    check_topk(ids[samp], dists[samp], oi, od, is_u8=w.dtype == "u8", X_by_id=x_by_id,
               Q=Qh[samp], allowed=lambda j: allowed_ids(cl2, rid, lists[j]))


def _free(*objs):
    for o in objs:
        if hasattr(o, "close"):
            o.close()
    gc.collect()
    torch.cuda.empty_cache()


# layout: "copy" = head plane + whole rows (the benchmark's), "split" = head
# plane + tails, "rows" = row-major
@pytest.mark.parametrize("cfg,P,mode,layout", [(4, 640, NR.NR_REFINE_AUTO, "copy"),
                                                (4, 640, NR.NR_REFINE_PER_QUERY, "copy"),
                                                (4, 520, NR.NR_REFINE_AUTO, "split"),
                                                (3, 256, NR.NR_REFINE_AUTO, "copy"),
                                                (3, 256, NR.NR_REFINE_AUTO, "rows"),
                                                (5, 64, NR.NR_REFINE_AUTO, "copy")])
def test_full_size_sampled_queries(cfg, P, mode, layout):
    dev = _dev()
    w = CF.WORKLOADS[cfg]
    ix = _build(w, dev, layout)
    try:
        gix = NR.Index.from_built(ix, dev)
        Q = GpuRows(w, "query", dev).range(0, w.n_queries)
        lg, mag = O.encode(_oracle_encoder(ix), Q.cpu().numpy(), with_mag=True)
        params = NR.Params(l_sel=16, r_max=w.r_max, k_c=w.k_c, refine_mode=mode, **GATE)
        samp = np.sort(G.seeded_permutation(w.seed("sample"), w.n_queries)[:24])
        _check_sample(w, ix, gix, Q, lg, mag, P, params, samp)
        gix.close()
    finally:
        del ix
        _free()


@pytest.mark.parametrize("P,k_c,seed", [(64, 512, 0), (128, 64, 256)])
def test_sift1m_every_query(P, k_c, seed):
    """1M x 128 uint8, b = 16, ~8 clusters per bucket: the one workload where
    the centroid stage scores hundreds of centroids per query.  All 10,000
    queries in one call equal the oracle's lists, bit for bit: at the
    benchmark's settings (P = 64 leaves ~1,000 rows per query, all in the
    seed pass) and with a 256-row seed, so that most clusters go through the
    batch-shared scan; K_c = 64 makes the heap fill, so the early stop fires."""
    dev = _dev()
    w = CF.WORKLOADS[2]
    ix = _build(w, dev, "copy")
    try:
        gix = NR.Index.from_built(ix, dev)
        Q = GpuRows(w, "query", dev).range(0, w.n_queries)
        Qh = Q.cpu().numpy()
        enc = _oracle_encoder(ix)
        lg = O.encode(enc, Qh)
        params = NR.Params(l_sel=16, r_max=w.r_max, k_c=k_c, shared_seed_rows=seed, **GATE)
        ids, dists, qs = gix.nr_search(Q, w.k, P, params, logits=torch.from_numpy(lg).to(dev),
                                       qstats=True)
        qs = qs.cpu().numpy()
        assert qs[:, NR.QS["scored"]].mean() > 10
        if seed:
            work = gix.nr_last_work()
            assert work["shared_pairs"] > 0 and work["flagged"] == 0
            assert qs[:, NR.QS["stopped"]].sum() > 0
        rows = IB.payload_range(ix, 0, w.n).cpu().numpy()
        oi, od, _, _ = O.search(enc, ix.tau, rows, ix.row_ids.cpu().numpy(),
                                ix.bc_off.cpu().numpy().astype(np.uint32),
                                ix.cl_off.cpu().numpy().astype(np.uint64),
                                ix.centroids.cpu().numpy(), Qh, w.k, 16, w.r_max, P,
                                _route_params(params),
                                n_threads=min(16, len(os.sched_getaffinity(0))))
        check_topk(ids.cpu().numpy(), dists.cpu().numpy(), oi, od, is_u8=True)
        gix.close()
    finally:
        del ix
        _free()


def test_sift1b_benchmark_index():
    """The 1B x 128 uint8 index as the benchmark builds it: the seeded
    encoder trained with L_sim (fewer steps than the benchmark's), the gate
    margin M fitted at the 95th percentile on 300 calibration queries whose
    targets come from the search itself at the largest budget with gate and
    early stop off (Sec. 3.4 "Calibration"), P = 304, head plane + whole
    rows, the batch-shared schedule; 256 sampled queries."""
    from paper_2608_15438_amd import train as TR
    dev = _dev()
    w = CF.WORKLOADS[4]
    data = GpuRows(w, "data", dev)
    enc = TR.train_encoder(IB.seeded_encoder(w), data, w.n, 300, batch=4096, lr=2e-4, gamma=0.6,
                           seed=w.seed("sample"), device=dev)
    ix = _build(w, dev, "copy", encoder=enc)
    try:
        gix = NR.Index.from_built(ix, dev)
        Qc = GpuRows(w, "calib", dev).range(0, 300)
        loose = NR.Params(l_sel=16, r_max=w.r_max, k_c=w.k_c, gate_on=False, early_stop_on=False)
        targets = CAL.bootstrap_targets(gix, Qc, w.k, 1024, loose)
        row_of_id = torch.empty_like(ix.row_ids)
        row_of_id[ix.row_ids] = torch.arange(w.n, device=dev)
        lgc = IB._TorchEncoder(ix.encoder, dev)(Qc)
        xs, ys = CAL.margin_points(lgc, targets, row_of_id, ix.cl_off, ix.bc_off, ix.centroids)
        del row_of_id
        m_x, m_y = CAL.fit_margin(xs, ys, 0.95)
        params = NR.Params(l_sel=16, r_max=w.r_max, k_c=w.k_c, m_x=m_x.tolist(),
                           m_y=m_y.tolist())
        Q = GpuRows(w, "query", dev).range(0, w.n_queries)
        lg, mag = O.encode(_oracle_encoder(ix), Q.cpu().numpy(), with_mag=True)
        samp = np.sort(G.seeded_permutation(w.seed("sample"), w.n_queries)[:256])
        _check_sample(w, ix, gix, Q, lg, mag, 304, params, samp)
        gix.close()
    finally:
        del ix
        _free()


# the sweep on the 100M x 96 fp32 index: probe budget x gate margin x early
# stop x batch size (a batch of 1 or 256 queries runs the per-query schedule,
# the whole batch the shared one); margins: loose / default / tight knots
_SWEEP_GATES = {"loose": dict(m_x=[0.0, 1.0], m_y=[1.0, 4.0]),
                "default": GATE,
                "tight": dict(m_x=[0.0, 1.0], m_y=[0.1, 0.5])}


@pytest.fixture(scope="module")
def deep100m():
    dev = _dev()
    w = CF.WORKLOADS[3]
    ix = _build(w, dev, "copy")
    gix = NR.Index.from_built(ix, dev)
    Q = GpuRows(w, "query", dev).range(0, w.n_queries)
    lg, mag = O.encode(_oracle_encoder(ix), Q.cpu().numpy(), with_mag=True)
    yield w, ix, gix, Q, lg, mag
    gix.close()
    del ix
    _free()


@pytest.mark.parametrize("P,gate,es,batch", [(4, "tight", True, 10_000), (16, "loose", False, 256),
                                             (64, "default", True, 1), (256, "tight", False, 10_000),
                                             (256, "loose", True, 256)])
def test_deep100m_sweep_points(deep100m, P, gate, es, batch):
    w, ix, gix, Q, lg, mag = deep100m
    dev = Q.device
    params = NR.Params(l_sel=16, r_max=w.r_max, k_c=w.k_c, early_stop_on=es, **_SWEEP_GATES[gate])
    samp = np.sort(G.seeded_permutation(w.seed("sample") + P, w.n_queries)[:16])
    if batch >= w.n_queries:
        _check_sample(w, ix, gix, Q, lg, mag, P, params, samp)
        return
    # the sampled queries inside batches of `batch` queries (one call each)
    lgd = torch.from_numpy(lg).to(dev)
    ids = torch.empty((w.n_queries, w.k), dtype=torch.int64, device=dev)
    dists = torch.empty((w.n_queries, w.k), dtype=torch.float32, device=dev)
    for q in samp:
        s0 = (int(q) // batch) * batch
        i, d = gix.nr_search(Q[s0:s0 + batch], w.k, P, params, logits=lgd[s0:s0 + batch])
        ids[s0:s0 + batch], dists[s0:s0 + batch] = i, d
    ids, dists = ids.cpu().numpy(), dists.cpu().numpy()
    bc = ix.bc_off.cpu().numpy().astype(np.uint32)
    codes, costs, bins, cnt = O.probes(lg[samp], ix.tau, 16, w.r_max, P)
    lists = O.route(lg[samp], codes, bins, cnt, bc, ix.centroids.cpu().numpy(),
                    _route_params(params))
    rows, rid, cl2 = stage_rows(ix, lists)
    oi, od, _ = O.refine(rows, rid, cl2, Q.cpu().numpy()[samp], lists, w.k)
    order = np.argsort(rid)
    rid_sorted = rid[order]
    Qh = Q.cpu().numpy()
    check_topk(ids[samp], dists[samp], oi, od, is_u8=False,
               X_by_id=lambda q_ids: rows[order[np.searchsorted(rid_sorted, q_ids)]],
               Q=Qh[samp], allowed=lambda j: allowed_ids(cl2, rid, lists[j]))
