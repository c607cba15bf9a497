"""Parity at the benchmark's full sizes and launch configuration: the whole
10,000-query batch goes through nr_search on the 1B x 128 uint8, the
100M x 96 fp32 and the 10M x 1536 fp32 indexes (built on the GPU from the seeded generators); a
seeded sample of queries is recomputed one by one by the oracle, with the
rows of their candidate clusters staged in host memory."""
import gc

import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_15438_amd import index_build as IB
from paper_2608_15438_amd import neuroute as NR
from synth import configs as CF
from synth import generators as G
from synth.gpu import GpuRows
from tests.instances import head_bytes_for, stage_rows

pytestmark = pytest.mark.gpu

GATE = dict(m_x=[0.0, 1.0], m_y=[0.5, 2.0])


# layout: "copy" = head plane + whole rows (the benchmark's), "split" = head
# plane + tails, "rows" = row-major
@pytest.mark.parametrize("cfg,P,mode,layout", [(4, 640, NR.NR_REFINE_AUTO, "copy"),
                                                (4, 640, NR.NR_REFINE_PER_QUERY, "copy"),
                                                (4, 520, NR.NR_REFINE_AUTO, "split"),
                                                (3, 256, NR.NR_REFINE_AUTO, "copy"),
                                                (3, 256, NR.NR_REFINE_AUTO, "rows"),
                                                (5, 64, NR.NR_REFINE_AUTO, "copy")])
def test_full_size_sampled_queries(cfg, P, mode, layout):
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    dev = torch.device("cuda")
    w = CF.WORKLOADS[cfg]
    data = GpuRows(w, "data", dev)
    ix = IB.build_index(w, data, device=dev, keep_codes=False, payload_fn=lambda p: data(p),
                        head_bytes=0 if layout == "rows" else head_bytes_for(w),
                        head_copy=layout == "copy")
    try:
        gix = NR.Index.from_built(ix, dev)
        Q = GpuRows(w, "query", dev).range(0, w.n_queries)
        Qh = Q.cpu().numpy()
        e = ix.encoder
        enc = O.Encoder(e.weights, e.biases, input_scale=e.input_scale)
        lg, mag = O.encode(enc, Qh, with_mag=True)
        params = NR.Params(l_sel=16, r_max=w.r_max, k_c=w.k_c, refine_mode=mode, **GATE)
        ids, dists = gix.nr_search(Q, w.k, P, params, logits=torch.from_numpy(lg).to(dev))
        ids, dists = ids.cpu().numpy(), dists.cpu().numpy()
        # a seeded sample spread over the batch
        samp = np.sort(G.seeded_permutation(w.seed("sample"), w.n_queries)[:24])
        glg = gix.nr_encode(Q).cpu().numpy()
        assert np.all(np.abs(glg.astype(np.float64) - lg) <= 1e-4 * mag)
        bc = ix.bc_off.cpu().numpy().astype(np.uint32)
        cent = ix.centroids.cpu().numpy()
        prm = O.RouteParams(k_c=w.k_c, m_x=np.array(GATE["m_x"], np.float32),
                            m_y=np.array(GATE["m_y"], np.float32))
        codes, costs, bins, cnt = O.probes(lg[samp], ix.tau, 16, w.r_max, P)
        lists = O.route(lg[samp], codes, bins, cnt, bc, cent, prm)
        rows, rid, cl2 = stage_rows(ix, lists)
        oi, od, _ = O.refine(rows, rid, cl2, Qh[samp], lists, w.k)
        if w.dtype == "u8":
            assert np.array_equal(ids[samp], oi)
            assert np.array_equal(dists[samp], od)
        else:
            for j, q in enumerate(samp):
                if np.array_equal(ids[q], oi[j]):
                    assert np.allclose(dists[q], od[j], rtol=1e-5, atol=1e-6)
                else:  # near-tie: the GPU list is still a valid top-k within 2e-5
                    assert np.all(dists[q] <= od[j][-1] * (1 + 2e-5) + 1e-6)
        gix.close()
    finally:
        del ix
        gc.collect()
        torch.cuda.empty_cache()
