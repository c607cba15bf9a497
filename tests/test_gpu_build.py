"""Index construction on the GPU (nr_build_tau / nr_build_codes /
nr_build_plan / nr_build_index, Sec. 3.3) against the reference builder run
on the CPU with the same fp32 latents (the encoder kernel's): thresholds,
codes, directory, cluster offsets and row order bit for bit, centroids
within 1e-5 (counted exact), and the search over the two indexes identical.
Cases: 1M x 128 uint8 at full size (b = 16, ~8 clusters per bucket); a
60k-row index with 16 large buckets (sorts past the LDS size, larger k-means
samples); the tiny fp32 case (tau = 0, four clusters per bucket)."""
import numpy as np
import pytest
import torch

from paper_2608_15438_amd import gpu_build as GB
from paper_2608_15438_amd import index_build as IB
from paper_2608_15438_amd import neuroute as NR
from synth import configs as CF
from synth.gpu import GpuRows
from tests.instances import instance

pytestmark = pytest.mark.gpu


def _dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda")


def _compare(w, ixg, lg, codes_g, ixr, dev, Q, P):
    assert np.array_equal(ixg.tau.view(np.uint32), ixr.tau.view(np.uint32))
    rid_r = np.asarray(ixr.row_ids.cpu() if hasattr(ixr.row_ids, "cpu") else ixr.row_ids)
    cg = codes_g.cpu().numpy().view(np.uint32)
    lgh = lg.cpu().numpy()
    exp_codes = ((lgh >= ixr.tau) * (1 << np.arange(w.b))).sum(1).astype(np.uint32)
    assert np.array_equal(cg, exp_codes)
    f = lambda t: t.cpu().numpy() if isinstance(t, torch.Tensor) else np.asarray(t)
    assert np.array_equal(f(ixg.bc_off).astype(np.int64), f(ixr.bc_off).astype(np.int64))
    assert np.array_equal(f(ixg.cl_off).astype(np.int64), f(ixr.cl_off).astype(np.int64))
    assert np.array_equal(f(ixg.row_ids), rid_r)
    cgc, crc = f(ixg.centroids), f(ixr.centroids)
    assert cgc.shape == crc.shape
    diff = np.abs(cgc.astype(np.float64) - crc)
    assert np.all(diff <= 1e-5 * np.maximum(1.0, np.abs(crc)))
    n_exact = int((cgc == crc).sum())
    print(f"build parity {w.name}: {ixg.n_clusters} clusters, {n_exact}/{cgc.size} "
          "centroid values bit-equal")
    # the search over both indexes
    gg = NR.Index.from_built(ixg, dev)
    gr = NR.Index.from_built(ixr, dev)
    qlg = gg.nr_encode(Q)
    p = NR.Params(l_sel=min(w.l_sel, w.b), r_max=w.r_max, k_c=w.k_c, m_x=[0.0, 1.0],
                  m_y=[0.5, 2.0])
    a = gg.nr_search(Q, w.k, P, p, logits=qlg)
    r = gr.nr_search(Q, w.k, P, p, logits=qlg)
    assert torch.equal(a[0], r[0]) and torch.equal(a[1], r[1])
    gg.close()
    gr.close()


@pytest.mark.parametrize("case", ["tiny", "big_buckets"])
def test_gpu_build_small(case):
    dev = _dev()
    if case == "tiny":
        w, _, X, Q = instance(1)
    else:
        w, _, X, Q = instance(2, 60_000, 200, widths=(128, 256, 4), cluster_rule="capacity",
                              capacity=500)
    src = IB.array_row_source(X)
    ixg, lg, codes = GB.build_index_gpu(w, src, device=dev, return_logits=True)
    lgh = lg.cpu().numpy()
    ixr = IB.build_index(w, src, device="cpu", logits_fn=lambda ids: lgh[np.asarray(ids)])
    _compare(w, ixg, lg, codes, ixr, dev, torch.from_numpy(Q).to(dev), 64)


def test_gpu_build_sift1m_full_size():
    dev = _dev()
    w = CF.WORKLOADS[2]
    data = GpuRows(w, "data", dev)
    ixg, lg, codes = GB.build_index_gpu(w, data, device=dev, return_logits=True,
                                        payload_fn=lambda perm: data(perm))
    lgh = lg.cpu().numpy()
    ixr = IB.build_index(w, None, device="cpu", keep_codes=False,
                         logits_fn=lambda ids: lgh[np.asarray(ids)],
                         payload_fn=lambda perm: data(perm.to(dev)))
    Q = GpuRows(w, "query", dev).range(0, w.n_queries)
    _compare(w, ixg, lg, codes, ixr, dev, Q, 64)
