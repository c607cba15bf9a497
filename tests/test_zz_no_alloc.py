"""nr_search_noalloc (the entry point for callers that cannot allocate)
returns exactly what nr_search returns, through the C ABI, on two calls in a
row, the second with a smaller batch; and in chunks when the batch does not
fit its fixed array at once."""
import numpy as np
import pytest
import torch

from paper_2608_15438_amd import neuroute as NR
from tests.instances import instance

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def case():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    dev = torch.device("cuda")
    w, ix, X, Q = instance(2, 60_000, 300, widths=(128, 256, 12))
    gix = NR.Index.from_built(ix, dev)
    yield w, gix, torch.from_numpy(Q).to(dev)
    gix.close()


def _params(w, **kw):
    base = dict(l_sel=min(w.b, 16), r_max=w.r_max, k_c=w.k_c, m_x=[0.0, 4.0], m_y=[1.0, 3.0])
    base.update(kw)
    return NR.Params(**base)


@pytest.mark.parametrize("mode", [NR.NR_REFINE_PER_QUERY, NR.NR_REFINE_SHARED])
def test_noalloc_matches_search_twice(case, mode):
    w, gix, Q = case
    p = _params(w, refine_mode=mode)
    for nq, P in ((300, 256), (37, 64)):   # the second call smaller
        ref_i, ref_d = gix.nr_search(Q[:nq], 10, P, p)
        ids = torch.full((nq, 10), -7, dtype=torch.int64, device=Q.device)
        dists = torch.full((nq, 10), -7.0, dtype=torch.float32, device=Q.device)
        gix.nr_search_noalloc(Q[:nq], 10, P, p, ids, dists)
        torch.cuda.synchronize()
        assert torch.equal(ids, ref_i) and torch.equal(dists, ref_d), (nq, P)


def test_noalloc_chunks_and_logits(case):
    """A batch larger than one chunk (P = 4096 and K_c = 5000 leave room for
    about 300 queries in the 64 MiB array), with caller-supplied logits."""
    w, gix, Q = case
    p = _params(w, k_c=5000, gate_on=False, early_stop_on=False)
    Qb = Q.repeat(3, 1)
    lg = gix.nr_encode(Qb)
    ref_i, ref_d = gix.nr_search(Qb, 16, 4096, p, logits=lg)
    ids = torch.empty((len(Qb), 16), dtype=torch.int64, device=Q.device)
    dists = torch.empty((len(Qb), 16), dtype=torch.float32, device=Q.device)
    gix.nr_search_noalloc(Qb, 16, 4096, p, ids, dists, logits=lg)
    torch.cuda.synchronize()
    assert torch.equal(ids, ref_i) and torch.equal(dists, ref_d)
    # then a small call again: the array keeps the last call's contents
    gix.nr_search_noalloc(Qb[:5], 16, 4096, p, ids[:5], dists[:5], logits=lg[:5])
    torch.cuda.synchronize()
    assert torch.equal(ids[:5], ref_i[:5]) and torch.equal(dists[:5], ref_d[:5])


def test_noalloc_argument_errors(case):
    w, gix, Q = case
    ids = torch.empty((4, 10), dtype=torch.int64, device=Q.device)
    dists = torch.empty((4, 10), dtype=torch.float32, device=Q.device)
    with pytest.raises(NR.NRError) as e:
        gix.nr_search_noalloc(Q[:4], 10, 5000, _params(w), ids, dists)
    assert e.value.status == NR.NR_EUNSUPPORTED
    ids64 = torch.empty((4, 65), dtype=torch.int64, device=Q.device)
    d64 = torch.empty((4, 65), dtype=torch.float32, device=Q.device)
    with pytest.raises(NR.NRError) as e:
        gix.nr_search_noalloc(Q[:4], 65, 16, _params(w), ids64, d64)
    assert e.value.status == NR.NR_EUNSUPPORTED
