"""The HIP row generator reproduces the NumPy generator (same Philox stream)."""
import numpy as np
import pytest
import torch

from synth import configs as CF
from synth import generators as G
from synth.gpu import GpuRows

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch.device("cuda")


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_gpu_rows_match_numpy(dev, cfg):
    w = CF.WORKLOADS[cfg]
    ids = np.concatenate([np.arange(300), np.array([w.n - 1, 123457 % w.n, 7])])
    for which in ("data", "query"):
        g = GpuRows(w, which, dev)
        got = g(torch.from_numpy(ids)).cpu().numpy()
        exp = __import__("paper_2608_15438_amd.index_build", fromlist=["x"]).cpu_row_source(w, which)(ids)
        if w.kind == "sift":
            assert np.array_equal(got, exp)
        elif w.kind == "gauss":
            assert np.array_equal(got, exp)
        else:
            # unit rows: the final fp64 square root may round differently;
            # allow one fp32 ulp
            assert np.all(np.abs(got - exp) <= np.spacing(np.abs(exp)))
        # a contiguous id range gives the same rows as the explicit ids
        assert np.array_equal(g.range(5, 40).cpu().numpy(), g(torch.arange(5, 45)).cpu().numpy())
