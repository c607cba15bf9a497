"""GPU row generator (synth/csrc/synth_gen.hip): the same rows as
synth.generators, produced on the device, e.g. directly in permuted order."""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np
import torch

from . import generators as G

_HERE = os.path.dirname(os.path.abspath(__file__))
SO = os.path.join(_HERE, "libsynth_gen.so")
_lib = None


def build() -> str:
    src = os.path.join(_HERE, "csrc", "synth_gen.hip")
    tmp = SO + ".tmp"
    subprocess.check_call(["/opt/rocm/bin/hipcc", "-O3", "-fPIC", "-shared", "--offload-arch=gfx950",
                           "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang",
                           "-packed-fp32-ops", "-o", tmp, src],
                          stderr=subprocess.DEVNULL)
    os.replace(tmp, SO)
    return SO


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(SO):
            raise RuntimeError(f"{SO} missing: run synth.gpu.build()")
        L = C.CDLL(SO)
        L.synth_rows.argtypes = [C.c_int, C.c_uint32, C.c_void_p, C.c_int64, C.c_int, C.c_double,
                                 C.c_void_p, C.c_void_p, C.c_int64, C.c_int64, C.c_void_p,
                                 C.c_void_p]
        L.synth_rows.restype = C.c_int
        _lib = L
    return _lib


class GpuRows:
    """rows(ids) on the device for one workload's data or query stream."""

    KIND = {"sift": 0, "deep": 1, "gauss": 2}

    def __init__(self, w, which="data", device="cuda"):
        self.w = w
        self.seed = w.seed(which)
        seed_c = w.seed("data")
        if w.kind == "sift":
            c = G.sift_centers(seed_c, w.n_centers, w.d)
            self.param = 12.0
        elif w.kind == "deep":
            c = G.unit_centers(seed_c, w.n_centers, w.d)
            self.param = 0.0
        else:
            c = G.gauss_centers(seed_c, w.n_centers, w.d)
            self.param = 1.0
        self.device = torch.device(device)
        self.centers = torch.from_numpy(np.ascontiguousarray(c, np.float64)).to(self.device)
        self.scale = None
        if w.kind == "deep":
            self.scale = torch.from_numpy(G.noise_scale(w.d, w.kappa, w.spectrum)).to(self.device)
        self.dtype = torch.uint8 if w.kind == "sift" else torch.float32

    def _run(self, ids_t, first, m, out):
        st = torch.cuda.current_stream(self.device).cuda_stream
        rc = lib().synth_rows(self.KIND[self.w.kind], self.seed, self.centers.data_ptr(),
                              self.centers.shape[0], self.w.d, self.param,
                              None if self.scale is None else self.scale.data_ptr(),
                              None if ids_t is None else ids_t.data_ptr(), first, m,
                              out.data_ptr(), C.c_void_p(st))
        if rc != 0:
            raise RuntimeError(f"synth_rows failed with hipError {rc}")
        return out

    def range(self, first, m, out=None):
        out = out if out is not None else torch.empty((m, self.w.d), dtype=self.dtype, device=self.device)
        return self._run(None, first, m, out)

    def __call__(self, ids, out=None):
        if isinstance(ids, np.ndarray):
            if ids.ndim == 1 and len(ids) > 0 and np.all(np.diff(ids) == 1):
                return self.range(int(ids[0]), len(ids), out)
            ids = torch.from_numpy(ids.astype(np.int64))
        ids_t = ids.to(self.device, torch.int64).contiguous()
        m = ids_t.shape[0]
        out = out if out is not None else torch.empty((m, self.w.d), dtype=self.dtype, device=self.device)
        return self._run(ids_t, 0, m, out)
