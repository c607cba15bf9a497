"""Workload table: sizes, generator kinds and seeds of the evaluation cases.

Pure data.  Seeds follow one scheme: data = 1000+cfg, queries = 2000+cfg,
calibration queries = 3000+cfg, encoder = 4000+cfg, sampling = 5000+cfg.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    cfg: int                   # 1..5
    kind: str                  # "gauss" | "sift" | "deep"
    n: int                     # base rows
    d: int                     # E_dim
    n_centers: int             # mixture components
    widths: Tuple[int, ...]    # encoder widths E_dim -> ... -> L_dim
    n_queries: int
    # index construction
    tau_mode: str              # "zero" (sign) | "median"
    cluster_rule: str          # "fixed4" | "per_bucket8" | "capacity" | "none" (one per bucket)
    capacity: int = 0          # t for cluster_rule == "capacity"
    kappa: float = 50.0        # "deep" rows: noise std (1+e)^-spectrum / sqrt(kappa) in
    spectrum: float = 0.0      #   dimension e around unit centres, then normalised
    # search defaults
    k: int = 10
    l_sel: int = 16
    r_max: int = 7
    k_c: int = 512
    probe_budgets: Tuple[int, ...] = ()
    notes: str = ""

    @property
    def b(self) -> int:
        return self.widths[-1]

    @property
    def dtype(self) -> str:
        return "u8" if self.kind == "sift" else "f32"

    @property
    def row_bytes(self) -> int:
        return self.d * (1 if self.kind == "sift" else 4)

    def seed(self, what: str) -> int:
        base = {"data": 1000, "query": 2000, "calib": 3000, "encoder": 4000, "sample": 5000}[what]
        return base + self.cfg


TINY = Workload(
    name="tiny-20k-f32-d32-b8", cfg=1, kind="gauss", n=20_000, d=32, n_centers=50,
    widths=(32, 64, 8), n_queries=100, tau_mode="zero", cluster_rule="fixed4",
    l_sel=8, r_max=8, k_c=16, probe_budgets=(4, 256),
    notes="P=256 with L_sel=R_max=8, S_max=inf, gate off, K_c=inf, no early stop probes every code",
)

SIFT1M = Workload(
    name="sift-like-1M-u8-d128-b16", cfg=2, kind="sift", n=1_000_000, d=128, n_centers=1_000,
    widths=(128, 256, 16), n_queries=10_000, tau_mode="median", cluster_rule="per_bucket8",
    l_sel=16, r_max=7, k_c=512, probe_budgets=(8, 16, 32, 64, 128, 256),
)

DEEP100M = Workload(
    name="deep-like-100M-f32-d96-b20", cfg=3, kind="deep", n=100_000_000, d=96, n_centers=10_000,
    widths=(96, 256, 20), n_queries=10_000, tau_mode="median", cluster_rule="capacity",
    capacity=2000, l_sel=16, r_max=7, k_c=3000, probe_budgets=(4, 16, 64, 256),
)

SIFT1B = Workload(
    name="sift-like-1B-u8-d128-b24", cfg=4, kind="sift", n=1_000_000_000, d=128, n_centers=100_000,
    widths=(128, 256, 24), n_queries=10_000, tau_mode="median", cluster_rule="capacity",
    capacity=4000, l_sel=16, r_max=7, k_c=3000, probe_budgets=(256, 512, 640, 768, 896, 1024),
)

GLD10M = Workload(
    name="gld-like-10M-f32-d1536-b16", cfg=5, kind="deep", n=10_000_000, d=1536, n_centers=10_000,
    widths=(1536, 512, 16), n_queries=10_000, tau_mode="median",
    cluster_rule="per_bucket8", kappa=10.0, spectrum=0.75, l_sel=13, r_max=5, k_c=4000,
    probe_budgets=(16, 32, 64, 128, 256, 512, 1024),
    notes="high-dimensional regime: 6 KB rows; noise std decaying as (1+e)^-3/4 (about 5.5 "
          "effective noise dimensions, total power 0.26 x the centre's); the encoder keeps the "
          "paper's first layer 1536->512 but not its deeper stack, whose untrained form loses "
          "the neighbourhoods",
)

WORKLOADS = {w.cfg: w for w in (TINY, SIFT1M, DEEP100M, SIFT1B, GLD10M)}


def scaled(w: Workload, n: int, n_queries: Optional[int] = None, **kw) -> Workload:
    """A smaller instance with the same generator, encoder shape and rules."""
    from dataclasses import replace
    return replace(w, n=n, n_queries=n_queries if n_queries is not None else w.n_queries,
                   name=f"{w.name}@{n}", **kw)
