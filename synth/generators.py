"""Seeded synthetic workloads that stand in for the paper's data sets.

Every random number comes from Philox4x32-10 keyed by a seed and addressed by
(call, row, tag), so any row can be regenerated alone and the HIP generator in
``synth/csrc/synth_gen.hip`` reproduces the same bytes.  The Gaussian noise is
the Irwin-Hall(12) sum of twelve 16-bit uniforms, centred and scaled to unit
variance; it is built from integer sums and exactly representable fp64 steps so
that the CPU and GPU generators agree bit for bit (uint8 rows) and to the last
fp32 bit except for the final square root of the fp32 (unit-norm) rows.

Workload shapes (the paper's evaluation data, Sec. 4.1 and Table 1):
* SIFT-like: uint8 rows, d=128, a mixture of centres uniform in [0,160]^d
  plus sigma=12 noise, rounded half-to-even and clipped to [0,255];
* Deep-like: fp32 unit-norm rows, d=96, a mixture of unit centres plus
  N(0, I/kappa) noise with kappa=50, then L2-normalised;
* GLD-like (the high-dimensional regime of Sec. 4.1): the same construction
  at d=1536, with a noise std that decays as (1+e)^-3/4 over the dimensions
  so that the rows have a low intrinsic dimension, as image embeddings do;
* Gaussian mixture: fp32 rows, centres ~ N(0, 4I), unit noise (tiny case).

Nothing here computes any part of the search method.
"""
from __future__ import annotations

import numpy as np

from .philox import philox4x32_10

TAG_COMP = 1      # mixture-component draw of a row
TAG_NOISE = 2     # per-element noise of a row
TAG_CENTER = 3    # mixture centres
TAG_WEIGHT = 4    # encoder weights (layer index in c2)
TAG_SAMPLE = 5    # sub-sampling permutations

IH_CENTRE = 393210          # 12 * (65536 - 1) / 2, the mean of twelve u16 draws
IH_SCALE = 1.0 / 65536.0    # unit variance after centring (Irwin-Hall(12) has var 12/12)


def _u32_words(seed, rows, n_words, tag):
    """Philox words for each row: array [len(rows), n_words] of uint32.

    Word w of row r is word (w % 4) of Philox(counter=(w // 4, r_lo, r_hi, tag),
    key=(seed, 0)).
    """
    rows = np.asarray(rows, dtype=np.uint64)
    n_calls = (n_words + 3) // 4
    lo = (rows & np.uint64(0xFFFFFFFF)).astype(np.uint32)[:, None]
    hi = (rows >> np.uint64(32)).astype(np.uint32)[:, None]
    calls = np.arange(n_calls, dtype=np.uint32)[None, :]
    w0, w1, w2, w3 = philox4x32_10(calls, lo, hi, np.uint32(tag), seed, 0)
    out = np.stack([w0, w1, w2, w3], axis=-1).reshape(len(rows), n_calls * 4)
    return out[:, :n_words]


def irwin_hall_normals(seed, rows, d, tag=TAG_NOISE, chunk=0):
    """Approximately standard-normal fp64 values [len(rows), d].

    Element e of a row sums the twelve u16 draws with indices 12e..12e+11 of
    that row's stream (u16 index t is half t%2 of word t//2, low half first),
    then centres and scales the exact integer sum.
    """
    rows = np.asarray(rows, dtype=np.int64)
    n16 = 12 * d
    # about 64K Philox calls per block keeps the working arrays cache-sized
    chunk = chunk or max(1, 65536 // ((n16 // 2 + 3) // 4))
    out = np.empty((len(rows), d), dtype=np.float64)
    for s0 in range(0, len(rows), chunk):
        words = _u32_words(seed, rows[s0:s0 + chunk], (n16 + 1) // 2, tag)
        halves = np.ascontiguousarray(words).view("<u2")[:, :n16]
        s = halves.reshape(-1, d, 12).sum(axis=2, dtype=np.int64)
        out[s0:s0 + chunk] = (s - IH_CENTRE).astype(np.float64) * IH_SCALE
    return out


def component_of(seed, rows, n_centers):
    """Mixture component of each row: floor(u32 * C / 2^32) (multiply-shift)."""
    w = _u32_words(seed, rows, 1, TAG_COMP)[:, 0].astype(np.uint64)
    return ((w * np.uint64(n_centers)) >> np.uint64(32)).astype(np.int64)


def uniform01(seed, rows, n, tag):
    """fp64 uniforms (u32 + 0.5) / 2^32 in (0, 1), shape [len(rows), n]."""
    w = _u32_words(seed, rows, n, tag).astype(np.float64)
    return (w + 0.5) * (1.0 / 4294967296.0)


# --------------------------------------------------------------------------
# mixture centres
# --------------------------------------------------------------------------

def sift_centers(seed, n_centers, d, hi=160.0):
    """Centres uniform in [0, hi]^d, fp64 [n_centers, d]."""
    return hi * uniform01(seed, np.arange(n_centers), d, TAG_CENTER)


def unit_centers(seed, n_centers, d):
    """Unit-norm centres normalize(N(0, I)), fp64 [n_centers, d]."""
    g = irwin_hall_normals(seed, np.arange(n_centers), d, TAG_CENTER)
    return g / np.sqrt((g * g).sum(axis=1, keepdims=True))


def gauss_centers(seed, n_centers, d, std=2.0):
    """Centres ~ N(0, std^2 I), fp64 [n_centers, d]."""
    return std * irwin_hall_normals(seed, np.arange(n_centers), d, TAG_CENTER)


# --------------------------------------------------------------------------
# rows
# --------------------------------------------------------------------------

def sift_rows(seed, centers, rows, sigma=12.0):
    """uint8 rows clip(rint(centre + sigma * z), 0, 255) for the given row ids."""
    rows = np.asarray(rows, dtype=np.int64)
    d = centers.shape[1]
    comp = component_of(seed, rows, centers.shape[0])
    z = irwin_hall_normals(seed, rows, d)
    # sigma * IH_SCALE is a power-of-two multiple of 3 for sigma=12, so the
    # product is exact and the only rounding is the final rint.
    x = centers[comp] + z * sigma
    return np.clip(np.rint(x), 0, 255).astype(np.uint8)


def noise_scale(d, kappa=50.0, spectrum=0.0):
    """Per-dimension noise std of unit rows: (1 + e)^-spectrum / sqrt(kappa),
    fp64 [d] (a constant 1 / sqrt(kappa) for spectrum 0).  Both generators
    take this table as an input."""
    e = np.arange(d, dtype=np.float64)
    return (1.0 / np.sqrt(kappa)) * (1.0 + e) ** (-spectrum) if spectrum else \
        np.full(d, 1.0 / np.sqrt(kappa))


def deep_rows(seed, centers, rows, kappa=50.0, spectrum=0.0):
    """fp32 unit rows normalize(centre + scale * z), scale = noise_scale()."""
    rows = np.asarray(rows, dtype=np.int64)
    d = centers.shape[1]
    comp = component_of(seed, rows, centers.shape[0])
    z = irwin_hall_normals(seed, rows, d)
    y = centers[comp] + z * noise_scale(d, kappa, spectrum)[None, :]
    nrm2 = np.zeros(len(rows), dtype=np.float64)
    for e in range(d):                      # fixed ascending order
        nrm2 = nrm2 + y[:, e] * y[:, e]
    return (y / np.sqrt(nrm2)[:, None]).astype(np.float32)


def gauss_rows(seed, centers, rows, sigma=1.0):
    """fp32 rows centre + sigma * z."""
    rows = np.asarray(rows, dtype=np.int64)
    d = centers.shape[1]
    comp = component_of(seed, rows, centers.shape[0])
    z = irwin_hall_normals(seed, rows, d)
    return (centers[comp] + z * sigma).astype(np.float32)


# --------------------------------------------------------------------------
# encoder weights
# --------------------------------------------------------------------------

def xavier_uniform(seed, layer, fan_out, fan_in):
    """fp32 [fan_out, fan_in] weights U(-a, a), a = sqrt(6 / (fan_in + fan_out))."""
    a = np.sqrt(6.0 / (fan_in + fan_out))
    idx = np.arange(fan_out * fan_in, dtype=np.int64)
    lo = (idx & 0xFFFFFFFF).astype(np.uint32)
    hi = (idx >> 32).astype(np.uint32)
    w0, _, _, _ = philox4x32_10(lo, hi, np.uint32(layer), np.uint32(TAG_WEIGHT), seed, 0)
    u = (w0.astype(np.float64) + 0.5) * (1.0 / 4294967296.0)
    return (a * (2.0 * u - 1.0)).reshape(fan_out, fan_in).astype(np.float32)


def seeded_permutation(seed, n, tag=TAG_SAMPLE):
    """A permutation of range(n): argsort of one Philox word per index (stable)."""
    w = _u32_words(seed, np.arange(n), 1, tag)[:, 0]
    return np.argsort(w, kind="stable")
