"""Seeded synthetic series for the five workload shapes.

This module only makes input data.  It holds none of the transform's
arithmetic and is shared by the tests, the benchmark and the smoke check, so
that the HIP path and the oracle see identical inputs.

The paper measures on randomly generated series of shape (n_instances,
l_series) (Sec. 4); the workloads below keep that and add the value structure
of typical time-series classification data.  Every series is z-normalised per
row in fp64 (population standard deviation) and stored as fp32, row-major.

  tiny            64 x 128,       1,000 kernels: Gaussian random walk
  small           1,000 x 500,   10,000 kernels: 1-3 sinusoids (amplitude
                  U(0.5, 2), phase U(0, 2 pi), U(1, 20) cycles per series)
                  plus N(0, 0.3) noise
  manufacturing   100,000 x 1,000, 10,000 kernels: AR(1), phi ~ U(0.5, 0.99),
                  N(0, 1) innovations, stationary start
  long            1,000 x 16,384, 10,000 kernels: Gaussian random walk plus 5
                  step changes of size N(0, 3) at positions U{1 .. L-1}
  many_short      1,000,000 x 64, 10,000 kernels: N(0, 1) noise plus a linear
                  trend of slope U(-0.05, 0.05)
  paper_sweep     1,000 x 10,000, 10,000 kernels: Gaussian random walk (the
                  default point of the paper's timing sweep, Sec. 4)
  multivariate    10,000 series x 6 channels x 500, 10,000 multivariate
                  kernels (Sec. 3.3): per series, 3 latent random walks mixed
                  into the 6 channels with random weights plus N(0, 0.3)
                  noise; every channel z-normalised
  minirocket      the manufacturing series with MINIROCKET (Sec. 5 names it):
                  10,000 features fitted on the first 1,000 series

Kernel seed 200 + i and data seed 100 + i for workload i = 1 .. 5.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    L: int
    n_kernels: int
    kernel_seed: int
    data_seed: int
    kind: str
    channels: int = 1


WORKLOADS = {
    "tiny": Workload("tiny", 64, 128, 1000, 201, 101, "random_walk"),
    "small": Workload("small", 1000, 500, 10000, 202, 102, "sinusoids"),
    "manufacturing": Workload("manufacturing", 100000, 1000, 10000, 203, 103, "ar1"),
    "long": Workload("long", 1000, 16384, 10000, 204, 104, "walk_steps"),
    "many_short": Workload("many_short", 1000000, 64, 10000, 205, 105, "trend"),
    "paper_sweep": Workload("paper_sweep", 1000, 10000, 10000, 206, 106, "random_walk"),
    "multivariate": Workload("multivariate", 10000, 500, 10000, 208, 108, "mixed_walks", 6),
    # MINIROCKET (Sec. 5): the Manufacturing series; n_kernels is the number of
    # features requested from the fit, kernel_seed the fit's seed; the fit uses
    # the first 1,000 series
    "minirocket": Workload("minirocket", 100000, 1000, 10000, 209, 103, "ar1"),
}


def znorm_rows(x: np.ndarray) -> np.ndarray:
    """Per-row z-normalisation in fp64 (ddof = 0), returned as fp32."""
    x = np.asarray(x, dtype=np.float64)
    mu = x.mean(axis=1, keepdims=True)
    sd = x.std(axis=1, keepdims=True)
    sd[sd == 0.0] = 1.0
    return ((x - mu) / sd).astype(np.float32)


def _random_walk(rng, n, L):
    return np.cumsum(rng.standard_normal((n, L)), axis=1)


def _sinusoids(rng, n, L):
    t = np.arange(L, dtype=np.float64) / L
    x = np.zeros((n, L))
    ncomp = rng.integers(1, 4, size=n)
    for c in range(3):
        amp = rng.uniform(0.5, 2.0, size=n) * (ncomp > c)
        freq = rng.uniform(1.0, 20.0, size=n)
        phase = rng.uniform(0.0, 2 * np.pi, size=n)
        x += amp[:, None] * np.sin(2 * np.pi * freq[:, None] * t[None, :] + phase[:, None])
    return x + rng.normal(0.0, 0.3, size=(n, L))


def _ar1(rng, n, L, chunk=1 << 16):
    out = np.empty((n, L), dtype=np.float32)
    for s in range(0, n, chunk):
        m = min(chunk, n - s)
        phi = rng.uniform(0.5, 0.99, size=m)
        e = rng.standard_normal((m, L))
        x = np.empty((m, L))
        x[:, 0] = e[:, 0] / np.sqrt(1.0 - phi * phi)
        for t in range(1, L):
            x[:, t] = phi * x[:, t - 1] + e[:, t]
        out[s:s + m] = znorm_rows(x)
    return out


def _walk_steps(rng, n, L):
    x = _random_walk(rng, n, L)
    for _ in range(5):
        pos = rng.integers(1, L, size=n)
        size = rng.normal(0.0, 3.0, size=n)
        mask = np.arange(L)[None, :] >= pos[:, None]
        x += mask * size[:, None]
    return x


def _trend(rng, n, L, chunk=1 << 18):
    out = np.empty((n, L), dtype=np.float32)
    t = np.arange(L, dtype=np.float64)
    for s in range(0, n, chunk):
        m = min(chunk, n - s)
        slope = rng.uniform(-0.05, 0.05, size=m)
        x = rng.standard_normal((m, L)) + slope[:, None] * t[None, :]
        out[s:s + m] = znorm_rows(x)
    return out


def make_multichannel(n: int, C: int, L: int, seed: int, chunk: int = 4096) -> np.ndarray:
    """fp32 [n, C, L]: per series, 3 latent Gaussian random walks mixed into
    C channels with N(0, 1) weights plus N(0, 0.3) noise, each channel
    z-normalised in fp64."""
    rng = np.random.default_rng(seed)
    out = np.empty((n, C, L), dtype=np.float32)
    for s0 in range(0, n, chunk):
        m = min(chunk, n - s0)
        lat = np.cumsum(rng.standard_normal((m, 3, L)), axis=2)
        mix = rng.standard_normal((m, C, 3))
        x = np.einsum("mcl,mlt->mct", mix, lat) + rng.normal(0.0, 0.3, size=(m, C, L))
        out[s0:s0 + m] = znorm_rows(x.reshape(m * C, L)).reshape(m, C, L)
    return out


def make_series(kind: str, n: int, L: int, seed: int) -> np.ndarray:
    """fp32 [n, L] z-normalised series of the given kind."""
    rng = np.random.default_rng(seed)
    if kind == "random_walk":
        return znorm_rows(_random_walk(rng, n, L))
    if kind == "sinusoids":
        return znorm_rows(_sinusoids(rng, n, L))
    if kind == "ar1":
        return _ar1(rng, n, L)
    if kind == "walk_steps":
        return znorm_rows(_walk_steps(rng, n, L))
    if kind == "trend":
        return _trend(rng, n, L)
    if kind == "gaussian":
        return znorm_rows(rng.standard_normal((n, L)))
    raise ValueError("unknown series kind %r" % kind)


def workload_series(name: str, n: int | None = None) -> np.ndarray:
    """Series of a named workload (optionally only its first n rows):
    [n, L], or [n, C, L] for multichannel workloads."""
    w = WORKLOADS[name]
    if w.channels > 1:
        return make_multichannel(w.n if n is None else n, w.channels, w.L, w.data_seed)
    return make_series(w.kind, w.n if n is None else n, w.L, w.data_seed)


def sample_rows(n: int, batch: int, extra: int = 0, seed: int = 7, total: int | None = None) -> np.ndarray:
    """Row sample used for parity and the CPU baseline: the first and last row,
    the first and last row of every batch, and ``extra`` seeded random rows
    (or, with ``total``, as many seeded random rows as bring the sample to
    ``total`` distinct rows, at most n)."""
    rows = {0, n - 1}
    for s in range(0, n, batch):
        rows.add(s)
        rows.add(min(n, s + batch) - 1)
    rng = np.random.default_rng(seed)
    if extra > 0:
        rows.update(int(r) for r in rng.integers(0, n, size=extra))
    if total is not None:
        total = min(int(total), n)
        while len(rows) < total:
            rows.update(int(r) for r in rng.integers(0, n, size=total - len(rows)))
    return np.array(sorted(rows), dtype=np.int64)
