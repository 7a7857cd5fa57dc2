"""Seeded synthetic two-class data shaped like the paper's workloads.

This module only draws and scales inputs. It holds none of the LS-SVM
arithmetic, so both the CPU oracle's tests and the GPU path's tests can take
their inputs from it without sharing any of the method's code.

Recipe (stands in for the paper's synthetic "planes" data of Section V-A,
whose generator is not available): two overlapping Gaussian classes on the
first ``round(inf_frac * d)`` features (unit variance, class means at
``+-mu``), uniform noise in [-1, 1] on the remaining features, per-column
min-max scaling to [-1, 1], balanced +-1 labels, and a fraction of labels
flipped after the points are drawn. The generator is numpy's PCG64 seeded
with ``seed``; the draw order below is part of the recipe and must not change.
"""
from __future__ import annotations

import dataclasses
import hashlib

import numpy as np

__all__ = ["Config", "CONFIGS", "gen_raw", "minmax_fit", "minmax_apply",
           "make_train", "make_test", "probe_vector", "sha256_arrays"]


@dataclasses.dataclass(frozen=True)
class Config:
    """One workload: data shape, generator knobs and solver settings."""
    name: str
    dtype: str          # "f64" or "f32": storage / compute type of the GPU path
    kernel: str         # "linear", "poly" or "rbf"
    n: int
    d: int
    mu: float
    inf_frac: float
    flip_frac: float
    C: float
    eps: float
    gamma: float = 1.0
    coef0: float = 0.0
    degree: int = 1
    max_iter: int = 0   # 0 means N = n - 1

    @property
    def np_dtype(self):
        return np.float64 if self.dtype == "f64" else np.float32

    def scaled(self, n: int, d: int | None = None, name: str | None = None) -> "Config":
        """Same recipe and solver settings at another size (gamma follows 1/d)."""
        d = self.d if d is None else d
        gamma = self.gamma
        if self.kernel in ("rbf", "poly"):
            gamma = 1.0 / d
        return dataclasses.replace(self, n=n, d=d, gamma=gamma,
                                   name=name or f"{self.name}@{n}x{d}", max_iter=0)


# The five workloads: two fp64 linear, one fp64 RBF, one fp32 cubic polynomial,
# one fp32 RBF whose reduced matrix (65535^2) is never materialised.
CONFIGS = {
    "linear_f64_256x64": Config("linear_f64_256x64", "f64", "linear", 256, 64,
                                mu=0.5, inf_frac=1.0, flip_frac=0.0,
                                C=1.0, eps=1e-10, max_iter=256),
    "linear_f64_4096x1024": Config("linear_f64_4096x1024", "f64", "linear", 4096, 1024,
                                   mu=1.0, inf_frac=0.3, flip_frac=0.05, C=1.0, eps=1e-8),
    "rbf_f64_16384x2048": Config("rbf_f64_16384x2048", "f64", "rbf", 16384, 2048,
                                 mu=1.0, inf_frac=0.3, flip_frac=0.05, C=1.0, eps=1e-8,
                                 gamma=1.0 / 2048),
    "poly_f32_32768x4096": Config("poly_f32_32768x4096", "f32", "poly", 32768, 4096,
                                  mu=1.0, inf_frac=0.3, flip_frac=0.05, C=1.0, eps=1e-5,
                                  gamma=1.0 / 4096, coef0=1.0, degree=3),
    "rbf_f32_65536x1024": Config("rbf_f32_65536x1024", "f32", "rbf", 65536, 1024,
                                 mu=1.0, inf_frac=0.3, flip_frac=0.10, C=10.0, eps=1e-4,
                                 gamma=1.0 / 1024),
}


def gen_raw(n: int, d: int, seed: int, mu: float, inf_frac: float, flip_frac: float):
    """Unscaled points (fp64, n x d row-major) and +-1 labels (fp64).

    Draw order: label permutation, informative block (n x k standard normals,
    row-major), noise block (n x (d-k) uniforms on [-1, 1), row-major), flip set.
    """
    rng = np.random.default_rng(seed)
    y = np.concatenate([np.ones(n // 2), -np.ones(n - n // 2)])
    y = y[rng.permutation(n)]
    k = int(round(inf_frac * d))
    X = np.empty((n, d), dtype=np.float64)
    if k > 0:
        blk = rng.standard_normal((n, k))
        blk += y[:, None] * mu
        X[:, :k] = blk
        del blk
    if d - k > 0:
        X[:, k:] = rng.uniform(-1.0, 1.0, (n, d - k))
    nflip = int(round(flip_frac * n))
    if nflip > 0:
        idx = rng.choice(n, nflip, replace=False)
        y[idx] *= -1.0
    return X, y


def minmax_fit(X: np.ndarray):
    """Per-column (min, max) of a point matrix."""
    return X.min(axis=0), X.max(axis=0)


def minmax_apply(X: np.ndarray, lo: np.ndarray, hi: np.ndarray, inplace: bool = False) -> np.ndarray:
    """Map each column linearly so that [lo, hi] becomes [-1, 1]; constant columns -> 0.

    Computed as (x - lo) * (2 / (hi - lo)) - 1 in fp64, column scale factors
    formed once.
    """
    span = hi - lo
    ok = span > 0
    scale = np.where(ok, 2.0 / np.where(ok, span, 1.0), 0.0)
    shift = np.where(ok, lo, 0.0)
    out = X if inplace else X.copy()
    out -= shift
    out *= scale
    out -= ok.astype(np.float64)      # the "- 1", only on non-constant columns
    return out


def make_train(cfg: Config, seed: int = 0):
    """(X, y, (lo, hi)) for a config: X in the config's dtype, C-contiguous."""
    Xr, y = gen_raw(cfg.n, cfg.d, seed, cfg.mu, cfg.inf_frac, cfg.flip_frac)
    lo, hi = minmax_fit(Xr)
    minmax_apply(Xr, lo, hi, inplace=True)
    X = Xr if cfg.np_dtype == np.float64 else Xr.astype(cfg.np_dtype)
    return X, y.astype(cfg.np_dtype), (lo, hi)


def make_test(cfg: Config, scale, n_test: int = 1024, seed: int = 1):
    """Held-out points drawn with seed 1 and scaled with the TRAINING min/max."""
    Xr, y = gen_raw(n_test, cfg.d, seed, cfg.mu, cfg.inf_frac, cfg.flip_frac)
    lo, hi = scale
    minmax_apply(Xr, lo, hi, inplace=True)
    X = Xr if cfg.np_dtype == np.float64 else Xr.astype(cfg.np_dtype)
    return X, y.astype(cfg.np_dtype)


def probe_vector(N: int, dtype, seed: int = 12345) -> np.ndarray:
    """Standard-normal direction vector of length N used to probe the matvec."""
    return np.random.default_rng(seed).standard_normal(N).astype(dtype)


def sha256_arrays(*arrays) -> str:
    """SHA-256 over the raw bytes of the given arrays (dtype and shape included)."""
    h = hashlib.sha256()
    for a in arrays:
        a = np.ascontiguousarray(a)
        h.update(str(a.dtype).encode())
        h.update(str(a.shape).encode())
        h.update(a.tobytes())
    return h.hexdigest()
