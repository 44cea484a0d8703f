"""Seeded synthetic inputs: points X (fp32, n x d row-major) and initial cluster ids.

This module holds input recipes only — none of the clustering arithmetic — so
both the GPU engine's tests/benchmark and the CPU oracle can draw the same
inputs from it.  The paper's datasets (libSVM KDD-sampled, HIGGS, MNIST8m;
Section VI-A, Table II) are not available; these five workloads stand in for
them with the shapes, value ranges and kernel parameters of the benchmark
configurations (the polynomial kernel with gamma=1, c=1, degree 2 is the one
the paper benchmarks, Section VI-A).

Every recipe uses ``numpy.random.default_rng``: data seed 1000+cfg, initial
assignment seed 2000+cfg unless overridden; after generation the points are
shuffled with the data generator, so cluster membership is not ordered.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    cfg: int
    name: str
    n: int
    d: int
    k: int
    iters: int
    kind: str          # "linear" | "poly" | "gauss"
    gamma: float
    coef0: float
    degree: int

    def describe(self) -> str:
        if self.kind == "poly":
            ker = f"poly(gamma={self.gamma:g},c={self.coef0:g},deg={self.degree})"
        elif self.kind == "gauss":
            ker = f"gauss(gamma={self.gamma:.6g})"
        else:
            ker = "linear"
        return f"{self.name}: n={self.n} d={self.d} k={self.k} iters={self.iters} {ker}"


WORKLOADS = {
    1: Workload(1, "blobs8", 2000, 16, 8, 20, "poly", 1.0, 1.0, 2),
    2: Workload(2, "proto10-d784", 20000, 784, 10, 30, "gauss", 1.0 / 784, 0.0, 1),
    3: Workload(3, "proto10-d780", 60000, 780, 10, 50, "poly", 1.0, 1.0, 2),
    4: Workload(4, "rings64", 100000, 128, 64, 50, "gauss", 0.5, 0.0, 1),
    5: Workload(5, "mix7-d54", 200000, 54, 7, 50, "gauss", 1.0 / 54, 0.0, 1),
}


def _blobs(rng, n, d, k):
    """k isotropic Gaussian blobs, centres uniform in [-10, 10]^d, sigma 1, i mod k labels."""
    centres = rng.uniform(-10.0, 10.0, size=(k, d))
    lab = np.arange(n) % k
    return centres[lab] + rng.standard_normal((n, d)), lab


def _prototypes(rng, n, d, k, amp=0.3):
    """k prototype vectors uniform in [0,1]^d plus uniform noise of amplitude amp, clipped to [0,1]."""
    protos = rng.uniform(0.0, 1.0, size=(k, d))
    lab = np.arange(n) % k
    return np.clip(protos[lab] + rng.uniform(-amp, amp, size=(n, d)), 0.0, 1.0), lab


def _rings(rng, n, d, k, radial_sigma=0.05, rest_var=0.01):
    """Dims 0-1 on k concentric rings of radius j = 1..k (uniform angle, radial noise);
    the other dims N(0, rest_var) (0.01 is read as a variance: sigma = 0.1)."""
    lab = np.arange(n) % k
    theta = rng.uniform(0.0, 2.0 * np.pi, size=n)
    r = (lab + 1) + radial_sigma * rng.standard_normal(n)
    X = np.empty((n, d))
    X[:, 0] = r * np.cos(theta)
    X[:, 1] = r * np.sin(theta)
    X[:, 2:] = np.sqrt(rest_var) * rng.standard_normal((n, d - 2))
    return X, lab


def _unequal_mix(rng, n, d, k):
    """k Gaussian clusters (means N(0,I), unit covariance) with sizes proportional to 1..k,
    then every feature standardised to mean 0, variance 1."""
    tot = k * (k + 1) // 2
    sizes = [n * j // tot for j in range(1, k)]
    sizes.append(n - sum(sizes))
    lab = np.repeat(np.arange(k), sizes)
    means = rng.standard_normal((k, d))
    X = means[lab] + rng.standard_normal((n, d))
    X = (X - X.mean(axis=0)) / X.std(axis=0)
    return X, lab


def make_points(cfg: int, n: int | None = None, d: int | None = None, seed: int | None = None):
    """Points of workload ``cfg`` (optionally at another n or d, same recipe).

    Returns (X float32 [n, d] C-contiguous, generating labels int32 [n]).
    """
    w = WORKLOADS[cfg]
    n = w.n if n is None else int(n)
    d = w.d if d is None else int(d)
    rng = np.random.default_rng(1000 + cfg if seed is None else seed)
    if cfg == 1:
        X, lab = _blobs(rng, n, d, 8)
    elif cfg in (2, 3):
        X, lab = _prototypes(rng, n, d, 10)
    elif cfg == 4:
        X, lab = _rings(rng, n, d, 64)
    elif cfg == 5:
        X, lab = _unequal_mix(rng, n, d, 7)
    else:
        raise ValueError(f"unknown workload {cfg}")
    p = rng.permutation(n)
    return np.ascontiguousarray(X[p], dtype=np.float32), lab[p].astype(np.int32)


def make_init(cfg: int, n: int, k: int, seed: int | None = None) -> np.ndarray:
    """Initial cluster ids: workload 1 uses round-robin ids after a seeded shuffle
    (the paper's round-robin initialisation, Section V); the others uniform random ids."""
    rng = np.random.default_rng(2000 + cfg if seed is None else seed)
    if cfg == 1:
        cl = np.empty(n, dtype=np.int32)
        cl[rng.permutation(n)] = np.arange(n) % k
        return cl
    return rng.integers(0, k, size=n).astype(np.int32)


def workload(cfg: int, n: int | None = None, d: int | None = None, k: int | None = None,
             seed: int | None = None):
    """(Workload, X, cl0) for a workload, optionally resized."""
    w = WORKLOADS[cfg]
    X, _ = make_points(cfg, n=n, d=d, seed=seed)
    kk = w.k if k is None else int(k)
    cl0 = make_init(cfg, X.shape[0], kk, seed=None if seed is None else seed + 1)
    return w, X, cl0


def separated_blobs(n: int, d: int, k: int, seed: int, spread: float = 10.0, sigma: float = 0.3):
    """Well separated blobs (centres uniform in [-spread, spread]^d, small sigma),
    shuffled; a generic test input.  Returns (X fp32, labels int32)."""
    rng = np.random.default_rng(seed)
    centres = rng.uniform(-spread, spread, size=(k, d))
    lab = np.arange(n) % k
    X = centres[lab] + sigma * rng.standard_normal((n, d))
    p = rng.permutation(n)
    return np.ascontiguousarray(X[p], dtype=np.float32), lab[p].astype(np.int32)


def random_init(n: int, k: int, seed: int) -> np.ndarray:
    return np.random.default_rng(seed).integers(0, k, size=n).astype(np.int32)
