"""Explicit feature maps used to pin the oracle independently of the kernel trick.

Kernel K-means with kernel kappa equals ordinary K-means on phi(x) whenever
kappa(x, y) = phi(x).phi(y) (Section II-A).  For the polynomial kernel phi is a
finite tensor power; for the Gaussian kernel a truncated Taylor series gives
phi to any accuracy on bounded inputs.  With phi in hand, centroids and
distances can be formed directly, which is what these helpers do.
"""
from __future__ import annotations

from itertools import product
from math import factorial

import numpy as np


def poly_features(X: np.ndarray, gamma: float, coef0: float, degree: int) -> np.ndarray:
    """phi(x) = (sqrt(gamma) x, sqrt(c))^{tensor degree}, so phi(x).phi(y) = (gamma x.y + c)^degree."""
    X = np.asarray(X, dtype=np.float64)
    base = np.hstack([np.sqrt(gamma) * X, np.full((X.shape[0], 1), np.sqrt(coef0))])
    phi = np.ones((X.shape[0], 1))
    for _ in range(degree):
        phi = np.einsum("ni,nj->nij", phi, base).reshape(X.shape[0], -1)
    return phi


def gauss_features(X: np.ndarray, gamma: float, order: int = 30) -> np.ndarray:
    """Truncated Taylor feature map of exp(-gamma |x-y|^2).

    exp(-g|x-y|^2) = e^{-g|x|^2} e^{-g|y|^2} sum_alpha (2g)^{|alpha|}/alpha! x^alpha y^alpha,
    summed over multi-indices alpha with |alpha| <= order.
    """
    X = np.asarray(X, dtype=np.float64)
    n, d = X.shape
    cols = []
    for alpha in product(range(order + 1), repeat=d):
        s = sum(alpha)
        if s > order:
            continue
        coef = (2.0 * gamma) ** s
        for a in alpha:
            coef /= factorial(a)
        cols.append(np.sqrt(coef) * np.prod(X ** np.array(alpha), axis=1))
    return np.exp(-gamma * np.sum(X * X, axis=1))[:, None] * np.stack(cols, axis=1)


def explicit_kmeans_terms(phi: np.ndarray, cl: np.ndarray, k: int):
    """Centroids mu_j = mean of phi over members, squared distances |phi_i - mu_j|^2,
    |mu_j|^2 and phi_i.mu_j, formed directly.  Empty clusters get mu_j = nan."""
    cl = np.asarray(cl)
    mu = np.full((k, phi.shape[1]), np.nan)
    for j in range(k):
        m = cl == j
        if m.any():
            mu[j] = phi[m].mean(axis=0)
    diff = phi[:, None, :] - mu[None, :, :]
    D = np.sum(diff * diff, axis=2)
    return mu, D, np.sum(mu * mu, axis=1), phi @ mu.T


def lloyd_step(X: np.ndarray, cl: np.ndarray, k: int):
    """One plain K-means (Lloyd) step in input space: means, squared distances, argmin."""
    X = np.asarray(X, dtype=np.float64)
    mu = np.stack([X[cl == j].mean(axis=0) for j in range(k)])
    D = ((X[:, None, :] - mu[None, :, :]) ** 2).sum(axis=2)
    return D, np.argmin(D, axis=1)
