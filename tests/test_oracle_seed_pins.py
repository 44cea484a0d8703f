"""Pins for the oracle's K-means++ seeding (D^2 sampling in feature space).

Independent routes only: a hand-worked fixture (tests/golden), squared
distances from the coordinates (scipy) for the linear kernel, the closed form
2 - 2 exp(-gamma r^2) of the Gaussian feature distance, explicit feature maps
for the polynomial kernel, numpy's searchsorted for the draw, the law of the
draw (index i is drawn for a fraction D(i)/S of the uniforms), and closed
forms (k = 1, k = n, all points equal).  The mutation tests at the end plant
plausible mistakes in the oracle and confirm that these pins catch each one.
"""
import json
import os

import numpy as np
import pytest
from scipy.spatial.distance import cdist

from featuremaps import poly_features

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _points(seed, n=40, d=3):
    return np.random.default_rng(seed).normal(size=(n, d)).astype(np.float32)


def _uniforms(seed, k):
    return np.random.default_rng(10_000 + seed).random(k)


def _seed_from_sqdist(Dall, u):
    """D^2 sampling from a full matrix of squared feature distances, written
    independently of the oracle: the draw is numpy's searchsorted on the
    cumulative weights (first index whose prefix exceeds u S)."""
    n, k = Dall.shape[0], u.size
    centers = [min(int(np.floor(u[0] * n)), n - 1)]
    D = Dall[:, centers[0]].copy()
    for t in range(1, k):
        P = np.cumsum(D)
        centers.append(int(np.searchsorted(P, u[t] * P[-1], side="right")))
        D = np.minimum(D, Dall[:, centers[-1]])
    cl = np.argmin(Dall[:, centers].astype(np.float32), axis=1)
    return np.array(centers), cl


# ------------------------------------------------------------------ checks

def check_golden(o):
    g = json.load(open(os.path.join(GOLDEN, "kmeanspp_linear_1d.json")))
    kp = g["kernel"]
    kern = o.Kernel(kp["kind"], kp["gamma"], kp["coef0"], kp["degree"])
    X = np.array(g["X"], dtype=np.float32)
    centers, cl = o.kmeanspp(kern, X, g["k"], g["u"])
    assert list(centers) == g["centers"], centers
    assert list(cl) == g["cl"], cl


def check_linear_coordinates(o):
    for seed in (0, 1, 2):
        X = _points(seed)
        u = _uniforms(seed, 6)
        centers, cl = o.kmeanspp(o.Kernel("linear", 1.0, 0.0, 1), X, 6, u)
        Dall = cdist(X.astype(np.float64), X.astype(np.float64), "sqeuclidean")
        ec, ecl = _seed_from_sqdist(Dall, u)
        np.testing.assert_array_equal(centers, ec)
        np.testing.assert_array_equal(cl, ecl)


def check_gauss_closed_form(o):
    gamma = 0.3
    for seed in (3, 4):
        X = _points(seed, n=50, d=2)
        u = _uniforms(seed, 5)
        centers, cl = o.kmeanspp(o.Kernel("gauss", gamma, 0.0, 1), X, 5, u)
        r2 = cdist(X.astype(np.float64), X.astype(np.float64), "sqeuclidean")
        ec, ecl = _seed_from_sqdist(2.0 - 2.0 * np.exp(-np.float64(np.float32(gamma)) * r2), u)
        np.testing.assert_array_equal(centers, ec)
        np.testing.assert_array_equal(cl, ecl)
        # feature distance is increasing in the input distance: nearest centers agree
        np.testing.assert_array_equal(cl, np.argmin(r2[:, centers], axis=1))


def check_poly_feature_map(o):
    gamma, coef0, degree = 0.5, 1.0, 2
    X = _points(5, n=30, d=2)
    u = _uniforms(5, 4)
    centers, cl = o.kmeanspp(o.Kernel("poly", gamma, coef0, degree), X, 4, u)
    phi = poly_features(X, np.float32(gamma), np.float32(coef0), degree)
    Dall = cdist(phi, phi, "sqeuclidean")
    ec, ecl = _seed_from_sqdist(Dall, u)
    np.testing.assert_array_equal(centers, ec)
    np.testing.assert_array_equal(cl, ecl)


def check_draw_law(o):
    """Second center: over a fine grid of uniforms, index i is drawn for a
    fraction D(i)/S of them, D the squared distances to the first center."""
    X = _points(6, n=7, d=2)
    Dfirst = cdist(X.astype(np.float64), X[:1].astype(np.float64), "sqeuclidean")[:, 0]
    M = 4000
    counts = np.zeros(X.shape[0])
    for m in range(M):
        centers, _ = o.kmeanspp(o.Kernel("linear", 1.0, 0.0, 1), X, 2, [0.0, (m + 0.5) / M])
        counts[centers[1]] += 1
    np.testing.assert_allclose(counts / M, Dfirst / Dfirst.sum(), atol=1.5 / M)


_CHECKS = [check_golden, check_linear_coordinates, check_gauss_closed_form, check_poly_feature_map,
           check_draw_law]


@pytest.mark.parametrize("check", _CHECKS, ids=lambda c: c.__name__)
def test_seed_pins(oracle, check):
    check(oracle)


def test_seed_single_cluster(oracle):
    X = _points(7)
    centers, cl = oracle.kmeanspp(oracle.Kernel("linear", 1.0, 0.0, 1), X, 1, [0.999])
    assert list(centers) == [39] and np.all(cl == 0)


def test_seed_every_point_a_center(oracle):
    X = _points(8, n=9)
    centers, cl = oracle.kmeanspp(oracle.Kernel("gauss", 0.5, 0.0, 1), X, 9, _uniforms(8, 9))
    assert sorted(centers) == list(range(9))
    np.testing.assert_array_equal(centers[cl], np.arange(9))


def test_seed_identical_points(oracle):
    """S = 0 after the first center: the lowest indices not yet chosen, all in cluster 0."""
    X = np.ones((10, 3), dtype=np.float32)
    centers, cl = oracle.kmeanspp(oracle.Kernel("linear", 1.0, 0.0, 1), X, 3, [0.5, 0.2, 0.9])
    assert list(centers) == [5, 0, 1] and np.all(cl == 0)


def test_seed_centers_distinct_while_spread(oracle):
    X = _points(9, n=60)
    for s in range(5):
        centers, _ = oracle.kmeanspp(oracle.Kernel("poly", 1.0, 1.0, 2), X, 12, _uniforms(s, 12))
        assert len(set(centers)) == 12


# ------------------------------------------------------------ planted mistakes

def _mutants(o):
    orig_draw, orig_dist = o.draw_index, o.feature_sq_dist

    def draw_linear_weights(D, ut, chosen):  # D^1 sampling instead of D^2
        return orig_draw(np.sqrt(D), ut, chosen)

    def draw_reversed(D, ut, chosen):        # prefix taken from the other end
        return D.size - 1 - orig_draw(D[::-1], ut, chosen)

    def dist_plus(kern, X, c, diagK):         # sign of the cross term flipped
        Kc = kern.block(X, rows=np.array([c]))[0]
        return np.maximum(diagK + 2.0 * Kc + diagK[c], 0.0)

    def dist_no_center_norm(kern, X, c, diagK):  # K(c,c) dropped
        Kc = kern.block(X, rows=np.array([c]))[0]
        return np.maximum(diagK - 2.0 * Kc, 0.0)

    def assign_max(D, decide_in=np.float32):
        return np.argmax(D, axis=1).astype(np.int32)

    return {"draw_index": [draw_linear_weights, draw_reversed],
            "feature_sq_dist": [dist_plus, dist_no_center_norm], "assign": [assign_max]}


@pytest.mark.parametrize("name,idx", [("draw_index", 0), ("draw_index", 1), ("feature_sq_dist", 0),
                                      ("feature_sq_dist", 1), ("assign", 0)])
def test_seed_pins_catch_planted_mistakes(oracle, monkeypatch, name, idx):
    mutant = _mutants(oracle)[name][idx]
    monkeypatch.setattr(oracle, name, mutant)
    caught = 0
    for chk in _CHECKS:
        try:
            chk(oracle)
        except (AssertionError, IndexError, ValueError, StopIteration):
            caught += 1
    assert caught >= 2, f"planted mistake in {name} caught by only {caught} pin(s)"
