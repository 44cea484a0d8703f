"""Pins for the CPU oracle: checks against what the paper and the mathematics fix.

Nothing here compares the oracle with itself or with the GPU engine.  Each
check uses an independent route: hand-worked fixtures of Eqs. 1-8
(tests/golden), library routines (BLAS Gram matrix, scipy's direct squared
distances), explicit feature maps with centroids formed directly, plain Lloyd
K-means for the linear kernel (Section II-A / Section IV), closed forms of
special cases (k = 1, k = n), and invariants (J non-increasing, row sums).
The mutation tests at the end plant plausible mistakes in the oracle and
confirm that these pins catch each one.
"""
import glob
import json
import os

import numpy as np
import pytest
from scipy.spatial.distance import cdist

from featuremaps import explicit_kmeans_terms, gauss_features, lloyd_step, poly_features
from paper_2601_17136_amd import datagen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------ checks
# Each check raises AssertionError on a mismatch; the mutation tests reuse them.

def check_golden(o, path):
    g = json.load(open(path))
    kp = g["kernel"]
    kern = o.Kernel(kp["kind"], kp["gamma"], kp["coef0"], kp["degree"])
    X = np.array(g["X"], dtype=np.float32)
    k = g["k"]
    K = kern.matrix(X)
    for it in g["iterations"]:
        if "K" in it:
            np.testing.assert_allclose(K, it["K"], rtol=1e-7, atol=1e-9)
        out = o.step_full(K, np.array(it["cl"]), k)
        counts = np.array(it["counts"], dtype=np.float64)
        np.testing.assert_array_equal(out["counts"], it["counts"])
        np.testing.assert_allclose(out["E"], it["E_onehot"], rtol=1e-7, atol=1e-9)
        # the paper's normalised E (Eq. 4 with V of Eq. 3) and its c (Eqs. 6-7)
        np.testing.assert_allclose(out["E"] / counts[None, :], it["E_paper"], rtol=1e-7, atol=1e-9)
        np.testing.assert_allclose(out["z"], it["c_paper"], rtol=1e-7, atol=1e-9)
        # Eq. 8 exactly (no diag K), then with diag K
        np.testing.assert_allclose(out["D"] - np.array(it["diagK"])[:, None], it["D_paper"],
                                   rtol=1e-7, atol=1e-8)
        np.testing.assert_allclose(out["D"], it["D"], rtol=1e-7, atol=1e-8)
        np.testing.assert_array_equal(out["cl"], it["cl_new"])
        np.testing.assert_array_equal(out["counts_new"], it["counts_new"])
        assert out["changed"] == it["changed"]
        np.testing.assert_allclose(out["J"], it["J"], rtol=1e-7, atol=1e-9)
        np.testing.assert_allclose(o.objective(np.trace(K), out["z"], out["counts"]), it["J"],
                                   rtol=1e-7, atol=1e-9)


def check_stop_golden(o, path):
    """A hand-worked trajectory of the loop (Alg. 1) and the stop rule under several tol."""
    g = json.load(open(path))
    kp = g["kernel"]
    kern = o.Kernel(kp["kind"], kp["gamma"], kp["coef0"], kp["degree"])
    X = np.array(g["X"], dtype=np.float32)
    K = kern.matrix(X)
    k = g["k"]
    for u in g["updates"]:
        out = o.step_full(K, np.array(u["cl"]), k)
        np.testing.assert_array_equal(out["cl"], u["cl_new"])
        assert out["changed"] == u["changed"]
        assert out["J"] == u["J"]
    for r in g["runs"]:
        cl, done, hist, traj = o.iterate_full(K, np.array(g["cl0"], dtype=np.int32), k, r["max_iter"], tol=r["tol"])
        assert done == r["done"], (path, r["tol"], done, r["done"])
        np.testing.assert_array_equal(cl, r["cl_final"])
        np.testing.assert_array_equal(hist, r["obj_hist"])


def check_poly_explicit(o, seed=0, n=48, d=4, k=5, degree=2, gamma=0.7, coef0=1.3):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d)).astype(np.float32)
    cl = rng.integers(0, k, n)
    cl[:k] = np.arange(k)
    kern = o.Kernel("poly", gamma, coef0, degree)
    phi = poly_features(X, kern.gamma, kern.coef0, degree)
    K = kern.matrix(X)
    np.testing.assert_allclose(K, phi @ phi.T, rtol=1e-10, atol=1e-10)
    mu, D_direct, z_direct, proj = explicit_kmeans_terms(phi, cl, k)
    out = o.step_full(K, cl, k)
    scale = np.abs(D_direct).max()
    np.testing.assert_allclose(out["z"], z_direct, rtol=1e-10, atol=1e-10 * scale)
    np.testing.assert_allclose(out["E"] / o.cluster_sizes(cl, k)[None, :], proj, rtol=1e-10,
                               atol=1e-10 * scale)
    np.testing.assert_allclose(out["D"], D_direct, rtol=1e-9, atol=1e-10 * scale)
    np.testing.assert_array_equal(out["cl"], np.argmin(D_direct.astype(np.float32), axis=1))
    np.testing.assert_allclose(out["J"], D_direct[np.arange(n), cl].sum(), rtol=1e-10)


def check_gauss_explicit(o, seed=1, n=40, d=2, k=4, gamma=0.5):
    rng = np.random.default_rng(seed)
    X = rng.uniform(-1.0, 1.0, (n, d)).astype(np.float32)
    cl = rng.integers(0, k, n)
    cl[:k] = np.arange(k)
    kern = o.Kernel("gauss", gamma)
    phi = gauss_features(X, kern.gamma)
    K = kern.matrix(X)
    np.testing.assert_allclose(K, phi @ phi.T, rtol=0, atol=1e-12)
    mu, D_direct, z_direct, proj = explicit_kmeans_terms(phi, cl, k)
    out = o.step_full(K, cl, k)
    np.testing.assert_allclose(out["z"], z_direct, atol=1e-11)
    np.testing.assert_allclose(out["D"], D_direct, atol=1e-11)
    np.testing.assert_array_equal(out["cl"], np.argmin(D_direct.astype(np.float32), axis=1))


def check_linear_lloyd(o, seed=3, n=300, d=3, k=6, iters=8):
    X, _ = datagen.separated_blobs(n, d, k, seed=seed, spread=3.0, sigma=1.0)
    cl0 = datagen.random_init(n, k, seed + 7)
    K = o.Kernel("linear").matrix(X)
    cl = cl0.copy()
    lloyd = []
    for _ in range(iters):
        D, new = lloyd_step(X, cl, k)
        lloyd.append((D, new, D[np.arange(n), cl].sum()))
        cl = new
    _, done, hist, traj = o.iterate_full(K, cl0, k, iters, tol=-1.0)
    assert done == iters
    cl = cl0
    for t in range(iters):
        D, new, sse = lloyd[t]
        out = o.step_full(K, cl, k)
        np.testing.assert_allclose(out["D"], D, rtol=1e-9, atol=1e-9 * np.abs(D).max())
        np.testing.assert_array_equal(traj[t], new)
        np.testing.assert_allclose(hist[t], sse, rtol=1e-10)
        cl = new


# ------------------------------------------------------------------ tests

@pytest.mark.parametrize("path", sorted(glob.glob(os.path.join(GOLDEN, "worked_*.json"))),
                         ids=os.path.basename)
def test_golden_worked_examples(oracle, path):
    check_golden(oracle, path)


@pytest.mark.parametrize("path", sorted(glob.glob(os.path.join(GOLDEN, "stop_rule_*.json"))),
                         ids=os.path.basename)
def test_golden_stop_rule(oracle, path):
    check_stop_golden(oracle, path)


def test_linear_kernel_is_blas_gram(oracle):
    X = np.random.default_rng(5).standard_normal((70, 9)).astype(np.float32)
    X64 = X.astype(np.float64)
    np.testing.assert_allclose(oracle.Kernel("linear").matrix(X), X64 @ X64.T, rtol=1e-12, atol=1e-12)


def test_gauss_kernel_matches_scipy_direct_distances(oracle):
    X = np.random.default_rng(6).uniform(0, 1, (60, 33)).astype(np.float32)
    g = np.float32(1.0 / 33)
    ref = np.exp(-float(g) * cdist(X.astype(np.float64), X.astype(np.float64), "sqeuclidean"))
    K = oracle.Kernel("gauss", g).matrix(X)
    np.testing.assert_allclose(K, ref, rtol=1e-12, atol=0)
    assert np.all(np.diag(K) == 1.0)


@pytest.mark.parametrize("degree", [1, 2, 3])
def test_poly_kernel_tensor_feature_map(oracle, degree):
    X = np.random.default_rng(7).standard_normal((30, 3)).astype(np.float32)
    kern = oracle.Kernel("poly", 0.5, 2.0, degree)
    phi = poly_features(X, kern.gamma, kern.coef0, degree)
    np.testing.assert_allclose(kern.matrix(X), phi @ phi.T, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(kern.diag(X), np.sum(phi * phi, axis=1), rtol=1e-11)


def test_block_pairs_and_matrix_agree(oracle):
    X = np.random.default_rng(8).standard_normal((50, 7)).astype(np.float32)
    for kind in ("linear", "poly", "gauss"):
        kern = oracle.Kernel(kind, 0.3, 1.0, 2)
        K = kern.matrix(X)
        np.testing.assert_array_equal(K, K.T)
        rows, cols = np.array([3, 9, 41]), np.array([0, 17, 18, 49])
        np.testing.assert_array_equal(kern.block(X, rows, cols), K[np.ix_(rows, cols)])
        np.testing.assert_array_equal(kern.pairs(X, rows, rows[::-1]), K[rows, rows[::-1]])


@pytest.mark.parametrize("seed", [0, 1])
def test_poly_step_equals_explicit_centroids(oracle, seed):
    check_poly_explicit(oracle, seed=seed)


def test_poly_degree3_step_equals_explicit_centroids(oracle):
    check_poly_explicit(oracle, seed=4, d=3, degree=3, gamma=0.4, coef0=0.5)


@pytest.mark.parametrize("seed", [1, 2])
def test_gauss_step_equals_taylor_feature_space(oracle, seed):
    check_gauss_explicit(oracle, seed=seed)


def test_linear_kernel_equals_lloyd_kmeans(oracle):
    check_linear_lloyd(oracle)


@pytest.mark.parametrize("kind,gamma,coef0", [("linear", 1, 0), ("poly", 1.0, 1.0),
                                              ("gauss", 0.05, 0.0), ("gauss", 2.0, 0.0)])
def test_objective_nonincreasing(oracle, kind, gamma, coef0):
    X = np.random.default_rng(11).standard_normal((200, 4)).astype(np.float32)
    cl0 = datagen.random_init(200, 7, 12)
    K = oracle.Kernel(kind, gamma, coef0, 2).matrix(X)
    _, done, hist, traj = oracle.iterate_full(K, cl0, 7, 25, tol=-1.0)
    assert done == 25
    assert np.all(np.diff(hist) <= 1e-9 * np.abs(hist[:-1]))
    assert hist[-1] < hist[0]


def test_single_cluster_closed_form(oracle):
    X = np.random.default_rng(13).standard_normal((40, 5)).astype(np.float32)
    K = oracle.Kernel("poly", 0.2, 1.0, 2).matrix(X)
    out = oracle.step_full(K, np.zeros(40, dtype=np.int32), 1)
    n = 40
    np.testing.assert_allclose(out["J"], np.trace(K) - K.sum() / n, rtol=1e-12)
    np.testing.assert_allclose(out["D"][:, 0], np.diag(K) - 2 * K.mean(axis=1) + K.mean(), rtol=1e-12)
    assert np.all(out["cl"] == 0)


def test_each_point_its_own_cluster(oracle):
    X = np.random.default_rng(14).standard_normal((25, 3)).astype(np.float32)
    for kind in ("linear", "poly", "gauss"):
        K = oracle.Kernel(kind, 0.5, 1.0, 2).matrix(X)
        out = oracle.step_full(K, np.arange(25), 25)
        assert abs(out["J"]) <= 1e-12 * np.abs(K).max()
        np.testing.assert_allclose(np.diag(out["D"]), 0.0, atol=1e-12 * np.abs(K).max())
        np.testing.assert_array_equal(out["cl"], np.arange(25))


def test_empty_cluster_is_never_chosen(oracle):
    X = np.random.default_rng(15).standard_normal((30, 2)).astype(np.float32)
    cl = np.random.default_rng(16).integers(0, 3, 30)
    cl[cl == 1] = 0                         # cluster 1 empty
    K = oracle.Kernel("gauss", 0.5).matrix(X)
    out = oracle.step_full(K, cl, 3)
    assert out["counts"][1] == 0 and out["z"][1] == 0.0
    assert np.all(np.isinf(out["D"][:, 1]))
    assert np.all(out["cl"] != 1) and out["counts_new"][1] == 0


def test_ties_take_lowest_index(oracle):
    # duplicated points in two clusters: both centroids coincide
    X = np.zeros((2, 1), dtype=np.float32)
    out = oracle.step_full(oracle.Kernel("linear").matrix(X), np.array([0, 1]), 2)
    assert out["D"][0, 0] == out["D"][0, 1]
    np.testing.assert_array_equal(out["cl"], [0, 0])
    # two centroids at -1/2 and +1/2, points at 0 are exactly equidistant
    X = np.array([[-1.0], [1.0], [0.0], [0.0]], dtype=np.float32)
    out = oracle.step_full(oracle.Kernel("linear").matrix(X), np.array([0, 1, 0, 1]), 2)
    assert out["D"][2, 0] == out["D"][2, 1] == 0.25
    np.testing.assert_array_equal(out["cl"], [0, 1, 0, 0])


def test_row_sums_and_counts(oracle):
    X = np.random.default_rng(17).standard_normal((64, 6)).astype(np.float32)
    cl = datagen.random_init(64, 5, 18)
    K = oracle.Kernel("poly", 1.0, 1.0, 2).matrix(X)
    out = oracle.step_full(K, cl, 5)
    np.testing.assert_allclose(out["E"].sum(axis=1), K.sum(axis=1), rtol=1e-12)
    assert out["counts"].sum() == 64 and out["counts_new"].sum() == 64
    # every new id attains the row minimum
    Dm = out["D"].astype(np.float32)
    assert np.all(Dm[np.arange(64), out["cl"]] == Dm.min(axis=1))


def test_step_rows_matches_full_step(oracle):
    w, X, cl = datagen.workload(4, n=600, d=10)
    kern = oracle.Kernel(w.kind, w.gamma, w.coef0, w.degree)
    K = kern.matrix(X)
    full = oracle.step_full(K, cl, w.k)
    rows = np.array([0, 5, 77, 599])
    part = oracle.step_rows(kern, X, cl, w.k, rows)
    np.testing.assert_allclose(part["E"], full["E"][rows], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(part["z"], full["z"], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(part["D"], full["D"][rows], rtol=1e-11, atol=1e-12)
    np.testing.assert_array_equal(part["cl"], full["cl"][rows])
    np.testing.assert_allclose(part["J"], full["J"], rtol=1e-11)


def test_stop_rules(oracle):
    X, _ = datagen.separated_blobs(120, 2, 3, seed=21)
    K = oracle.Kernel("linear").matrix(X)
    cl0 = datagen.random_init(120, 3, 22)
    cl_a, done_a, hist_a, traj = oracle.iterate_full(K, cl0, 3, 50, tol=0.0)
    assert done_a < 50
    assert np.array_equal(traj[-1], cl_a)
    assert np.array_equal(traj[-2], traj[-1])     # the last update changed nothing
    _, done_b, hist_b, _ = oracle.iterate_full(K, cl0, 3, 50, tol=-1.0)
    assert done_b == 50
    _, done_c, hist_c, _ = oracle.iterate_full(K, cl0, 3, 50, tol=0.5)
    assert done_c <= done_a


def test_workload_recipes_shape_and_determinism():
    for cfg in (1, 2, 3, 4, 5):
        w = datagen.WORKLOADS[cfg]
        X1, l1 = datagen.make_points(cfg, n=512)
        X2, l2 = datagen.make_points(cfg, n=512)
        assert X1.dtype == np.float32 and X1.shape == (512, w.d) and X1.flags.c_contiguous
        assert np.array_equal(X1, X2) and np.array_equal(l1, l2)
        cl = datagen.make_init(cfg, 512, w.k)
        assert cl.dtype == np.int32 and cl.min() >= 0 and cl.max() < w.k
    cl = datagen.make_init(1, 2000, 8)
    assert np.all(np.bincount(cl) == 250)            # round-robin after shuffle
    X, _ = datagen.make_points(2, n=1000)
    assert X.min() >= 0.0 and X.max() <= 1.0


# ------------------------------------------------------------------ mutation tests

def _mutants(o):
    def no_diag(diagK_rows, E_rows, z, counts):
        return o.__dict__["_orig_distances"](np.zeros_like(diagK_rows), E_rows, z, counts)

    def sign_flip(diagK_rows, E_rows, z, counts):
        return o.__dict__["_orig_distances"](diagK_rows, -E_rows, z, counts)

    def z_single_norm(own, cl, counts):
        return o.__dict__["_orig_self_terms"](own, cl, counts) * np.maximum(counts, 1)

    def argmax(D, decide_in=np.float32):
        return np.argmax(np.where(np.isinf(D), -np.inf, D), axis=1).astype(np.int32)

    def wrong_index(E_rows, cl_rows):
        return E_rows[np.arange(len(cl_rows)), (np.asarray(cl_rows) + 1) % E_rows.shape[1]]

    def shifted_ids(K_rows, cl, k):
        return K_rows @ o.one_hot((np.asarray(cl) + 1) % k, k)

    def stop_sign_flip(tol, changed, J_prev, J_cur):
        if tol < 0:
            return False
        if changed == 0:
            return True
        return bool(tol > 0 and J_prev is not None and (J_cur - J_prev) <= tol * abs(J_prev))

    def stop_current_ref(tol, changed, J_prev, J_cur):
        if tol < 0:
            return False
        if changed == 0:
            return True
        return bool(tol > 0 and J_prev is not None and (J_prev - J_cur) <= tol * abs(J_cur))

    def stop_strict(tol, changed, J_prev, J_cur):
        if tol < 0:
            return False
        if changed == 0:
            return True
        return bool(tol > 0 and J_prev is not None and (J_prev - J_cur) < tol * abs(J_prev))

    return {"distances": [no_diag, sign_flip], "self_terms": [z_single_norm], "assign": [argmax],
            "mask": [wrong_index], "one_hot_product": [shifted_ids],
            "stop_now": [stop_sign_flip, stop_current_ref, stop_strict]}


_CHECKS = [
    lambda o: check_golden(o, os.path.join(GOLDEN, "worked_poly_2d.json")),
    lambda o: check_golden(o, os.path.join(GOLDEN, "worked_linear_1d.json")),
    check_poly_explicit,
    check_gauss_explicit,
    check_linear_lloyd,
    lambda o: check_stop_golden(o, os.path.join(GOLDEN, "stop_rule_linear_1d_a.json")),
    lambda o: check_stop_golden(o, os.path.join(GOLDEN, "stop_rule_linear_1d_b.json")),
]


@pytest.mark.parametrize("name,idx", [("distances", 0), ("distances", 1), ("self_terms", 0),
                                      ("assign", 0), ("mask", 0), ("one_hot_product", 0),
                                      ("stop_now", 0), ("stop_now", 1), ("stop_now", 2)])
def test_pins_catch_planted_mistakes(oracle, monkeypatch, name, idx):
    oracle.__dict__.setdefault("_orig_distances", oracle.distances)
    oracle.__dict__.setdefault("_orig_self_terms", oracle.self_terms)
    mutant = _mutants(oracle)[name][idx]
    monkeypatch.setattr(oracle, name, mutant)
    caught = 0
    for chk in _CHECKS:
        try:
            chk(oracle)
        except (AssertionError, IndexError, ValueError):
            caught += 1
    assert caught >= 2, f"planted mistake in {name} caught by only {caught} pin(s)"
