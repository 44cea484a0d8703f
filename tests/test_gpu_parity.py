"""GPU parity: the HIP engine through its C ABI against the CPU oracle.

Small problems (the oracle forms all of K in seconds) with ragged sizes that
span several 128 x 128 tiles and partial 1024-column stripes, every kernel
kind, and the degenerate cases (n = 1, k = 1, k = n, empty clusters, exact
ties, invalid ids).  The bar: K, E and D within 1e-4 row-scaled, z and J
within 1e-4 relative, sizes exact, assignments exact except at near-ties of
the oracle's distances, and exact trajectories on well-separated input.
"""
import numpy as np
import pytest

from gpu_helpers import TOL, Engine, assignment_mismatches, rel_err, rowscaled_err
from paper_2601_17136_amd import datagen

pytestmark = pytest.mark.gpu


def _norm_spread(X, seed):
    """The points with row norms spread over four decades (10^-3 .. 10 times
    their own) and one point at the origin: the packed column side's
    power-of-two row scales then range widely, one row of K is zero (its
    bound falls back to 1), and the Cauchy-Schwarz bound of a small row is
    loose against its entries."""
    rng = np.random.default_rng(seed)
    Y = (X * 10.0 ** rng.uniform(-3.0, 1.0, size=(X.shape[0], 1))).astype(np.float32)
    Y[17] = 0.0
    return Y


def _torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.fail("GPU test on a machine without a GPU")
    return torch


CASES = {
    # name: (points, k, kind, gamma, coef0, degree, init seed)
    "blobs-n2000-poly": (lambda: datagen.make_points(1)[0], 8, "poly", 1.0, 1.0, 2, None),
    "ragged-poly3": (lambda: datagen.separated_blobs(1037, 13, 5, seed=3, spread=2.0, sigma=1.0)[0],
                     5, "poly", 0.5, 1.0, 3, 11),
    "ragged-gauss": (lambda: datagen.make_points(2, n=777, d=37)[0], 9, "gauss", 0.3, 0.0, 1, 12),
    "linear-n300": (lambda: datagen.separated_blobs(300, 3, 4, seed=4, spread=3.0, sigma=1.0)[0],
                    4, "linear", 1.0, 0.0, 1, 13),
    "rings-n3000-gauss": (lambda: datagen.make_points(4, n=3000)[0], 64, "gauss", 0.5, 0.0, 1, 14),
    # the same rings at a small width (the sweep build and sweep update), fix-up entries listed
    "rings-n3000-d24-gauss": (lambda: datagen.make_points(4, n=3000, d=24)[0], 64, "gauss", 0.5, 0.0, 1, 24),
    # widths above 64: the sweep build's contraction in two chunks (second chunk
    # of half-width 32, 20 and 4), ragged row tails
    "rings-n2000-d120-gauss": (lambda: datagen.make_points(4, n=2000, d=120)[0], 16, "gauss", 0.5, 0.0, 1, 25),
    "d100-n1300-poly": (lambda: datagen.make_points(2, n=1300, d=100)[0], 6, "poly", 0.01, 1.0, 2, 26),
    "d72-n700-linear": (lambda: datagen.separated_blobs(700, 72, 5, seed=7, spread=2.0, sigma=1.0)[0],
                        5, "linear", 1.0, 0.0, 1, 27),
    # the packed SpMM's segment length changes at 4096 points (k <= 16): the last
    # size with 2-tile segments (and the largest label count they take), and one
    # just above it with a ragged tail
    "n4096-k16-gauss": (lambda: datagen.make_points(2, n=4096, d=20)[0], 16, "gauss", 1.0 / 20, 0.0, 1, 28),
    "n4500-k12-poly": (lambda: datagen.make_points(2, n=4500, d=20)[0], 12, "poly", 0.05, 1.0, 2, 29),
    "n129-d1": (lambda: datagen.separated_blobs(129, 1, 3, seed=5)[0], 3, "poly", 0.25, 2.0, 2, 15),
    "n128-d16": (lambda: datagen.make_points(5, n=128, d=16)[0], 7, "gauss", 1.0 / 16, 0.0, 1, 16),
    "n2-k2": (lambda: np.array([[0.0, 1.0], [2.0, -1.0]], np.float32), 2, "poly", 1.0, 1.0, 2, 17),
    "n1-k1": (lambda: np.array([[0.5]], np.float32), 1, "gauss", 1.0, 0.0, 1, 18),
    "stripes-n2100-k1": (lambda: datagen.make_points(3, n=2100, d=20)[0], 1, "poly", 0.1, 1.0, 2, 19),
    # the largest cluster count (KKM_MAX_K); with n=3000 many clusters hold 1-5 points or none
    "kmax1024-n3000": (lambda: datagen.make_points(5, n=3000, d=8)[0], 1024, "gauss", 0.125, 0.0, 1, 20),
    # a wide point (d_pad = 2512, 157 k chunks)
    "d2500-n300": (lambda: datagen.make_points(2, n=300, d=2500)[0], 6, "poly", 1.0 / 2500, 1.0, 3, 21),
    # two and three 16-label blocks in the packed SpMM's column side
    "k20-n1500-gauss": (lambda: datagen.make_points(2, n=1500, d=24)[0], 20, "gauss", 1.0 / 24, 0.0, 1, 22),
    "k40-n1800-poly": (lambda: datagen.separated_blobs(1800, 6, 40, seed=6, spread=2.5, sigma=1.0)[0],
                       40, "poly", 0.2, 1.0, 2, 23),
    # more than 16 labels above 4096 points: the packed SpMM's 16-tile segments
    # (ragged last segment); the polynomial's rows scaled by powers of two for
    # the split column side
    "k40-n6000-gauss": (lambda: datagen.make_points(4, n=6000, d=16)[0], 40, "gauss", 0.5, 0.0, 1, 30),
    "k24-n5000-poly": (lambda: datagen.make_points(2, n=5000, d=20)[0], 24, "poly", 0.05, 1.0, 2, 31),
    # the row scales of the split column side over widely spread row norms
    "k33-n5000-linear-spread": (lambda: _norm_spread(datagen.make_points(2, n=5000, d=12)[0], 32),
                                33, "linear", 1.0, 0.0, 1, 32),
    "k20-n3000-poly-spread": (lambda: _norm_spread(datagen.make_points(4, n=3000, d=10)[0], 33),
                              20, "poly", 0.1, 0.5, 3, 33),
}


def _setup(name, oracle):
    pts, k, kind, g, c, p, seed = CASES[name]
    X = pts()
    n = X.shape[0]
    cl = datagen.make_init(1, n, k) if seed is None else datagen.random_init(n, k, seed)
    kern = oracle.Kernel(kind, g, c, p)
    return X, k, kind, g, c, p, cl, kern


MODES = ["resident", "onthefly", "packed"]
PACKED_MAX_K = 64


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", list(CASES))
def test_kernel_matrix(oracle, name, mode):
    """K (resident: the stored matrix; packed: the stored upper block triangle,
    the rest read by symmetry; on the fly: rows from the same tile kernel and
    epilogue the update sweep uses) against the oracle."""
    _torch_cuda()
    print(f"[gpu] K parity {name} {mode}", flush=True)
    X, k, kind, g, c, p, cl, kern = _setup(name, oracle)
    with Engine(X, kind, g, c, p, mode=mode) as eng:
        K = eng.K_rows()
        diag = eng.diag()
        info = eng.info()
    from paper_2601_17136_amd import kkm
    assert info["mode"] == kkm.MODES[mode]
    Kref = kern.matrix(X)
    err = rowscaled_err(K, Kref)
    assert err <= TOL, f"K row-scaled error {err:.3e}"
    if mode in ("resident", "packed"):
        assert np.array_equal(K, K.T), "K is not exactly symmetric"
        np.testing.assert_array_equal(diag, np.diag(K))
    assert rel_err(diag, np.diag(Kref)) <= TOL
    if kind == "gauss":
        assert np.all(diag == 1.0) and np.all(np.diag(K) == 1.0)
    print(f"[gpu] {name} {mode}: K err {err:.2e}, fixups {info['fixups']}", flush=True)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", list(CASES))
def test_step(oracle, name, mode):
    _torch_cuda()
    print(f"[gpu] step parity {name} {mode}", flush=True)
    X, k, kind, g, c, p, cl, kern = _setup(name, oracle)
    if mode == "packed" and k > PACKED_MAX_K:
        from paper_2601_17136_amd import kkm
        with Engine(X, kind, g, c, p, mode=mode) as eng:
            with pytest.raises(kkm.KKMError) as e:
                eng.step(cl, k)
        assert e.value.code == kkm.KKM_ERR_ARG and "packed" in str(e.value)
        return
    ref = oracle.step_full(kern.matrix(X), cl, k)
    with Engine(X, kind, g, c, p, mode=mode) as eng:
        out = eng.step(cl, k)
    np.testing.assert_array_equal(out["counts"], ref["counts"])
    eE, eD = rowscaled_err(out["E"], ref["E"]), rowscaled_err(out["D"], ref["D"])
    ez, eJ = rel_err(out["z"], ref["z"]), rel_err(out["J"], ref["J"]) if ref["J"] != 0 else abs(out["J"])
    assert eE <= TOL and eD <= TOL and ez <= TOL and eJ <= TOL, (eE, eD, ez, eJ)
    mism = assignment_mismatches(out["cl"], ref["cl"], ref["D"])
    print(f"[gpu] {name}: E {eE:.2e} D {eD:.2e} z {ez:.2e} J {eJ:.2e} near-tie flips {mism}", flush=True)


def _margins(oracle, K, cl, k, iters):
    """Smallest row-scaled gap between the best and second-best distance at each
    update of the oracle's trajectory from cl (0 where a row has one finite D)."""
    out_m = []
    for _ in range(iters):
        out = oracle.step_full(K, cl, k)
        D = out["D"]
        fin = np.isfinite(D)
        s = np.sort(np.where(fin, D, np.inf), axis=1)
        gap = np.where(np.isfinite(s[:, 1]), s[:, 1] - s[:, 0], np.inf)
        out_m.append(float((gap / np.where(fin, np.abs(D), 0).max(axis=1)).min()))
        cl = out["cl"]
        if out["changed"] == 0:
            break
    return out_m


WELL_SEPARATED = [  # (kernel, gamma, coef0, degree, scrambled fraction of the init, seed)
    ("poly", 1.0, 1.0, 2, 0.9, 0), ("poly", 0.01, 1.0, 2, 0.9, 1), ("gauss", 1 / 128, 0.0, 1, 0.95, 0),
    ("linear", 1.0, 0.0, 1, 0.8, 0), ("gauss", 1 / 128, 0.0, 1, 0.9, 2),
]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("case", WELL_SEPARATED, ids=lambda c: f"{c[0]}-{c[1]:g}-{c[4]}-{c[5]}")
def test_well_separated_trajectory_is_exact(oracle, case, mode):
    """On input the oracle certifies as well separated (every point's best and
    second-best distance differ by more than 1e-3 of its row at every update)
    the whole trajectory matches bit for bit, including where it stops."""
    _torch_cuda()
    kind, g, c, p, frac, seed = case
    X, lab = datagen.make_points(1)
    rng = np.random.default_rng(seed)
    cl0 = lab.copy()
    scr = rng.random(lab.size) < frac
    cl0[scr] = rng.integers(0, 8, int(scr.sum()))
    K = oracle.Kernel(kind, g, c, p).matrix(X)
    m = _margins(oracle, K, cl0, 8, 30)
    assert min(m) > 1e-3, f"input not well separated (margins {m})"
    cl_ref, done_ref, hist_ref, traj = oracle.iterate_full(K, cl0, 8, 30, tol=0.0)
    with Engine(X, kind, g, c, p, mode=mode) as eng:
        cl = cl0
        for t in range(done_ref):
            nxt, it, _ = eng.iterate(cl, 8, 1)
            assert np.array_equal(nxt, traj[t]), f"update {t} differs"
            cl = nxt
        final, done, hist = eng.iterate(cl0, 8, 30, tol=0.0)
    assert done == done_ref
    np.testing.assert_array_equal(final, cl_ref)
    assert np.max(np.abs(hist - hist_ref) / np.abs(hist_ref)) <= TOL


def test_blobs_stepwise_along_engine_trajectory(oracle):
    """Workload 1 (20 updates of the paper's kernel from round-robin ids): it
    passes near-ties of ~1e-7 relative, below fp32 resolution, so each update
    is compared with the oracle's update from the engine's own ids."""
    _torch_cuda()
    w, X, _ = datagen.workload(1)
    cl0 = datagen.make_init(1, w.n, w.k)
    K = oracle.Kernel(w.kind, w.gamma, w.coef0, w.degree).matrix(X)
    flips = 0
    with Engine(X, w.kind, w.gamma, w.coef0, w.degree) as eng:
        cl = cl0
        for t in range(w.iters):
            ref = oracle.step_full(K, cl, w.k)
            nxt, it, hist = eng.iterate(cl, w.k, 1)
            assert it == 1 and rel_err(hist[0], ref["J"]) <= TOL
            flips += assignment_mismatches(nxt, ref["cl"], ref["D"])
            cl = nxt
        final, it, hist = eng.iterate(cl0, w.k, w.iters)
    assert it == w.iters and np.array_equal(final, cl)   # the loop equals its single steps
    print(f"[gpu] workload 1: {flips} near-tie flips over {w.iters} updates", flush=True)


STOP_GOLDEN = ["stop_rule_linear_1d_a.json", "stop_rule_linear_1d_b.json"]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", STOP_GOLDEN)
def test_stop_rule_hand_worked(name, mode):
    """The loop and its stop rule (Alg. 1 'while not converged'; the tol reading)
    on the hand-worked trajectories of tests/golden: the relative drop of J
    reaches tol at update t = 2, one update before tol = 0 stops, and at
    tol = 0.25 (fixture a) and 1/16 (fixture b) with equality.  Every value is
    exact in fp32 and fp64, so done, the final ids and J must match exactly."""
    import json
    import os
    _torch_cuda()
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", name)))
    X = np.array(g["X"], dtype=np.float32)
    cl0 = np.array(g["cl0"], dtype=np.int32)
    with Engine(X, "linear", mode=mode) as eng:
        for r in g["runs"]:
            cl, done, hist = eng.iterate(cl0, g["k"], r["max_iter"], tol=r["tol"])
            assert done == r["done"], (r["tol"], done, r["done"])
            np.testing.assert_array_equal(cl, r["cl_final"])
            np.testing.assert_array_equal(hist, r["obj_hist"])


def _chain(oracle):
    """Twelve tight groups of 40 points on a line (3-D, sigma 0.05), two clusters
    from a misplaced split: Lloyd moves the boundary over 7 updates, and the
    relative drops of J are 0.239, 0.118, 0.057, 0.110, 0.168, 0.206."""
    pos = [4, 8, 14, 16, 18, 20, 24, 25, 27, 31, 53, 54]
    lab = [0, 0, 1, 0, 1, 1, 1, 1, 1, 1, 1, 1]
    rng = np.random.default_rng(31)
    X = np.zeros((len(pos) * 40, 3), np.float32)
    X[:, 0] = np.repeat(pos, 40)
    X = (X + 0.05 * rng.standard_normal(X.shape)).astype(np.float32)
    cl0 = np.repeat(lab, 40).astype(np.int32)
    perm = rng.permutation(X.shape[0])
    return X[perm], cl0[perm]


@pytest.mark.parametrize("mode", MODES)
def test_stop_rules_match_oracle(oracle, mode):
    """tol = 0 stops when no id changed, tol > 0 also on a small relative drop of
    J, tol < 0 runs every update.  On a certified well-separated trajectory of 7
    updates, tol = 0.08 stops after update 3 and tol = 0.15 after update 2:
    both differ from tol = 0 and from the first update where the rule can fire,
    so a rule with the drop's sign flipped (which fires there) fails."""
    _torch_cuda()
    X, cl0 = _chain(oracle)
    K = oracle.Kernel("linear").matrix(X)
    assert min(_margins(oracle, K, cl0, 2, 40)) > 1e-3
    expect = {0.0: 7, 0.08: 4, 0.15: 3, -1.0: 40}
    with Engine(X, "linear", mode=mode) as eng:
        for tol, want in expect.items():
            cl_ref, done_ref, hist_ref, _ = oracle.iterate_full(K, cl0, 2, 40, tol=tol)
            assert done_ref == want, (tol, done_ref)
            cl, done, hist = eng.iterate(cl0, 2, 40, tol=tol)
            assert done == done_ref, (tol, done, done_ref)
            np.testing.assert_array_equal(cl, cl_ref)
            assert np.max(np.abs(hist - hist_ref) / np.abs(hist_ref)) <= TOL


@pytest.mark.parametrize("mode", MODES)
def test_empty_cluster_and_ties(oracle, mode):
    _torch_cuda()
    X = np.array([[-1.0], [1.0], [0.0], [0.0], [3.0]], np.float32)
    cl = np.array([0, 1, 0, 1, 1], np.int32)    # cluster 2 empty
    kern = oracle.Kernel("linear")
    ref = oracle.step_full(kern.matrix(X), cl, 3)
    with Engine(X, "linear", mode=mode) as eng:
        out = eng.step(cl, 3)
    assert out["counts"][2] == 0 and np.all(np.isinf(out["D"][:, 2])) and out["z"][2] == 0
    np.testing.assert_array_equal(out["cl"], ref["cl"])
    assert rowscaled_err(out["D"], ref["D"]) <= TOL


@pytest.mark.parametrize("mode", MODES)
def test_each_point_its_own_cluster(oracle, mode):
    """k = n (packed: n = k = its largest k, four full label blocks)."""
    _torch_cuda()
    n = PACKED_MAX_K if mode == "packed" else 70
    X = datagen.make_points(2, n=n, d=9)[0]
    with Engine(X, "gauss", 0.2, mode=mode) as eng:
        out = eng.step(np.arange(n, dtype=np.int32), n)
    assert abs(out["J"]) <= 1e-4 * n
    np.testing.assert_array_equal(out["cl"], np.arange(n))
    assert np.all(np.abs(np.diag(out["D"])) <= 1e-5)


@pytest.mark.parametrize("mode", MODES)
def test_invalid_ids_are_reported(oracle, mode):
    _torch_cuda()
    from paper_2601_17136_amd import kkm
    X = datagen.make_points(1, n=300)[0]
    with Engine(X, "poly", 1.0, 1.0, 2, mode=mode) as eng:
        for bad in (8, -1):
            cl = datagen.random_init(300, 8, 3)
            cl[123] = bad
            with pytest.raises(kkm.KKMError) as e:
                eng.iterate(cl, 8, 3)
            assert e.value.code == kkm.KKM_ERR_DEVICE_DATA
        cl, it, _ = eng.iterate(datagen.random_init(300, 8, 3), 8, 2)   # context still usable
        assert it == 2


@pytest.mark.parametrize("mode", MODES)
def test_bitwise_reproducible(oracle, mode):
    _torch_cuda()
    X = datagen.make_points(4, n=2500)[0]
    cl = datagen.random_init(2500, 64, 40)
    runs = []
    for _ in range(2):
        with Engine(X, "gauss", 0.5, mode=mode) as eng:
            runs.append((eng.K_rows(0, 64), eng.step(cl, 64), eng.iterate(cl, 64, 5)))
    (K1, s1, i1), (K2, s2, i2) = runs
    assert np.array_equal(K1, K2)
    for key in ("E", "D", "z", "cl", "counts"):
        assert np.array_equal(s1[key], s2[key]), key
    assert s1["J"] == s2["J"]
    assert np.array_equal(i1[0], i2[0]) and np.array_equal(i1[2], i2[2])


@pytest.mark.parametrize("d", [128, 24])
@pytest.mark.parametrize("mode", ["resident", "packed"])
def test_gauss_fixup_overflow_path(oracle, mode, d):
    """With a memory budget that leaves room for only a few ten thousand fix-up
    list entries, more entries qualify than the list holds and the fix-up
    re-tests the whole triangle; K must still match the oracle.  The points
    are shifted by a common offset: the Gaussian K does not change, but the
    norms grow, so the expansion loses digits on most pairs and nearly every
    entry with a non-negligible value is listed."""
    _torch_cuda()
    from paper_2601_17136_amd import kkm
    X = datagen.make_points(4, n=3000, d=d)[0] + np.float32(30.0)
    _, need = kkm.kkm_plan(3000, X.shape[1], 1, kkm.KKM_GAUSS, 1 << 40, kkm.MODES[mode])
    with Engine(X, "gauss", 0.5, mode=mode, mem_budget=need + 4096) as eng:
        K = eng.K_rows()
        info = eng.info()
    assert info["fixups"] > info["fixup_capacity"] > 0, info
    err = rowscaled_err(K, oracle.Kernel("gauss", 0.5).matrix(X))
    assert err <= TOL, err
    # the re-test pass runs after the listed pairs and recomputes with the same
    # routine: K is exactly symmetric and the same bits come back on a rebuild
    np.testing.assert_array_equal(K, K.T)
    with Engine(X, "gauss", 0.5, mode=mode, mem_budget=need + 4096) as eng:
        np.testing.assert_array_equal(eng.K_rows(), K)
    with Engine(X, "gauss", 0.5, mode=mode) as eng:
        K2 = eng.K_rows()
    assert rowscaled_err(K2, oracle.Kernel("gauss", 0.5).matrix(X)) <= TOL


@pytest.mark.parametrize("kind,k_hint,want", [("gauss", 8, "packed"), ("gauss", 40, "packed"),
                                               ("poly", 64, "packed"), ("poly", 65, "resident"),
                                               ("gauss", 0, "resident")])
def test_auto_mode_follows_the_k_hint(oracle, kind, k_hint, want):
    """AUTO stores K packed when the announced k is at most 64 and fully
    otherwise or without a hint (memory allowing); either way the step
    matches the oracle."""
    _torch_cuda()
    from paper_2601_17136_amd import kkm
    X = datagen.make_points(2, n=700, d=12)[0]
    k = k_hint or 5
    cl = datagen.random_init(700, k, 3)
    g, c, p = (0.1, 0.0, 1) if kind == "gauss" else (0.05, 1.0, 2)
    ref = oracle.step_full(oracle.Kernel(kind, g, c, p).matrix(X), cl, k)
    with Engine(X, kind, g, c, p, mode="auto", k_hint=k_hint) as eng:
        assert eng.info()["mode"] == kkm.MODES[want]
        out = eng.step(cl, k)
    assert rowscaled_err(out["E"], ref["E"]) <= TOL and rowscaled_err(out["D"], ref["D"]) <= TOL


def test_nonpsd_polynomial_build_warns(oracle):
    """A polynomial kernel with coef0 < 0 builds, warns that J need not fall,
    and still matches the oracle's step."""
    _torch_cuda()
    X = datagen.make_points(2, n=300, d=6)[0]
    cl = datagen.random_init(300, 4, 5)
    with pytest.warns(RuntimeWarning, match="positive semidefinite"):
        eng = Engine(X, "poly", 1.0, -2.0, 2)
    with eng:
        out = eng.step(cl, 4)
    ref = oracle.step_full(oracle.Kernel("poly", 1.0, -2.0, 2).matrix(X), cl, 4)
    assert rowscaled_err(out["E"], ref["E"]) <= TOL and rowscaled_err(out["D"], ref["D"]) <= TOL


def test_packed_k_limit(oracle):
    """Packed storage takes k <= 64 (four 16-label MFMA blocks); k = 65 is
    refused before anything is enqueued, and the context stays usable."""
    _torch_cuda()
    from paper_2601_17136_amd import kkm
    X = datagen.make_points(2, n=500, d=9)[0]
    with Engine(X, "gauss", 0.2, mode="packed") as eng:
        for k in (PACKED_MAX_K + 1, 1024):
            with pytest.raises(kkm.KKMError) as e:
                eng.iterate(datagen.random_init(500, k, 1), k, 2)
            assert e.value.code == kkm.KKM_ERR_ARG
        _, it, _ = eng.iterate(datagen.random_init(500, PACKED_MAX_K, 1), PACKED_MAX_K, 2)
        assert it == 2
