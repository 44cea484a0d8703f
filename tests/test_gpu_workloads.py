"""GPU parity at the full workload sizes, in the launch configurations the
benchmark times (packed and resident K, K on the fly: the same build and
update kernels).

The oracle cannot form K at these sizes, so each check is on outputs it can
compute one by one:
  * K and E and D on 48 sampled rows (tile and stripe boundaries included);
  * every cluster self-term z_j (the oracle sums each cluster's block of K);
  * J, the cluster sizes (exact) and the new ids on the sampled rows;
and on properties that hold at any size for a whole loop: J non-increasing
within fp32 noise, sizes summing to n, ids in range, loop == its single steps.
"""
import numpy as np
import pytest

from gpu_helpers import TOL, Engine, assignment_mismatches, rel_err, rowscaled_err
from paper_2601_17136_amd import datagen

pytestmark = pytest.mark.gpu


def _rows(n, seed):
    fixed = [0, 1, 127, 128, 129, 1023, 1024, n // 2, n - 2, n - 1]
    rng = np.random.default_rng(seed)
    extra = rng.choice(n, size=48 - len(fixed), replace=False)
    return np.unique(np.concatenate([fixed, extra]).astype(np.int64))


@pytest.mark.parametrize("cfg,mode", [(2, "packed"), (3, "packed"), (4, "packed"), (5, "packed"),
                                      (2, "resident"), (3, "resident"), (4, "resident"),
                                      (5, "resident"), (5, "onthefly"), (2, "onthefly")])
def test_workload_step_full_size(oracle, cfg, mode):
    torch = pytest.importorskip("torch")
    assert torch.cuda.is_available()
    w, X, cl = datagen.workload(cfg)
    n, k = w.n, w.k
    print(f"[gpu] full-size step parity: {w.describe()} K {mode}", flush=True)
    kern = oracle.Kernel(w.kind, w.gamma, w.coef0, w.degree)
    rows = _rows(n, cfg)
    with Engine(X, w.kind, w.gamma, w.coef0, w.degree, mode=mode) as eng:
        info = eng.info()
        assert info["mode"] == eng.kkm.MODES[mode]
        K_rows = np.stack([eng.K_rows(int(r), int(r) + 1)[0] for r in rows])
        diag = eng.diag()
        out = eng.step(cl, k)
        print(f"[gpu] cfg {cfg}: built and stepped (fixups {info['fixups']})", flush=True)
    ref = oracle.step_rows(kern, X, cl, k, rows)
    eK = rowscaled_err(K_rows, ref["K_rows"])
    assert eK <= TOL, f"K rows error {eK:.3e}"
    np.testing.assert_array_equal(out["counts"], ref["counts"])
    ez = rel_err(out["z"], ref["z"])
    eJ = rel_err(out["J"], ref["J"])
    eE = rowscaled_err(out["E"][rows], ref["E"])
    eD = rowscaled_err(out["D"][rows], ref["D"])
    assert ez <= TOL and eJ <= TOL and eE <= TOL and eD <= TOL, (ez, eJ, eE, eD)
    flips = assignment_mismatches(out["cl"][rows], ref["cl"], ref["D"])
    if w.kind == "gauss":
        assert np.all(diag == 1.0)
    else:
        assert rel_err(diag[rows], kern.diag(X)[rows]) <= TOL
    # the new ids are a valid argmin of the engine's own D everywhere
    D = out["D"]
    assert np.all(D[np.arange(n), out["cl"]] == D.min(axis=1))
    print(f"[gpu] cfg {cfg}: K {eK:.2e} E {eE:.2e} D {eD:.2e} z {ez:.2e} J {eJ:.2e} flips {flips}",
          flush=True)


@pytest.mark.parametrize("kind,k", [("poly", 40), ("linear", 20), ("gauss", 33), ("gauss", 64)])
def test_many_labels_tall_chunks(oracle, kind, k):
    """More than 16 labels above 40000 points: the packed SpMM's 128-row
    chunks and 32-tile segments with three or four 16-label blocks; the
    polynomial's rows scaled by powers of two for the split column side, the
    Gaussian's not; checked on sampled rows as above."""
    torch = pytest.importorskip("torch")
    assert torch.cuda.is_available()
    n, d = 45000, 48
    X = datagen.make_points(5, n=n, d=d)[0]
    cl = datagen.random_init(n, k, 40 + k)
    g, c, p = {"poly": (1.0 / d, 1.0, 2), "linear": (1.0, 0.0, 1), "gauss": (1.0 / d, 0.0, 1)}[kind]
    print(f"[gpu] packed, n={n} d={d} k={k} {kind}", flush=True)
    kern = oracle.Kernel(kind, g, c, p)
    rows = _rows(n, k)
    with Engine(X, kind, g, c, p, mode="packed") as eng:
        out = eng.step(cl, k)
        again = eng.step(cl, k)
    assert np.array_equal(out["E"], again["E"]) and out["J"] == again["J"]
    ref = oracle.step_rows(kern, X, cl, k, rows)
    np.testing.assert_array_equal(out["counts"], ref["counts"])
    ez, eJ = rel_err(out["z"], ref["z"]), rel_err(out["J"], ref["J"])
    eE = rowscaled_err(out["E"][rows], ref["E"])
    eD = rowscaled_err(out["D"][rows], ref["D"])
    assert ez <= TOL and eJ <= TOL and eE <= TOL and eD <= TOL, (ez, eJ, eE, eD)
    D = out["D"]
    assert np.all(D[np.arange(n), out["cl"]] == D.min(axis=1))
    print(f"[gpu] k={k} {kind}: E {eE:.2e} D {eD:.2e} z {ez:.2e} J {eJ:.2e}", flush=True)


@pytest.mark.parametrize("cfg,mode", [(2, "packed"), (4, "packed"), (2, "resident"), (4, "resident"),
                                      (2, "onthefly")])
def test_workload_loop_properties(oracle, cfg, mode):
    torch = pytest.importorskip("torch")
    assert torch.cuda.is_available()
    w, X, cl0 = datagen.workload(cfg)
    print(f"[gpu] full-size loop: {w.describe()} K {mode}", flush=True)
    with Engine(X, w.kind, w.gamma, w.coef0, w.degree, mode=mode) as eng:
        final, it, hist = eng.iterate(cl0, w.k, w.iters)
        cl = cl0
        for t in range(3):
            cl, _, _ = eng.iterate(cl, w.k, 1)
        three, _, _ = eng.iterate(cl0, w.k, 3)
        J_final = eng.kkm.kkm_objective(eng.ctx, torch.from_numpy(final).cuda(), w.k)
    assert it == w.iters
    assert final.min() >= 0 and final.max() < w.k
    assert np.array_equal(three, cl)
    # J(cl_t) non-increasing up to fp32 noise on the objective
    assert np.all(np.diff(hist) <= 1e-5 * np.abs(hist[:-1])), hist
    assert J_final <= hist[-1] * (1 + 1e-5)
    print(f"[gpu] cfg {cfg}: J {hist[0]:.6g} -> {hist[-1]:.6g} -> {J_final:.6g}", flush=True)
