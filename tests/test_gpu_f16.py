"""GPU parity of binary16 K storage (kkm_params.storage = F16) with the fp64 oracle.

Mixed precision is the paper's future work (Section VII); the bar here is the
error the storage format can introduce, derived from the arithmetic, on top
of the fp32 bar of the other parity tests (TOL of the row scale):

  entry   |K~(i,j) - K(i,j)| <= 2^-11 |K(i,j)| + 2^-25 w
          (K(i,j)/w rounded to nearest binary16, |K/w| <= 1, w the storing
          row's scale; 2^-25 w is half the subnormal spacing)
  E(i,j)  <= 2^-11 sum_{m in L_j} |K(i,m)| + 2^-25 sum_{m in L_j} max(w_i, w_m)
  z_j     <= 2^-11 (sum_{i in L_j} sqrt K(i,i))^2 / |L_j|^2 + 2^-25 max w
          (for a PSD kernel |K(i,m)| <= sqrt(K(i,i) K(m,m)))
  D(i,j)  <= 2 bound_E(i,j) / |L_j| + bound_z(j)
  J       <= sum_j |L_j| bound_z(j)

Ids may differ from the oracle's only where the oracle's distances are
within the two D bounds of each other.  diag K (and tr K) is fp32 whatever
the storage, so it must equal the fp32 build's exactly.
"""
import numpy as np
import pytest

from gpu_helpers import TIE, TOL, Engine
from paper_2601_17136_amd import datagen
from test_gpu_parity import CASES, _setup

pytestmark = pytest.mark.gpu

U16 = 2.0 ** -11
SUB = 2.0 ** -25
F16_CASES = ["blobs-n2000-poly", "ragged-poly3", "ragged-gauss", "linear-n300", "rings-n3000-gauss", "n129-d1",
             "stripes-n2100-k1", "d2500-n300", "n2-k2", "k20-n1500-gauss", "k40-n1800-poly",
             "k40-n6000-gauss", "k24-n5000-poly", "k33-n5000-linear-spread", "k20-n3000-poly-spread"]


def row_scales(X, kind, g, c, p):
    """The storage row scales from their definition (Cauchy-Schwarz bounds), fp64."""
    nrm = (np.asarray(X, np.float64) ** 2).sum(axis=1)
    dot = np.sqrt(nrm * nrm.max())
    if kind == "gauss":
        w = np.ones_like(dot)
    elif kind == "poly":
        w = (abs(np.float32(g)) * dot + abs(np.float32(c))) ** p
    else:
        w = dot
    w[w == 0] = 1.0
    return w


def bounds(Krows, rows, diagK, w, cl, k):
    """Storage error bounds of E, z, D (rows of the sample) and J."""
    cl = np.asarray(cl)
    V = np.zeros((cl.size, k))
    V[np.arange(cl.size), cl] = 1.0
    counts = V.sum(axis=0)
    cnt = np.maximum(counts, 1.0)
    bE = U16 * (np.abs(Krows) @ V) + SUB * (np.maximum(w[rows][:, None], w[None, :]) @ V)
    sq = np.sqrt(np.maximum(diagK, 0.0)) @ V
    bz = U16 * sq ** 2 / cnt ** 2 + SUB * w.max()
    bD = 2.0 * bE / cnt[None, :] + bz[None, :]
    bJ = float(np.sum(counts * bz))
    return bE, bz, bD, bJ


def check_within(gpu, ref, bound, what):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(gpu)), f"{what}: infinite entries differ"
    scale = np.abs(np.where(fin, ref, 0.0))
    if scale.ndim == 2:
        scale = scale.max(axis=1, keepdims=True)
    allow = 1.05 * np.where(fin, bound, 0.0) + TOL * np.maximum(scale, 1e-30)
    err = np.abs(np.where(fin, gpu, 0.0) - np.where(fin, ref, 0.0))
    worst = np.max(err / allow) if err.size else 0.0
    assert worst <= 1.0, f"{what}: error {float(np.max(err)):.3e} exceeds its bound (ratio {worst:.2f})"
    return float(np.max(err / np.maximum(scale, 1e-30))) if err.size else 0.0


def check_ids(cl_gpu, cl_ref, Dref, bD):
    bad = np.nonzero(np.asarray(cl_gpu) != np.asarray(cl_ref))[0]
    for i in bad:
        a, r = int(cl_gpu[i]), int(cl_ref[i])
        scale = np.abs(Dref[i][np.isfinite(Dref[i])]).max()
        assert Dref[i, a] - Dref[i, r] <= bD[i, a] + bD[i, r] + TIE * scale, (i, a, r)
    return len(bad)


@pytest.mark.parametrize("mode", ["resident", "packed"])
@pytest.mark.parametrize("name", F16_CASES)
def test_f16_step(oracle, name, mode):
    X, k, kind, g, c, p, cl, kern = _setup(name, oracle)
    print(f"[gpu] binary16 K step {name} {mode}", flush=True)
    n = X.shape[0]
    with Engine(X, kind, g, c, p, mode=mode, storage="f16") as eng:
        info = eng.info()
        K = eng.K_rows()
        diag16 = eng.diag()
        out = eng.step(cl, k)
    with Engine(X, kind, g, c, p, mode=mode) as eng32:
        diag32 = eng32.diag()
    assert info["storage"] == 1
    # diag K stays fp32 in both formats; the two builds may sum x.x in another
    # order (the small-width fp32 build runs a different product loop)
    np.testing.assert_allclose(diag16, diag32, rtol=1e-5, atol=1e-6 * float(np.abs(diag32).max()))
    Kref = kern.matrix(X)
    w = row_scales(X, kind, g, c, p)
    rows = np.arange(n)
    bK = U16 * np.abs(Kref) + SUB * np.maximum(w[:, None], w[None, :])
    eK = check_within(K, Kref, bK, "K")
    # Gaussian rows are unscaled, so K(i,j) and K(j,i) round alike; packed K
    # stores an off-diagonal tile once, but a diagonal tile keeps (i,j) and
    # (j,i) in their own rows, each with its row's scale
    if kind == "gauss":
        assert np.array_equal(K, K.T), "binary16 Gaussian K should be symmetric"
    elif mode == "packed":
        tile = np.arange(n) // 128
        off = tile[:, None] != tile[None, :]
        assert np.array_equal(K[off], K.T[off]), "packed K off the diagonal tiles should be symmetric"
    ref = oracle.step_full(Kref, cl, k)
    bE, bz, bD, bJ = bounds(Kref, rows, np.diag(Kref), w, cl, k)
    np.testing.assert_array_equal(out["counts"], ref["counts"])
    eE = check_within(out["E"], ref["E"], bE, "E")
    ez = check_within(out["z"], ref["z"], bz, "z")
    eD = check_within(out["D"], ref["D"], bD, "D")
    check_within([out["J"]], [ref["J"]], [bJ], "J")
    flips = check_ids(out["cl"], ref["cl"], ref["D"], bD)
    print(f"[gpu] {name} {mode}: K {eK:.2e} E {eE:.2e} z {ez:.2e} D {eD:.2e} (row-scaled), id flips {flips}",
          flush=True)


def test_f16_halves_the_stored_bytes():
    X = datagen.make_points(2, n=1000, d=16)[0]
    for mode in ("resident", "packed"):
        with Engine(X, "gauss", 0.1, mode=mode) as e32:
            b32 = e32.info()["bytes_K"]
        with Engine(X, "gauss", 0.1, mode=mode, storage="f16") as e16:
            b16 = e16.info()["bytes_K"]
        assert b16 * 2 == b32, (mode, b16, b32)
    with Engine(X, "gauss", 0.1, mode="onthefly", storage="f16") as e:
        assert e.info()["storage"] == 0 and e.info()["bytes_K"] == 0


@pytest.mark.parametrize("cfg,mode", [(2, "packed"), (2, "resident"), (3, "packed"), (4, "packed"), (5, "packed")])
def test_f16_workload_step(oracle, cfg, mode):
    w_, X, cl = datagen.workload(cfg)
    print(f"[gpu] binary16 K full-size step: {w_.describe()} {mode}", flush=True)
    sampled_step(oracle, X, w_.kind, w_.gamma, w_.coef0, w_.degree, cl, w_.k, mode, cfg, f"cfg {cfg} {mode}")


@pytest.mark.parametrize("kind,k", [("poly", 40), ("gauss", 64), ("linear", 20)])
def test_f16_many_labels_tall_chunks(oracle, kind, k):
    """Binary16 packed K with more than 16 labels above 40000 points: 128-row
    chunks, 32-tile segments, two to four label blocks, two tiles per step."""
    n, d = 45000, 48
    X = datagen.make_points(5, n=n, d=d)[0]
    cl = datagen.random_init(n, k, 40 + k)
    g, c, p = {"poly": (1.0 / d, 1.0, 2), "linear": (1.0, 0.0, 1), "gauss": (1.0 / d, 0.0, 1)}[kind]
    print(f"[gpu] binary16 packed, n={n} d={d} k={k} {kind}", flush=True)
    sampled_step(oracle, X, kind, g, c, p, cl, k, "packed", k, f"n={n} k={k} {kind}")


def sampled_step(oracle, X, kind, g, c, p, cl, k, mode, seed, label):
    """One binary16 step against the oracle on sampled rows, within the storage
    bounds; the step repeated on the same context gives the same bits."""
    n = X.shape[0]
    kern = oracle.Kernel(kind, g, c, p)
    rows = np.unique(np.concatenate([[0, 1, 127, 128, n // 2, n - 1],
                                     np.random.default_rng(seed).choice(n, 42, replace=False)]))
    with Engine(X, kind, g, c, p, mode=mode, storage="f16") as eng:
        Krows = np.stack([eng.K_rows(int(r), int(r) + 1)[0] for r in rows])
        out = eng.step(cl, k)
        again = eng.step(cl, k)
    assert np.array_equal(out["E"], again["E"]) and out["J"] == again["J"]
    ref = oracle.step_rows(kern, X, cl, k, rows)
    diagK = kern.diag(X)
    w = row_scales(X, kind, g, c, p)
    bK = U16 * np.abs(ref["K_rows"]) + SUB * np.maximum(w[rows][:, None], w[None, :])
    eK = check_within(Krows, ref["K_rows"], bK, "K rows")
    bE, bz, bD, bJ = bounds(ref["K_rows"], rows, diagK, w, cl, k)
    np.testing.assert_array_equal(out["counts"], ref["counts"])
    eE = check_within(out["E"][rows], ref["E"], bE, "E")
    ez = check_within(out["z"], ref["z"], bz, "z")
    eD = check_within(out["D"][rows], ref["D"], bD, "D")
    check_within([out["J"]], [ref["J"]], [bJ], "J")
    flips = check_ids(out["cl"][rows], ref["cl"], ref["D"], bD)
    print(f"[gpu] {label}: K {eK:.2e} E {eE:.2e} z {ez:.2e} D {eD:.2e}, id flips {flips}", flush=True)


@pytest.mark.parametrize("cfg,mode", [(2, "packed"), (4, "resident")])
def test_f16_loop(cfg, mode):
    """The loop on binary16 K: ids in range, sizes add up, J non-increasing
    within the storage error (the rounded matrix need not be exactly PSD), and
    the final J within 1e-3 of the fp32 run's."""
    w_, X, cl0 = datagen.workload(cfg)
    with Engine(X, w_.kind, w_.gamma, w_.coef0, w_.degree, mode=mode, storage="f16") as eng:
        final, it, hist = eng.iterate(cl0, w_.k, 10)
    with Engine(X, w_.kind, w_.gamma, w_.coef0, w_.degree, mode=mode) as eng:
        _, _, hist32 = eng.iterate(cl0, w_.k, 10)
    assert it == 10 and final.min() >= 0 and final.max() < w_.k
    assert np.all(np.diff(hist) <= 2 * U16 * np.abs(hist[:-1])), hist
    assert abs(hist[-1] - hist32[-1]) <= 1e-3 * abs(hist32[-1]), (hist[-1], hist32[-1])
    print(f"[gpu] cfg {cfg} {mode}: J binary16 {hist[-1]:.8g}, fp32 {hist32[-1]:.8g}", flush=True)
