"""GPU parity for one GPU's share of the 1D split (kkm_build_panel,
kkm_panel_spmm, kkm_panel_assign): G column panels of K, each built and
stepped on a context of its own, with the two exchanges a multi-GPU run would
make (the all-reduce of the z parts, the all-gather of the new ids) done here
on the host.

Small problems against the full oracle step: every panel's K columns, the
panels' rows of E, the global z from the summed parts, the cluster sizes, and
the new ids (exact except at the oracle's near-ties).  At workload 5's shape
(n = 200,000 split over 8 GPUs: panels of 25,000 points, 20 GB each): K, E
and the new ids on sampled points and z against the oracle's sampled-row step.
"""
import numpy as np
import pytest

from gpu_helpers import TOL, assignment_mismatches, rel_err, rowscaled_err
from paper_2601_17136_amd import datagen

pytestmark = pytest.mark.gpu


def panel_bounds(n, G):
    """G contiguous point ranges, each starting at a multiple of 128 (empty ones dropped)."""
    b = [(g * n // G) // 128 * 128 for g in range(G)] + [n]
    return [(b[g], b[g + 1]) for g in range(G) if b[g + 1] > b[g]]


class Panel:
    """One GPU's share: a context holding the column panel K[:, c0:c1]."""

    def __init__(self, kkm, Xd, n, d, kind, gamma, coef0, degree, c0, c1):
        self.kkm, self.n, self.c0, self.c1 = kkm, n, c0, c1
        self.ctx = kkm.kkm_create(kkm.current_stream_handle())
        kkm.kkm_build_panel(self.ctx, Xd, n, d, kkm.KINDS[kind],
                            kkm.make_params(gamma, coef0, degree, kkm.KKM_MODE_RESIDENT), c0, c1)

    def K_rows(self, r0, r1):
        import torch
        out = torch.empty((r1 - r0, self.c1 - self.c0), device="cuda")
        self.kkm.kkm_copy_kernel_rows(self.ctx, r0, r1, out)
        return out.cpu().numpy()

    def close(self):
        if self.ctx is not None:
            self.kkm.kkm_destroy(self.ctx)
            self.ctx = None


def run_panels(X, kind, gamma, coef0, degree, cl, k, G, k_rows=None):
    """The update from ids cl split over G panels; returns the assembled outputs."""
    import torch

    from paper_2601_17136_amd import kkm
    n, d = X.shape
    Xd = torch.from_numpy(np.ascontiguousarray(X, dtype=np.float32)).cuda()
    cl_d = torch.from_numpy(np.ascontiguousarray(cl, dtype=np.int32)).cuda()
    panels = []
    try:
        for c0, c1 in panel_bounds(n, G):
            panels.append(Panel(kkm, Xd, n, d, kind, gamma, coef0, degree, c0, c1))
        zsum = np.zeros(k)
        counts = None
        for P in panels:  # each GPU's SpMM; the all-reduce of its z parts
            zpart, cnt = kkm.kkm_panel_spmm(P.ctx, cl_d, k)
            zsum += zpart
            if counts is None:
                counts = cnt
            np.testing.assert_array_equal(cnt, counts)  # every GPU counts all n ids
        c = counts.astype(np.float64)
        z = np.where(counts > 0, zsum / np.where(counts > 0, c * c, 1.0), 0.0)
        new = np.empty(n, dtype=np.int32)
        E = np.empty((n, k), dtype=np.float32)
        took = np.zeros(k, dtype=np.int64)
        for P in panels:  # each GPU's assignment; the all-gather of the ids
            w = P.c1 - P.c0
            out = torch.empty(w, dtype=torch.int32, device="cuda")
            Eo = torch.empty((w, k), device="cuda")
            took += kkm.kkm_panel_assign(P.ctx, k, z, out, Eo)
            new[P.c0:P.c1] = out.cpu().numpy()
            E[P.c0:P.c1] = Eo.cpu().numpy()
        K = None
        if k_rows is not None:  # rows of K, the panels' columns side by side
            every = len(k_rows) == n and np.array_equal(k_rows, np.arange(n))
            K = np.concatenate([P.K_rows(0, n) if every else
                                np.concatenate([P.K_rows(int(r), int(r) + 1) for r in k_rows])
                                for P in panels], axis=1)
        return dict(z=z, counts=counts, cl=new, E=E, took=took, K=K, npanels=len(panels))
    finally:
        for P in panels:
            P.close()


CASES = {
    # name: (points, k, kind, gamma, coef0, degree, init seed)
    "ragged-gauss": (lambda: datagen.make_points(2, n=777, d=37)[0], 9, "gauss", 0.3, 0.0, 1, 31),
    "blobs-poly": (lambda: datagen.make_points(1)[0], 8, "poly", 1.0, 1.0, 2, 32),
    # Gaussian entries the epilogue flags and the fix-up recomputes
    "rings-gauss": (lambda: datagen.make_points(4, n=2600)[0], 40, "gauss", 0.5, 0.0, 1, 33),
    "linear-n300": (lambda: datagen.separated_blobs(300, 3, 4, seed=4, spread=3.0, sigma=1.0)[0],
                    4, "linear", 1.0, 0.0, 1, 34),
}


@pytest.mark.parametrize("G", [1, 3])
@pytest.mark.parametrize("name", list(CASES))
def test_panels_match_full_step(oracle, name, G):
    pts, k, kind, g, c, p, seed = CASES[name]
    X = pts()
    n = X.shape[0]
    cl = datagen.random_init(n, k, seed)
    print(f"[gpu] panels {name} n={n} k={k} G={G}", flush=True)
    kern = oracle.Kernel(kind, g, c, p)
    Kref = kern.matrix(X)
    ref = oracle.step_full(Kref, cl, k)
    out = run_panels(X, kind, g, c, p, cl, k, G, k_rows=np.arange(n))
    eK = rowscaled_err(out["K"], Kref)
    np.testing.assert_array_equal(out["counts"], ref["counts"])
    eE = rowscaled_err(out["E"], ref["E"])
    ez = rel_err(out["z"], ref["z"])
    assert eK <= TOL and eE <= TOL and ez <= TOL, (eK, eE, ez)
    flips = assignment_mismatches(out["cl"], ref["cl"], ref["D"])
    np.testing.assert_array_equal(out["took"], np.bincount(out["cl"], minlength=k))
    print(f"[gpu] panels {name} G={out['npanels']}: K {eK:.2e} E {eE:.2e} z {ez:.2e} flips {flips}", flush=True)


def test_panel_errors(oracle):
    torch = pytest.importorskip("torch")
    from paper_2601_17136_amd import kkm
    X = datagen.make_points(2, n=500, d=8)[0]
    Xd = torch.from_numpy(X).cuda()
    ctx = kkm.kkm_create(kkm.current_stream_handle())
    try:
        prm = kkm.make_params(0.5, 0.0, 1, kkm.KKM_MODE_RESIDENT)
        for c0, c1 in [(100, 300), (0, 0), (256, 128), (0, 501), (-128, 100)]:
            with pytest.raises(kkm.KKMError) as e:
                kkm.kkm_build_panel(ctx, Xd, 500, 8, kkm.KINDS["gauss"], prm, c0, c1)
            assert e.value.code == kkm.KKM_ERR_ARG
        with pytest.raises(kkm.KKMError) as e:
            kkm.kkm_build_panel(ctx, Xd, 500, 8, kkm.KINDS["gauss"],
                                kkm.make_params(0.5, 0.0, 1, kkm.KKM_MODE_RESIDENT, kkm.KKM_STORE_F16), 0, 256)
        assert e.value.code == kkm.KKM_ERR_ARG
        kkm.kkm_build_panel(ctx, Xd, 500, 8, kkm.KINDS["gauss"], prm, 128, 384)
        cl = torch.zeros(500, dtype=torch.int32, device="cuda")
        out = torch.empty(256, dtype=torch.int32, device="cuda")
        with pytest.raises(kkm.KKMError) as e:  # assign before the SpMM
            kkm.kkm_panel_assign(ctx, 3, np.zeros(3), out)
        assert e.value.code == kkm.KKM_ERR_STATE
        with pytest.raises(kkm.KKMError) as e:  # the full-K calls refuse a panel
            kkm.kkm_iterate(ctx, cl, 3, 1)
        assert e.value.code == kkm.KKM_ERR_STATE
        bad = torch.full((500,), 7, dtype=torch.int32, device="cuda")
        with pytest.raises(kkm.KKMError) as e:
            kkm.kkm_panel_spmm(ctx, bad, 3)
        assert e.value.code == kkm.KKM_ERR_DEVICE_DATA
    finally:
        kkm.kkm_destroy(ctx)


def test_panels_workload5_shape(oracle):
    """n = 200,000 over G = 8: each panel is one GPU's share at its real shape."""
    torch = pytest.importorskip("torch")
    assert torch.cuda.is_available()
    w, X, cl = datagen.workload(5)
    n, k = w.n, w.k
    G = 8
    print(f"[gpu] panels at {w.describe()}, G={G}", flush=True)
    kern = oracle.Kernel(w.kind, w.gamma, w.coef0, w.degree)
    rng = np.random.default_rng(5)
    fixed = [0, 1, 127, 128, 24999, 25000, 25087, 25088, n // 2, n - 2, n - 1]
    rows = np.unique(np.concatenate([fixed, rng.choice(n, size=37, replace=False)]).astype(np.int64))
    out = run_panels(X, w.kind, w.gamma, w.coef0, w.degree, cl, k, G, k_rows=rows)
    print(f"[gpu] panels built and stepped", flush=True)
    ref = oracle.step_rows(kern, X, cl, k, rows)
    eK = rowscaled_err(out["K"], ref["K_rows"])
    np.testing.assert_array_equal(out["counts"], ref["counts"])
    eE = rowscaled_err(out["E"][rows], ref["E"])
    ez = rel_err(out["z"], ref["z"])
    assert eK <= TOL and eE <= TOL and ez <= TOL, (eK, eE, ez)
    flips = assignment_mismatches(out["cl"][rows], ref["cl"], ref["D"])
    np.testing.assert_array_equal(out["took"], np.bincount(out["cl"], minlength=k))
    print(f"[gpu] panels cfg 5: K {eK:.2e} E {eE:.2e} z {ez:.2e} flips {flips}", flush=True)


def test_panels_rebuilt_on_one_context(oracle):
    """All G panels of equal width built one after another on ONE context, so
    every rebuild after the first keeps the buffers of the first: the panel's
    column offset must still reach the self-term parts (ids of its own points)
    and the assignment (diag K of its own points).  A polynomial kernel makes
    diag K differ from point to point."""
    import torch

    from paper_2601_17136_amd import kkm
    n, d, k, G = 768, 11, 5, 3                 # three panels of 256 points
    X = datagen.separated_blobs(n, d, k, seed=8, spread=2.0, sigma=1.0)[0]
    cl = datagen.random_init(n, k, 35)
    kern = oracle.Kernel("poly", 0.3, 1.0, 2)
    ref = oracle.step_full(kern.matrix(X), cl, k)
    Xd = torch.from_numpy(X).cuda()
    cl_d = torch.from_numpy(cl).cuda()
    params = kkm.make_params(0.3, 1.0, 2, kkm.KKM_MODE_RESIDENT)
    bounds = panel_bounds(n, G)
    assert len({c1 - c0 for c0, c1 in bounds}) == 1
    ctx = kkm.kkm_create(kkm.current_stream_handle())
    try:
        zsum = np.zeros(k)
        for c0, c1 in bounds:
            kkm.kkm_build_panel(ctx, Xd, n, d, kkm.KKM_POLY, params, c0, c1)
            zpart, counts = kkm.kkm_panel_spmm(ctx, cl_d, k)
            zsum += zpart
        c = counts.astype(np.float64)
        z = np.where(counts > 0, zsum / np.where(counts > 0, c * c, 1.0), 0.0)
        new = np.empty(n, dtype=np.int32)
        E = np.empty((n, k), dtype=np.float32)
        for c0, c1 in bounds:
            kkm.kkm_build_panel(ctx, Xd, n, d, kkm.KKM_POLY, params, c0, c1)
            kkm.kkm_panel_spmm(ctx, cl_d, k)
            out = torch.empty(c1 - c0, dtype=torch.int32, device="cuda")
            Eo = torch.empty((c1 - c0, k), device="cuda")
            kkm.kkm_panel_assign(ctx, k, z, out, Eo)
            new[c0:c1] = out.cpu().numpy()
            E[c0:c1] = Eo.cpu().numpy()
    finally:
        kkm.kkm_destroy(ctx)
    np.testing.assert_array_equal(counts, ref["counts"])
    assert rel_err(z, ref["z"]) <= TOL
    assert rowscaled_err(E, ref["E"]) <= TOL
    flips = assignment_mismatches(new, ref["cl"], ref["D"])
    print(f"[gpu] panels rebuilt on one context: {flips} near-tie flips", flush=True)
