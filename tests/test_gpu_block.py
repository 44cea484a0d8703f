"""GPU parity for one GPU's share of the 1.5D split (kkm_build_block,
kkm_block_spmm, kkm_block_zpart, kkm_block_assign): a q x q grid of blocks of
K (P = q^2 processes), each built and stepped on a context of its own, with
the exchanges a multi-GPU run would make done here on the host: the
row-block ids handed to each block, the column sums of the partial E split
into the q pieces of each column block (the reduce-scatter), and the sums of
the pieces' self-term parts and sizes (the all-reduce).

Small problems against the full oracle step: K assembled from the blocks,
every block's partial E against the oracle's partial sums, E, z, the sizes
and the new ids (exact except at the oracle's near-ties).  At workload 5's
shape (n = 200,000 over P = 64: blocks of 25,000 x 25,000 points, 2.5 GB
each) the 64 shares run one after another on one context, checked on
sampled points against the oracle's sampled-row step.
"""
import numpy as np
import pytest

from gpu_helpers import TOL, assignment_mismatches, rel_err, rowscaled_err
from paper_2601_17136_amd import datagen

pytestmark = pytest.mark.gpu


def block_bounds(n, q):
    """q contiguous point ranges, each starting at a multiple of 128 (empty ones dropped)."""
    b = [(g * n // q) // 128 * 128 for g in range(q)] + [n]
    return [(b[g], b[g + 1]) for g in range(q) if b[g + 1] > b[g]]


def pieces(lo, hi, q):
    """[lo, hi) cut into q contiguous pieces (the 1D partition inside a column block)."""
    b = [lo + (hi - lo) * l // q for l in range(q + 1)]
    return [(b[l], b[l + 1]) for l in range(q)]


def params(kkm, gamma, coef0, degree):
    return kkm.make_params(gamma, coef0, degree, kkm.KKM_MODE_RESIDENT)


def partial_err(oracle, part, Kb, cl_rows, k, E_full):
    """A block's partial E against the oracle's, each row held to the scale of
    the full row of E it sums into (or its own, if larger): K's entries are
    accurate to their row's scale, not to a block's share of it."""
    ref = oracle.one_hot_product(np.ascontiguousarray(Kb.T), cl_rows, k)
    scale = np.maximum(np.abs(E_full).max(axis=1), np.abs(ref).max(axis=1))[:, None]
    return float((np.abs(part - ref) / scale).max())


def run_grid(X, kind, gamma, coef0, degree, cl, k, q, oracle=None, Kref=None, Eref=None):
    """One update from ids cl over a q x q grid of blocks; returns the assembled outputs."""
    import torch

    from paper_2601_17136_amd import kkm
    n, d = X.shape
    Xd = torch.from_numpy(np.ascontiguousarray(X, dtype=np.float32)).cuda()
    cl_d = torch.from_numpy(np.ascontiguousarray(cl, dtype=np.int32)).cuda()
    blocks = block_bounds(n, q)
    nb = len(blocks)
    ctx = {}
    try:
        for i, (r0, r1) in enumerate(blocks):
            for j, (c0, c1) in enumerate(blocks):
                ctx[i, j] = kkm.kkm_create(kkm.current_stream_handle())
                kkm.kkm_build_block(ctx[i, j], Xd, n, d, kkm.KINDS[kind], params(kkm, gamma, coef0, degree),
                                    r0, r1, c0, c1)
        K = np.empty((n, n), dtype=np.float32)
        E = np.zeros((n, k), dtype=np.float32)
        part_err = 0.0
        for j, (c0, c1) in enumerate(blocks):
            for i, (r0, r1) in enumerate(blocks):  # process (i, j): its block's partial E
                out = torch.empty((r1 - r0, c1 - c0), device="cuda")
                kkm.kkm_copy_kernel_rows(ctx[i, j], r0, r1, out)
                K[r0:r1, c0:c1] = out.cpu().numpy()
                part = torch.empty((c1 - c0, k), device="cuda")
                kkm.kkm_block_spmm(ctx[i, j], cl_d[r0:r1], k, part)
                part = part.cpu().numpy()
                E[c0:c1] += part  # the reduce over grid column j, in row order
                if Kref is not None:
                    part_err = max(part_err, partial_err(oracle, part, Kref[r0:r1, c0:c1], cl[r0:r1], k,
                                                         Eref[c0:c1]))
        zsum = np.zeros(k)
        counts = np.zeros(k, dtype=np.int64)
        owner = []
        for j, (c0, c1) in enumerate(blocks):  # the scatter: piece l of column block j to process (l, j)
            for l, (a0, a1) in enumerate(pieces(c0, c1, nb)):
                if a1 > a0:
                    Ep = torch.from_numpy(E[a0:a1]).cuda()
                    zp, cnt = kkm.kkm_block_zpart(ctx[l, j], Ep, cl_d[a0:a1], a0, a1, k)
                    zsum += zp
                    counts += cnt
                    owner.append((l, j, a0, a1, Ep))
        np.testing.assert_array_equal(counts, np.bincount(cl, minlength=k))
        c = counts.astype(np.float64)
        z = np.where(counts > 0, zsum / np.where(counts > 0, c * c, 1.0), 0.0)
        new = np.full(n, -1, dtype=np.int32)
        took = np.zeros(k, dtype=np.int64)
        for l, j, a0, a1, Ep in owner:  # every process assigns its own piece
            out = torch.empty(a1 - a0, dtype=torch.int32, device="cuda")
            took += kkm.kkm_block_assign(ctx[l, j], Ep, a0, a1, k, z, counts.astype(np.int32), out)
            new[a0:a1] = out.cpu().numpy()
        assert (new >= 0).all()
        return dict(K=K, E=E, z=z, counts=counts, cl=new, took=took, part_err=part_err, nb=nb)
    finally:
        for cx in ctx.values():
            kkm.kkm_destroy(cx)


CASES = {
    # name: (points, k, kind, gamma, coef0, degree, init seed)
    "ragged-gauss": (lambda: datagen.make_points(2, n=777, d=37)[0], 9, "gauss", 0.3, 0.0, 1, 41),
    "blobs-poly": (lambda: datagen.make_points(1)[0], 8, "poly", 1.0, 1.0, 2, 42),
    # Gaussian entries the epilogue flags and the fix-up recomputes
    "rings-gauss": (lambda: datagen.make_points(4, n=2600)[0], 40, "gauss", 0.5, 0.0, 1, 43),
    "linear-n300": (lambda: datagen.separated_blobs(300, 3, 4, seed=4, spread=3.0, sigma=1.0)[0],
                    4, "linear", 1.0, 0.0, 1, 44),
}


@pytest.mark.parametrize("q", [2, 3])
@pytest.mark.parametrize("name", list(CASES))
def test_grid_matches_full_step(oracle, name, q):
    pts, k, kind, g, c, p, seed = CASES[name]
    X = pts()
    n = X.shape[0]
    cl = datagen.random_init(n, k, seed)
    print(f"[gpu] 1.5D grid {name} n={n} k={k} q={q}", flush=True)
    kern = oracle.Kernel(kind, g, c, p)
    Kref = kern.matrix(X)
    ref = oracle.step_full(Kref, cl, k)
    out = run_grid(X, kind, g, c, p, cl, k, q, oracle=oracle, Kref=Kref, Eref=ref["E"])
    eK = rowscaled_err(out["K"], Kref)
    np.testing.assert_array_equal(out["counts"], ref["counts"])
    eE = rowscaled_err(out["E"], ref["E"])
    ez = rel_err(out["z"], ref["z"])
    assert eK <= TOL and eE <= TOL and ez <= TOL and out["part_err"] <= TOL, (eK, eE, ez, out["part_err"])
    flips = assignment_mismatches(out["cl"], ref["cl"], ref["D"])
    np.testing.assert_array_equal(out["took"], np.bincount(out["cl"], minlength=k))
    print(f"[gpu] 1.5D grid {name} {out['nb']}x{out['nb']}: K {eK:.2e} partial E {out['part_err']:.2e} "
          f"E {eE:.2e} z {ez:.2e} flips {flips}", flush=True)


def test_block_errors(oracle):
    torch = pytest.importorskip("torch")
    from paper_2601_17136_amd import kkm
    X = datagen.make_points(2, n=500, d=8)[0]
    Xd = torch.from_numpy(X).cuda()
    ctx = kkm.kkm_create(kkm.current_stream_handle())
    G = kkm.KINDS["gauss"]
    try:
        prm = params(kkm, 0.5, 0.0, 1)
        for r0, r1, c0, c1 in [(100, 300, 0, 128), (0, 128, 100, 300), (0, 0, 0, 128), (256, 128, 0, 128),
                               (0, 501, 0, 128), (-128, 100, 0, 128), (0, 128, 0, 501)]:
            with pytest.raises(kkm.KKMError) as e:
                kkm.kkm_build_block(ctx, Xd, 500, 8, G, prm, r0, r1, c0, c1)
            assert e.value.code == kkm.KKM_ERR_ARG, (r0, r1, c0, c1)
        with pytest.raises(kkm.KKMError) as e:
            kkm.kkm_build_block(ctx, Xd, 500, 8, G,
                                kkm.make_params(0.5, 0.0, 1, kkm.KKM_MODE_RESIDENT, kkm.KKM_STORE_F16),
                                0, 128, 0, 128)
        assert e.value.code == kkm.KKM_ERR_ARG
        # a block or panel wider than the K build's 32-bit store offsets allow
        # is refused before anything runs (X is not read, so a small buffer
        # stands in for the 9M points)
        import ctypes
        L = kkm.lib()
        for c1 in (8_388_480 + 1, 8_400_000):
            assert L.kkm_build_block(ctx, Xd.data_ptr(), 9_000_000, 8, G, ctypes.byref(prm),
                                     0, 128, 0, c1) == kkm.KKM_ERR_ARG
            assert L.kkm_build_panel(ctx, Xd.data_ptr(), 9_000_000, 8, G, ctypes.byref(prm),
                                     0, c1) == kkm.KKM_ERR_ARG
        kkm.kkm_build_block(ctx, Xd, 500, 8, G, prm, 128, 384, 256, 500)
        info = kkm.kkm_get_info(ctx)
        assert (info["r0"], info["r1"], info["c0"], info["c1"]) == (128, 384, 256, 500)
        rows = torch.zeros(256, dtype=torch.int32, device="cuda")
        E = torch.empty((244, 3), device="cuda")
        cl = torch.empty(500, dtype=torch.int32, device="cuda")
        with pytest.raises(kkm.KKMError) as e:  # the full-K and panel calls refuse a block
            kkm.kkm_iterate(ctx, cl, 3, 1)
        assert e.value.code == kkm.KKM_ERR_STATE
        with pytest.raises(kkm.KKMError) as e:
            kkm.kkm_panel_spmm(ctx, torch.zeros(256, dtype=torch.int32, device="cuda"), 3)
        assert e.value.code == kkm.KKM_ERR_STATE
        with pytest.raises(ValueError):  # the binding checks lengths against the stored block
            kkm.kkm_block_spmm(ctx, cl, 3, E)
        with pytest.raises(ValueError):
            kkm.kkm_block_spmm(ctx, rows, 3, torch.empty((244, 2), device="cuda"))
        bad = torch.full((256,), 3, dtype=torch.int32, device="cuda")
        with pytest.raises(kkm.KKMError) as e:
            kkm.kkm_block_spmm(ctx, bad, 3, E)
        assert e.value.code == kkm.KKM_ERR_DEVICE_DATA
        kkm.kkm_block_spmm(ctx, rows, 3, E)
        ids = torch.zeros(100, dtype=torch.int32, device="cuda")
        Ep = torch.zeros((100, 3), device="cuda")
        for a0, a1 in [(128, 228), (450, 550), (300, 300)]:  # pieces outside [256, 500) or empty
            with pytest.raises((kkm.KKMError, ValueError)) as e:
                kkm.kkm_block_zpart(ctx, Ep, ids, a0, a1, 3)
            if e.type is kkm.KKMError:
                assert e.value.code == kkm.KKM_ERR_ARG
        with pytest.raises(kkm.KKMError) as e:
            kkm.kkm_block_zpart(ctx, Ep, torch.full((100,), -1, dtype=torch.int32, device="cuda"), 300, 400, 3)
        assert e.value.code == kkm.KKM_ERR_DEVICE_DATA
        zp, cnt = kkm.kkm_block_zpart(ctx, Ep, ids, 300, 400, 3)
        assert cnt.tolist() == [100, 0, 0] and zp.tolist() == [0.0, 0.0, 0.0]
        out = torch.empty(100, dtype=torch.int32, device="cuda")
        with pytest.raises(kkm.KKMError) as e:
            kkm.kkm_block_assign(ctx, Ep, 300, 400, 3, np.zeros(3), np.array([1, -1, 0]), out)
        assert e.value.code == kkm.KKM_ERR_ARG
        took = kkm.kkm_block_assign(ctx, Ep, 300, 400, 3, np.zeros(3), np.array([0, 5, 5]), out)
        assert took.tolist() == [0, 100, 0]  # cluster 0 is empty; 1 and 2 tie, the lower wins
        with pytest.raises(kkm.KKMError) as e:  # rows outside the block
            kkm.kkm_copy_kernel_rows(ctx, 0, 1, torch.empty(244, device="cuda"))
        assert e.value.code == kkm.KKM_ERR_ARG
    finally:
        kkm.kkm_destroy(ctx)


def test_grid_workload5_shape(oracle):
    """n = 200,000 over P = 64 (q = 8): the 64 shares at their real shape, one after another."""
    torch = pytest.importorskip("torch")
    from paper_2601_17136_amd import kkm
    w, X, cl = datagen.workload(5)
    n, d, k = w.n, X.shape[1], w.k
    q = 8
    print(f"[gpu] 1.5D grid at {w.describe()}, q={q}", flush=True)
    kern = oracle.Kernel(w.kind, w.gamma, w.coef0, w.degree)
    rng = np.random.default_rng(6)
    blocks = block_bounds(n, q)
    edges = [b for r in blocks for b in (r[0], r[1] - 1)]
    rows = np.unique(np.concatenate([edges, rng.choice(n, size=29, replace=False)]).astype(np.int64))
    Xd = torch.from_numpy(np.ascontiguousarray(X, dtype=np.float32)).cuda()
    cl_d = torch.from_numpy(np.ascontiguousarray(cl, dtype=np.int32)).cuda()
    prm = params(kkm, w.gamma, w.coef0, w.degree)
    E = np.zeros((n, k), dtype=np.float32)
    K_rows = np.empty((rows.size, n), dtype=np.float32)
    ctx = kkm.kkm_create(kkm.current_stream_handle())
    try:
        part = None
        for j, (c0, c1) in enumerate(blocks):
            for i, (r0, r1) in enumerate(blocks):
                kkm.kkm_build_block(ctx, Xd, n, d, kkm.KINDS[w.kind], prm, r0, r1, c0, c1)
                if part is None or part.shape[0] != c1 - c0:
                    part = torch.empty((c1 - c0, k), device="cuda")
                kkm.kkm_block_spmm(ctx, cl_d[r0:r1], k, part)
                E[c0:c1] += part.cpu().numpy()
                for t in np.nonzero((rows >= r0) & (rows < r1))[0]:
                    out = torch.empty(c1 - c0, device="cuda")
                    kkm.kkm_copy_kernel_rows(ctx, int(rows[t]), int(rows[t]) + 1, out)
                    K_rows[t, c0:c1] = out.cpu().numpy()
            print(f"[gpu] column block {j} done", flush=True)
        # the pieces of column block j, on a context holding a block of that
        # column (each of the q processes of grid column j holds one)
        zsum = np.zeros(k)
        counts = np.zeros(k, dtype=np.int64)
        for j, (c0, c1) in enumerate(blocks):
            kkm.kkm_build_block(ctx, Xd, n, d, kkm.KINDS[w.kind], prm, *blocks[j], c0, c1)
            for a0, a1 in pieces(c0, c1, q):
                zp, cnt = kkm.kkm_block_zpart(ctx, torch.from_numpy(E[a0:a1]).cuda(), cl_d[a0:a1], a0, a1, k)
                zsum += zp
                counts += cnt
        c = counts.astype(np.float64)
        z = np.where(counts > 0, zsum / np.where(counts > 0, c * c, 1.0), 0.0)
        new = np.full(n, -1, dtype=np.int32)
        for j, (c0, c1) in enumerate(blocks):
            kkm.kkm_build_block(ctx, Xd, n, d, kkm.KINDS[w.kind], prm, *blocks[j], c0, c1)
            for a0, a1 in pieces(c0, c1, q):
                out = torch.empty(a1 - a0, dtype=torch.int32, device="cuda")
                kkm.kkm_block_assign(ctx, torch.from_numpy(E[a0:a1]).cuda(), a0, a1, k, z,
                                     counts.astype(np.int32), out)
                new[a0:a1] = out.cpu().numpy()
    finally:
        kkm.kkm_destroy(ctx)
    print("[gpu] 64 shares built and stepped", flush=True)
    ref = oracle.step_rows(kern, X, cl, k, rows)
    eK = rowscaled_err(K_rows, ref["K_rows"])
    np.testing.assert_array_equal(counts, ref["counts"])
    eE = rowscaled_err(E[rows], ref["E"])
    ez = rel_err(z, ref["z"])
    assert eK <= TOL and eE <= TOL and ez <= TOL, (eK, eE, ez)
    assert (new >= 0).all()
    flips = assignment_mismatches(new[rows], ref["cl"], ref["D"])
    print(f"[gpu] 1.5D grid cfg 5: K {eK:.2e} E {eE:.2e} z {ez:.2e} flips {flips}", flush=True)
