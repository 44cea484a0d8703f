"""Helpers shared by the GPU parity tests (engine setup and comparisons)."""
from __future__ import annotations

import numpy as np

# Tolerance of the parity bar: |gpu - ref| <= TOL * max_l |ref(i, l)| per row for
# K, E and D (row-scaled: an entry near zero inside a row of large entries is
# held to the row's scale), relative error for J and z.
TOL = 1e-4
# Near-tie band for assignments: a differing id must be within this
# (row-scaled) distance of the oracle's minimum.
TIE = 2e-4


def rowscaled_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(gpu)), "infinite entries differ"
    assert np.array_equal(gpu[~fin], ref[~fin]), "infinite entries differ in sign"
    if not fin.any():
        return 0.0
    a = np.where(fin, np.abs(ref), 0.0)
    scale = a.max(axis=1, keepdims=True)
    scale[scale == 0] = 1.0
    err = np.abs(np.where(fin, gpu, 0.0) - np.where(fin, ref, 0.0)) / scale
    return float(err.max())


def rel_err(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.max(np.abs(a - b) / np.maximum(np.abs(b).max(), 1e-300)))


def assignment_mismatches(cl_gpu, cl_ref, D_ref, tie=TIE) -> int:
    """Count differing ids; fail if any difference is not a near-tie of the oracle's D."""
    cl_gpu = np.asarray(cl_gpu)
    cl_ref = np.asarray(cl_ref)
    bad = np.nonzero(cl_gpu != cl_ref)[0]
    for i in bad:
        row = D_ref[i]
        scale = np.abs(row[np.isfinite(row)]).max()
        gap = row[cl_gpu[i]] - row[cl_ref[i]]
        assert np.isfinite(row[cl_gpu[i]]) and gap <= tie * scale, \
            f"point {i}: gpu id {cl_gpu[i]} vs oracle {cl_ref[i]}, gap {gap:.3e} (scale {scale:.3e})"
    return int(bad.size)


class Engine:
    """A context with a built kernel matrix on torch's current stream."""

    def __init__(self, X: np.ndarray, kind: str, gamma=1.0, coef0=0.0, degree=1, mode="resident",
                 mem_budget=0, storage="f32", k_hint=0):
        import torch

        from paper_2601_17136_amd import kkm
        self.kkm = kkm
        self.n, self.d = X.shape
        self.X = torch.from_numpy(np.ascontiguousarray(X, dtype=np.float32)).cuda()
        self.ctx = kkm.kkm_create(kkm.current_stream_handle(), mem_budget)
        kkm.kkm_build_kernel(self.ctx, self.X, self.n, self.d, kkm.KINDS[kind],
                             kkm.make_params(gamma, coef0, degree, kkm.MODES[mode], kkm.STORAGES[storage],
                                             k_hint))

    def K_rows(self, r0=0, r1=None):
        import torch
        r1 = self.n if r1 is None else r1
        out = torch.empty((r1 - r0, self.n), device="cuda")
        self.kkm.kkm_copy_kernel_rows(self.ctx, r0, r1, out)
        return out.cpu().numpy()

    def diag(self):
        import torch
        out = torch.empty(self.n, device="cuda")
        self.kkm.kkm_copy_diag(self.ctx, out)
        return out.cpu().numpy()

    def step(self, cl: np.ndarray, k: int, want_E=True, want_D=True):
        import torch
        n = self.n
        cl_d = torch.from_numpy(np.ascontiguousarray(cl, dtype=np.int32)).cuda()
        E = torch.empty((n, k), device="cuda") if want_E else None
        D = torch.empty((n, k), device="cuda") if want_D else None
        z = torch.empty(k, device="cuda")
        nxt = torch.empty(n, dtype=torch.int32, device="cuda")
        cnt = torch.empty(k, dtype=torch.int32, device="cuda")
        J = self.kkm.kkm_step(self.ctx, cl_d, k, E=E, z=z, D=D, cl_out=nxt, counts_out=cnt)
        out = dict(z=z.cpu().numpy(), cl=nxt.cpu().numpy(), counts=cnt.cpu().numpy(), J=J)
        if want_E:
            out["E"] = E.cpu().numpy()
        if want_D:
            out["D"] = D.cpu().numpy()
        return out

    def iterate(self, cl0: np.ndarray, k: int, max_iter: int, tol=-1.0):
        import torch
        V = torch.from_numpy(np.ascontiguousarray(cl0, dtype=np.int32)).cuda()
        it, hist = self.kkm.kkm_iterate(self.ctx, V, k, max_iter, tol)
        return V.cpu().numpy(), it, hist

    def seed(self, k: int, u):
        """K-means++ seeding: (centers, initial ids) as numpy arrays."""
        import torch
        V = torch.full((self.n,), -1, dtype=torch.int32, device="cuda")
        centers = self.kkm.kkm_init_kmeanspp(self.ctx, k, u, V)
        return centers, V.cpu().numpy()

    def info(self):
        return self.kkm.kkm_get_info(self.ctx)

    def close(self):
        if self.ctx is not None:
            self.kkm.kkm_destroy(self.ctx)
            self.ctx = None

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()
