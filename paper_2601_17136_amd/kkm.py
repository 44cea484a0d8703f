"""Thin ctypes binding to libkkm.so: the C ABI of include/kkm.h under the same names.

Only argument marshalling happens here: device tensors become raw pointers
(after dtype/device/contiguity checks), host results come back as Python
values, and a non-zero status raises KKMError with the library's message.
Every step of the computation runs in the library's HIP kernels.  If the
library has not been built, loading it fails loudly; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkkm.so")

KKM_OK, KKM_ERR_ARG, KKM_ERR_OOM, KKM_ERR_HIP, KKM_ERR_STATE, KKM_ERR_DEVICE_DATA = 0, -1, -2, -3, -4, -5
KKM_LINEAR, KKM_POLY, KKM_GAUSS = 0, 1, 2
KKM_MODE_AUTO, KKM_MODE_RESIDENT, KKM_MODE_ONTHEFLY, KKM_MODE_PACKED = 0, 1, 2, 3
KKM_STORE_F32, KKM_STORE_F16 = 0, 1
STORAGES = {"f32": KKM_STORE_F32, "f16": KKM_STORE_F16}
KKM_MAX_K = 1024
KKM_PACKED_MAX_K = 64
KKM_PACKED_FAST_K = 64
KKM_ABI_VERSION = 8
KKM_NOALLOC_SCRATCH_BYTES = 64 << 20
PHASES = ("stage", "gemm", "fixup", "labels", "scatter", "spmm", "assign", "onthefly", "reduce", "other",
          "seed")
KINDS = {"linear": KKM_LINEAR, "poly": KKM_POLY, "gauss": KKM_GAUSS}
MODES = {"auto": KKM_MODE_AUTO, "resident": KKM_MODE_RESIDENT, "onthefly": KKM_MODE_ONTHEFLY,
         "packed": KKM_MODE_PACKED}


class KKMError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"kkm error {code}: {msg}")
        self.code = code


class kkm_params(ctypes.Structure):
    _fields_ = [("gamma", ctypes.c_float), ("coef0", ctypes.c_float),
                ("degree", ctypes.c_int32), ("mode", ctypes.c_int32), ("storage", ctypes.c_int32),
                ("k_hint", ctypes.c_int32)]


class kkm_timing(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * len(PHASES)), ("launches", ctypes.c_int64 * len(PHASES))]


class kkm_info(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("d", ctypes.c_int32), ("d_pad", ctypes.c_int32),
                ("kind", ctypes.c_int32), ("mode", ctypes.c_int32), ("storage", ctypes.c_int32),
                ("ld", ctypes.c_int64),
                ("bytes_K", ctypes.c_size_t), ("bytes_total", ctypes.c_size_t),
                ("fixups", ctypes.c_int64), ("fixup_capacity", ctypes.c_int64),
                ("r0", ctypes.c_int64), ("r1", ctypes.c_int64), ("c0", ctypes.c_int64), ("c1", ctypes.c_int64)]


_lib = None
_vp, _i32, _i64, _f64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_size_t
_SIGS = {
    "kkm_abi_version": ([], _i32),
    "kkm_last_error": ([_vp], ctypes.c_char_p),
    "kkm_last_warning": ([_vp], ctypes.c_char_p),
    "kkm_create": ([ctypes.POINTER(_vp), _vp, _sz], _i32),
    "kkm_destroy": ([_vp], _i32),
    "kkm_plan": ([_i64, _i32, _i32, _i32, _sz, _i32, _i32, ctypes.POINTER(_i32), ctypes.POINTER(_sz)], _i32),
    "kkm_check_build_args": ([_i64, _i32, _i32, ctypes.POINTER(kkm_params)], _i32),
    "kkm_check_iterate_args": ([_i64, _i32, _i32], _i32),
    "kkm_build_kernel": ([_vp, _vp, _i64, _i32, _i32, ctypes.POINTER(kkm_params)], _i32),
    "kkm_iterate": ([_vp, _vp, _i32, _i32, _f64, ctypes.POINTER(_i32), _vp], _i32),
    "kkm_iterate_noalloc": ([_vp, _vp, _i32, _i32, _f64, ctypes.POINTER(_i32), _vp], _i32),
    "kkm_objective": ([_vp, _vp, _i32, ctypes.POINTER(_f64)], _i32),
    "kkm_step": ([_vp, _vp, _i32, _vp, _vp, _vp, _vp, _vp, ctypes.POINTER(_f64)], _i32),
    "kkm_init_kmeanspp": ([_vp, _i32, _vp, _vp, _vp], _i32),
    "kkm_build_panel": ([_vp, _vp, _i64, _i32, _i32, ctypes.POINTER(kkm_params), _i64, _i64], _i32),
    "kkm_panel_spmm": ([_vp, _vp, _i32, _vp, _vp], _i32),
    "kkm_panel_assign": ([_vp, _i32, _vp, _vp, _vp, _vp], _i32),
    "kkm_build_block": ([_vp, _vp, _i64, _i32, _i32, ctypes.POINTER(kkm_params), _i64, _i64, _i64, _i64], _i32),
    "kkm_block_spmm": ([_vp, _vp, _i32, _vp], _i32),
    "kkm_block_zpart": ([_vp, _vp, _vp, _i64, _i64, _i32, _vp, _vp], _i32),
    "kkm_block_assign": ([_vp, _vp, _i64, _i64, _i32, _vp, _vp, _vp, _vp], _i32),
    "kkm_copy_kernel_rows": ([_vp, _i64, _i64, _vp], _i32),
    "kkm_copy_diag": ([_vp, _vp], _i32),
    "kkm_set_timing": ([_vp, _i32], _i32),
    "kkm_peak_read": ([_vp, _vp, _sz, _vp, _i32, ctypes.POINTER(ctypes.c_float)], _i32),
    "kkm_peak_read_rows": ([_vp, _vp, ctypes.c_int64, ctypes.c_int64, _vp, _i32, _i32, _vp, _i32,
                            ctypes.POINTER(ctypes.c_float)], _i32),
    "kkm_peak_write": ([_vp, _vp, _sz, ctypes.c_float, _i32, ctypes.POINTER(ctypes.c_float)], _i32),
    "kkm_peak_mfma": ([_vp, _i32, _vp, _i32, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(_f64)], _i32),
    "kkm_get_timing": ([_vp, ctypes.POINTER(kkm_timing)], _i32),
    "kkm_get_info": ([_vp, ctypes.POINTER(kkm_info)], _i32),
}


def lib():
    """Load libkkm.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python __graft_entry__.py build` "
                               "(hipcc --offload-arch=gfx950); the engine has no fallback")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            f = getattr(L, name)
            f.argtypes, f.restype = args, res
        if L.kkm_abi_version() != KKM_ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} has ABI {L.kkm_abi_version()}, this binding {KKM_ABI_VERSION}: "
                               "rebuild it with `python __graft_entry__.py build`")
        _lib = L
    return _lib


def _check(rc: int, ctx=None):
    if rc != KKM_OK:
        msg = lib().kkm_last_error(ctx)
        raise KKMError(rc, msg.decode() if msg else "")


def _dev_ptr(t, dtype, name, numel=None):
    """Raw device address of a contiguous CUDA/HIP tensor, with its checks."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} must have {numel} elements, got {t.numel()}")
    return t.data_ptr()


def current_stream_handle():
    """hipStream_t of torch's current stream on the current device."""
    import torch
    return torch.cuda.current_stream().cuda_stream


# ------------------------------------------------------------------ the C ABI

def kkm_abi_version() -> int:
    return lib().kkm_abi_version()


def kkm_last_error(ctx=None) -> str:
    m = lib().kkm_last_error(ctx)
    return m.decode() if m else ""


def kkm_create(stream=None, mem_budget: int = 0):
    ctx = _vp()
    _check(lib().kkm_create(ctypes.byref(ctx), stream, int(mem_budget)))
    return ctx


def kkm_destroy(ctx) -> None:
    _check(lib().kkm_destroy(ctx))


def kkm_plan(n: int, d: int, k: int, kind: int, mem_budget: int, mode: int = KKM_MODE_AUTO,
             storage: int = KKM_STORE_F32):
    """(resolved mode, device bytes); raises KKMError(KKM_ERR_OOM) if it cannot fit."""
    m, b = _i32(), _sz()
    _check(lib().kkm_plan(int(n), int(d), int(k), int(kind), int(mem_budget), int(mode), int(storage),
                          ctypes.byref(m), ctypes.byref(b)))
    return m.value, b.value


def make_params(gamma=1.0, coef0=0.0, degree=1, mode=KKM_MODE_AUTO, storage=KKM_STORE_F32,
                k_hint=0) -> kkm_params:
    return kkm_params(float(gamma), float(coef0), int(degree), int(mode), int(storage), int(k_hint))


def kkm_last_warning(ctx=None) -> str:
    m = lib().kkm_last_warning(ctx)
    return m.decode() if m else ""


def _warn_if_any(ctx):
    msg = kkm_last_warning(ctx)
    if msg:
        import warnings
        warnings.warn(msg, RuntimeWarning, stacklevel=3)


def kkm_check_build_args(n, d, kind, params: kkm_params) -> int:
    return lib().kkm_check_build_args(int(n), int(d), int(kind), ctypes.byref(params))


def kkm_check_iterate_args(n, k, max_iter) -> int:
    return lib().kkm_check_iterate_args(int(n), int(k), int(max_iter))


def kkm_build_kernel(ctx, X, n: int, d: int, kind: int, params: kkm_params) -> None:
    import torch
    _check(lib().kkm_build_kernel(ctx, _dev_ptr(X, torch.float32, "X", int(n) * int(d)), int(n), int(d),
                                  int(kind), ctypes.byref(params)), ctx)
    _warn_if_any(ctx)


def kkm_iterate(ctx, V, k: int, max_iter: int, tol: float = -1.0):
    """Returns (iters_done, obj_hist[:iters_done] as numpy fp64)."""
    import torch
    it = _i32()
    hist = np.zeros(max(int(max_iter), 1), dtype=np.float64)
    _check(lib().kkm_iterate(ctx, _dev_ptr(V, torch.int32, "V"), int(k), int(max_iter), float(tol),
                             ctypes.byref(it), hist.ctypes.data), ctx)
    return it.value, hist[:it.value].copy()


def kkm_iterate_noalloc(ctx, V, k: int, max_iter: int, tol: float = -1.0):
    """kkm_iterate on the library's static device scratch (no device allocation
    in the call).  Returns (iters_done, obj_hist[:iters_done] as numpy fp64)."""
    import torch
    it = _i32()
    hist = np.zeros(max(int(max_iter), 1), dtype=np.float64)
    _check(lib().kkm_iterate_noalloc(ctx, _dev_ptr(V, torch.int32, "V"), int(k), int(max_iter), float(tol),
                                     ctypes.byref(it), hist.ctypes.data), ctx)
    return it.value, hist[:it.value].copy()


def kkm_objective(ctx, V, k: int) -> float:
    import torch
    J = _f64()
    _check(lib().kkm_objective(ctx, _dev_ptr(V, torch.int32, "V"), int(k), ctypes.byref(J)), ctx)
    return J.value


def kkm_step(ctx, cl_in, k: int, E=None, z=None, D=None, cl_out=None, counts_out=None) -> float:
    """One step with every intermediate; returns J(cl_in).  Outputs are device tensors or None."""
    import torch
    J = _f64()
    _check(lib().kkm_step(ctx, _dev_ptr(cl_in, torch.int32, "cl_in"), int(k),
                          _dev_ptr(E, torch.float32, "E"), _dev_ptr(z, torch.float32, "z", int(k)),
                          _dev_ptr(D, torch.float32, "D"), _dev_ptr(cl_out, torch.int32, "cl_out"),
                          _dev_ptr(counts_out, torch.int32, "counts_out", int(k)), ctypes.byref(J)), ctx)
    return J.value


def kkm_build_panel(ctx, X, n: int, d: int, kind: int, params: kkm_params, c0: int, c1: int) -> None:
    """One GPU's share: the column panel K[:, c0:c1] (c0 a multiple of 128)."""
    import torch
    _check(lib().kkm_build_panel(ctx, _dev_ptr(X, torch.float32, "X", int(n) * int(d)), int(n), int(d),
                                 int(kind), ctypes.byref(params), int(c0), int(c1)), ctx)
    _warn_if_any(ctx)


def _stored(ctx):
    """(r0, r1, c0, c1) of the K the context holds, or None before a build."""
    info = kkm_info()
    if lib().kkm_get_info(ctx, ctypes.byref(info)) != KKM_OK:
        return None
    return info.r0, info.r1, info.c0, info.c1


def kkm_panel_spmm(ctx, cl, k: int):
    """E for the panel's points (kept); returns (zpart as numpy fp64[k], sizes as numpy int32[k])."""
    import torch
    st = _stored(ctx)
    zpart = np.zeros(int(k), dtype=np.float64)
    counts = np.zeros(int(k), dtype=np.int32)
    _check(lib().kkm_panel_spmm(ctx, _dev_ptr(cl, torch.int32, "cl", st and st[1] - st[0]), int(k),
                                zpart.ctypes.data, counts.ctypes.data), ctx)
    return zpart, counts


def kkm_panel_assign(ctx, k: int, z, cl_out, E_out=None) -> np.ndarray:
    """New ids of the panel's points into cl_out from the global z; returns
    how many of them took each id (numpy int32[k])."""
    import torch
    z = np.ascontiguousarray(z, dtype=np.float64)
    if z.shape != (int(k),):
        raise KKMError(KKM_ERR_ARG, f"z must hold k={k} values, got shape {z.shape}")
    st = _stored(ctx)
    w = st and st[3] - st[2]
    counts = np.zeros(int(k), dtype=np.int32)
    _check(lib().kkm_panel_assign(ctx, int(k), z.ctypes.data, _dev_ptr(cl_out, torch.int32, "cl_out", w),
                                  _dev_ptr(E_out, torch.float32, "E_out", w and w * int(k)),
                                  counts.ctypes.data), ctx)
    return counts


def kkm_build_block(ctx, X, n: int, d: int, kind: int, params: kkm_params, r0: int, r1: int, c0: int,
                    c1: int) -> None:
    """One GPU's share of the 1.5D split: the block K[r0:r1, c0:c1] (r0, c0 multiples of 128)."""
    import torch
    _check(lib().kkm_build_block(ctx, _dev_ptr(X, torch.float32, "X", int(n) * int(d)), int(n), int(d),
                                 int(kind), ctypes.byref(params), int(r0), int(r1), int(c0), int(c1)), ctx)
    _warn_if_any(ctx)


def kkm_block_spmm(ctx, cl, k: int, E_out) -> None:
    """The block's partial E (its c1 - c0 columns x k, point-major) into
    E_out from the ids cl of its rows r0 .. r1-1."""
    import torch
    st = _stored(ctx)
    _check(lib().kkm_block_spmm(ctx, _dev_ptr(cl, torch.int32, "cl", st and st[1] - st[0]), int(k),
                                _dev_ptr(E_out, torch.float32, "E_out", st and (st[3] - st[2]) * int(k))), ctx)


def kkm_block_zpart(ctx, E, cl, a0: int, a1: int, k: int):
    """Self-term parts and sizes of the piece [a0, a1) of the block's columns
    from its rows of E (device, (a1-a0) x k) and its ids; returns (zpart as
    numpy fp64[k], sizes as numpy int32[k])."""
    import torch
    m = max(int(a1) - int(a0), 0)
    zpart = np.zeros(int(k), dtype=np.float64)
    counts = np.zeros(int(k), dtype=np.int32)
    _check(lib().kkm_block_zpart(ctx, _dev_ptr(E, torch.float32, "E", m * int(k)),
                                 _dev_ptr(cl, torch.int32, "cl", m), int(a0), int(a1), int(k),
                                 zpart.ctypes.data, counts.ctypes.data), ctx)
    return zpart, counts


def kkm_block_assign(ctx, E, a0: int, a1: int, k: int, z, counts, cl_out) -> np.ndarray:
    """New ids of the piece [a0, a1) into cl_out from its rows of E and the
    global z and sizes; returns how many of its points took each id."""
    import torch
    m = max(int(a1) - int(a0), 0)
    z = np.ascontiguousarray(z, dtype=np.float64)
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    if z.shape != (int(k),) or counts.shape != (int(k),):
        raise KKMError(KKM_ERR_ARG, f"z and counts must hold k={k} values, got {z.shape}, {counts.shape}")
    took = np.zeros(int(k), dtype=np.int32)
    _check(lib().kkm_block_assign(ctx, _dev_ptr(E, torch.float32, "E", m * int(k)), int(a0), int(a1), int(k),
                                  z.ctypes.data, counts.ctypes.data, _dev_ptr(cl_out, torch.int32, "cl_out", m),
                                  took.ctypes.data), ctx)
    return took


def kkm_init_kmeanspp(ctx, k: int, u, V) -> np.ndarray:
    """K-means++ seeding from the uniforms u (k floats in [0, 1)); writes the
    initial ids into V (device int32[n]) and returns the chosen centers."""
    import torch
    u = np.ascontiguousarray(u, dtype=np.float64)
    if u.shape != (int(k),):
        raise KKMError(KKM_ERR_ARG, f"u must hold k={k} uniforms, got shape {u.shape}")
    centers = np.zeros(int(k), dtype=np.int32)
    _check(lib().kkm_init_kmeanspp(ctx, int(k), u.ctypes.data, centers.ctypes.data,
                                   _dev_ptr(V, torch.int32, "V")), ctx)
    return centers


def kkm_copy_kernel_rows(ctx, r0: int, r1: int, out) -> None:
    """Rows r0 .. r1-1 of the stored K (of a panel or block: its columns) into out."""
    import torch
    st = _stored(ctx)
    numel = (int(r1) - int(r0)) * (st[3] - st[2]) if st and r1 > r0 else None
    _check(lib().kkm_copy_kernel_rows(ctx, int(r0), int(r1), _dev_ptr(out, torch.float32, "out", numel)), ctx)


def kkm_copy_diag(ctx, out) -> None:
    import torch
    st = _stored(ctx)
    n = kkm_get_info(ctx)["n"] if st else None
    _check(lib().kkm_copy_diag(ctx, _dev_ptr(out, torch.float32, "out", n)), ctx)


PEAK_READ_GROUPS = 2040  # workgroups of the streaming read and write


def kkm_peak_read(ctx, buf, sums, reps: int = 1) -> float:
    """Streaming-read microbenchmark over the fp32 device tensor buf; the sum read by
    workgroup g goes to sums[g], g < PEAK_READ_GROUPS.  Returns ms per launch."""
    import torch
    if sums.numel() < PEAK_READ_GROUPS:
        raise KKMError(KKM_ERR_ARG, f"sums must hold at least {PEAK_READ_GROUPS} floats (one per workgroup)")
    ms = ctypes.c_float()
    _check(lib().kkm_peak_read(ctx, _dev_ptr(buf, torch.float32, "buf"), buf.numel() * 4,
                               _dev_ptr(sums, torch.float32, "sums"), int(reps), ctypes.byref(ms)), ctx)
    return ms.value


def kkm_peak_read_rows(ctx, buf, rows, seg: int, sums, reps: int = 1) -> float:
    """Streaming read of rows in the packed SpMM's load pattern over the 2-D fp32
    device tensor buf (nrows x ld): workgroup (c, s) reads rows[128c .. 128c + 127]
    (int32 device tensor, clamped into range) over columns [s*seg, (s+1)*seg) and
    writes its sum to sums[c * (ld // seg) + s].  Returns ms per launch."""
    import torch
    if buf.dim() != 2 or not buf.is_contiguous():
        raise KKMError(KKM_ERR_ARG, "buf must be a contiguous 2-D tensor")
    nrows, ld = buf.shape
    if rows.numel() % 128 or rows.numel() == 0:
        raise KKMError(KKM_ERR_ARG, "rows must hold a positive multiple of 128 indices")
    nchunks = rows.numel() // 128
    if seg > 0 and sums.numel() < nchunks * (ld // seg):
        raise KKMError(KKM_ERR_ARG, f"sums must hold at least {nchunks * (ld // seg)} floats")
    ms = ctypes.c_float()
    _check(lib().kkm_peak_read_rows(ctx, _dev_ptr(buf, torch.float32, "buf"), nrows, ld,
                                    _dev_ptr(rows, torch.int32, "rows"), nchunks, int(seg),
                                    _dev_ptr(sums, torch.float32, "sums"), int(reps), ctypes.byref(ms)), ctx)
    return ms.value


def kkm_peak_write(ctx, buf, value: float, reps: int = 1) -> float:
    """Streaming-write microbenchmark: value into every element of buf.  Returns ms per launch."""
    import torch
    ms = ctypes.c_float()
    _check(lib().kkm_peak_write(ctx, _dev_ptr(buf, torch.float32, "buf"), buf.numel() * 4, float(value),
                                int(reps), ctypes.byref(ms)), ctx)
    return ms.value


def kkm_peak_mfma(ctx, iters: int, out, reps: int = 1):
    """fp32 MFMA register loop; out >= 4096 floats.  Returns (ms per launch, flop per launch)."""
    import torch
    if out.numel() < 4096:
        raise KKMError(KKM_ERR_ARG, "out must hold at least 4096 floats (one per wavefront)")
    ms, fl = ctypes.c_float(), _f64()
    _check(lib().kkm_peak_mfma(ctx, int(iters), _dev_ptr(out, torch.float32, "out"), int(reps),
                               ctypes.byref(ms), ctypes.byref(fl)), ctx)
    return ms.value, fl.value


KKM_TIME_ALL = (1 << len(PHASES)) - 1


def phase_mask(*names) -> int:
    """Bit mask of the named phases for kkm_set_timing."""
    return sum(1 << PHASES.index(n) for n in names)


def kkm_set_timing(ctx, phase_mask_: int) -> None:
    """phase_mask_: phases to bracket with HIP events (KKM_TIME_ALL, 0 = off)."""
    _check(lib().kkm_set_timing(ctx, int(phase_mask_)), ctx)


def kkm_get_timing(ctx) -> dict:
    t = kkm_timing()
    _check(lib().kkm_get_timing(ctx, ctypes.byref(t)), ctx)
    return {p: (t.ms[i], t.launches[i]) for i, p in enumerate(PHASES)}


def kkm_get_info(ctx) -> dict:
    i = kkm_info()
    _check(lib().kkm_get_info(ctx, ctypes.byref(i)), ctx)
    return {f: getattr(i, f) for f, _ in kkm_info._fields_}
