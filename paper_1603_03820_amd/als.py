"""Thin ctypes binding of libals.so (include/als.h), marshalling torch tensors.

Every call forwards device pointers (``tensor.data_ptr()``) and the current HIP stream to the
C ABI; all arithmetic runs in the library's kernels.  PyTorch only provides device memory
and streams.  Importing this module fails loudly when libals.so is not built: there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libals.so")

ALS_OK = 0
ALS_F_MAX = 128
EXPORTED = ("als_workspace_bytes", "als_init", "als_destroy", "als_half_sweep", "als_rmse",
            "als_status", "als_plan", "als_csr_to_csc", "als_rmse_waves", "als_gather_dump",
            "als_profile_begin", "als_profile_end", "als_last_hip_error", "als_strerror",
            "als_rmse_noalloc")


class ALSError(RuntimeError):
    def __init__(self, fn: str, code: int, hip: int = 0):
        msg = f"{fn}: {_lib.als_strerror(code).decode()} ({code})"
        if hip:
            msg += f", HIP error {hip}"
        super().__init__(msg)
        self.code = code


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libals.so is not built ({LIB_PATH}); run __graft_entry__.build() or "
                          "python paper_1603_03820_amd/build.py")
    lib = ctypes.CDLL(LIB_PATH)
    P, i64, i32, f32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float
    lib.als_workspace_bytes.argtypes = [ctypes.c_int, i32]
    lib.als_workspace_bytes.restype = ctypes.c_size_t
    lib.als_init.argtypes = [ctypes.POINTER(P), ctypes.c_int, P, ctypes.c_size_t, i32]
    lib.als_destroy.argtypes = [P]
    lib.als_half_sweep.argtypes = [P, P, P, P, i64, i64, i32, f32, P, P, P]
    lib.als_rmse.argtypes = [P, P, P, P, i64, i64, i32, P, P, P, P]
    lib.als_rmse_noalloc.argtypes = [ctypes.c_int, P, P, P, i64, i64, i32, P, P, P, P]
    lib.als_status.argtypes = [P, P, ctypes.POINTER(i64)]
    lib.als_plan.argtypes = [P, P, i64, i32, P, i64, P, P]
    lib.als_csr_to_csc.argtypes = [P, P, P, P, i64, i64, P, P, P, P]
    lib.als_rmse_waves.argtypes = [P, i32]
    lib.als_gather_dump.argtypes = [P, P, P, P, i64, i64, i32, P, i64, P, i64, P]
    lib.als_profile_begin.argtypes = [P, i32]
    lib.als_profile_end.argtypes = [P, P, i32, ctypes.POINTER(i32)]
    lib.als_last_hip_error.argtypes = [P]
    lib.als_strerror.argtypes = [ctypes.c_int]
    lib.als_strerror.restype = ctypes.c_char_p
    for fn in ("als_init", "als_destroy", "als_half_sweep", "als_rmse", "als_status", "als_plan",
               "als_csr_to_csc", "als_rmse_waves", "als_gather_dump", "als_profile_begin",
               "als_profile_end", "als_last_hip_error", "als_rmse_noalloc"):
        getattr(lib, fn).restype = ctypes.c_int
    return lib


_lib = _load()


def _stream(device: torch.device, stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream(device) if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t: torch.Tensor, dtype, name: str, numel: int | None = None) -> ctypes.c_void_p:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, needs {numel}")
    return ctypes.c_void_p(t.data_ptr())


def _check(fn: str, rc: int, ctx=None):
    if rc != ALS_OK:
        hip = _lib.als_last_hip_error(ctx) if ctx is not None else 0
        raise ALSError(fn, rc, hip)


def als_workspace_bytes(device: int = 0, f_max: int = ALS_F_MAX) -> int:
    return int(_lib.als_workspace_bytes(device, f_max))


class Context:
    """An als_ctx plus the workspace tensor it runs in (one per device)."""

    def __init__(self, device: int = 0, f_max: int = ALS_F_MAX):
        self.device = torch.device("cuda", device)
        nbytes = als_workspace_bytes(device, f_max)
        if nbytes == 0:
            raise RuntimeError(f"als_workspace_bytes failed for device {device} (not gfx950?)")
        # torch's caching allocator hands out 512-byte aligned blocks
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        h = ctypes.c_void_p()
        _check("als_init", _lib.als_init(ctypes.byref(h), device,
                                         ctypes.c_void_p(self.workspace.data_ptr()), nbytes, f_max))
        self.handle = h
        self.f_max = f_max

    def close(self):
        if getattr(self, "handle", None):
            _lib.als_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def als_init(device: int = 0, f_max: int = ALS_F_MAX) -> Context:
    return Context(device, f_max)


def als_destroy(ctx: Context):
    ctx.close()


def als_half_sweep(ctx: Context, rowptr, colidx, vals, m: int, n: int, f: int, lam: float,
                   theta_in, x_out, stream=None):
    """x_out[u] = (sum theta_v theta_v^T + lam n_u I)^{-1} sum r_uv theta_v for all rows u."""
    nnz = None
    args = (ctx.handle,
            _dev(rowptr, torch.int64, "rowptr", m + 1),
            _dev(colidx, torch.int32, "colidx", nnz),
            _dev(vals, torch.float32, "vals", nnz),
            m, n, f, float(lam),
            _dev(theta_in, torch.float32, "theta_in", n * f),
            _dev(x_out, torch.float32, "x_out", m * f),
            _stream(ctx.device, stream))
    _check("als_half_sweep", _lib.als_half_sweep(*args), ctx.handle)
    return x_out


def als_rmse(ctx: Context, rowptr, colidx, vals, m: int, n: int, f: int, x, theta, out=None,
             stream=None):
    """Training RMSE over the stored entries, as a 1-element float64 device tensor."""
    if out is None:
        out = torch.empty(1, dtype=torch.float64, device=ctx.device)
    rc = _lib.als_rmse(ctx.handle, _dev(rowptr, torch.int64, "rowptr", m + 1),
                       _dev(colidx, torch.int32, "colidx"), _dev(vals, torch.float32, "vals"),
                       m, n, f, _dev(x, torch.float32, "x", m * f),
                       _dev(theta, torch.float32, "theta", n * f),
                       _dev(out, torch.float64, "out", 1), _stream(ctx.device, stream))
    _check("als_rmse", rc, ctx.handle)
    return out


def als_rmse_noalloc(device: int, rowptr, colidx, vals, m: int, n: int, f: int, x, theta, out,
                     stream=None):
    """als_rmse without a context or workspace: the library's fixed per-device scratch, no
    allocation in the call.  `out` (a 1-element float64 device tensor) is the caller's."""
    dev = torch.device("cuda", device)
    rc = _lib.als_rmse_noalloc(device, _dev(rowptr, torch.int64, "rowptr", m + 1),
                               _dev(colidx, torch.int32, "colidx"),
                               _dev(vals, torch.float32, "vals"), m, n, f,
                               _dev(x, torch.float32, "x", m * f),
                               _dev(theta, torch.float32, "theta", n * f),
                               _dev(out, torch.float64, "out", 1), _stream(dev, stream))
    _check("als_rmse_noalloc", rc)
    return out


def als_rmse_waves(ctx: Context, waves_per_simd: int):
    """Cap later als_rmse calls on this context at `waves_per_simd` resident waves per SIMD
    (0: as many as fit).  The result does not depend on the width."""
    _check("als_rmse_waves", _lib.als_rmse_waves(ctx.handle, waves_per_simd), ctx.handle)


def als_status(ctx: Context, stream=None) -> int:
    """Synchronise the stream; rows found not positive definite since the last call."""
    cnt = ctypes.c_int64(0)
    _check("als_status", _lib.als_status(ctx.handle, _stream(ctx.device, stream),
                                         ctypes.byref(cnt)), ctx.handle)
    return int(cnt.value)


def als_plan(ctx: Context, rowptr, m: int, f: int, stream=None):
    """(bounds int64 [C+1, 2] device tensor, (C, c_nnz, c_row, q, W, tail_div))."""
    params = (ctypes.c_int64 * 6)()
    # first call with zero capacity to learn C
    rc = _lib.als_plan(ctx.handle, _dev(rowptr, torch.int64, "rowptr", m + 1), m, f,
                       ctypes.c_void_p(rowptr.data_ptr()), 0, params, _stream(ctx.device, stream))
    if rc not in (ALS_OK, -1):
        _check("als_plan", rc, ctx.handle)
    C = int(params[0])
    bounds = torch.empty((C + 1, 2), dtype=torch.int64, device=ctx.device)
    rc = _lib.als_plan(ctx.handle, _dev(rowptr, torch.int64, "rowptr", m + 1), m, f,
                       _dev(bounds, torch.int64, "bounds"), C + 1, params,
                       _stream(ctx.device, stream))
    _check("als_plan", rc, ctx.handle)
    return bounds, tuple(int(v) for v in params)


def als_csr_to_csc(ctx: Context, rowptr, colidx, vals, m: int, n: int, nnz: int | None = None,
                   out=None, stream=None):
    """The CSC of the m x n CSR matrix (stable: rows ascending within each column), as device
    tensors (colptr int64 [n+1], rowidx int32 [nnz], vals_t float32 [nnz]).  nnz defaults to
    rowptr[m] (read from the device); `out` may supply the three output tensors."""
    if nnz is None:
        nnz = int(rowptr[m].item()) if m > 0 else 0
    if out is None:
        # at least one element each (an empty tensor's data pointer is null)
        out = (torch.empty(n + 1, dtype=torch.int64, device=ctx.device),
               torch.empty(max(nnz, 1), dtype=torch.int32, device=ctx.device),
               torch.empty(max(nnz, 1), dtype=torch.float32, device=ctx.device))
    colptr, rowidx, vals_t = out
    rc = _lib.als_csr_to_csc(ctx.handle, _dev(rowptr, torch.int64, "rowptr", m + 1),
                             _dev(colidx, torch.int32, "colidx", nnz),
                             _dev(vals, torch.float32, "vals", nnz), m, n,
                             _dev(colptr, torch.int64, "colptr", n + 1),
                             _dev(rowidx, torch.int32, "rowidx", nnz),
                             _dev(vals_t, torch.float32, "vals_t", nnz),
                             _stream(ctx.device, stream))
    _check("als_csr_to_csc", rc, ctx.handle)
    return colptr, rowidx[:nnz], vals_t[:nnz]


def als_gather_dump(ctx: Context, rowptr, colidx, vals, m: int, n: int, f: int, theta, u: int,
                    n_u: int, stream=None):
    """The gather stage of the half-sweep on row u, as a float32 device tensor [n_u, NB + 3, 16]
    (NB = f // 16 + 1): per entry the MFMA operand blocks, the quad-form operands and the
    rating (see als_gather_dump in include/als.h).  Zero-filled before the call."""
    nb = f // 16 + 1
    out = torch.zeros((max(n_u, 1), nb + 3, 16), dtype=torch.float32, device=ctx.device)
    rc = _lib.als_gather_dump(ctx.handle, _dev(rowptr, torch.int64, "rowptr", m + 1),
                              _dev(colidx, torch.int32, "colidx"),
                              _dev(vals, torch.float32, "vals"), m, n, f,
                              _dev(theta, torch.float32, "theta", n * f), u,
                              ctypes.c_void_p(out.data_ptr()), n_u * (nb + 3) * 16,
                              _stream(ctx.device, stream))
    _check("als_gather_dump", rc, ctx.handle)
    return out[:n_u]


def als_profile_begin(ctx: Context, capacity: int):
    """Record HIP events around the kernels of the next `capacity` half-sweeps."""
    _check("als_profile_begin", _lib.als_profile_begin(ctx.handle, capacity), ctx.handle)


def als_profile_end(ctx: Context, capacity: int):
    """[(plan_ms, herm_solve_ms, reduce_solve_ms) per profiled half-sweep, in call order]."""
    import numpy as np
    ms = np.zeros(3 * max(capacity, 1), dtype=np.float32)
    cnt = ctypes.c_int32(0)
    _check("als_profile_end", _lib.als_profile_end(ctx.handle, ctypes.c_void_p(ms.ctypes.data),
                                                 capacity, ctypes.byref(cnt)), ctx.handle)
    return [tuple(float(v) for v in ms[3 * i:3 * i + 3]) for i in range(cnt.value)]
