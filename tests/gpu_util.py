"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI on host arrays,
and the per-row error measure the parity bar is stated in."""
from __future__ import annotations

import sys

import numpy as np
import torch


def log(msg: str):
    """Name the case before each GPU step, flushed, so a failure points at it."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def gpu_half_sweep(ctx, rowptr, colidx, vals, m, n, f, lam, theta, sentinel=float("nan")):
    """x (float32 numpy, m x f) from one als_half_sweep; x is pre-filled with `sentinel` so an
    unwritten row shows up."""
    from paper_1603_03820_amd import als
    dev = ctx.device
    rp, ci, v = to_dev(rowptr, dev), to_dev(colidx, dev), to_dev(vals, dev)
    th = to_dev(np.asarray(theta, dtype=np.float32).reshape(n, f), dev)
    x = torch.full((m, f), sentinel, dtype=torch.float32, device=dev)
    als.als_half_sweep(ctx, rp, ci, v, m, n, f, lam, th, x)
    torch.cuda.synchronize()
    return x.cpu().numpy()


def row_rel_err(x_gpu: np.ndarray, x_ref: np.ndarray) -> np.ndarray:
    """Per row: max_i |x_gpu - x_ref| / max(max_i |x_ref|, 1e-6 max_{u,i} |x_ref|)."""
    x_ref = np.asarray(x_ref, dtype=np.float64)
    gmax = float(np.abs(x_ref).max()) if x_ref.size else 0.0
    den = np.maximum(np.abs(x_ref).max(axis=1), max(1e-6 * gmax, 1e-30))
    return np.abs(x_gpu.astype(np.float64) - x_ref).max(axis=1) / den
