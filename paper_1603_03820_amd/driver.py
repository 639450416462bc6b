"""ALS iterations on the device: update-X (eq. 2) then update-Theta (eq. 3), each one
als_half_sweep call, with the training RMSE after each iteration.  Inputs are torch device
tensors; nothing here computes on the host."""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import als


@dataclass
class DeviceProblem:
    m: int
    n: int
    f: int
    lam: float
    rowptr: torch.Tensor    # CSR of R
    colidx: torch.Tensor
    vals: torch.Tensor
    colptr: torch.Tensor    # CSC of R (CSR of R^T)
    rowidx: torch.Tensor
    vals_t: torch.Tensor

    @classmethod
    def from_host(cls, m, n, f, lam, rowptr, colidx, vals, colptr, rowidx, vals_t, device):
        t = lambda a: torch.from_numpy(a).to(device)  # noqa: E731
        return cls(m, n, f, lam, t(rowptr), t(colidx), t(vals), t(colptr), t(rowidx), t(vals_t))


def update_x(ctx, p: DeviceProblem, theta, x, stream=None):
    return als.als_half_sweep(ctx, p.rowptr, p.colidx, p.vals, p.m, p.n, p.f, p.lam, theta, x,
                              stream)


def update_theta(ctx, p: DeviceProblem, x, theta, stream=None):
    return als.als_half_sweep(ctx, p.colptr, p.rowidx, p.vals_t, p.n, p.m, p.f, p.lam, x, theta,
                              stream)


def train(ctx, p: DeviceProblem, theta0, iters: int, rmse_every: bool = True):
    """Run `iters` ALS iterations from theta0; returns (x, theta, [rmse per iteration])."""
    theta = theta0.clone()
    x = torch.empty((p.m, p.f), dtype=torch.float32, device=theta0.device)
    hist = []
    out = torch.empty(1, dtype=torch.float64, device=theta0.device)
    for _ in range(iters):
        update_x(ctx, p, theta, x)
        update_theta(ctx, p, x, theta)
        if rmse_every:
            als.als_rmse(ctx, p.rowptr, p.colidx, p.vals, p.m, p.n, p.f, x, theta, out)
            hist.append(float(out.item()))
    return x, theta, hist
