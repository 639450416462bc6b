"""ALS iterations on the device: update-X (eq. 2) then update-Theta (eq. 3), each one
als_half_sweep call, with the training RMSE -- and, given a held-out set, the test RMSE (the
paper's evaluation metric, experiments section) -- after each iteration, and optional
asynchronous checkpoints of X and Theta with resume.  Inputs are torch device tensors; nothing
here computes on the host."""
from __future__ import annotations

import json
import os
import threading
import time
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

    @classmethod
    def from_host_csr(cls, ctx, m, n, f, lam, rowptr, colidx, vals):
        """Upload the CSR of R only; its CSC (the item side's input) is built on the device by
        als_csr_to_csc (stable, so identical to any stable host transpose)."""
        t = lambda a: torch.from_numpy(a).to(ctx.device)  # noqa: E731
        rp, ci, v = t(rowptr), t(colidx), t(vals)
        colptr, rowidx, vals_t = als.als_csr_to_csc(ctx, rp, ci, v, m, n, nnz=int(rowptr[-1]))
        return cls(m, n, f, lam, rp, ci, v, colptr, rowidx, vals_t)


@dataclass
class RatingSet:
    """A set of ratings over the same m x n shape (e.g. a held-out test split), CSR on device."""
    m: int
    n: int
    rowptr: torch.Tensor
    colidx: torch.Tensor
    vals: torch.Tensor

    @classmethod
    def from_host(cls, m, n, rowptr, colidx, vals, device):
        t = lambda a: torch.from_numpy(a).to(device)  # noqa: E731
        return cls(m, n, t(rowptr), t(colidx), t(vals))


def update_x(ctx, p: DeviceProblem, theta, x, stream=None):
    return als.als_half_sweep(ctx, p.rowptr, p.colidx, p.vals, p.m, p.n, p.f, p.lam, theta, x,
                              stream)


def update_theta(ctx, p: DeviceProblem, x, theta, stream=None):
    return als.als_half_sweep(ctx, p.colptr, p.rowidx, p.vals_t, p.n, p.m, p.f, p.lam, x, theta,
                              stream)


CHECKPOINT_FILE = "als_{:06d}.safetensors"


class AsyncCheckpointer:
    """Saves (iteration, X, Theta) without holding up the compute stream: a device-to-device
    snapshot on the compute stream (so later iterations may overwrite X and Theta at once), a
    copy of the snapshot to pinned host memory on a side stream, and a host thread that writes
    the file (safetensors + a JSON manifest) once that copy has completed.  One save is in
    flight at a time: the next one first waits for the previous file.  Files are written to a
    temporary name and renamed, so a file that exists is complete."""

    def __init__(self, directory: str, x_like: torch.Tensor, theta_like: torch.Tensor):
        self.dir = directory
        os.makedirs(directory, exist_ok=True)
        self.snap_x = torch.empty_like(x_like)
        self.snap_t = torch.empty_like(theta_like)
        cuda = x_like.is_cuda
        self.host_x = torch.empty(x_like.shape, dtype=x_like.dtype, pin_memory=cuda)
        self.host_t = torch.empty(theta_like.shape, dtype=theta_like.dtype, pin_memory=cuda)
        self.side = torch.cuda.Stream(device=x_like.device) if cuda else None
        self._thread: threading.Thread | None = None
        self._error: BaseException | None = None
        self.saved: list[str] = []

    def save(self, iteration: int, x: torch.Tensor, theta: torch.Tensor) -> None:
        self.wait()
        if self.side is None:   # host tensors: write synchronously
            self.host_x.copy_(x)
            self.host_t.copy_(theta)
            self._write(iteration, None)
            return
        cur = torch.cuda.current_stream(x.device)
        self.snap_x.copy_(x, non_blocking=True)
        self.snap_t.copy_(theta, non_blocking=True)
        snapped = torch.cuda.Event()
        snapped.record(cur)
        self.side.wait_event(snapped)
        with torch.cuda.stream(self.side):
            self.host_x.copy_(self.snap_x, non_blocking=True)
            self.host_t.copy_(self.snap_t, non_blocking=True)
            copied = torch.cuda.Event()
            copied.record(self.side)
        self._thread = threading.Thread(target=self._write_guarded, args=(iteration, copied),
                                        daemon=True)
        self._thread.start()

    def _write_guarded(self, iteration, event):
        try:
            self._write(iteration, event)
        except BaseException as e:  # reported by wait()
            self._error = e

    def _write(self, iteration, event):
        from safetensors.torch import save_file
        if event is not None:
            event.synchronize()
        name = CHECKPOINT_FILE.format(iteration)
        tmp = os.path.join(self.dir, name + ".tmp")
        save_file({"x": self.host_x, "theta": self.host_t}, tmp,
                  metadata={"iteration": str(iteration)})
        os.replace(tmp, os.path.join(self.dir, name))
        with open(os.path.join(self.dir, "latest.json.tmp"), "w") as fh:
            json.dump({"iteration": iteration, "file": name,
                       "x_shape": list(self.host_x.shape),
                       "theta_shape": list(self.host_t.shape)}, fh)
        os.replace(os.path.join(self.dir, "latest.json.tmp"), os.path.join(self.dir, "latest.json"))
        self.saved.append(name)

    def wait(self) -> None:
        """Block until the save in flight (if any) is on disk; re-raise its error."""
        if self._thread is not None:
            self._thread.join()
            self._thread = None
        if self._error is not None:
            e, self._error = self._error, None
            raise e


def load_checkpoint(directory: str, device, iteration: int | None = None):
    """(iteration, x, theta) from a checkpoint directory: the latest, or a given iteration."""
    from safetensors.torch import load_file
    if iteration is None:
        with open(os.path.join(directory, "latest.json")) as fh:
            iteration = int(json.load(fh)["iteration"])
    t = load_file(os.path.join(directory, CHECKPOINT_FILE.format(iteration)))
    return iteration, t["x"].to(device), t["theta"].to(device)


def run(ctx, p: DeviceProblem, theta0, iters: int, *, test: RatingSet | None = None,
        rmse_every: bool = True, checkpointer: AsyncCheckpointer | None = None,
        checkpoint_every: int = 0, start_iteration: int = 0, x0=None):
    """Run ALS iterations start_iteration+1 .. start_iteration+iters from theta0 (and x0, which
    update-X overwrites, so it only matters for a zero-iteration run).  Per iteration: the
    iteration's device time (HIP events around its two half-sweeps), the wall time since the
    start once its results are back, the training RMSE and the test RMSE (when `test` is given),
    and a checkpoint every `checkpoint_every` iterations.  Returns (x, theta, history) with one
    dict per iteration."""
    dev = theta0.device
    theta = theta0.clone()
    x = x0.clone() if x0 is not None else torch.zeros((p.m, p.f), dtype=torch.float32,
                                                      device=dev)
    out = torch.empty(2, dtype=torch.float64, device=dev)
    hist = []
    t_start = time.perf_counter()
    for k in range(iters):
        it = start_iteration + k + 1
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        update_x(ctx, p, theta, x)
        update_theta(ctx, p, x, theta)
        e1.record()
        rec = {"iteration": it}
        if rmse_every:
            als.als_rmse(ctx, p.rowptr, p.colidx, p.vals, p.m, p.n, p.f, x, theta, out[0:1])
            if test is not None:
                als.als_rmse(ctx, test.rowptr, test.colidx, test.vals, test.m, test.n, p.f, x,
                             theta, out[1:2])
        if checkpointer is not None and checkpoint_every > 0 and it % checkpoint_every == 0:
            checkpointer.save(it, x, theta)
        e1.synchronize()
        rec["ms"] = e0.elapsed_time(e1)
        if rmse_every:
            vals = out.tolist()
            rec["train_rmse"] = vals[0]
            if test is not None:
                rec["test_rmse"] = vals[1]
        rec["wall_s"] = time.perf_counter() - t_start
        hist.append(rec)
    if checkpointer is not None:
        checkpointer.wait()
    return x, theta, hist


def train(ctx, p: DeviceProblem, theta0, iters: int, rmse_every: bool = True):
    """Run `iters` ALS iterations from theta0; returns (x, theta, [training RMSE per
    iteration])."""
    x, theta, hist = run(ctx, p, theta0, iters, rmse_every=rmse_every)
    return x, theta, [h["train_rmse"] for h in hist] if rmse_every else []
