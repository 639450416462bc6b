"""Row-batched half-sweep with R streamed from host memory, for rating matrices larger than the
device's memory (the paper's out-of-core / batched setting: only the factors and a working set
of R stay on the GPU).  The rows are cut into batches of whole rows holding about
`batch_entries` ratings (a longer row is a batch of its own); batch i+1's indices and ratings
are copied from pinned host memory on a side stream while batch i's half-sweep runs, through two
device buffers.  Each batch is one als_half_sweep call on a sub-CSR of the batch's rows (row
pointers rebased to 0), writing those rows of x_out; theta_in stays resident.  Nothing here
computes on the host beyond rebasing the row pointers of a batch."""
from __future__ import annotations

import numpy as np
import torch

from . import als


def plan_batches(rowptr: np.ndarray, batch_entries: int):
    """[(u0, u1)]: consecutive whole-row ranges covering all rows, each holding at most
    `batch_entries` ratings unless it is a single longer row."""
    if batch_entries < 1:
        raise ValueError("batch_entries must be positive")
    m = len(rowptr) - 1
    out, u0 = [], 0
    while u0 < m:
        # the last row u1 - 1 with rowptr[u1] - rowptr[u0] <= batch_entries, at least one row
        u1 = int(np.searchsorted(rowptr, rowptr[u0] + batch_entries, side="right")) - 1
        u1 = min(max(u1, u0 + 1), m)
        out.append((u0, u1))
        u0 = u1
    return out


class HostCSR:
    """One side of R (a CSR) in host memory: row pointers as int64 numpy, column indices and
    ratings in pinned (page-locked) tensors so that copies to the device are asynchronous."""

    def __init__(self, rowptr, colidx, vals):
        self.rowptr = np.ascontiguousarray(rowptr, dtype=np.int64)
        self.colidx = torch.from_numpy(np.ascontiguousarray(colidx, dtype=np.int32)).pin_memory()
        self.vals = torch.from_numpy(np.ascontiguousarray(vals, dtype=np.float32)).pin_memory()
        self.m = len(self.rowptr) - 1


class StreamedSweep:
    """Half-sweeps of one side of R held in host memory (see the module docstring).  Device
    memory: two buffers of the largest batch (indices, ratings, row pointers)."""

    def __init__(self, ctx, host: HostCSR, n: int, f: int, batch_entries: int):
        self.ctx, self.host, self.n, self.f = ctx, host, n, f
        self.batches = plan_batches(host.rowptr, batch_entries)
        rp = host.rowptr
        cap_e = max(int(rp[u1] - rp[u0]) for u0, u1 in self.batches) if self.batches else 0
        cap_r = max(u1 - u0 for u0, u1 in self.batches) if self.batches else 0
        dev = ctx.device
        self.d_col = [torch.empty(max(cap_e, 1), dtype=torch.int32, device=dev) for _ in range(2)]
        self.d_val = [torch.empty(max(cap_e, 1), dtype=torch.float32, device=dev)
                      for _ in range(2)]
        self.d_ptr = [torch.empty(cap_r + 1, dtype=torch.int64, device=dev) for _ in range(2)]
        self.h_ptr = [torch.empty(cap_r + 1, dtype=torch.int64, pin_memory=True)
                      for _ in range(2)]
        self.copy_stream = torch.cuda.Stream(device=dev)
        self.copied = [None, None]     # event: batch copy into buffer s done
        self.consumed = [None, None]   # event: the half-sweep reading buffer s done
        self.h2d_bytes = 0

    def _issue_copy(self, i: int) -> None:
        s = i % 2
        u0, u1 = self.batches[i]
        rp = self.host.rowptr
        k0, k1 = int(rp[u0]), int(rp[u1])
        if self.copied[s] is not None:
            self.copied[s].synchronize()          # the staging buffer's previous copy is done
        hp = self.h_ptr[s].numpy()
        np.subtract(rp[u0:u1 + 1], rp[u0], out=hp[:u1 - u0 + 1])
        if self.consumed[s] is not None:
            self.copy_stream.wait_event(self.consumed[s])
        with torch.cuda.stream(self.copy_stream):
            self.d_ptr[s][:u1 - u0 + 1].copy_(self.h_ptr[s][:u1 - u0 + 1], non_blocking=True)
            if k1 > k0:
                self.d_col[s][:k1 - k0].copy_(self.host.colidx[k0:k1], non_blocking=True)
                self.d_val[s][:k1 - k0].copy_(self.host.vals[k0:k1], non_blocking=True)
            ev = torch.cuda.Event()
            ev.record(self.copy_stream)
        self.copied[s] = ev
        self.h2d_bytes += 8 * (u1 - u0 + 1) + 8 * (k1 - k0)

    def half_sweep(self, lam: float, theta_in: torch.Tensor, x_out: torch.Tensor) -> torch.Tensor:
        """x_out[u] for every row u of the host CSR, as als_half_sweep computes it."""
        comp = torch.cuda.current_stream(self.ctx.device)
        nb = len(self.batches)
        if nb:
            self._issue_copy(0)
        for i in range(nb):
            s = i % 2
            if i + 1 < nb:
                self._issue_copy(i + 1)
            comp.wait_event(self.copied[s])
            u0, u1 = self.batches[i]
            ne = int(self.host.rowptr[u1] - self.host.rowptr[u0])
            als.als_half_sweep(self.ctx, self.d_ptr[s][:u1 - u0 + 1], self.d_col[s][:max(ne, 1)],
                               self.d_val[s][:max(ne, 1)], u1 - u0, self.n, self.f, lam,
                               theta_in, x_out[u0:u1])
            ev = torch.cuda.Event()
            ev.record(comp)
            self.consumed[s] = ev
        return x_out
