"""The gather stage of the half-sweep, bit for bit: als_gather_dump runs a row through the same
gather form, index ring and pipeline as the half-sweep kernel and writes the MFMA operands each
entry received.  They must equal theta[colidx[k]] (with the rating in column f and zeros past it),
the quad-form operands and the rating, exactly, for every gather form and for row lengths around
the step (4), group (16) and index-batch (48) boundaries and beyond one batch."""
import os

import numpy as np
import pytest
import torch

from tests.gpu_util import log, to_dev

pytestmark = pytest.mark.gpu

LENGTHS = [1, 2, 3, 4, 5, 15, 16, 17, 47, 48, 49, 95, 96, 97, 191, 1000]


def make_ctx(form):
    from paper_1603_03820_amd import als
    env = {"global": ("ALS_GATHER", "global"), "tiles": ("ALS_LAST_BLOCK", "tiles"),
           "lds": ("ALS_GATHER", "lds")}.get(form)
    if env:
        os.environ[env[0]] = env[1]
    try:
        return als.Context(0, 128)
    finally:
        if env:
            del os.environ[env[0]]


def quads(f, form):
    """Quad operands the library uses for this f and form (0: 16x16 tiles for the last block)."""
    nb = f // 16 + 1
    f_last = f - 16 * (nb - 1)
    if form in ("tiles", "lds") or f_last not in (0, 4):
        return 0
    return f_last // 4 + 1


def expected(theta, cols, ratings, f, P):
    nb = f // 16 + 1
    k = len(cols)
    rec = np.zeros((k, nb + 3, 16), np.float32)
    lane = np.arange(16)
    for I in range(nb):
        j = 16 * I + lane
        blk = np.zeros((k, 16), np.float32)
        blk[:, j < f] = theta[cols][:, j[j < f]]
        blk[:, j == f] = ratings[:, None]
        rec[:, I] = blk
    for p in range(P):
        if p < P - 1:
            rec[:, nb + p] = theta[cols][:, 16 * (nb - 1) + 4 * p + (lane & 3)]
        else:
            rec[:, nb + p] = np.where((lane & 3) == 0, ratings[:, None], 0.0)
    rec[:, nb + 2] = ratings[:, None]
    return rec


@pytest.mark.parametrize("f,form", [(1, "buffer"), (7, "buffer"), (16, "buffer"), (33, "buffer"),
                                    (100, "buffer"), (100, "tiles"), (100, "global"),
                                    (112, "buffer"), (128, "buffer"), (128, "global"),
                                    (7, "global"), (16, "global"), (21, "global"),
                                    (47, "global"), (90, "global"), (116, "global"),
                                    (4, "lds"), (32, "lds"), (100, "lds"), (128, "lds")])
def test_gather_dump_bit_exact(f, form):
    from paper_1603_03820_amd import als
    ctx = make_ctx(form)
    rng = np.random.default_rng(1000 + f)
    n = 3000
    lengths = np.array(LENGTHS + [0, 7], np.int64)
    rowptr = np.zeros(len(lengths) + 1, np.int64)
    rowptr[1:] = np.cumsum(lengths)
    colidx = np.concatenate([rng.choice(n, size=c, replace=False) for c in lengths]).astype(np.int32)
    vals = rng.standard_normal(rowptr[-1]).astype(np.float32)
    theta = rng.standard_normal((n, f)).astype(np.float32)
    dev = ctx.device
    rp, ci, v, th = to_dev(rowptr, dev), to_dev(colidx, dev), to_dev(vals, dev), to_dev(theta, dev)
    P = quads(f, form)
    for u, nu in enumerate(lengths):
        log(f"gather dump f={f} form={form} row {u} (n_u={nu}, quads={P})")
        got = als.als_gather_dump(ctx, rp, ci, v, len(lengths), n, f, th, u, int(nu))
        torch.cuda.synchronize()
        got = got.cpu().numpy()
        k0, k1 = rowptr[u], rowptr[u + 1]
        ref = expected(theta, colidx[k0:k1], vals[k0:k1], f, P)
        assert got.shape == ref.shape
        bad = np.argwhere(got.view(np.uint32) != ref.view(np.uint32))
        assert bad.size == 0, f"row {u}: first mismatches (entry, block, lane) {bad[:5].tolist()}"
    ctx.close()


def test_gather_dump_respects_capacity():
    """Records past the caller's capacity are not written."""
    from paper_1603_03820_amd import als
    import ctypes
    ctx = make_ctx("buffer")
    f, n = 100, 500
    rng = np.random.default_rng(5)
    rowptr = np.array([0, 200], np.int64)
    colidx = rng.choice(n, size=200, replace=False).astype(np.int32)
    vals = rng.standard_normal(200).astype(np.float32)
    theta = rng.standard_normal((n, f)).astype(np.float32)
    dev = ctx.device
    rec = (f // 16 + 1 + 3) * 16
    out = torch.full((200, rec), -1.0, dtype=torch.float32, device=dev)
    log("gather dump with capacity for 37 records")
    keep = [to_dev(a, dev) for a in (rowptr, colidx, vals, theta)]   # alive until the sync
    torch.cuda.synchronize()
    rp, ci, v, th = (ctypes.c_void_p(t.data_ptr()) for t in keep)
    rc = als._lib.als_gather_dump(ctx.handle, rp, ci, v, 1, n, f, th, 0,
                                  ctypes.c_void_p(out.data_ptr()), 37 * rec, None)
    torch.cuda.synchronize()
    assert rc == 0
    o = out.cpu().numpy()
    assert np.all(o[37:] == -1.0) and not np.all(o[:37] == -1.0)
    ctx.close()
