"""als_rmse_noalloc (the RMSE entry point that allocates nothing: fixed per-device scratch
instead of a workspace) against als_rmse, through the C ABI: two calls in a row, the second on
a smaller input, each bit-identical to als_rmse on the same input (same kernels, chunks and
summation order) and within 1e-6 of the fp64 oracle.  Also: argument errors, and a call
between two calls of als_rmse on the same stream does not disturb them."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import log, to_dev

pytestmark = pytest.mark.gpu


def _inputs(m, n, nnz, f, seed):
    p = synth.make(m, n, nnz, rows="lognormal", zipf=0.9, f=f, model="movie", plant_f=16,
                   seed=seed)
    x = synth.normal(seed + 1, 8, (p.m, f), 0.3)
    th = synth.normal(seed + 2, 8, (p.n, f), 0.3)
    return p, x, th


def test_noalloc_rmse_matches_rmse_twice_second_smaller():
    from paper_1603_03820_amd import als
    assert torch.cuda.is_available()
    orc = oracle.get()
    ctx = als.Context(0, 128)
    dev = ctx.device
    out_a = torch.full((1,), -1.0, dtype=torch.float64, device=dev)
    out_b = torch.full((1,), -1.0, dtype=torch.float64, device=dev)
    cases = [(20_000, 3_000, 1_500_000, 100, 41), (700, 90, 9_000, 33, 43)]
    for m, n, nnz, f, seed in cases:
        p, x, th = _inputs(m, n, nnz, f, seed)
        rp, ci, v = to_dev(p.rowptr, dev), to_dev(p.colidx, dev), to_dev(p.vals, dev)
        xd, td = to_dev(x, dev), to_dev(th, dev)
        log(f"rmse_noalloc m={m} n={n} nnz={nnz} f={f}")
        als.als_rmse_noalloc(0, rp, ci, v, p.m, p.n, f, xd, td, out_a)
        als.als_rmse(ctx, rp, ci, v, p.m, p.n, f, xd, td, out=out_b)
        torch.cuda.synchronize()
        a, b = out_a.item(), out_b.item()
        ref = orc.rmse(p.rowptr, p.colidx, p.vals, p.m, f, x.astype(np.float64),
                       th.astype(np.float64))
        log(f"noalloc {a:.12f} rmse {b:.12f} oracle {ref:.12f}")
        assert np.float64(a).tobytes() == np.float64(b).tobytes()
        assert abs(a - ref) <= 1e-6 * ref
    ctx.close()


def test_noalloc_rmse_interleaved_and_errors():
    from paper_1603_03820_amd import als
    dev = torch.device("cuda", 0)
    p, x, th = _inputs(5_000, 800, 200_000, 64, 47)
    rp, ci, v = to_dev(p.rowptr, dev), to_dev(p.colidx, dev), to_dev(p.vals, dev)
    xd, td = to_dev(x, dev), to_dev(th, dev)
    outs = [torch.zeros(1, dtype=torch.float64, device=dev) for _ in range(3)]
    log("rmse_noalloc three calls in a row on one stream")
    for o in outs:
        als.als_rmse_noalloc(0, rp, ci, v, p.m, p.n, 64, xd, td, o)
    torch.cuda.synchronize()
    vals = {np.float64(o.item()).tobytes() for o in outs}
    assert len(vals) == 1
    # empty matrix: 0
    z = torch.zeros(6, dtype=torch.int64, device=dev)
    als.als_rmse_noalloc(0, z, ci, v, 5, p.n, 64, xd, td, outs[0])
    torch.cuda.synchronize()
    assert outs[0].item() == 0.0
    lib = als._lib
    P = ctypes.c_void_p
    args = [P(rp.data_ptr()), P(ci.data_ptr()), P(v.data_ptr()), p.m, p.n, 64,
            P(xd.data_ptr()), P(td.data_ptr()), P(outs[1].data_ptr()), None]
    assert lib.als_rmse_noalloc(-1, *args) == -7
    assert lib.als_rmse_noalloc(4096, *args) == -7
    bad = list(args)
    bad[5] = 0
    assert lib.als_rmse_noalloc(0, *bad) == -2
    bad = list(args)
    bad[8] = P(outs[1].data_ptr() + 4)
    assert lib.als_rmse_noalloc(0, *bad) == -4
    bad = list(args)
    bad[0] = None
    assert lib.als_rmse_noalloc(0, *bad) == -1
