"""Row-batched half-sweeps with R streamed from pinned host memory (NEXT row f2): against the
fp64 oracle and against the resident half-sweep, with batches small enough that there are many
of them and one row is longer than a batch."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import log, row_rel_err, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    from paper_1603_03820_amd import als
    assert torch.cuda.is_available()
    return als.Context(0, 128)


@pytest.mark.parametrize("f", [16, 100])
def test_streamed_half_sweeps_match_oracle(ctx, f):
    from paper_1603_03820_amd import als, stream
    orc = oracle.get()
    p = synth.make(6_000, 900, 400_000, rows="lognormal", zipf=0.9, f=f, model="movie",
                   plant_f=16, seed=71)
    colptr, rowidx, vt = p.csc()
    dev = ctx.device
    xin = synth.normal(72, 8, (p.m, f), 0.3)
    for side, (rp, ci, v, m, n, th) in {
            "user": (p.rowptr, p.colidx, p.vals, p.m, p.n, p.theta0),
            "item": (colptr, rowidx, vt, p.n, p.m, xin)}.items():
        longest = int(np.diff(rp).max())
        batch = max(longest // 2, 1)
        sw = stream.StreamedSweep(ctx, stream.HostCSR(rp, ci, v), n, f, batch)
        log(f"{side} f={f}: {len(sw.batches)} batches of <= {batch} ratings (longest row "
            f"{longest})")
        assert len(sw.batches) > 4
        assert any(int(rp[u1] - rp[u0]) > batch for u0, u1 in sw.batches)
        th_d = to_dev(np.ascontiguousarray(th, np.float32), dev)
        x = torch.full((m, f), float("nan"), device=dev)
        sw.half_sweep(p.lam, th_d, x)
        torch.cuda.synchronize()
        assert not torch.isnan(x).any().item()
        assert sw.h2d_bytes == 8 * (m + len(sw.batches)) + 8 * int(rp[-1])
        # the resident half-sweep of the same side
        xr = torch.full((m, f), float("nan"), device=dev)
        als.als_half_sweep(ctx, to_dev(rp, dev), to_dev(ci, dev), to_dev(v, dev), m, n, f,
                           p.lam, th_d, xr)
        torch.cuda.synchronize()
        xs, xrs = x.cpu().numpy(), xr.cpu().numpy()
        assert row_rel_err(xs, xrs.astype(np.float64)).max() <= 1e-4
        # against the oracle on the longest rows and a random sample
        rng = np.random.default_rng(f)
        rows = np.unique(np.concatenate([np.argsort(np.diff(rp))[-8:],
                                         rng.choice(m, 200, replace=False)])).astype(np.int64)
        xo, st = orc.half_sweep(rp, ci, v, m, n, f, p.lam, np.asarray(th, np.float64),
                                rows=rows)
        assert np.all(st == 0)
        err = row_rel_err(xs[rows], xo)
        log(f"{side} f={f}: streamed vs oracle max row rel err {err.max():.2e}")
        assert err.max() <= 1e-3
