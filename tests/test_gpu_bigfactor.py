"""A gathered factor larger than 2 GiB at a small number of ratings.

Algorithm 1 reads theta_v for every rated column v of a row; the read-only factor it reads from
can exceed the 2 GiB range that one bounded buffer descriptor covers (the item side of the
Hugewiki-shaped workload gathers from a 20 GB X).  Here the factor is 3.1-3.2 GB while the
matrix holds only ~10^5 ratings, so the oracle checks every row in seconds: most columns lie
past the first 2 GiB of the factor, and a few rows rate only the factor's last columns.
Checked: the half-sweep per row (<= 1e-3 against the fp64 oracle), the training RMSE (1e-6
relative) and the gather stage bit for bit (als_gather_dump) on rows at the factor's end, the
quad-form operands included.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import log, row_rel_err, to_dev
from tests.test_gpu_gather import expected, quads

pytestmark = pytest.mark.gpu

BUFFER_RANGE = 0x7FFFF000   # bytes of factor one buffer descriptor serves


@pytest.fixture(scope="module")
def ctx():
    from paper_1603_03820_amd import als
    assert torch.cuda.is_available()
    return als.Context(0, 128)


def problem(n, f, seed):
    """Seeded lognormal rows over n columns (Zipf 0.3, so entries spread over the whole factor),
    plus handmade rows: one entry at the last column, 50 of the last 1,000 columns, an empty row,
    and 300 columns spread from the first to the last."""
    p = synth.make(2_000, n, 80_000, rows="lognormal", zipf=0.3, f=f, model="movie", plant_f=16,
                   seed=seed)
    rng = np.random.default_rng(seed)
    extra = [np.array([n - 1]),
             np.sort(n - 1000 + rng.choice(1000, 50, replace=False)),
             np.zeros(0, np.int64),
             np.sort(rng.choice(n, 300, replace=False))]
    lens = np.concatenate([np.diff(p.rowptr), [len(e) for e in extra]])
    rowptr = np.zeros(len(lens) + 1, np.int64)
    np.cumsum(lens, out=rowptr[1:])
    colidx = np.concatenate([p.colidx] + [e.astype(np.int32) for e in extra])
    vals = np.concatenate([p.vals, rng.uniform(1, 5, int(sum(len(e) for e in extra)))
                           .astype(np.float32)])
    theta = synth.normal(seed + 1, 8, (n, f), 0.3)
    return rowptr, colidx, vals, len(lens), theta


@pytest.mark.parametrize("f,n", [(100, 8_000_000), (128, 6_000_000)])
def test_factor_above_2gib(ctx, f, n):
    from paper_1603_03820_amd import als
    orc = oracle.get()
    assert 4 * n * f > BUFFER_RANGE
    rowptr, colidx, vals, m, theta = problem(n, f, 9100 + f)
    far = np.mean(colidx.astype(np.int64) * 4 * f >= (1 << 31))
    log(f"factor {4 * n * f / 2**30:.2f} GiB, n={n} f={f}, m={m}, nnz={int(rowptr[-1])}, "
        f"{100 * far:.0f}% of entries past 2 GiB")
    assert far > 0.2
    dev = ctx.device
    rp, ci, v = to_dev(rowptr, dev), to_dev(colidx, dev), to_dev(vals, dev)
    th = to_dev(theta, dev)
    x = torch.full((m, f), float("nan"), dtype=torch.float32, device=dev)
    log("half-sweep")
    als.als_half_sweep(ctx, rp, ci, v, m, n, f, 0.05, th, x)
    torch.cuda.synchronize()
    assert als.als_status(ctx) == 0
    xg = x.cpu().numpy()
    th64 = theta.astype(np.float64)
    xo, st = orc.half_sweep(rowptr, colidx, vals, m, n, f, 0.05, th64)
    assert not np.isnan(xg).any()
    err = row_rel_err(xg, xo)
    log(f"max row rel err {err.max():.3e}")
    assert err.max() <= 1e-3
    assert np.all(xg[m - 2] == 0.0)   # the empty row
    # training RMSE with this factor gathered (x: a synthetic row factor)
    xs = synth.normal(9200 + f, 8, (m, f), 0.3)
    log("rmse")
    got = float(als.als_rmse(ctx, rp, ci, v, m, n, f, to_dev(xs, dev), th).item())
    ref = orc.rmse(rowptr, colidx, vals, m, f, xs.astype(np.float64), th64)
    log(f"rmse gpu {got:.9f} oracle {ref:.9f}")
    assert abs(got - ref) <= 1e-6 * ref
    # the gather stage, bit for bit, on the rows at the factor's end and the spread row
    for u in (m - 4, m - 3, m - 1):
        k0, k1 = int(rowptr[u]), int(rowptr[u + 1])
        log(f"gather dump row {u} (n_u={k1 - k0})")
        got = als.als_gather_dump(ctx, rp, ci, v, m, n, f, th, u, k1 - k0)
        torch.cuda.synchronize()
        got = got.cpu().numpy()
        ref = expected(theta, colidx[k0:k1], vals[k0:k1], f, quads(f, "global"))
        bad = np.argwhere(got.view(np.uint32) != ref.view(np.uint32))
        assert bad.size == 0, f"row {u}: first mismatches {bad[:5].tolist()}"
