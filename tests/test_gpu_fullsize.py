"""Full-size parity: the workloads at their full sizes, through the same calls bench.py times,
against the fp64 oracle on sampled rows (each sampled x_u is recomputed from its definition) and
on the training RMSE over every stored entry.

Rows sampled per side: the longest rows (the heaviest Grams, cut into the most chunk pieces),
random rows and empty rows.  Item-side inputs and RMSE factors are synthetic factors from the
generator, never GPU output.  The wiki shape runs at its full size, 50M x 40,000 with 3.1B
ratings: it alone has more than 2^31 entries (64-bit entry offsets, the device transpose's
column-relative positions) and an item-side factor X of 20 GB, past the 2 GiB range of one
buffer descriptor.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import log, row_rel_err, to_dev

pytestmark = pytest.mark.gpu

TOL = 1e-3


@pytest.fixture(scope="module")
def ctx():
    from paper_1603_03820_amd import als
    assert torch.cuda.is_available()
    return als.Context(0, 128)


@pytest.fixture(scope="module")
def orc():
    return oracle.get()


def sample_rows(rowptr, k_random, k_long, seed):
    cnt = np.diff(rowptr)
    rng = np.random.default_rng(seed)
    longest = np.argsort(cnt, kind="stable")[len(cnt) - k_long:]
    rand = rng.choice(len(cnt), size=min(k_random, len(cnt)), replace=False)
    empty = np.flatnonzero(cnt == 0)[:5]
    return np.unique(np.concatenate([longest, rand, empty])).astype(np.int64)


class Side:
    """One side of a workload: host CSR arrays and their device copies."""

    def __init__(self, rowptr, colidx, vals, m, n, dev, d=None):
        self.rowptr, self.colidx, self.vals, self.m, self.n = rowptr, colidx, vals, m, n
        self.d = d if d is not None else (to_dev(rowptr, dev), to_dev(colidx, dev),
                                          to_dev(vals, dev))


def check_side(ctx, orc, side, f, lam, theta, label, k_random=600, k_long=8, seed=1):
    from paper_1603_03820_amd import als
    dev = ctx.device
    log(f"{label}: half-sweep m={side.m} n={side.n} nnz={int(side.rowptr[-1])} f={f}")
    th = to_dev(np.ascontiguousarray(theta, np.float32).reshape(side.n, f), dev)
    x = torch.full((side.m, f), float("nan"), dtype=torch.float32, device=dev)
    als.als_half_sweep(ctx, *side.d, side.m, side.n, f, lam, th, x)
    torch.cuda.synchronize()
    assert not torch.isnan(x).any().item(), f"{label}: unwritten or NaN rows"
    assert als.als_status(ctx) == 0
    rows = sample_rows(side.rowptr, k_random, k_long, seed)
    xg = x[torch.from_numpy(rows).to(dev)].cpu().numpy()
    del x, th
    log(f"{label}: oracle on {len(rows)} sampled rows (longest {int(np.diff(side.rowptr).max())})")
    th64 = np.asarray(theta, np.float64).reshape(side.n, f)
    # in chunks (the oracle threads over a chunk's rows), logging after each: a row of tens of
    # millions of ratings takes the oracle about a minute
    order = np.argsort(-np.diff(side.rowptr)[rows], kind="stable")
    xo = np.empty((len(rows), f))
    for k in range(0, len(rows), 16):
        sel = order[k:k + 16]
        xc, st = orc.half_sweep(side.rowptr, side.colidx, side.vals, side.m, side.n, f, lam,
                                th64, rows=rows[sel])
        assert np.all(st == 0)
        xo[sel] = xc
        log(f"{label}: oracle rows {k + len(sel)}/{len(rows)}")
    err = row_rel_err(xg, xo)
    worst = int(np.argmax(err))
    log(f"{label}: max row rel err {err.max():.3e} (row {int(rows[worst])})")
    assert err.max() <= TOL, f"{label}: row {int(rows[worst])} rel err {err.max():.3e}"


def check_rmse(ctx, orc, side, f, x, theta, label):
    from paper_1603_03820_amd import als
    dev = ctx.device
    log(f"{label}: rmse over {int(side.rowptr[-1])} entries")
    xd = to_dev(np.ascontiguousarray(x, np.float32), dev)
    td = to_dev(np.ascontiguousarray(theta, np.float32), dev)
    got = float(als.als_rmse(ctx, *side.d, side.m, side.n, f, xd, td).item())
    ref = orc.rmse(side.rowptr, side.colidx, side.vals, side.m, f, x.astype(np.float64),
                   theta.astype(np.float64))
    log(f"{label}: rmse gpu {got:.9f} oracle {ref:.9f}")
    assert abs(got - ref) <= 1e-6 * max(1.0, ref)


def load(name, f=None, m_scale=1):
    log(f"generate {name} (f={f}, rows/{m_scale})")
    if m_scale == 1:
        p = synth.config(name, f=f)
    else:
        c = synth.CONFIGS[name]
        p = synth.make(c["m"] // m_scale, c["n"], c["nnz"] // m_scale, rows=c["rows"],
                       mean=c["mean"], zipf=c["zipf"], f=c["f"], lam=c["lam"], model=c["model"],
                       seed=c["seed"], name=f"{name}/{m_scale}")
    return p


@pytest.fixture(scope="module")
def movie(ctx):
    p = load("movie")
    colptr, rowidx, vt = p.csc()
    return p, Side(p.rowptr, p.colidx, p.vals, p.m, p.n, ctx.device), \
        Side(colptr, rowidx, vt, p.n, p.m, ctx.device)


def test_movie_full_size(ctx, orc, movie):
    p, user, item = movie
    check_side(ctx, orc, user, p.f, p.lam, p.theta0, "movie user", seed=11)
    xin = synth.normal(p.recipe["seed"], 8, (p.m, p.f), 0.3)
    check_side(ctx, orc, item, p.f, p.lam, xin, "movie item", seed=12)
    th = synth.normal(p.recipe["seed"] + 1, 8, (p.n, p.f), 0.3)
    check_rmse(ctx, orc, user, p.f, xin, th, "movie")


@pytest.mark.parametrize("f", [32, 64, 128])
def test_movie_rank_sweep_full_size(ctx, orc, movie, f):
    p, user, item = movie
    theta0 = synth.normal(synth.RANK_SWEEP_THETA_SEED, synth.THETA0_STREAM, (p.n, f),
                          synth.THETA0_STD)
    check_side(ctx, orc, user, f, p.lam, theta0, f"movie f={f} user", seed=20 + f)
    xin = synth.normal(p.recipe["seed"] + f, 8, (p.m, f), 1.0 / np.sqrt(f))
    check_side(ctx, orc, item, f, p.lam, xin, f"movie f={f} item", seed=21 + f)


def test_music_full_size(ctx, orc):
    p = load("music")
    user = Side(p.rowptr, p.colidx, p.vals, p.m, p.n, ctx.device)
    check_side(ctx, orc, user, p.f, p.lam, p.theta0, "music user", seed=31)
    colptr, rowidx, vt = p.csc()
    del user
    item = Side(colptr, rowidx, vt, p.n, p.m, ctx.device)
    xin = synth.normal(p.recipe["seed"], 8, (p.m, p.f), 0.3)
    check_side(ctx, orc, item, p.f, p.lam, xin, "music item", seed=32)


def test_wiki_full_size(ctx, orc):
    """Hugewiki-shaped (Table 5), full size: user side, the device transpose at 3.1B entries
    (bit-exact against the host transpose), item side (the 20 GB X gathered), and the RMSE
    summed over the CSC so that it gathers from the 20 GB factor too."""
    from paper_1603_03820_amd import als
    p = load("wiki")
    dev = ctx.device
    user = Side(p.rowptr, p.colidx, p.vals, p.m, p.n, dev)
    check_side(ctx, orc, user, p.f, p.lam, p.theta0, "wiki user", seed=41)
    log("wiki: device transpose of 3.1B entries")
    colptr, rowidx, vt = p.csc()
    dcsc = als.als_csr_to_csc(ctx, *user.d, p.m, p.n, nnz=p.nnz)
    torch.cuda.synchronize()
    same = (np.array_equal(dcsc[0].cpu().numpy(), colptr)
            and torch.equal(dcsc[1], to_dev(rowidx, dev))
            and torch.equal(dcsc[2].view(torch.int32), to_dev(vt.view(np.int32), dev)))
    log(f"wiki: device CSC equals the host transpose: {same}")
    assert same
    del user
    item = Side(colptr, rowidx, vt, p.n, p.m, dev, d=dcsc)
    xin = synth.normal(p.recipe["seed"], 8, (p.m, p.f), 0.3)
    # at full size the longest item rows hold up to 45M ratings, a minute or more each for the
    # oracle (it gathers from a 40 GB fp64 factor): the longest row and random rows
    check_side(ctx, orc, item, p.f, p.lam, xin, "wiki item", k_random=200, k_long=1, seed=42)
    th = synth.normal(p.recipe["seed"] + 1, 8, (p.n, p.f), 0.3)
    check_rmse_columns(ctx, orc, colptr, rowidx, vt, p.m, p.f, th, xin, seed=43,
                       label="wiki (columns, gathering from the 20 GB X)")


def check_rmse_columns(ctx, orc, colptr, rowidx, vt, m, f, th, xin, seed, label, k=60):
    """The RMSE over the ratings of k random columns, computed from the CSC side so that the
    GPU gathers x_u from the full m x f factor (row indices unchanged); the oracle sums the same
    entries with the rows renumbered onto the distinct rows they touch (the same terms)."""
    from paper_1603_03820_amd import als
    dev = ctx.device
    rng = np.random.default_rng(seed)
    cols = np.sort(rng.choice(len(colptr) - 1, size=k, replace=False))
    lens = colptr[cols + 1] - colptr[cols]
    sub_ptr = np.zeros(k + 1, np.int64)
    np.cumsum(lens, out=sub_ptr[1:])
    idx = np.concatenate([np.arange(colptr[c], colptr[c + 1]) for c in cols])
    sub_rows, sub_vals = rowidx[idx], vt[idx]
    log(f"{label}: rmse over {int(sub_ptr[-1])} entries of {k} columns")
    xd = to_dev(xin, dev)
    got = float(als.als_rmse(ctx, to_dev(sub_ptr, dev), to_dev(sub_rows, dev),
                             to_dev(sub_vals, dev), k, m, f, to_dev(th[cols], dev), xd).item())
    del xd
    uniq, inv = np.unique(sub_rows, return_inverse=True)
    ref = orc.rmse(sub_ptr, inv.astype(np.int32), sub_vals, k, f, th[cols].astype(np.float64),
                   xin[uniq].astype(np.float64))
    log(f"{label}: rmse gpu {got:.9f} oracle {ref:.9f}")
    assert abs(got - ref) <= 1e-6 * max(1.0, ref)
