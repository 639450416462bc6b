"""GPU parity of als_csr_to_csc (the R -> R^T transpose the update-Theta half-sweep reads, eq. 3):
bit-exact against the oracle's stable counting-sort transpose on the same seeded inputs, including
empty rows and columns, rows longer than a wave, small row-block counts forced by a small
workspace, the workspace error, skipped out-of-range columns, and the full movie shape."""
import numpy as np
import pytest
import torch

import synth
from tests.gpu_util import log, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    from paper_1603_03820_amd import als
    assert torch.cuda.is_available()
    return als.Context(0, 128)


@pytest.fixture(scope="module")
def orc():
    import oracle
    return oracle.get()


def gpu_transpose(ctx, rowptr, colidx, vals, m, n):
    from paper_1603_03820_amd import als
    dev = ctx.device
    cp, ri, vt = als.als_csr_to_csc(ctx, to_dev(rowptr, dev), to_dev(colidx, dev),
                                    to_dev(vals, dev), m, n, nnz=int(rowptr[-1]))
    torch.cuda.synchronize()
    return cp.cpu().numpy(), ri.cpu().numpy(), vt.cpu().numpy()


def assert_same(got, ref, label):
    for name, a, b in zip(("colptr", "rowidx", "vals"), got, ref):
        assert a.shape == b.shape, f"{label}: {name} shape {a.shape} vs {b.shape}"
        if a.dtype == np.float32:
            assert np.array_equal(a.view(np.uint32), np.asarray(b, np.float32).view(np.uint32)), \
                f"{label}: {name} differs"
        else:
            assert np.array_equal(a, b), f"{label}: {name} differs at {np.flatnonzero(a != b)[:5]}"


def random_csr(m, n, seed, p_empty_row=0.1, long_rows=()):
    rng = np.random.default_rng(seed)
    counts = rng.integers(0, min(n, 40) + 1, size=m)
    counts[rng.random(m) < p_empty_row] = 0
    for u, c in long_rows:
        counts[u] = c
    rowptr = np.zeros(m + 1, np.int64)
    rowptr[1:] = np.cumsum(counts)
    def row_cols(c):
        if n <= 100_000:
            return np.sort(rng.choice(n, size=c, replace=False))
        cols = np.unique(rng.integers(0, n, size=2 * c + 8))   # distinct, ascending
        return np.sort(rng.permutation(cols)[:c])
    colidx = np.concatenate([row_cols(c) for c in counts]
                            or [np.zeros(0, np.int64)]).astype(np.int32)
    vals = rng.standard_normal(rowptr[-1]).astype(np.float32)
    return rowptr, colidx, vals


def test_tiny_config(ctx, orc):
    p = synth.config("tiny")
    log(f"transpose tiny m={p.m} n={p.n} nnz={p.nnz}")
    got = gpu_transpose(ctx, p.rowptr, p.colidx, p.vals, p.m, p.n)
    assert_same(got, orc.transpose(p.rowptr, p.colidx, p.vals, p.m, p.n), "tiny")


@pytest.mark.parametrize("m,n,seed", [(3000, 700, 1), (1, 1, 2), (500, 1, 3), (257, 5000, 4)])
def test_ragged_with_empty_rows_and_columns(ctx, orc, m, n, seed):
    long_rows = [(0, min(n, 300)), (m - 1, min(n, 129))] if n >= 129 else [(0, n)]
    rowptr, colidx, vals = random_csr(m, n, seed, long_rows=long_rows)
    log(f"transpose ragged m={m} n={n} nnz={int(rowptr[-1])}")
    got = gpu_transpose(ctx, rowptr, colidx, vals, m, n)
    assert_same(got, orc.transpose(rowptr, colidx, vals, m, n), f"ragged {m}x{n}")


def test_round_trip_is_identity(ctx):
    rowptr, colidx, vals = random_csr(2000, 900, 7)
    log("transpose round trip 2000 x 900")
    cp, ri, vt = gpu_transpose(ctx, rowptr, colidx, vals, 2000, 900)
    rp2, ci2, v2 = gpu_transpose(ctx, cp, ri, vt, 900, 2000)
    assert np.array_equal(rp2, rowptr) and np.array_equal(ci2, colidx)
    assert np.array_equal(v2.view(np.uint32), vals.view(np.uint32))


def test_empty_inputs(ctx):
    log("transpose empty inputs")
    cp, ri, vt = gpu_transpose(ctx, np.zeros(1, np.int64), np.zeros(0, np.int32),
                               np.zeros(0, np.float32), 0, 6)
    assert np.array_equal(cp, np.zeros(7, np.int64)) and ri.size == 0 and vt.size == 0
    # an m x n matrix with m, n > 0 and no entries: index and value arrays of one unused element
    cp, ri, vt = gpu_transpose(ctx, np.zeros(5, np.int64), np.zeros(1, np.int32),
                               np.zeros(1, np.float32), 4, 3)
    assert np.array_equal(cp, np.zeros(4, np.int64)) and ri.size == 0
    cp, ri, vt = gpu_transpose(ctx, np.zeros(4, np.int64), np.zeros(0, np.int32),
                               np.zeros(0, np.float32), 3, 0)
    assert np.array_equal(cp, np.zeros(1, np.int64))


def test_few_row_blocks_from_a_small_workspace(orc):
    """A context sized for f_max = 1 holds few per-column counters: many columns leave room for
    only a couple of row blocks, and too many columns for even one is ALS_ERR_WORKSPACE."""
    from paper_1603_03820_amd import als
    small = als.Context(0, 1)
    avail = small.workspace.numel()
    n = max(1000, avail // 4 // 3)   # about 3 row blocks of counters fit
    rowptr, colidx, vals = random_csr(4000, n, 11)
    log(f"transpose with small workspace ({avail} B) m=4000 n={n} nnz={int(rowptr[-1])}")
    got = gpu_transpose(small, rowptr, colidx, vals, 4000, n)
    assert_same(got, orc.transpose(rowptr, colidx, vals, 4000, n), "small workspace")
    big_n = avail // 4 + 1024
    with pytest.raises(als.ALSError) as e:
        dev = small.device
        als.als_csr_to_csc(small, to_dev(rowptr, dev), to_dev(colidx, dev), to_dev(vals, dev),
                           4000, big_n, nnz=int(rowptr[-1]))
    assert e.value.code == -3
    small.close()


def test_out_of_range_columns_are_skipped(ctx, orc):
    rowptr, colidx, vals = random_csr(300, 50, 13, p_empty_row=0.0)
    bad = colidx.copy()
    bad[::7] = 50 + (np.arange(bad[::7].size) % 3)      # columns n, n+1, n+2
    bad[3::11] = -1
    keep = (bad >= 0) & (bad < 50)
    row_of = np.repeat(np.arange(300), np.diff(rowptr))
    counts = np.bincount(row_of[keep], minlength=300)
    rp_ok = np.zeros_like(rowptr)
    rp_ok[1:] = np.cumsum(counts)
    ref = orc.transpose(rp_ok, bad[keep], vals[keep], 300, 50)
    log("transpose with out-of-range columns")
    from paper_1603_03820_amd import als
    dev = ctx.device
    nnz_ok = int(keep.sum())
    out = (torch.empty(51, dtype=torch.int64, device=dev),
           torch.full((int(rowptr[-1]),), -7, dtype=torch.int32, device=dev),
           torch.zeros(int(rowptr[-1]), dtype=torch.float32, device=dev))
    cp, ri, vt = als.als_csr_to_csc(ctx, to_dev(rowptr, dev), to_dev(bad, dev), to_dev(vals, dev),
                                    300, 50, nnz=int(rowptr[-1]), out=out)
    torch.cuda.synchronize()
    got = (cp.cpu().numpy(), ri.cpu().numpy()[:nnz_ok], vt.cpu().numpy()[:nnz_ok])
    assert_same(got, ref, "skipped columns")
    assert np.all(ri.cpu().numpy()[nnz_ok:] == -7)     # nothing written past colptr[n]


def test_movie_shape_full_size(ctx, orc):
    p = synth.config("movie")
    log(f"transpose movie m={p.m} n={p.n} nnz={p.nnz}")
    got = gpu_transpose(ctx, p.rowptr, p.colidx, p.vals, p.m, p.n)
    log("transpose movie: oracle")
    assert_same(got, orc.transpose(p.rowptr, p.colidx, p.vals, p.m, p.n), "movie")
    log("transpose movie: back")
    rp2, ci2, v2 = gpu_transpose(ctx, *got, p.n, p.m)
    assert np.array_equal(rp2, p.rowptr) and np.array_equal(ci2, p.colidx)
    assert np.array_equal(v2.view(np.uint32), p.vals.view(np.uint32))
