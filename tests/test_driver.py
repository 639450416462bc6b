"""The driver's host-side parts (CPU only): the seeded held-out split and the checkpoint file
format."""
import numpy as np
import pytest
import torch

import synth


def _rows(rowptr):
    return np.repeat(np.arange(len(rowptr) - 1), np.diff(rowptr))


@pytest.mark.parametrize("frac", [0.0, 0.1, 0.5])
def test_split_partitions_the_entries(frac):
    p = synth.config("tiny")
    (tr, te) = synth.split(p.rowptr, p.colidx, p.vals, frac, 11)
    for ptr, ci, v in (tr, te):
        assert ptr[0] == 0 and np.all(np.diff(ptr) >= 0) and len(ptr) == p.m + 1
        assert ci.dtype == np.int32 and v.dtype == np.float32 and len(ci) == ptr[-1]
        # columns stay ascending within each row (entries keep their order)
        r = _rows(ptr)
        same = r[1:] == r[:-1]
        assert np.all(ci[1:][same] > ci[:-1][same])
    assert tr[0][-1] + te[0][-1] == p.nnz
    # every (row, column, value) lands in exactly one side
    whole = set(zip(_rows(p.rowptr).tolist(), p.colidx.tolist(), p.vals.tolist()))
    a = list(zip(_rows(tr[0]).tolist(), tr[1].tolist(), tr[2].tolist()))
    b = list(zip(_rows(te[0]).tolist(), te[1].tolist(), te[2].tolist()))
    assert set(a) | set(b) == whole and not set(a) & set(b)
    if frac == 0.0:
        assert te[0][-1] == 0
    else:
        assert abs(te[0][-1] / p.nnz - frac) < 0.02


def test_split_is_seeded():
    p = synth.config("tiny")
    a = synth.split(p.rowptr, p.colidx, p.vals, 0.2, 5)[1]
    b = synth.split(p.rowptr, p.colidx, p.vals, 0.2, 5)[1]
    c = synth.split(p.rowptr, p.colidx, p.vals, 0.2, 6)[1]
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    assert not np.array_equal(a[1], c[1])


def test_split_with_empty_rows():
    rowptr = np.array([0, 0, 3, 3, 5, 5], dtype=np.int64)
    colidx = np.array([0, 2, 4, 1, 3], dtype=np.int32)
    vals = np.arange(5, dtype=np.float32)
    (tr, te) = synth.split(rowptr, colidx, vals, 0.5, 3)
    assert tr[0][-1] + te[0][-1] == 5
    assert np.all(np.diff(tr[0])[[0, 2, 4]] == 0) and np.all(np.diff(te[0])[[0, 2, 4]] == 0)


def test_checkpoint_round_trip_host(tmp_path):
    from paper_1603_03820_amd import driver
    x = torch.randn(37, 5)
    th = torch.randn(11, 5)
    ck = driver.AsyncCheckpointer(str(tmp_path), x, th)
    ck.save(3, x, th)
    ck.save(7, x * 2, th * 2)
    ck.wait()
    it, x7, th7 = driver.load_checkpoint(str(tmp_path), "cpu")
    assert it == 7 and torch.equal(x7, x * 2) and torch.equal(th7, th * 2)
    it, x3, th3 = driver.load_checkpoint(str(tmp_path), "cpu", iteration=3)
    assert it == 3 and torch.equal(x3, x) and torch.equal(th3, th)
    assert not list(tmp_path.glob("*.tmp"))


@pytest.mark.parametrize("batch", [1, 7, 60, 10**9])
def test_stream_batches_cover_whole_rows(batch):
    from paper_1603_03820_amd import stream
    p = synth.make(500, 80, 20_000, rows="lognormal", zipf=0.9, f=8, model="movie", seed=5)
    rp = p.rowptr.copy()
    rp[1:] += 0   # (copy: the plan must not modify its input)
    b = stream.plan_batches(p.rowptr, batch)
    assert np.array_equal(rp, p.rowptr)
    assert b[0][0] == 0 and b[-1][1] == p.m
    assert all(u1 > u0 for u0, u1 in b) and all(b[i][1] == b[i + 1][0] for i in range(len(b) - 1))
    for u0, u1 in b:
        ne = int(p.rowptr[u1] - p.rowptr[u0])
        assert ne <= batch or u1 == u0 + 1
        # maximal: the next row would not have fit
        if u1 < p.m:
            assert int(p.rowptr[u1 + 1] - p.rowptr[u0]) > batch


def test_stream_batches_with_empty_rows():
    from paper_1603_03820_amd import stream
    rowptr = np.array([0, 0, 0, 5, 5, 6, 6], dtype=np.int64)
    b = stream.plan_batches(rowptr, 3)
    assert b[0][0] == 0 and b[-1][1] == 6
    assert all(b[i][1] == b[i + 1][0] for i in range(len(b) - 1))
