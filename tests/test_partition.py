"""The work partition that the HIP path uses to balance rows across waves (CPU only).

The oracle restates the partition from its definition; these tests pin that restatement to
properties any correct partition must have: every stored entry goes to exactly one worker,
every row (empty ones included) is finished exactly once, boundaries are monotone, cut points
sit on the snapping grid, and no worker's cost strays far from T/W."""
import random

import numpy as np
import pytest

from tests import pins


def portions(bounds, rowptr):
    """Expand worker boundaries into (worker, row, k_begin, k_end) pieces, the way each wave
    walks its range: rows u0..u1, the first from k0, the last (u1) up to k1 when k1 > 0."""
    out = []
    m = len(rowptr) - 1
    for w in range(len(bounds) - 1):
        (u0, k0), (u1, k1) = bounds[w], bounds[w + 1]
        u = u0
        while u <= u1 and u < m:
            nu = int(rowptr[u + 1] - rowptr[u])
            ka = k0 if u == u0 else 0
            if u == u1:
                if k1 == 0:
                    break
                kb = k1
            else:
                kb = nu
            if ka < kb or (nu == 0 and ka == 0):
                out.append((w, u, ka, kb))
            u += 1
    return out


def _cases():
    rng = random.Random(3)
    cases = []
    for t in range(10):
        m = rng.randint(1, 60)
        n = rng.randint(1, 900)
        rowptr, _, _ = pins.random_csr(rng, m, n, rng.choice([0.0, 0.01, 0.2, 0.9]))
        cases.append((rowptr, rng.randint(1, 40), rng.randint(1, 20), rng.randint(1, 300),
                      rng.choice([2, 4, 64, 256])))
    # heavy-tailed: a few huge rows among short ones, many workers
    rp = np.concatenate([[0], np.cumsum([3, 0, 5000, 1, 0, 0, 12000, 7, 300, 0])]).astype(np.int64)
    cases.append((rp, 64, 16, 16 * 100, 256))
    cases.append((np.zeros(5, np.int64), 8, 16, 1600, 256))  # all rows empty
    return cases


@pytest.mark.parametrize("case", range(len(_cases())))
def test_partition_properties(oracle_lib, case):
    rowptr, W, c_nnz, c_row, q = _cases()[case]
    m = len(rowptr) - 1
    bounds = oracle_lib.partition(rowptr, m, W, c_nnz, c_row, q)
    assert tuple(bounds[0]) == (0, 0) and tuple(bounds[W]) == (m, 0)
    for b in range(W):
        assert tuple(bounds[b]) <= tuple(bounds[b + 1]), "boundaries must be monotone"
    nus = np.diff(rowptr)
    for u, kk in bounds[1:W]:
        if u < m:
            assert 0 <= kk <= nus[u]
            assert kk == nus[u] or kk % q == 0
            assert kk == 0 or kk == nus[u] or nus[u] - kk >= q // 2
    # coverage: every entry exactly once, every row finished exactly once
    seen = np.zeros(int(rowptr[-1]), np.int64)
    pieces_per_row = np.zeros(m, np.int64)
    for w, u, ka, kb in portions(bounds, rowptr):
        seen[rowptr[u] + ka: rowptr[u] + kb] += 1
        pieces_per_row[u] += 1
    assert np.all(seen == 1)
    assert np.all(pieces_per_row >= 1)
    assert np.all(pieces_per_row[nus == 0] == 1), "an empty row must be written exactly once"
    # balance: each worker's share of the cost axis is within one row cost plus one snap of T/W
    T = c_nnz * int(rowptr[-1]) + c_row * m
    cost = np.zeros(W)
    for w, u, ka, kb in portions(bounds, rowptr):
        cost[w] += c_nnz * (kb - ka) + (c_row if ka == 0 else 0)
    # each realised cut lies within c_row + c_nnz (q/2 + 1) of its ideal point s_b
    slack = 2 * (c_row + c_nnz * (q // 2 + 1))
    assert np.all(np.abs(cost - T / W) <= slack)


def test_partition_is_pure_integer_and_deterministic(oracle_lib):
    rowptr = np.cumsum(np.r_[0, np.arange(1, 400) % 37]).astype(np.int64)
    a = oracle_lib.partition(rowptr, 399, 97, 16, 1760, 256)
    b = oracle_lib.partition(rowptr, 399, 97, 16, 1760, 256)
    assert a.dtype == np.int64 and np.array_equal(a, b)


def reducer_pieces(bounds, rowptr):
    """The second pass's view: for each boundary that first cuts a row, the (wave, slot) pieces
    it sums, as the reduce kernel selects them (slot 0 = a wave's first piece, 1 = its last)."""
    m, W = len(rowptr) - 1, len(bounds) - 1

    def cuts(b):
        u, k = bounds[b]
        return u < m and 0 < k < rowptr[u + 1] - rowptr[u]

    out = {}
    for b in range(1, W):
        if not cuts(b):
            continue
        u = int(bounds[b][0])
        if b > 1 and cuts(b - 1) and bounds[b - 1][0] == u:
            continue
        nu = int(rowptr[u + 1] - rowptr[u])
        pieces = [(b - 1, 0 if bounds[b - 1][0] == u else 1)]
        bb = b
        while True:
            more = bb + 1 < W and cuts(bb + 1) and bounds[bb + 1][0] == u
            end = int(bounds[bb + 1][1]) if more else nu
            if bounds[bb][1] < end:
                pieces.append((bb, 0))
            if not more:
                break
            bb += 1
        out[u] = pieces
    return out


def writer_pieces(bounds, rowptr):
    """What the first pass stores: (wave, slot) -> row, for every piece that is not a whole row."""
    m = len(rowptr) - 1
    stored = {}
    for w, u, ka, kb in portions(bounds, rowptr):
        nu = int(rowptr[u + 1] - rowptr[u])
        if ka == 0 and kb == nu:
            continue
        slot = 0 if u == bounds[w][0] else 1
        assert (w, slot) not in stored
        stored[(w, slot)] = u
    return stored


@pytest.mark.parametrize("W", [3, 17, 200, 2000])
def test_reducer_reads_exactly_the_stored_pieces(oracle_lib, W):
    # few entries per wave: many boundaries snap onto the same cut point
    rp = np.concatenate([[0], np.cumsum([3, 0, 5000, 1, 0, 300, 12000, 7, 900, 0, 4100])])
    rp = rp.astype(np.int64)
    bounds = oracle_lib.partition(rp, len(rp) - 1, W, 16, 16 * 60, 256)
    stored = writer_pieces(bounds, rp)
    read = reducer_pieces(bounds, rp)
    read_set = {(w, s): u for u, ps in read.items() for (w, s) in ps}
    assert read_set == stored
    for u, ps in read.items():
        assert [w for w, _ in ps] == sorted(w for w, _ in ps), "pieces summed in wave order"
