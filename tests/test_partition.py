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


@pytest.mark.parametrize("tiers", [1, 5])
@pytest.mark.parametrize("case", range(len(_cases())))
def test_partition_properties(oracle_lib, case, tiers):
    rowptr, W, c_nnz, c_row, q = _cases()[case]
    C = tiers * W   # tiers = 5: W large chunks, then 4 W small ones over the last T / 8
    m = len(rowptr) - 1
    bounds = oracle_lib.partition(rowptr, m, W, c_nnz, c_row, q, C=C, tail_div=8)
    assert bounds.shape == (C + 1, 2)
    assert tuple(bounds[0]) == (0, 0) and tuple(bounds[C]) == (m, 0)
    for b in range(C):
        assert tuple(bounds[b]) <= tuple(bounds[b + 1]), "boundaries must be monotone"
    nus = np.diff(rowptr)
    for u, kk in bounds[1:C]:
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
    # balance: each chunk's share of the cost axis is within one row cost plus one snap of its
    # tier's ideal size (T1 / W for the large chunks, T2 / (C - W) for the small ones)
    T = c_nnz * int(rowptr[-1]) + c_row * m
    T2 = T // 8 if C > W else 0
    T1 = T - T2
    ideal = np.array([T1 / W] * W + ([T2 / (C - W)] * (C - W) if C > W else []))
    cost = np.zeros(C)
    for w, u, ka, kb in portions(bounds, rowptr):
        cost[w] += c_nnz * (kb - ka) + (c_row if ka == 0 else 0)
    # each realised cut lies within c_row + c_nnz (q/2 + 1) of its ideal point s_b
    slack = 2 * (c_row + c_nnz * (q // 2 + 1))
    assert np.all(np.abs(cost - ideal) <= slack)


def test_single_tier_matches_equal_split(oracle_lib):
    # C = W: boundaries at floor(T b / W), the equal split
    rowptr = np.cumsum(np.r_[0, np.arange(1, 300) % 23]).astype(np.int64)
    a = oracle_lib.partition(rowptr, 299, 41, 16, 900, 64)
    b = oracle_lib.partition(rowptr, 299, 41, 16, 900, 64, C=41, tail_div=3)
    assert np.array_equal(a, b)
    # the large tier of a two-tier plan cuts T - floor(T/8) into W equal parts: where T / 8 is
    # a whole number of rows at the end, the first W boundaries equal an equal split of the rest
    rp = np.arange(0, 8 * 10 * 4 + 1, 4, dtype=np.int64)          # 80 rows of 4 entries
    two = oracle_lib.partition(rp, 80, 5, 16, 64, 2, C=15, tail_div=8)
    one = oracle_lib.partition(rp[:71], 70, 5, 16, 64, 2)          # first 70 rows = 7/8 of T
    assert np.array_equal(two[:6], one)
    assert tuple(two[15]) == (80, 0)


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


@pytest.mark.parametrize("tiers", [1, 5])
@pytest.mark.parametrize("W", [3, 17, 200, 2000])
def test_reducer_reads_exactly_the_stored_pieces(oracle_lib, W, tiers):
    # few entries per wave: many boundaries snap onto the same cut point
    rp = np.concatenate([[0], np.cumsum([3, 0, 5000, 1, 0, 300, 12000, 7, 900, 0, 4100])])
    rp = rp.astype(np.int64)
    bounds = oracle_lib.partition(rp, len(rp) - 1, W, 16, 16 * 60, 256, C=tiers * W)
    stored = writer_pieces(bounds, rp)
    read = reducer_pieces(bounds, rp)
    read_set = {(w, s): u for u, ps in read.items() for (w, s) in ps}
    assert read_set == stored
    for u, ps in read.items():
        assert [w for w, _ in ps] == sorted(w for w, _ in ps), "pieces summed in wave order"


def grouped_reduce(bounds, rowptr, G):
    """The two-pass reduce's view (groups of G boundary pieces for rows with more than G):
    returns (pass1, pass2), pass1: leader b -> (slots read in order, slot written),
    pass2: row -> slots read in order.  Slots are (chunk, 0|1) like writer_pieces."""
    m, C = len(rowptr) - 1, len(bounds) - 1

    def cuts(b):
        u, k = bounds[b]
        return u < m and 0 < k < rowptr[u + 1] - rowptr[u]

    runs = {}   # row -> consecutive boundaries cutting it
    for b in range(1, C):
        if cuts(b):
            runs.setdefault(int(bounds[b][0]), []).append(b)
    pass1, pass2 = {}, {}
    for u, bs in runs.items():
        assert bs == list(range(bs[0], bs[-1] + 1)), "cuts of one row are consecutive"
        nu = int(rowptr[u + 1] - rowptr[u])
        b_first, b_last = bs[0], bs[-1]

        def piece_slots(lo, hi):
            out = []
            for bb in range(lo, hi + 1):
                end = int(bounds[bb + 1][1]) if bb < b_last else nu
                if bounds[bb][1] < end:
                    out.append((bb, 0))
            return out

        first = (b_first - 1, 0 if bounds[b_first - 1][0] == u else 1)
        if len(bs) <= G:
            pass2[u] = [first] + piece_slots(b_first, b_last)
        else:
            reads = [first]
            for g in range(b_first, b_last + 1, G):
                pass1[g] = (piece_slots(g, min(g + G - 1, b_last)), (g, 0))
                reads.append((g, 0))
            pass2[u] = reads
    return pass1, pass2


@pytest.mark.parametrize("G", [1, 2, 16])
@pytest.mark.parametrize("W", [3, 17, 200, 2000])
def test_grouped_reduce_consumes_every_piece_once(oracle_lib, W, G):
    rp = np.concatenate([[0], np.cumsum([3, 0, 5000, 1, 0, 300, 12000, 7, 900, 0, 4100, 60000])])
    rp = rp.astype(np.int64)
    bounds = oracle_lib.partition(rp, len(rp) - 1, W, 16, 16 * 60, 256, C=5 * W)
    stored = writer_pieces(bounds, rp)
    pass1, pass2 = grouped_reduce(bounds, rp, G)
    written1 = {w for _, w in pass1.values()}
    consumed = []
    for reads, _ in pass1.values():
        consumed += reads
    for u, reads in pass2.items():
        consumed += [s for s in reads if s not in written1]
        # group sums are read in chunk order, after the first piece
        assert [c for c, _ in reads] == sorted(c for c, _ in reads)
    assert sorted(consumed) == sorted(stored), "every stored piece summed exactly once"
    for s_, u in stored.items():
        # a group slot only ever overwrites its own leader's piece, which it reads first
        if s_ in written1:
            reads, w = pass1[s_[0]]
            assert not reads or reads[0] == s_ or s_ not in reads
    for reads, w in pass1.values():
        assert [c for c, _ in reads] == sorted(c for c, _ in reads)
