"""The seeded input generator (CPU only): Philox known answers, CSR well-formedness, shape
statistics, thread-count independence, and its transpose against the oracle's."""
import hashlib
import os
import subprocess
import sys

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_philox_known_answers():
    # known-answer vectors published with the Random123 library (philox4x32, 10 rounds)
    assert [hex(v) for v in synth.philox4x32_10([0, 0, 0, 0], [0, 0])] == \
        ["0x6627e8d5", "0xe169c58d", "0xbc57ac4c", "0x9b00dbd8"]
    assert [hex(v) for v in synth.philox4x32_10([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2)] == \
        ["0x408f276d", "0x41c83b0e", "0xa20bc7c6", "0x6d5451fd"]
    assert [hex(v) for v in synth.philox4x32_10(
        [0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0])] == \
        ["0xd16cfe09", "0x94fdcceb", "0x5001e420", "0x24126ea1"]


def _check_csr(p):
    rp, ci = p.rowptr, p.colidx
    assert rp[0] == 0 and rp[-1] == p.nnz and np.all(np.diff(rp) >= 0)
    assert ci.min() >= 0 and ci.max() < p.n
    d = np.diff(ci.astype(np.int64))
    starts = rp[1:-1]
    starts = starts[(starts > 0) & (starts < p.nnz)]
    mask = np.ones(p.nnz - 1, bool)
    mask[starts - 1] = False           # differences across row boundaries are free
    assert np.all(d[mask] > 0), "columns must be distinct and ascending within a row"
    assert np.all(np.isfinite(p.vals))


def test_tiny_config_well_formed():
    p = synth.config("tiny")
    assert (p.m, p.n, p.nnz, p.f) == (2000, 500, 50_000, 16)
    _check_csr(p)
    assert p.theta0.shape == (500, 16) and p.theta0.dtype == np.float32
    assert abs(p.theta0.std() - 0.01) < 5e-4 and abs(p.theta0.mean()) < 5e-4


def test_lognormal_rows_and_zipf_columns():
    p = synth.make(20_000, 3_000, 1_000_000, rows="lognormal", zipf=0.9, f=8, model="movie",
                   seed=123)
    _check_csr(p)
    cnt = np.diff(p.rowptr)
    assert cnt.min() >= 1 and cnt.max() <= p.n and cnt.sum() == 1_000_000
    # lognormal sigma = 1: the std of log-lengths is about 1 (clamping trims it a little)
    assert 0.85 < np.log(cnt).std() < 1.05
    # Zipf popularity: the most popular column is far above the mean column count
    col_cnt = np.bincount(p.colidx, minlength=p.n)
    assert col_cnt.max() > 20 * col_cnt.mean()
    assert np.all((p.vals >= 1.0) & (p.vals <= 5.0))


def test_transpose_matches_oracle(oracle_lib):
    p = synth.make(5_000, 700, 120_000, rows="lognormal", zipf=1.1, f=4, model="music", seed=7)
    a = synth.transpose(p.m, p.n, p.rowptr, p.colidx, p.vals)
    b = oracle_lib.transpose(p.rowptr, p.colidx, p.vals, p.m, p.n)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


_HASH_SNIPPET = r"""
import hashlib, sys
sys.path.insert(0, %r)
import synth
p = synth.make(30_000, 2_000, 900_000, rows="lognormal", zipf=1.0, f=8, model="wiki", seed=99)
h = hashlib.sha256()
for a in (p.rowptr, p.colidx, p.vals, p.theta0, *p.csc()):
    h.update(a.tobytes())
print(h.hexdigest())
"""


def test_independent_of_thread_count():
    outs = []
    for nt in ("1", "3"):
        env = dict(os.environ, OMP_NUM_THREADS=nt)
        r = subprocess.run([sys.executable, "-c", _HASH_SNIPPET % ROOT], env=env,
                           capture_output=True, text=True, check=True)
        outs.append(r.stdout.strip())
    assert outs[0] == outs[1]
