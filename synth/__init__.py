"""Seeded synthetic ALS inputs shaped like the paper's workloads (experiments section, data-set
table: Netflix-, YahooMusic- and Hugewiki-shaped rating matrices).

The public data sets are not used: these generators stand in for their *shapes* only (m, n,
N_z, skewed row lengths, Zipf column popularity, planted low-rank ratings).  Both the fp64
oracle and the HIP path take their inputs from here; this module holds none of the ALS
arithmetic.  The C kernel (``synth.c``) is built into ``libsynth.so`` next to this file.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

BASE_SEED = 160303820

# Named workloads.  Shapes follow the paper's data-set table; the rating model, row-length law
# and Zipf exponent are this project's synthetic recipe.
CONFIGS = {
    # correctness-sized: the fp64 oracle runs ten iterations of it in seconds
    "tiny": dict(m=2_000, n=500, nnz=50_000, rows="uniform", mean=25.0, zipf=1.0, f=16,
                 lam=0.05, model="tiny", iters=10, seed=BASE_SEED + 1),
    # Netflix-shaped (480,189 x 17,770, 99M ratings, f=100, lambda=0.05)
    "movie": dict(m=480_000, n=17_770, nnz=100_000_000, rows="lognormal", mean=210.0, zipf=0.9,
                  f=100, lam=0.05, model="movie", iters=10, seed=BASE_SEED + 2),
    # YahooMusic-shaped (1,000,990 x 624,961, 252.8M ratings, f=100)
    "music": dict(m=1_000_000, n=625_000, nnz=250_000_000, rows="lognormal", mean=250.0,
                  zipf=1.1, f=100, lam=1.0, model="music", iters=10, seed=BASE_SEED + 3),
    # Hugewiki-shaped (50,082,603 x 39,780, 3.1B ratings, f=100, lambda=0.05)
    "wiki": dict(m=50_000_000, n=40_000, nnz=3_100_000_000, rows="lognormal", mean=62.0,
                 zipf=1.0, f=100, lam=0.05, model="wiki", iters=5, seed=BASE_SEED + 4),
}
# the rank sweep reuses the movie-shaped matrix with a fresh initial factor per f
RANK_SWEEP_F = (32, 64, 128)
RANK_SWEEP_THETA_SEED = BASE_SEED + 5

_MODELS = {"tiny": 0, "movie": 1, "music": 2, "wiki": 3}
_ROWS = {"uniform": 0, "lognormal": 1}
THETA0_STREAM = 7
THETA0_STD = 0.01
SPLIT_STREAM = 9   # held-out test split (stream 8 draws test factors)


def build(force: bool = False) -> str:
    """Compile libsynth.so (gcc, OpenMP)."""
    src = os.path.join(_HERE, "synth.c")
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(src):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11",
                               "-Wall", "-Wno-unknown-pragmas", src, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i64, i32, u64, u32, dbl = (ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64,
                                   ctypes.c_uint32, ctypes.c_double)
        lib.synth_row_counts.argtypes = [ctypes.c_int, i64, i64, i64, dbl, dbl, u64, P]
        lib.synth_columns.argtypes = [i64, i64, dbl, u64, P, P]
        lib.synth_values.argtypes = [ctypes.c_int, i64, i64, i32, u64, P, P, P]
        lib.synth_normal.argtypes = [u64, u32, i64, dbl, P]
        lib.synth_transpose.argtypes = [i64, i64, P, P, P, P, P, P]
        lib.synth_philox4x32_10.argtypes = [P, P, P]
        lib.synth_split_mask.argtypes = [u64, u32, i64, u32, P]
        for fn in ("synth_row_counts", "synth_columns", "synth_values", "synth_normal",
                   "synth_transpose", "synth_split_mask"):
            getattr(lib, fn).restype = ctypes.c_int
        lib.synth_philox4x32_10.restype = None
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def _check(rc: int, what: str):
    if rc != 0:
        raise RuntimeError(f"synth: {what} failed with code {rc}")


def philox4x32_10(ctr, key):
    """One Philox4x32-10 block (exposed for its known-answer test)."""
    c = np.asarray(ctr, dtype=np.uint32)
    k = np.asarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    _load().synth_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


@dataclass
class Problem:
    """A rating matrix in CSR (plus its CSC on demand) and an initial factor for update-X."""
    name: str
    m: int
    n: int
    f: int
    lam: float
    iters: int
    rowptr: np.ndarray   # int64 [m+1]
    colidx: np.ndarray   # int32 [nnz], ascending within a row
    vals: np.ndarray     # float32 [nnz]
    theta0: np.ndarray   # float32 [n, f], N(0, 0.01^2)
    recipe: dict = field(default_factory=dict)
    _csc: tuple | None = None

    @property
    def nnz(self) -> int:
        return int(self.rowptr[-1])

    def csc(self):
        """(colptr int64[n+1], rowidx int32[nnz], vals float32[nnz]), rows ascending per column."""
        if self._csc is None:
            self._csc = transpose(self.m, self.n, self.rowptr, self.colidx, self.vals)
        return self._csc


def row_counts(kind: str, m: int, n: int, nnz: int, mean: float, seed: int, sigma: float = 1.0):
    rowptr = np.zeros(m + 1, dtype=np.int64)
    _check(_load().synth_row_counts(_ROWS[kind], m, n, nnz, mean, sigma, seed, _ptr(rowptr)),
           "row_counts")
    return rowptr


def columns(m: int, n: int, zipf: float, seed: int, rowptr: np.ndarray):
    colidx = np.empty(int(rowptr[-1]), dtype=np.int32)
    _check(_load().synth_columns(m, n, zipf, seed, _ptr(rowptr), _ptr(colidx)), "columns")
    return colidx


def values(model: str, m: int, n: int, fp: int, seed: int, rowptr, colidx):
    vals = np.empty(int(rowptr[-1]), dtype=np.float32)
    _check(_load().synth_values(_MODELS[model], m, n, fp, seed, _ptr(rowptr), _ptr(colidx),
                                _ptr(vals)), "values")
    return vals


def normal(seed: int, stream: int, shape, std: float):
    out = np.empty(shape, dtype=np.float32)
    _check(_load().synth_normal(seed, stream, out.size, std, _ptr(out)), "normal")
    return out


def split(rowptr, colidx, vals, frac: float, seed: int):
    """Seeded held-out split of the stored entries: entry k is a test entry iff Philox word
    (seed, SPLIT_STREAM, k) < frac * 2^32.  Returns (train, test), each a CSR triple
    (rowptr int64, colidx int32, vals float32) over the same m rows, entries in their original
    order; the two are disjoint and together hold every entry."""
    nnz = int(rowptr[-1])
    if not 0.0 <= frac < 1.0:
        raise ValueError("frac must lie in [0, 1)")
    mask = np.empty(nnz, dtype=np.uint8)
    thr = min(int(round(frac * 2.0 ** 32)), 2 ** 32 - 1)
    _check(_load().synth_split_mask(seed, SPLIT_STREAM, nnz, thr, _ptr(mask)), "split")
    test = mask.view(bool)
    lens = np.diff(rowptr)
    n_test = np.zeros(len(lens), dtype=np.int64)
    nonempty = lens > 0
    if nnz:
        # per-row sums over [rowptr[u], rowptr[u+1]) (reduceat is wrong on empty rows: masked)
        n_test[nonempty] = np.add.reduceat(mask, rowptr[:-1][nonempty], dtype=np.int64)

    def csr(counts, sel):
        ptr = np.zeros(len(rowptr), dtype=np.int64)
        np.cumsum(counts, out=ptr[1:])
        return ptr, colidx[sel], vals[sel]

    return csr(lens - n_test, ~test), csr(n_test, test)


def transpose(m: int, n: int, rowptr, colidx, vals):
    nnz = int(rowptr[-1])
    colptr = np.zeros(n + 1, dtype=np.int64)
    rowidx = np.empty(nnz, dtype=np.int32)
    vt = np.empty(nnz, dtype=np.float32)
    _check(_load().synth_transpose(m, n, _ptr(rowptr), _ptr(colidx), _ptr(vals), _ptr(colptr),
                                   _ptr(rowidx), _ptr(vt)), "transpose")
    return colptr, rowidx, vt


def make(m: int, n: int, nnz: int, *, rows: str = "lognormal", mean: float | None = None,
         zipf: float = 1.0, f: int = 16, lam: float = 0.05, model: str = "movie",
         plant_f: int | None = None, seed: int = BASE_SEED, theta_seed: int | None = None,
         iters: int = 10, name: str = "custom") -> Problem:
    """Generate a problem with an explicit shape (scaled-down workloads for parity tests)."""
    if mean is None:
        mean = nnz / m
    plant_f = plant_f or f
    rowptr = row_counts(rows, m, n, nnz, mean, seed)
    colidx = columns(m, n, zipf, seed, rowptr)
    vals = values(model, m, n, plant_f, seed, rowptr, colidx)
    theta0 = normal(seed if theta_seed is None else theta_seed, THETA0_STREAM, (n, f), THETA0_STD)
    recipe = dict(m=m, n=n, nnz=nnz, rows=rows, mean=mean, zipf=zipf, f=f, lam=lam, model=model,
                  plant_f=plant_f, seed=seed, theta_seed=theta_seed)
    return Problem(name, m, n, f, lam, iters, rowptr, colidx, vals, theta0, recipe)


def config(name: str, f: int | None = None) -> Problem:
    """A named workload; ``f`` other than the config's own selects a rank-sweep initial factor."""
    c = CONFIGS[name]
    ff = c["f"] if f is None else f
    theta_seed = None if ff == c["f"] else RANK_SWEEP_THETA_SEED
    p = make(c["m"], c["n"], c["nnz"], rows=c["rows"], mean=c["mean"], zipf=c["zipf"], f=ff,
             lam=c["lam"], model=c["model"], plant_f=c["f"], seed=c["seed"],
             theta_seed=theta_seed, iters=c["iters"], name=name if ff == c["f"] else f"{name}_f{ff}")
    return p
