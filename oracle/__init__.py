"""ORACLE -- test infrastructure only.

Python face of the plain fp64 CPU oracle in ``oracle.c`` (one ALS half-sweep per the paper's
eq. 2/3 and Algorithm 1, RMSE, the cost function J of eq. 1, CSR->CSC, and a restatement of
the HIP path's work partition).  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package; the HIP library never does.

``build()`` compiles ``liboracle.so`` (gcc -O2, IEEE, no fast-math, OpenMP over rows) and the
planted-mistake variants ``_mutants/liboracle_m<k>.so`` used to show that the pins bite.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")
MUTANT_DIR = os.path.join(_HERE, "_mutants")
MUTANTS = {
    1: "plain lambda*I instead of lambda*n_u*I",
    2: "right-hand side drops the rating",
    3: "Gram matrix uses the wrong index",
    4: "wrong sign in forward substitution",
    5: "back substitution with L instead of L^T",
    6: "RMSE averaged over rows instead of entries",
    7: "regulariser of J not weighted by n_u, n_v",
    8: "transpose not stable",
}

ROW_OK, ROW_EMPTY, ROW_NOT_SPD = 0, 1, 2


def _compile(out: str, defines=()):
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=gnu11", "-Wall",
           "-Wno-unknown-pragmas", *[f"-D{d}" for d in defines], _SRC, "-o", tmp, "-lm"]
    subprocess.check_call(cmd)
    os.replace(tmp, out)


def _stale(path: str) -> bool:
    return not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC)


def build(force: bool = False, mutants: bool = True) -> str:
    if force or _stale(LIB_PATH):
        _compile(LIB_PATH)
    if mutants:
        os.makedirs(MUTANT_DIR, exist_ok=True)
        for k in MUTANTS:
            p = os.path.join(MUTANT_DIR, f"liboracle_m{k}.so")
            if force or _stale(p):
                _compile(p, [f"ORACLE_MUTANT={k}"])
    return LIB_PATH


class Oracle:
    """ctypes wrapper around one build of oracle.c (the real one, or a planted mutant)."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        P, i64, i32, dbl = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double
        lib.oracle_half_sweep.argtypes = [P, P, P, i64, i64, i32, dbl, P, P, i64, P, P]
        lib.oracle_half_sweep.restype = ctypes.c_int
        lib.oracle_rmse.argtypes = [P, P, P, i64, i32, P, P]
        lib.oracle_rmse.restype = dbl
        lib.oracle_objective.argtypes = [P, P, P, i64, i64, i32, dbl, P, P]
        lib.oracle_objective.restype = dbl
        lib.oracle_transpose.argtypes = [P, P, P, i64, i64, P, P, P]
        lib.oracle_transpose.restype = ctypes.c_int
        lib.oracle_partition.argtypes = [P, i64, i64, i64, i64, i64, i64, i64, P]
        lib.oracle_partition.restype = ctypes.c_int
        lib.oracle_threads.argtypes = []
        lib.oracle_threads.restype = ctypes.c_int
        lib.oracle_set_threads.argtypes = [ctypes.c_int]
        lib.oracle_set_threads.restype = None
        self._lib = lib

    def threads(self) -> int:
        """OpenMP threads the oracle's row loops use."""
        return int(self._lib.oracle_threads())

    def set_threads(self, n: int) -> None:
        """Use n threads in later calls (from this thread)."""
        self._lib.oracle_set_threads(int(n))

    @staticmethod
    def _p(a):
        return ctypes.c_void_p(a.ctypes.data) if a is not None else None

    def half_sweep(self, rowptr, colidx, vals, m, n, f, lam, theta, rows=None):
        """x (fp64, [m or len(rows), f]) and per-row status for one half-sweep."""
        rowptr = np.ascontiguousarray(rowptr, dtype=np.int64)
        colidx = np.ascontiguousarray(colidx, dtype=np.int32)
        vals = np.ascontiguousarray(vals, dtype=np.float32)
        theta = np.ascontiguousarray(theta, dtype=np.float64).reshape(n, f)
        if rows is not None:
            rows = np.ascontiguousarray(rows, dtype=np.int64)
        cnt = m if rows is None else len(rows)
        x = np.empty((cnt, f), dtype=np.float64)
        st = np.empty(cnt, dtype=np.int32)
        rc = self._lib.oracle_half_sweep(self._p(rowptr), self._p(colidx), self._p(vals), m, n,
                                         f, float(lam), self._p(theta), self._p(rows),
                                         0 if rows is None else len(rows), self._p(x), self._p(st))
        if rc != 0:
            raise RuntimeError(f"oracle_half_sweep failed: {rc}")
        return x, st

    def rmse(self, rowptr, colidx, vals, m, f, x, theta):
        x = np.ascontiguousarray(x, dtype=np.float64)
        theta = np.ascontiguousarray(theta, dtype=np.float64)
        return self._lib.oracle_rmse(self._p(np.ascontiguousarray(rowptr, dtype=np.int64)),
                                     self._p(np.ascontiguousarray(colidx, dtype=np.int32)),
                                     self._p(np.ascontiguousarray(vals, dtype=np.float32)),
                                     m, f, self._p(x), self._p(theta))

    def objective(self, rowptr, colidx, vals, m, n, f, lam, x, theta):
        x = np.ascontiguousarray(x, dtype=np.float64)
        theta = np.ascontiguousarray(theta, dtype=np.float64)
        return self._lib.oracle_objective(self._p(np.ascontiguousarray(rowptr, dtype=np.int64)),
                                          self._p(np.ascontiguousarray(colidx, dtype=np.int32)),
                                          self._p(np.ascontiguousarray(vals, dtype=np.float32)),
                                          m, n, f, float(lam), self._p(x), self._p(theta))

    def transpose(self, rowptr, colidx, vals, m, n):
        nnz = int(rowptr[m])
        colptr = np.empty(n + 1, dtype=np.int64)
        rowidx = np.empty(nnz, dtype=np.int32)
        vt = np.empty(nnz, dtype=np.float32)
        rc = self._lib.oracle_transpose(self._p(np.ascontiguousarray(rowptr, dtype=np.int64)),
                                        self._p(np.ascontiguousarray(colidx, dtype=np.int32)),
                                        self._p(np.ascontiguousarray(vals, dtype=np.float32)),
                                        m, n, self._p(colptr), self._p(rowidx), self._p(vt))
        if rc != 0:
            raise RuntimeError(f"oracle_transpose failed: {rc}")
        return colptr, rowidx, vt

    def partition(self, rowptr, m, W, c_nnz, c_row, q, C=None, tail_div=8):
        """int64 [C+1, 2]: (row, entry offset) of each chunk boundary; C = W (the default)
        gives W equal chunks."""
        C = W if C is None else C
        out = np.empty((C + 1, 2), dtype=np.int64)
        rc = self._lib.oracle_partition(self._p(np.ascontiguousarray(rowptr, dtype=np.int64)),
                                        m, W, C, tail_div, c_nnz, c_row, q, self._p(out))
        if rc != 0:
            raise RuntimeError(f"oracle_partition failed: {rc}")
        return out


_default = None


def get() -> Oracle:
    global _default
    if _default is None:
        if not os.path.exists(LIB_PATH):
            build(mutants=False)
        _default = Oracle(LIB_PATH)
    return _default


def mutant(k: int) -> Oracle:
    p = os.path.join(MUTANT_DIR, f"liboracle_m{k}.so")
    if not os.path.exists(p):
        build(mutants=True)
    return Oracle(p)


def iterate(rowptr, colidx, vals, m, n, f, lam, theta, csc=None):
    """One ALS iteration in fp64: update-X (eq. 2) then update-Theta (eq. 3)."""
    o = get()
    x, _ = o.half_sweep(rowptr, colidx, vals, m, n, f, lam, theta)
    if csc is None:
        csc = o.transpose(rowptr, colidx, vals, m, n)
    colptr, rowidx, vt = csc
    th, _ = o.half_sweep(colptr, rowidx, vt, n, m, f, lam, x)
    return x, th
