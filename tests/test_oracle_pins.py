"""The fp64 oracle against what the paper and the mathematics fix (CPU only).

Each pin must hold for the real oracle, and each planted mistake (oracle built with
-DORACLE_MUTANT=k) must be caught by at least one pin.
"""
import numpy as np
import pytest

import oracle
from tests import pins

TOL = {
    "least_squares": 1e-10,
    "exact_rational": 1e-12,
    "gradient_zero": 1e-12,
    "closed_forms": 1e-12,
    "scaling": 1e-12,
    "rmse_and_objective": 1e-12,
    "monotone_objective": 1e-12,
    "planted_recovery": 1e-9,
    "transpose": 0.0,
}


def _pin(name):
    return getattr(pins, "pin_" + name)


@pytest.mark.parametrize("name", sorted(TOL))
def test_pin_holds(oracle_lib, name):
    err = _pin(name)(oracle_lib)
    assert err <= TOL[name], f"{name}: {err:.3e} > {TOL[name]:.1e}"


# which pins each planted mistake must trip (at least one of them)
CATCHERS = {
    1: ["least_squares", "exact_rational", "gradient_zero", "closed_forms"],
    2: ["least_squares", "exact_rational", "closed_forms"],
    3: ["least_squares", "exact_rational", "gradient_zero"],
    4: ["least_squares", "exact_rational", "gradient_zero"],
    5: ["least_squares", "exact_rational", "gradient_zero"],
    6: ["rmse_and_objective"],
    7: ["rmse_and_objective"],
    8: ["transpose"],
}


@pytest.fixture(scope="module")
def built_mutants():
    oracle.build(mutants=True)


@pytest.mark.parametrize("k", sorted(oracle.MUTANTS))
def test_planted_mistake_is_caught(built_mutants, k):
    mut = oracle.mutant(k)
    tripped = []
    for name in CATCHERS[k]:
        try:
            err = _pin(name)(mut)
        except Exception:          # a mistake that crashes a pin is caught too
            err = np.inf
        if not (err <= TOL[name]):
            tripped.append(name)
    assert tripped, f"mutant {k} ({oracle.MUTANTS[k]}) passed every pin"
    # the first listed catcher is the pin designed for it
    assert CATCHERS[k][0] in tripped


def test_empty_row_is_zero_and_flagged(oracle_lib):
    rowptr = np.array([0, 0, 2], np.int64)
    colidx = np.array([0, 1], np.int32)
    vals = np.array([1.0, 2.0], np.float32)
    x, st = oracle_lib.half_sweep(rowptr, colidx, vals, 2, 2, 2, 0.1, np.eye(2))
    assert np.all(x[0] == 0.0) and st[0] == oracle.ROW_EMPTY and st[1] == oracle.ROW_OK


def test_not_spd_row_is_nan(oracle_lib):
    # lambda = 0 and a single rating in f = 2: the Gram matrix is singular
    rowptr = np.array([0, 1], np.int64)
    x, st = oracle_lib.half_sweep(rowptr, np.array([0], np.int32), np.array([1.0], np.float32),
                                  1, 1, 2, 0.0, np.array([[1.0, 2.0]]))
    assert st[0] == oracle.ROW_NOT_SPD and np.all(np.isnan(x[0]))


def test_row_subset_matches_full(oracle_lib):
    import random
    rng = random.Random(11)
    rowptr, colidx, vals = pins.random_csr(rng, 20, 15, 0.3)
    theta = np.random.default_rng(0).normal(size=(15, 5))
    full, _ = oracle_lib.half_sweep(rowptr, colidx, vals, 20, 15, 5, 0.1, theta)
    rows = np.array([19, 3, 7, 7, 0], np.int64)
    sub, _ = oracle_lib.half_sweep(rowptr, colidx, vals, 20, 15, 5, 0.1, theta, rows=rows)
    assert np.array_equal(sub, full[rows])
