"""Pins for the fp64 oracle: checks against what the paper and the mathematics fix, not
against the oracle's own formulas.  Each ``pin_*`` returns an error measure; the tests assert
it is tiny for the real oracle and large for each planted-mistake build.

* least squares by Householder QR, pure Python (a different algorithm from the normal
  equations): the row update minimises J of eq. 1 restricted to x_u, i.e.
  || [Theta_u; sqrt(lambda n_u) I] x - [r_u; 0] ||;
* exact rational solves with ``fractions`` (Gaussian elimination over Q);
* the first-order condition dJ/dx_u = 0 that the paper starts from (section 2.1);
* closed forms: f = 1, a single rating (Sherman-Morrison), Theta = I;
* monotone J across half-sweeps; exact recovery of a planted rank-f matrix;
* brute-force RMSE and J; CSR->CSC round trip and stability.
"""
from __future__ import annotations

import math
import random
from fractions import Fraction

import numpy as np


# ------------------------------------------------------------------ helpers (pure Python)

def householder_lstsq(M, y):
    """argmin_x ||M x - y|| for a p x q list-of-lists M (p >= q, full column rank)."""
    p, q = len(M), len(M[0])
    A = [list(map(float, M[i])) + [float(y[i])] for i in range(p)]
    for j in range(q):
        norm = math.sqrt(sum(A[i][j] ** 2 for i in range(j, p)))
        if norm == 0.0:
            continue
        alpha = -norm if A[j][j] >= 0 else norm
        v = [0.0] * p
        v[j] = A[j][j] - alpha
        for i in range(j + 1, p):
            v[i] = A[i][j]
        vv = sum(v[i] ** 2 for i in range(j, p))
        if vv == 0.0:
            continue
        for c in range(j, q + 1):
            s = sum(v[i] * A[i][c] for i in range(j, p))
            t = 2.0 * s / vv
            for i in range(j, p):
                A[i][c] -= t * v[i]
    x = [0.0] * q
    for i in reversed(range(q)):
        s = A[i][q] - sum(A[i][k] * x[k] for k in range(i + 1, q))
        x[i] = s / A[i][i]
    return x


def exact_solve(A, b):
    """Solve A x = b over the rationals (A: list of lists of Fractions)."""
    n = len(A)
    M = [list(A[i]) + [b[i]] for i in range(n)]
    for c in range(n):
        piv = next(r for r in range(c, n) if M[r][c] != 0)
        M[c], M[piv] = M[piv], M[c]
        for r in range(n):
            if r != c and M[r][c] != 0:
                fac = M[r][c] / M[c][c]
                M[r] = [M[r][k] - fac * M[c][k] for k in range(n + 1)]
    return [M[i][n] / M[i][i] for i in range(n)]


def random_csr(rng: random.Random, m, n, density, allow_empty=True, min_row=0):
    """Tiny random CSR with distinct ascending columns per row."""
    rowptr, cols, vals = [0], [], []
    for _ in range(m):
        k = sum(1 for _ in range(n) if rng.random() < density)
        k = max(k, min_row)
        if not allow_empty:
            k = max(k, 1)
        k = min(k, n)
        cs = sorted(rng.sample(range(n), k))
        cols += cs
        vals += [rng.uniform(-2.0, 3.0) for _ in cs]
        rowptr.append(len(cols))
    return (np.array(rowptr, np.int64), np.array(cols, np.int32),
            np.array(vals, np.float32))


def csr_rows(rowptr, colidx, vals, u):
    b, e = int(rowptr[u]), int(rowptr[u + 1])
    return [int(c) for c in colidx[b:e]], [float(v) for v in vals[b:e]]


# ------------------------------------------------------------------ pins

def pin_least_squares(orc, seed=1, cases=6):
    """max relative difference between the oracle's x_u and Householder least squares."""
    rng = random.Random(seed)
    worst = 0.0
    for case in range(cases):
        m, n, f = rng.randint(3, 12), rng.randint(4, 14), rng.randint(1, 7)
        lam = rng.choice([0.05, 0.3, 1.0])
        rowptr, colidx, vals = random_csr(rng, m, n, rng.uniform(0.15, 0.8))
        theta = np.array([[rng.gauss(0, 1) for _ in range(f)] for _ in range(n)])
        x, st = orc.half_sweep(rowptr, colidx, vals, m, n, f, lam, theta)
        for u in range(m):
            cols, rs = csr_rows(rowptr, colidx, vals, u)
            nu = len(cols)
            if nu == 0:
                worst = max(worst, float(np.abs(x[u]).max()))
                continue
            M = [list(theta[c]) for c in cols]
            s = math.sqrt(lam * nu)
            M += [[s if i == j else 0.0 for j in range(f)] for i in range(f)]
            y = rs + [0.0] * f
            ref = householder_lstsq(M, y)
            den = max(max(abs(t) for t in ref), 1e-300)
            worst = max(worst, max(abs(x[u][i] - ref[i]) for i in range(f)) / den)
    return worst


def pin_exact_rational(orc, seed=2):
    """max relative difference to the exact solution over Q of sum(theta theta^T + lam I) x =
    sum r theta, with dyadic (exactly representable) data."""
    rng = random.Random(seed)
    m, n, f, lam = 5, 6, 3, 0.25
    rowptr, colidx, vals = random_csr(rng, m, n, 0.6, allow_empty=False)
    vals = np.array([rng.randint(-8, 8) / 4 for _ in range(len(vals))], np.float32)
    theta = np.array([[rng.randint(-4, 4) / 2 for _ in range(f)] for _ in range(n)])
    x, _ = orc.half_sweep(rowptr, colidx, vals, m, n, f, lam, theta)
    worst = 0.0
    for u in range(m):
        cols, rs = csr_rows(rowptr, colidx, vals, u)
        A = [[Fraction(0)] * f for _ in range(f)]
        b = [Fraction(0)] * f
        for c, r in zip(cols, rs):
            t = [Fraction(float(v)) for v in theta[c]]
            for i in range(f):
                for j in range(f):
                    A[i][j] += t[i] * t[j]
                A[i][i] += Fraction(lam)
                b[i] += Fraction(r) * t[i]
        ref = [float(v) for v in exact_solve(A, b)]
        den = max(max(abs(v) for v in ref), 1e-300)
        worst = max(worst, max(abs(x[u][i] - ref[i]) for i in range(f)) / den)
    return worst


def pin_gradient_zero(orc, seed=3):
    """max over rows of |dJ/dx_u| / scale, with the gradient of eq. 1 written in residual
    form: -2 sum_v (r_uv - x_u.theta_v) theta_v + 2 lambda n_u x_u."""
    rng = np.random.default_rng(seed)
    m, n, f, lam = 40, 30, 6, 0.1
    r = random.Random(seed)
    rowptr, colidx, vals = random_csr(r, m, n, 0.3)
    theta = rng.normal(size=(n, f))
    x, _ = orc.half_sweep(rowptr, colidx, vals, m, n, f, lam, theta)
    worst = 0.0
    for u in range(m):
        b, e = rowptr[u], rowptr[u + 1]
        if e == b:
            continue
        T = theta[colidx[b:e]]
        res = vals[b:e].astype(np.float64) - T @ x[u]
        g = -2.0 * (T.T @ res) + 2.0 * lam * (e - b) * x[u]
        scale = 2.0 * (np.abs(T).sum(axis=0).max() * np.abs(T).max() * np.abs(x[u]).max()
                       + np.abs(vals[b:e]).max() * np.abs(T).max() * (e - b))
        worst = max(worst, float(np.abs(g).max() / scale))
    return worst


def pin_closed_forms(orc):
    """f = 1; one rating per row (Sherman-Morrison); Theta = I with full observation."""
    worst = 0.0
    # f = 1: x_u = sum r theta / (sum theta^2 + lambda n_u)
    rng = random.Random(4)
    rowptr, colidx, vals = random_csr(rng, 8, 9, 0.5, allow_empty=False)
    theta = np.array([[rng.uniform(-2, 2)] for _ in range(9)])
    lam = 0.2
    x, _ = orc.half_sweep(rowptr, colidx, vals, 8, 9, 1, lam, theta)
    for u in range(8):
        cols, rs = csr_rows(rowptr, colidx, vals, u)
        num = sum(r * theta[c][0] for c, r in zip(cols, rs))
        den = sum(theta[c][0] ** 2 for c in cols) + lam * len(cols)
        worst = max(worst, abs(x[u][0] - num / den) / max(abs(num / den), 1e-300))
    # one rating: (theta theta^T + lambda I) x = r theta  =>  x = r theta / (|theta|^2 + lambda)
    f, n = 5, 7
    theta = np.array([[rng.uniform(-1, 1) for _ in range(f)] for _ in range(n)])
    rowptr = np.arange(n + 1, dtype=np.int64)
    colidx = np.arange(n, dtype=np.int32)[::-1].copy()
    vals = np.array([rng.uniform(1, 5) for _ in range(n)], np.float32)
    x, _ = orc.half_sweep(rowptr, colidx, vals, n, n, f, lam, theta)
    for u in range(n):
        t = theta[colidx[u]]
        ref = float(vals[u]) * t / (t @ t + lam)
        worst = max(worst, float(np.abs(x[u] - ref).max() / np.abs(ref).max()))
    # Theta = I (n = f), every column rated: A = (1 + lambda f) I, b = r_u
    f = 6
    m = 4
    rowptr = np.arange(0, (m + 1) * f, f, dtype=np.int64)
    colidx = np.tile(np.arange(f, dtype=np.int32), m)
    vals = np.array([rng.uniform(-3, 3) for _ in range(m * f)], np.float32)
    x, _ = orc.half_sweep(rowptr, colidx, vals, m, f, f, lam, np.eye(f))
    ref = vals.reshape(m, f).astype(np.float64) / (1.0 + lam * f)
    worst = max(worst, float(np.abs(x - ref).max() / np.abs(ref).max()))
    return worst


def pin_scaling(orc, c=4.0):
    """x_u(c R) = c x_u(R): the solution is linear in the ratings (c a power of two, so the
    scaled fp32 ratings are exact)."""
    rng = random.Random(5)
    rowptr, colidx, vals = random_csr(rng, 10, 12, 0.4, allow_empty=False)
    theta = np.array([[rng.gauss(0, 1) for _ in range(4)] for _ in range(12)])
    x1, _ = orc.half_sweep(rowptr, colidx, vals, 10, 12, 4, 0.1, theta)
    x2, _ = orc.half_sweep(rowptr, colidx, (vals * np.float32(c)).astype(np.float32), 10, 12, 4,
                           0.1, theta)
    return float(np.abs(x2 - c * x1).max() / np.abs(c * x1).max())


def brute_objective(rowptr, colidx, vals, m, n, f, lam, x, theta):
    """J of eq. 1 by direct loops over the stored entries."""
    fit = 0.0
    nu = [0] * m
    nv = [0] * n
    for u in range(m):
        for k in range(int(rowptr[u]), int(rowptr[u + 1])):
            v = int(colidx[k])
            d = sum(float(x[u][i]) * float(theta[v][i]) for i in range(f))
            fit += (float(vals[k]) - d) ** 2
            nu[u] += 1
            nv[v] += 1
    reg = sum(nu[u] * sum(float(x[u][i]) ** 2 for i in range(f)) for u in range(m))
    reg += sum(nv[v] * sum(float(theta[v][i]) ** 2 for i in range(f)) for v in range(n))
    return fit + lam * reg, fit


def pin_rmse_and_objective(orc, seed=6):
    """relative error of the oracle's RMSE and J against direct loops."""
    rng = random.Random(seed)
    m, n, f, lam = 9, 11, 3, 0.3
    rowptr, colidx, vals = random_csr(rng, m, n, 0.5)
    x = np.array([[rng.gauss(0, 1) for _ in range(f)] for _ in range(m)])
    theta = np.array([[rng.gauss(0, 1) for _ in range(f)] for _ in range(n)])
    J, fit = brute_objective(rowptr, colidx, vals, m, n, f, lam, x, theta)
    nnz = int(rowptr[m])
    rm = math.sqrt(fit / nnz)
    e1 = abs(orc.rmse(rowptr, colidx, vals, m, f, x, theta) - rm) / rm
    e2 = abs(orc.objective(rowptr, colidx, vals, m, n, f, lam, x, theta) - J) / J
    return max(e1, e2)


def pin_monotone_objective(orc, seed=7, sweeps=8):
    """largest relative increase of J over consecutive half-sweeps (each half-sweep is an exact
    block minimisation of J, so J must not increase)."""
    rng = np.random.default_rng(seed)
    r = random.Random(seed)
    m, n, f, lam = 30, 20, 4, 0.05
    rowptr, colidx, vals = random_csr(r, m, n, 0.35, allow_empty=False)
    colptr, rowidx, vt = orc.transpose(rowptr, colidx, vals, m, n)
    theta = rng.normal(0, 0.5, size=(n, f))
    x = np.zeros((m, f))
    J_prev = orc.objective(rowptr, colidx, vals, m, n, f, lam, x, theta)
    worst = -np.inf
    for s in range(sweeps):
        if s % 2 == 0:
            x, _ = orc.half_sweep(rowptr, colidx, vals, m, n, f, lam, theta)
        else:
            theta, _ = orc.half_sweep(colptr, rowidx, vt, n, m, f, lam, x)
        J = orc.objective(rowptr, colidx, vals, m, n, f, lam, x, theta)
        worst = max(worst, (J - J_prev) / abs(J_prev))
        J_prev = J
    return worst


def pin_planted_recovery(orc, seed=8):
    """R = X* Theta*^T dense (every entry stored), rank f, noise-free, lambda = 0: after one
    iteration X Theta^T reproduces R (update-X puts col(X) = col(X*); update-Theta is then an
    exact fit).  Returns max |X Theta^T - R| / rms(R)."""
    rng = np.random.default_rng(seed)
    m, n, f = 14, 11, 3
    # small-integer factors, so R is exactly rank f even after rounding to fp32
    Xs = rng.integers(-3, 4, size=(m, f)).astype(np.float64)
    Ts = rng.integers(-3, 4, size=(n, f)).astype(np.float64)
    R = (Xs @ Ts.T).astype(np.float32)
    rowptr = np.arange(0, (m + 1) * n, n, dtype=np.int64)
    colidx = np.tile(np.arange(n, dtype=np.int32), m)
    vals = R.reshape(-1)
    theta0 = rng.normal(size=(n, f))
    x, _ = orc.half_sweep(rowptr, colidx, vals, m, n, f, 0.0, theta0)
    colptr, rowidx, vt = orc.transpose(rowptr, colidx, vals, m, n)
    th, _ = orc.half_sweep(colptr, rowidx, vt, n, m, f, 0.0, x)
    Rd = R.astype(np.float64)
    return float(np.abs(x @ th.T - Rd).max() / np.sqrt((Rd ** 2).mean()))


def pin_transpose(orc, seed=9):
    """0 iff CSR->CSC->CSR is the identity and each column lists rows ascending."""
    rng = random.Random(seed)
    m, n = 23, 17
    rowptr, colidx, vals = random_csr(rng, m, n, 0.3)
    colptr, rowidx, vt = orc.transpose(rowptr, colidx, vals, m, n)
    bad = 0
    for v in range(n):
        seg = rowidx[colptr[v]:colptr[v + 1]]
        bad += int(np.any(np.diff(seg.astype(np.int64)) <= 0))
    rp2, ci2, v2 = orc.transpose(colptr, rowidx, vt, n, m)
    bad += int(not (np.array_equal(rp2, rowptr) and np.array_equal(ci2, colidx)
                    and np.array_equal(v2, vals)))
    return float(bad)
