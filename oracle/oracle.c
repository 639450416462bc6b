/*
 * ORACLE -- test infrastructure only.
 *
 * A plain, slow, fp64 CPU statement of what one ALS half-sweep computes, written from the
 * paper (Tan, Cao, Fong, "Faster and Cheaper: Parallelizing Large-Scale Matrix Factorization
 * on GPUs", HPDC'16).  Only the tests, the smoke check and the CPU-baseline leg of the
 * benchmark may load it; the product path never does.  It shares no code with the HIP
 * library.
 *
 * Readings of the paper taken here (each is listed in the design notes):
 *   - the regulariser is lambda * n_u * I: Algorithm 1 adds (theta_v theta_v^T + lambda I)
 *     once per rated column, i.e. the weighted-lambda term of the cost function (eq. 1);
 *   - "r_uv != 0" means "stored in the sparse matrix", whatever the stored value;
 *   - a row with no stored entries gets x_u = 0 (the paper is silent; J does not depend on
 *     such an x_u and 0 is its minimum-norm minimiser);
 *   - the solver is Cholesky (A_u is symmetric positive definite when lambda > 0, n_u > 0),
 *     followed by forward and back substitution; a non-positive pivot marks the row NOT_SPD
 *     and its x_u is NaN;
 *   - indices are 0-based and Theta^T (f x n, theta_v as columns) is held as an n x f
 *     row-major array (the same bytes as column-major Theta^T).
 *
 * Building with -DORACLE_MUTANT=k plants mistake number k (see the MUTANT blocks); the
 * tests use those builds to show that the pins catch each mistake.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#ifndef ORACLE_MUTANT
#define ORACLE_MUTANT 0
#endif

enum { ORACLE_ROW_OK = 0, ORACLE_ROW_EMPTY = 1, ORACLE_ROW_NOT_SPD = 2 };
enum { ORACLE_OK = 0, ORACLE_ERR_ARG = -1, ORACLE_ERR_NOMEM = -2 };

/*
 * One row of update-X: Algorithm 1 (base ALS), procedures Get_Hermitian_X and Batch_Solve,
 * for a single u; the normal equations are eq. 2.
 *   A_u = sum over stored (u,v) of (theta_v theta_v^T + lambda I)   [lower triangle kept]
 *   B_u = Theta^T R_u*^T = sum over stored (u,v) of r_uv theta_v
 *   solve A_u x_u = B_u
 * A, L are f*f scratch (row-major), b, y are f scratch.  Returns a row status.
 */
static int solve_row(const int32_t* cols, const float* vals, int64_t nu, int32_t f,
                     double lambda, const double* theta, double* A, double* L, double* b,
                     double* y, double* x) {
    if (nu == 0) {
        for (int32_t i = 0; i < f; ++i) x[i] = 0.0;
        return ORACLE_ROW_EMPTY;
    }
    memset(A, 0, sizeof(double) * (size_t)f * (size_t)f);
    memset(b, 0, sizeof(double) * (size_t)f);
    for (int64_t k = 0; k < nu; ++k) {
        const double* tv = theta + (size_t)cols[k] * (size_t)f;
        const double r = (double)vals[k];
        for (int32_t i = 0; i < f; ++i) {
            for (int32_t j = 0; j <= i; ++j) {
#if ORACLE_MUTANT == 3 /* MUTANT 3: Gram uses theta_i^2 everywhere (wrong index) */
                A[(size_t)i * f + j] += tv[i] * tv[i];
#else
                A[(size_t)i * f + j] += tv[i] * tv[j];
#endif
            }
#if ORACLE_MUTANT == 1 /* MUTANT 1: plain lambda I once, not once per rated column */
            if (k == 0) A[(size_t)i * f + i] += lambda;
#else
            A[(size_t)i * f + i] += lambda; /* the "+ lambda I" inside the sum of Alg. 1 */
#endif
#if ORACLE_MUTANT == 2 /* MUTANT 2: right-hand side drops the rating */
            b[i] += tv[i] + 0.0 * r;
#else
            b[i] += r * tv[i];
#endif
        }
    }
    /* Cholesky-Banachiewicz, row by row: A = L L^T */
    for (int32_t i = 0; i < f; ++i) {
        for (int32_t j = 0; j <= i; ++j) {
            double s = A[(size_t)i * f + j];
            for (int32_t p = 0; p < j; ++p) s -= L[(size_t)i * f + p] * L[(size_t)j * f + p];
            if (i == j) {
                if (!(s > 0.0)) {
                    for (int32_t t = 0; t < f; ++t) x[t] = NAN;
                    return ORACLE_ROW_NOT_SPD;
                }
                L[(size_t)i * f + i] = sqrt(s);
            } else {
                L[(size_t)i * f + j] = s / L[(size_t)j * f + j];
            }
        }
    }
    /* forward substitution: L y = b */
    for (int32_t i = 0; i < f; ++i) {
        double s = b[i];
#if ORACLE_MUTANT == 4 /* MUTANT 4: wrong sign in forward substitution */
        for (int32_t p = 0; p < i; ++p) s += L[(size_t)i * f + p] * y[p];
#else
        for (int32_t p = 0; p < i; ++p) s -= L[(size_t)i * f + p] * y[p];
#endif
        y[i] = s / L[(size_t)i * f + i];
    }
    /* back substitution: L^T x = y */
    for (int32_t i = f - 1; i >= 0; --i) {
        double s = y[i];
#if ORACLE_MUTANT == 5 /* MUTANT 5: back substitution with L instead of L^T (transposed operand) */
        for (int32_t p = i + 1; p < f; ++p) s -= L[(size_t)i * f + p] * x[p];
#else
        for (int32_t p = i + 1; p < f; ++p) s -= L[(size_t)p * f + i] * x[p];
#endif
        x[i] = s / L[(size_t)i * f + i];
    }
    return ORACLE_ROW_OK;
}

/*
 * One half-sweep (update-X by eq. 2; the same routine on the transposed matrix with the roles
 * of X and Theta exchanged is update-Theta by eq. 3).  Rows are independent, so the loop over
 * rows runs in parallel; each row is computed serially, so the result does not depend on the
 * thread count.
 *   rows == NULL: all m rows, x_out is m x f.  Otherwise only rows[0..nrows), x_out is
 *   nrows x f in that order (used for sampled checks of full-size problems).
 *   status_out (optional) receives a row status per output row.
 */
int oracle_half_sweep(const int64_t* rowptr, const int32_t* colidx, const float* vals,
                      int64_t m, int64_t n, int32_t f, double lambda, const double* theta,
                      const int64_t* rows, int64_t nrows, double* x_out, int32_t* status_out) {
    if (!rowptr || m < 0 || n < 0 || f <= 0 || !x_out || (n > 0 && !theta)) return ORACLE_ERR_ARG;
    const int64_t cnt = rows ? nrows : m;
    int rc = ORACLE_OK;
#pragma omp parallel
    {
        double* A = (double*)malloc(sizeof(double) * (size_t)f * (size_t)f);
        double* L = (double*)malloc(sizeof(double) * (size_t)f * (size_t)f);
        double* b = (double*)malloc(sizeof(double) * (size_t)f);
        double* y = (double*)malloc(sizeof(double) * (size_t)f);
        if (!A || !L || !b || !y) {
#pragma omp atomic write
            rc = ORACLE_ERR_NOMEM;
        }
#pragma omp for schedule(dynamic, 64)
        for (int64_t t = 0; t < cnt; ++t) {
            if (!A || !L || !b || !y) continue;
            const int64_t u = rows ? rows[t] : t;
            const int64_t beg = rowptr[u], nu = rowptr[u + 1] - rowptr[u];
            int st = solve_row(colidx + beg, vals + beg, nu, f, lambda, theta, A, L, b, y,
                               x_out + (size_t)t * (size_t)f);
            if (status_out) status_out[t] = st;
        }
        free(A); free(L); free(b); free(y);
    }
    return rc;
}

/* squared residual sum over stored entries, rows ascending, entries ascending */
static double residual_sq_sum(const int64_t* rowptr, const int32_t* colidx, const float* vals,
                              int64_t m, int32_t f, const double* x, const double* theta) {
    double total = 0.0;
    for (int64_t u = 0; u < m; ++u) {
        for (int64_t k = rowptr[u]; k < rowptr[u + 1]; ++k) {
            const double* tv = theta + (size_t)colidx[k] * (size_t)f;
            const double* xu = x + (size_t)u * (size_t)f;
            double d = 0.0;
            for (int32_t i = 0; i < f; ++i) d += xu[i] * tv[i];
            double e = (double)vals[k] - d;
            total += e * e;
        }
    }
    return total;
}

/* Root-mean-square error over the stored entries (the evaluation metric of the experiments
   section, here over the training entries): sqrt(sum (r_uv - x_u^T theta_v)^2 / N_z). */
double oracle_rmse(const int64_t* rowptr, const int32_t* colidx, const float* vals, int64_t m,
                   int32_t f, const double* x, const double* theta) {
    const int64_t nnz = rowptr[m];
    if (nnz == 0) return 0.0;
    double s = residual_sq_sum(rowptr, colidx, vals, m, f, x, theta);
#if ORACLE_MUTANT == 6 /* MUTANT 6: mean over rows instead of over stored entries */
    return sqrt(s / (double)m);
#else
    return sqrt(s / (double)nnz);
#endif
}

/* The cost function J of eq. 1 with weighted-lambda regularisation:
   sum (r_uv - x_u^T theta_v)^2 + lambda (sum_u n_u |x_u|^2 + sum_v n_v |theta_v|^2),
   n_u and n_v counted from the stored entries. */
double oracle_objective(const int64_t* rowptr, const int32_t* colidx, const float* vals,
                        int64_t m, int64_t n, int32_t f, double lambda, const double* x,
                        const double* theta) {
    double fit = residual_sq_sum(rowptr, colidx, vals, m, f, x, theta);
    int64_t* nv = (int64_t*)calloc((size_t)(n > 0 ? n : 1), sizeof(int64_t));
    if (!nv) return NAN;
    for (int64_t k = 0; k < rowptr[m]; ++k) nv[colidx[k]]++;
    double reg = 0.0;
    for (int64_t u = 0; u < m; ++u) {
        double s = 0.0;
        for (int32_t i = 0; i < f; ++i) s += x[(size_t)u * f + i] * x[(size_t)u * f + i];
#if ORACLE_MUTANT == 7 /* MUTANT 7: unweighted regulariser */
        reg += s;
#else
        reg += (double)(rowptr[u + 1] - rowptr[u]) * s;
#endif
    }
    for (int64_t v = 0; v < n; ++v) {
        double s = 0.0;
        for (int32_t i = 0; i < f; ++i) s += theta[(size_t)v * f + i] * theta[(size_t)v * f + i];
#if ORACLE_MUTANT == 7
        reg += s;
#else
        reg += (double)nv[v] * s;
#endif
    }
    free(nv);
    return fit + lambda * reg;
}

/* R -> R^T (CSR -> CSC): for update-Theta, which the paper solves by the same method on the
   columns R_*v (eq. 3).  Stable: rows ascending within each column, values carried along. */
int oracle_transpose(const int64_t* rowptr, const int32_t* colidx, const float* vals,
                     int64_t m, int64_t n, int64_t* colptr, int32_t* rowidx, float* vals_t) {
    if (!rowptr || !colptr || m < 0 || n < 0) return ORACLE_ERR_ARG;
    const int64_t nnz = rowptr[m];
    memset(colptr, 0, sizeof(int64_t) * (size_t)(n + 1));
    for (int64_t k = 0; k < nnz; ++k) colptr[colidx[k] + 1]++;
    for (int64_t v = 0; v < n; ++v) colptr[v + 1] += colptr[v];
    int64_t* cur = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    if (!cur) return ORACLE_ERR_NOMEM;
    memcpy(cur, colptr, sizeof(int64_t) * (size_t)n);
#if ORACLE_MUTANT == 8 /* MUTANT 8: unstable order (rows descending within a column) */
    for (int64_t u = m - 1; u >= 0; --u)
#else
    for (int64_t u = 0; u < m; ++u)
#endif
        for (int64_t k = rowptr[u]; k < rowptr[u + 1]; ++k) {
            int64_t d = cur[colidx[k]]++;
            rowidx[d] = (int32_t)u;
            vals_t[d] = vals[k];
        }
    free(cur);
    return ORACLE_OK;
}

/* Threads the row loops run on (OpenMP's team size for a parallel region here). */
int oracle_threads(void) { return omp_get_max_threads(); }

/* Set that team size for later calls from this thread (timing a single core). */
void oracle_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }

/*
 * The work partition of the HIP path, restated from its definition so that the library's
 * integer planning can be checked bit for bit.  Each row u costs c_row + c_nnz * n_u units
 * on a cost axis with prefix P(u) = c_nnz * rowptr[u] + c_row * u (T = P(m)).  The axis is cut
 * into C chunks: W equal "large" chunks cover T1 = T - T2 and C - W equal "small" chunks cover
 * the tail T2 = floor(T / tail_div) (T2 = 0 when C = W).  Boundary b sits at
 *     s_b = floor(T1 b / W)                          for b <= W,
 *     s_b = T1 + floor(T2 (b - W) / (C - W))         for b >= W,
 * in row u_b, the largest u with P(u) <= s_b, at entry offset ceil((s_b - P(u_b) - c_row) /
 * c_nnz) clamped to [0, n_u], rounded to the nearest multiple of q and, if that is not 0, moved
 * to the row end when fewer than q/2 entries would remain.
 * bounds_out[2b] = u_b, bounds_out[2b+1] = that offset; b = 0..C.
 */
int oracle_partition(const int64_t* rowptr, int64_t m, int64_t W, int64_t C, int64_t tail_div,
                     int64_t c_nnz, int64_t c_row, int64_t q, int64_t* bounds_out) {
    if (!rowptr || m < 0 || W < 1 || C < W || tail_div < 1 || c_nnz < 1 || c_row < 1 || q < 2 ||
        (q & 1) || !bounds_out)
        return ORACLE_ERR_ARG;
    const __int128 T = (__int128)c_nnz * rowptr[m] + (__int128)c_row * m;
    const __int128 T2 = C > W ? T / tail_div : 0, T1 = T - T2;
    int64_t u = 0; /* s_b grows with b, so u_b does too: scan on from the previous one */
    for (int64_t b = 0; b <= C; ++b) {
        const __int128 s = b <= W ? T1 * b / W : T1 + T2 * (b - W) / (C - W);
        while (u < m && (__int128)c_nnz * rowptr[u + 1] + (__int128)c_row * (u + 1) <= s) ++u;
        int64_t kk = 0;
        if (u < m) {
            const int64_t nu = rowptr[u + 1] - rowptr[u];
            __int128 over = s - ((__int128)c_nnz * rowptr[u] + (__int128)c_row * u) - c_row;
            __int128 raw = over <= 0 ? 0 : (over + c_nnz - 1) / c_nnz;
            if (raw > nu) raw = nu;
            kk = (int64_t)((raw + q / 2) / q * q);
            if (kk > 0 && kk + q / 2 > nu) kk = nu;
        }
        bounds_out[2 * b] = u;
        bounds_out[2 * b + 1] = kk;
    }
    return ORACLE_OK;
}
