/*
 * Seeded synthetic inputs for the ALS half-sweep.
 *
 * Builds sparse rating matrices shaped like the paper's workloads (the data-set table of the
 * experiments section: m x n with N_z ratings, skewed row lengths, popular columns), planted
 * low-rank ratings, and the initial factor matrix.  Both the fp64 oracle and the HIP path take
 * their inputs from here.  This file holds none of the ALS arithmetic (no Gram matrix, no
 * solve, no error metric): it only draws numbers and lays them out as CSR/CSC.
 *
 * Randomness: Philox4x32-10, the counter-based generator of Salmon, Moraes, Dror and Shaw,
 * "Parallel random numbers: as easy as 1, 2, 3" (SC'11), implemented from that definition.
 * Key = (seed low word, seed high word + 65536 * stream); counter = (index low, index high,
 * sub-draw, 0).  Every value is a pure function of (seed, stream, index), so the result does
 * not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

/* ------------------------------------------------------------------ Philox4x32-10 ---- */

typedef struct { uint32_t v[4]; } p4x32;

static inline p4x32 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                   uint32_t k0, uint32_t k1) {
    for (int r = 0; r < 10; ++r) {
        uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    p4x32 out = {{c0, c1, c2, c3}};
    return out;
}

/* exported for the known-answer test of the generator itself */
void synth_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    p4x32 r = philox4x32_10(ctr[0], ctr[1], ctr[2], ctr[3], key[0], key[1]);
    memcpy(out, r.v, sizeof r.v);
}

typedef struct { uint32_t k0, k1; } skey;

static inline skey make_key(uint64_t seed, uint32_t stream) {
    skey k = {(uint32_t)seed, (uint32_t)(seed >> 32) + (stream << 16)};
    return k;
}

static inline p4x32 draw(skey k, uint64_t idx, uint32_t sub) {
    return philox4x32_10((uint32_t)idx, (uint32_t)(idx >> 32), sub, 0u, k.k0, k.k1);
}

/* 53-bit uniform in [0,1) from two words */
static inline double u01(uint32_t a, uint32_t b) {
    return ((double)(a >> 5) * 67108864.0 + (double)(b >> 6)) * (1.0 / 9007199254740992.0);
}
/* 53-bit uniform in (0,1] */
static inline double u01_open0(uint32_t a, uint32_t b) {
    return ((double)(a >> 5) * 67108864.0 + (double)(b >> 6) + 1.0) * (1.0 / 9007199254740992.0);
}

/* Standard normal number idx of a stream: Box-Muller on one Philox block, which yields
   the pair (2j, 2j+1). */
static inline double normal_at(skey k, uint64_t idx) {
    p4x32 r = draw(k, idx >> 1, 0);
    double u1 = u01_open0(r.v[0], r.v[1]);
    double u2 = u01(r.v[2], r.v[3]);
    double rad = sqrt(-2.0 * log(u1));
    double ang = 6.283185307179586 * u2;
    return (idx & 1) ? rad * sin(ang) : rad * cos(ang);
}

/* ------------------------------------------------------------------ row lengths ------ */

enum { SYNTH_OK = 0, SYNTH_ERR_ARG = -1, SYNTH_ERR_NOMEM = -2, SYNTH_ERR_INFEASIBLE = -3 };
enum { ROWS_UNIFORM = 0, ROWS_LOGNORMAL = 1 };

/* Multinomial row lengths: each of the nnz entries picks a row uniformly (stream 1, counter =
   entry index).  Rows that would exceed n entries (impossible without duplicates) pass the
   excess on to the next rows with room, in ascending order, wrapping around. */
static int counts_uniform(int64_t m, int64_t n, int64_t nnz, uint64_t seed, int64_t* cnt) {
    skey k = make_key(seed, 1);
    memset(cnt, 0, sizeof(int64_t) * (size_t)m);
    int64_t* part = NULL;
    int nt = omp_get_max_threads();
    part = (int64_t*)calloc((size_t)nt * (size_t)m, sizeof(int64_t));
    if (!part) return SYNTH_ERR_NOMEM;
#pragma omp parallel
    {
        int64_t* h = part + (size_t)omp_get_thread_num() * (size_t)m;
#pragma omp for schedule(static)
        for (int64_t t = 0; t < nnz; ++t) {
            p4x32 r = draw(k, (uint64_t)t, 0);
            int64_t u = (int64_t)(u01(r.v[0], r.v[1]) * (double)m);
            if (u >= m) u = m - 1;
            h[u]++;
        }
    }
    for (int t = 0; t < nt; ++t)
        for (int64_t u = 0; u < m; ++u) cnt[u] += part[(size_t)t * (size_t)m + u];
    free(part);
    int64_t carry = 0;
    for (int pass = 0; pass < 2; ++pass)
        for (int64_t u = 0; u < m; ++u) {
            cnt[u] += carry;
            carry = 0;
            if (cnt[u] > n) { carry = cnt[u] - n; cnt[u] = n; }
        }
    return carry ? SYNTH_ERR_INFEASIBLE : SYNTH_OK;
}

static double clamp_d(double x, double lo, double hi) { return x < lo ? lo : (x > hi ? hi : x); }

/* Lognormal row lengths: w_u = exp(mu + sigma z_u) with z_u ~ N(0,1) (stream 1, counter u),
   mu = ln(mean) - sigma^2/2 so E[w] = mean.  A common scale a is found by bisection so that
   sum_u clamp(a w_u, 1, n) = nnz; lengths are the floors of those targets, and the remaining
   entries go one each to the rows with the largest fractional parts (ties to lower u; rows
   already at n are skipped). */
static int counts_lognormal(int64_t m, int64_t n, int64_t nnz, double mean, double sigma,
                            uint64_t seed, int64_t* cnt) {
    if (nnz < m || nnz > m * n) return SYNTH_ERR_INFEASIBLE;
    skey k = make_key(seed, 1);
    double mu = log(mean) - 0.5 * sigma * sigma;
    double* w = (double*)malloc(sizeof(double) * (size_t)m);
    if (!w) return SYNTH_ERR_NOMEM;
#pragma omp parallel for schedule(static)
    for (int64_t u = 0; u < m; ++u) w[u] = exp(mu + sigma * normal_at(k, (uint64_t)u));
    double lo = 0.0, hi = 1.0;
    for (;;) {  /* grow hi until the clamped sum reaches nnz */
        double s = 0.0;
#pragma omp parallel for reduction(+ : s) schedule(static)
        for (int64_t u = 0; u < m; ++u) s += clamp_d(hi * w[u], 1.0, (double)n);
        if (s >= (double)nnz) break;
        lo = hi;
        hi *= 2.0;
        if (hi > 1e300) { free(w); return SYNTH_ERR_INFEASIBLE; }
    }
    for (int it = 0; it < 200; ++it) {
        double mid = 0.5 * (lo + hi), s = 0.0;
#pragma omp parallel for reduction(+ : s) schedule(static)
        for (int64_t u = 0; u < m; ++u) s += clamp_d(mid * w[u], 1.0, (double)n);
        if (s >= (double)nnz) hi = mid; else lo = mid;
    }
    double a = lo;  /* sum of floors <= nnz */
    int64_t total = 0;
#pragma omp parallel for reduction(+ : total) schedule(static)
    for (int64_t u = 0; u < m; ++u) {
        double t = clamp_d(a * w[u], 1.0, (double)n);
        cnt[u] = (int64_t)floor(t);
        w[u] = t - floor(t);  /* reuse w for the fractional part */
        total += cnt[u];
    }
    int64_t rem = nnz - total;
    if (rem < 0) { free(w); return SYNTH_ERR_INFEASIBLE; }
    if (rem > 0) {
        /* largest fractional parts first: quantise to 2^24 buckets, find the threshold
           bucket from the top, then break ties inside it in ascending u */
        const int64_t NBK = (int64_t)1 << 24;
        int64_t* hist = (int64_t*)calloc((size_t)NBK, sizeof(int64_t));
        if (!hist) { free(w); return SYNTH_ERR_NOMEM; }
        for (int64_t u = 0; u < m; ++u)
            if (cnt[u] < n) hist[(int64_t)(w[u] * (double)NBK)]++;
        int64_t acc = 0, thr = NBK - 1;
        for (; thr >= 0; --thr) {
            if (acc + hist[thr] >= rem) break;
            acc += hist[thr];
        }
        free(hist);
        if (thr < 0) { free(w); return SYNTH_ERR_INFEASIBLE; }
        int64_t left_at_thr = rem - acc;
        for (int64_t u = 0; u < m; ++u) {
            if (cnt[u] >= n) continue;
            int64_t q = (int64_t)(w[u] * (double)NBK);
            if (q > thr) cnt[u]++;
            else if (q == thr && left_at_thr > 0) { cnt[u]++; left_at_thr--; }
        }
    }
    free(w);
    return SYNTH_OK;
}

/* rowptr_out[m+1] (int64) for the given row-length model */
int synth_row_counts(int kind, int64_t m, int64_t n, int64_t nnz, double mean, double sigma,
                     uint64_t seed, int64_t* rowptr_out) {
    if (m <= 0 || n <= 0 || nnz < 0 || !rowptr_out) return SYNTH_ERR_ARG;
    int64_t* cnt = (int64_t*)malloc(sizeof(int64_t) * (size_t)m);
    if (!cnt) return SYNTH_ERR_NOMEM;
    int rc = kind == ROWS_UNIFORM ? counts_uniform(m, n, nnz, seed, cnt)
                                  : counts_lognormal(m, n, nnz, mean, sigma, seed, cnt);
    if (rc == SYNTH_OK) {
        rowptr_out[0] = 0;
        for (int64_t u = 0; u < m; ++u) rowptr_out[u + 1] = rowptr_out[u] + cnt[u];
    }
    free(cnt);
    return rc;
}

/* ------------------------------------------------------------------ columns ---------- */

typedef struct { double key; int32_t rank; } keyrank;

static int cmp_i32(const void* a, const void* b) {
    int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
    return (x > y) - (x < y);
}

/* deterministic quickselect: afterwards the k smallest keys (ties by rank) occupy [0,k) */
static inline int kr_less(const keyrank* a, const keyrank* b) {
    return a->key < b->key || (a->key == b->key && a->rank < b->rank);
}
static void kr_select(keyrank* v, int64_t len, int64_t k) {
    int64_t lo = 0, hi = len - 1;
    while (lo < hi) {
        keyrank piv = v[lo + (hi - lo) / 2];
        int64_t i = lo, j = hi;
        while (i <= j) {
            while (kr_less(&v[i], &piv)) ++i;
            while (kr_less(&piv, &v[j])) --j;
            if (i <= j) { keyrank t = v[i]; v[i] = v[j]; v[j] = t; ++i; --j; }
        }
        if (k <= j) hi = j;
        else if (k >= i) lo = i;
        else return;
    }
}

/* Column ids: Zipf(s) popularity over ranks 0..n-1 (weight (rank+1)^-s), mapped to column
   ids through a seeded Fisher-Yates permutation (stream 2) so popularity is not index-ordered.
   Each row draws its n_u distinct ranks by successive weighted sampling without replacement
   (stream 3, counter = row, sub-draw = attempt): rejection of repeats while that is cheap,
   otherwise exponential keys -ln(U_r)/w_r (stream 3, counter = row, sub-draw = 2^31 + rank)
   and the n_u smallest -- both realise the same sampling law.  Columns are stored ascending. */
int synth_columns(int64_t m, int64_t n, double zipf_s, uint64_t seed, const int64_t* rowptr,
                  int32_t* colidx_out) {
    if (m <= 0 || n <= 0 || n > INT32_MAX || !rowptr || !colidx_out) return SYNTH_ERR_ARG;
    for (int64_t u = 0; u < m; ++u)
        if (rowptr[u + 1] - rowptr[u] > n || rowptr[u + 1] < rowptr[u]) return SYNTH_ERR_ARG;
    int32_t* perm = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
    double* cdf = (double*)malloc(sizeof(double) * (size_t)n);
    double* wgt = (double*)malloc(sizeof(double) * (size_t)n);
    if (!perm || !cdf || !wgt) { free(perm); free(cdf); free(wgt); return SYNTH_ERR_NOMEM; }
    skey kp = make_key(seed, 2), ks = make_key(seed, 3);
    for (int64_t i = 0; i < n; ++i) perm[i] = (int32_t)i;
    for (int64_t i = n - 1; i > 0; --i) {
        p4x32 r = draw(kp, (uint64_t)i, 0);
        int64_t j = (int64_t)(u01(r.v[0], r.v[1]) * (double)(i + 1));
        if (j > i) j = i;
        int32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t;
    }
    double run = 0.0;
    for (int64_t r = 0; r < n; ++r) {
        wgt[r] = pow((double)(r + 1), -zipf_s);
        run += wgt[r];
        cdf[r] = run;
    }
    const double total = run;
    int rc = SYNTH_OK;
#pragma omp parallel
    {
        int32_t* stamp = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
        keyrank* kr = NULL;
        if (!stamp) {
#pragma omp atomic write
            rc = SYNTH_ERR_NOMEM;
        } else {
            for (int64_t i = 0; i < n; ++i) stamp[i] = -1;
        }
#pragma omp for schedule(dynamic, 256)
        for (int64_t u = 0; u < m; ++u) {
            if (!stamp) continue;
            int64_t beg = rowptr[u], nu = rowptr[u + 1] - beg;
            int32_t* out = colidx_out + beg;
            int32_t mark = (int32_t)(u & 0x7fffffff);
            int use_keys = nu > n / 8;
            if (!use_keys) {
                int64_t got = 0, cap = 8 * nu + 256;
                uint32_t att = 0;
                while (got < nu && (int64_t)att < cap) {
                    p4x32 r = draw(ks, (uint64_t)u, att++);
                    double x = u01(r.v[0], r.v[1]) * total;
                    int64_t lo = 0, hi = n - 1;  /* first rank with cdf > x */
                    while (lo < hi) {
                        int64_t mid = (lo + hi) >> 1;
                        if (cdf[mid] > x) hi = mid; else lo = mid + 1;
                    }
                    if (stamp[lo] != mark) { stamp[lo] = mark; out[got++] = (int32_t)lo; }
                }
                if (got < nu) {  /* too many repeats: redo this row with exponential keys */
                    for (int64_t i = 0; i < got; ++i) stamp[out[i]] = -1;
                    use_keys = 1;
                } else {
                    for (int64_t i = 0; i < nu; ++i) stamp[out[i]] = -1;
                }
            }
            if (use_keys && nu > 0) {
                if (!kr) kr = (keyrank*)malloc(sizeof(keyrank) * (size_t)n);
                if (!kr) {
#pragma omp atomic write
                    rc = SYNTH_ERR_NOMEM;
                    continue;
                }
                for (int64_t r = 0; r < n; ++r) {
                    p4x32 d = draw(ks, (uint64_t)u, 0x80000000u + (uint32_t)r);
                    kr[r].key = -log(u01_open0(d.v[0], d.v[1])) / wgt[r];
                    kr[r].rank = (int32_t)r;
                }
                if (nu < n) kr_select(kr, n, nu);
                for (int64_t i = 0; i < nu; ++i) out[i] = kr[i].rank;
            }
            for (int64_t i = 0; i < nu; ++i) out[i] = perm[out[i]];
            qsort(out, (size_t)nu, sizeof(int32_t), cmp_i32);
        }
        free(stamp);
        free(kr);
    }
    free(perm); free(cdf); free(wgt);
    return rc;
}

/* ------------------------------------------------------------------ values ----------- */

enum { MODEL_TINY = 0, MODEL_MOVIE = 1, MODEL_MUSIC = 2, MODEL_WIKI = 3 };

/* Planted ratings.  X* (m x fp) and Theta* (n x fp) have N(0, 1/fp) entries (streams 4 and 5,
   counter = row*fp + j); noise e ~ N(0,1) per stored entry (stream 6, counter = entry index).
   With d = x*_u . theta*_v and z = sqrt(fp) d (unit variance):
     tiny : r = d + 0.1 e
     movie: r = clip(3 + z + 0.5 e, 1, 5)
     music: r = clip(50 + 20 (z + e), 0, 100)
     wiki : r = z + 0.5 e                                                                    */
int synth_values(int model, int64_t m, int64_t n, int32_t fp, uint64_t seed,
                 const int64_t* rowptr, const int32_t* colidx, float* vals_out) {
    if (m <= 0 || n <= 0 || fp <= 0 || !rowptr || !colidx || !vals_out) return SYNTH_ERR_ARG;
    skey kx = make_key(seed, 4), kt = make_key(seed, 5), ke = make_key(seed, 6);
    const double sd = 1.0 / sqrt((double)fp);
    float* th = (float*)malloc(sizeof(float) * (size_t)n * (size_t)fp);
    if (!th) return SYNTH_ERR_NOMEM;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n * fp; ++i) th[i] = (float)(sd * normal_at(kt, (uint64_t)i));
    int rc = SYNTH_OK;
#pragma omp parallel
    {
        double* xu = (double*)malloc(sizeof(double) * (size_t)fp);
        if (!xu) {
#pragma omp atomic write
            rc = SYNTH_ERR_NOMEM;
        }
#pragma omp for schedule(dynamic, 512)
        for (int64_t u = 0; u < m; ++u) {
            if (!xu) continue;
            for (int32_t j = 0; j < fp; ++j)
                xu[j] = sd * normal_at(kx, (uint64_t)u * (uint64_t)fp + (uint64_t)j);
            for (int64_t t = rowptr[u]; t < rowptr[u + 1]; ++t) {
                const float* tv = th + (size_t)colidx[t] * (size_t)fp;
                double d = 0.0;
                for (int32_t j = 0; j < fp; ++j) d += xu[j] * (double)tv[j];
                double z = sqrt((double)fp) * d, e = normal_at(ke, (uint64_t)t), r;
                switch (model) {
                    case MODEL_TINY: r = d + 0.1 * e; break;
                    case MODEL_MOVIE: r = clamp_d(3.0 + z + 0.5 * e, 1.0, 5.0); break;
                    case MODEL_MUSIC: r = clamp_d(50.0 + 20.0 * (z + e), 0.0, 100.0); break;
                    default: r = z + 0.5 * e; break;
                }
                vals_out[t] = (float)r;
            }
        }
        free(xu);
    }
    free(th);
    return rc;
}

/* count values of N(0, std^2) from a stream (counter = element index), as fp32 */
int synth_normal(uint64_t seed, uint32_t stream, int64_t count, double std, float* out) {
    if (count < 0 || (count > 0 && !out)) return SYNTH_ERR_ARG;
    skey k = make_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) out[i] = (float)(std * normal_at(k, (uint64_t)i));
    return SYNTH_OK;
}

/* Held-out split: stored entry k goes to the test set iff the first word of Philox block
   (k, 0) of the stream is below `threshold` (threshold / 2^32 = the test fraction). */
int synth_split_mask(uint64_t seed, uint32_t stream, int64_t count, uint32_t threshold,
                     uint8_t* out) {
    if (count < 0 || (count > 0 && !out)) return SYNTH_ERR_ARG;
    skey k = make_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) out[i] = draw(k, (uint64_t)i, 0u).v[0] < threshold;
    return SYNTH_OK;
}

/* ------------------------------------------------------------------ CSR -> CSC ------- */

/* Stable counting-sort transpose: within each column the row indices stay ascending and
   the values travel with them.  Threads own contiguous row blocks and private histograms. */
int synth_transpose(int64_t m, int64_t n, const int64_t* rowptr, const int32_t* colidx,
                    const float* vals, int64_t* colptr, int32_t* rowidx, float* vals_t) {
    if (m < 0 || n <= 0 || !rowptr || !colptr) return SYNTH_ERR_ARG;
    int nt = omp_get_max_threads();
    int64_t* hist = (int64_t*)calloc((size_t)nt * (size_t)n, sizeof(int64_t));
    if (!hist) return SYNTH_ERR_NOMEM;
    const int64_t nnz = rowptr[m];
    int64_t* rb = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nt + 1));
    if (!rb) { free(hist); return SYNTH_ERR_NOMEM; }
    /* row blocks with about nnz/nt entries each */
    rb[0] = 0;
    for (int t = 1; t < nt; ++t) {
        int64_t target = nnz / nt * t, lo = rb[t - 1], hi = m;
        while (lo < hi) {
            int64_t mid = (lo + hi) >> 1;
            if (rowptr[mid] < target) lo = mid + 1; else hi = mid;
        }
        rb[t] = lo;
    }
    rb[nt] = m;
#pragma omp parallel num_threads(nt)
    {
        int t = omp_get_thread_num();
        int64_t* h = hist + (size_t)t * (size_t)n;
        for (int64_t k = rowptr[rb[t]]; k < rowptr[rb[t + 1]]; ++k) h[colidx[k]]++;
    }
    colptr[0] = 0;
    for (int64_t c = 0; c < n; ++c) {
        int64_t s = 0;
        for (int t = 0; t < nt; ++t) s += hist[(size_t)t * (size_t)n + c];
        colptr[c + 1] = colptr[c] + s;
    }
    for (int64_t c = 0; c < n; ++c) {  /* hist becomes each thread's write cursor */
        int64_t cur = colptr[c];
        for (int t = 0; t < nt; ++t) {
            int64_t s = hist[(size_t)t * (size_t)n + c];
            hist[(size_t)t * (size_t)n + c] = cur;
            cur += s;
        }
    }
#pragma omp parallel num_threads(nt)
    {
        int t = omp_get_thread_num();
        int64_t* h = hist + (size_t)t * (size_t)n;
        for (int64_t u = rb[t]; u < rb[t + 1]; ++u)
            for (int64_t k = rowptr[u]; k < rowptr[u + 1]; ++k) {
                int64_t d = h[colidx[k]]++;
                rowidx[d] = (int32_t)u;
                vals_t[d] = vals[k];
            }
    }
    free(hist);
    free(rb);
    return SYNTH_OK;
}
