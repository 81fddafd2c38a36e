/*
 * CPU oracle for CCD++ -- TEST INFRASTRUCTURE ONLY (see ccdpp_oracle.h).
 *
 * Plain double-precision C written from the paper's equations and the order
 * of Algorithm 3 (Section 3.2.2).  Nothing here is blocked, fused or
 * reordered beyond what those definitions state: R-hat is built for all of
 * Omega, then u and v are updated inner times, then the factors are committed
 * and the residual is updated, exactly in that order.
 *
 * Storage: the observed entries are kept once, in row order (rows ascending,
 * columns ascending inside a row).  Column access goes through a list of row
 * positions sorted by (column, row).  Every sum runs in ascending index order
 * inside one thread.
 */
#include "ccdpp_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

struct oracle_ccdpp {
    int64_t m, n, nnz;
    int32_t k;
    double lambda;
    /* row-ordered entries */
    int64_t *rp;    /* [m+1] row start */
    int32_t *rcol;  /* [nnz] column of each row-ordered entry */
    int64_t *src;   /* [nnz] input (triplet) index of each row-ordered entry */
    /* column access */
    int64_t *cp;    /* [n+1] column start */
    int32_t *crow;  /* [nnz] row of each column-ordered entry */
    int64_t *cpos;  /* [nnz] row-ordered position of each column-ordered entry */
    double *A;      /* [nnz] ratings, row order */
    double *R;      /* [nnz] residual A - W H^T, row order */
    double *Rh;     /* [nnz] R-hat of the rank being updated, row order */
    double *W;      /* [m*k] row-major */
    double *H;      /* [n*k] row-major */
    double *u, *v;  /* [m], [n] */
    int32_t threads;
    int32_t from_scratch;
};

static int nthreads(const oracle_ccdpp *o) {
#ifdef _OPENMP
    return o->threads > 0 ? o->threads : omp_get_max_threads();
#else
    (void)o;
    return 1;
#endif
}

/* Stable counting sort of the index list `in` by key[in[e]] (0 <= key < nkeys). */
static void counting_sort(int64_t N, const int32_t *key, int64_t nkeys,
                          const int64_t *in, int64_t *out, int64_t *start) {
    int64_t *cnt = calloc((size_t)nkeys + 1, sizeof(int64_t));
    for (int64_t e = 0; e < N; ++e) cnt[key[in[e]] + 1]++;
    for (int64_t b = 0; b < nkeys; ++b) cnt[b + 1] += cnt[b];
    if (start) memcpy(start, cnt, ((size_t)nkeys + 1) * sizeof(int64_t));
    for (int64_t e = 0; e < N; ++e) out[cnt[key[in[e]]]++] = in[e];
    free(cnt);
}

void oracle_destroy(oracle_ccdpp *o) {
    if (!o) return;
    free(o->rp); free(o->rcol); free(o->src);
    free(o->cp); free(o->crow); free(o->cpos);
    free(o->A); free(o->R); free(o->Rh);
    free(o->W); free(o->H); free(o->u); free(o->v);
    free(o);
}

/* w_i^T h_j */
static double dot_wh(const oracle_ccdpp *o, int64_t i, int64_t j) {
    double s = 0.0;
    for (int32_t t = 0; t < o->k; ++t) s += o->W[i * o->k + t] * o->H[j * o->k + t];
    return s;
}

oracle_ccdpp *oracle_create(int64_t m, int64_t n, int32_t k, double lambda,
                            int64_t nnz, const int32_t *row, const int32_t *col,
                            const double *a, const double *W0, const double *H0) {
    if (m < 1 || n < 1 || k < 1 || nnz < 0 || !(lambda >= 0.0) || !H0) return NULL;
    if (nnz > 0 && (!row || !col || !a)) return NULL;
    for (int64_t e = 0; e < nnz; ++e)
        if (row[e] < 0 || row[e] >= m || col[e] < 0 || col[e] >= n) return NULL;

    oracle_ccdpp *o = calloc(1, sizeof *o);
    o->m = m; o->n = n; o->nnz = nnz; o->k = k; o->lambda = lambda;
    size_t N = (size_t)nnz ? (size_t)nnz : 1;
    o->rp = malloc(((size_t)m + 1) * sizeof(int64_t));
    o->cp = malloc(((size_t)n + 1) * sizeof(int64_t));
    o->rcol = malloc(N * sizeof(int32_t));
    o->crow = malloc(N * sizeof(int32_t));
    o->src = malloc(N * sizeof(int64_t));
    o->cpos = malloc(N * sizeof(int64_t));
    o->A = malloc(N * sizeof(double));
    o->R = malloc(N * sizeof(double));
    o->Rh = malloc(N * sizeof(double));
    o->W = calloc((size_t)m * k, sizeof(double));
    o->H = malloc((size_t)n * k * sizeof(double));
    o->u = calloc((size_t)m, sizeof(double));
    o->v = calloc((size_t)n, sizeof(double));

    /* Row order (row, then column): two stable counting sorts, column first. */
    int64_t *id = malloc(N * sizeof(int64_t));
    int64_t *tmp = malloc(N * sizeof(int64_t));
    for (int64_t e = 0; e < nnz; ++e) id[e] = e;
    counting_sort(nnz, col, n, id, tmp, NULL);
    counting_sort(nnz, row, m, tmp, o->src, o->rp);
    /* Column order (column, then row). */
    counting_sort(nnz, row, m, id, tmp, NULL);
    int64_t *csrc = id; /* reuse: column-ordered input indices */
    counting_sort(nnz, col, n, tmp, csrc, o->cp);
    /* input index -> row-ordered position */
    for (int64_t p = 0; p < nnz; ++p) tmp[o->src[p]] = p;
    for (int64_t q = 0; q < nnz; ++q) {
        o->cpos[q] = tmp[csrc[q]];
        o->crow[q] = row[csrc[q]];
    }
    free(id); free(tmp);
    for (int64_t p = 0; p < nnz; ++p) {
        o->rcol[p] = col[o->src[p]];
        o->A[p] = a[o->src[p]];
    }
    /* Omega is a set: reject repeated (i, j). */
    for (int64_t i = 0; i < m; ++i)
        for (int64_t p = o->rp[i] + 1; p < o->rp[i + 1]; ++p)
            if (o->rcol[p] == o->rcol[p - 1]) { oracle_destroy(o); return NULL; }

    if (W0) memcpy(o->W, W0, (size_t)m * k * sizeof(double));
    memcpy(o->H, H0, (size_t)n * k * sizeof(double));
    /* R_ij = A_ij - w_i^T h_j on Omega. */
    for (int64_t i = 0; i < m; ++i)
        for (int64_t p = o->rp[i]; p < o->rp[i + 1]; ++p)
            o->R[p] = o->A[p] - dot_wh(o, i, o->rcol[p]);
    return o;
}

void oracle_set_threads(oracle_ccdpp *o, int32_t threads) { o->threads = threads; }
void oracle_set_from_scratch(oracle_ccdpp *o, int32_t on) { o->from_scratch = on; }

/* Closed-form minimiser of sum (rhat - z x)^2 + lambda z^2: num / (lambda + den).
 * With lambda = 0 and nothing observed the minimiser is taken as 0. */
static double coord(double num, double den, double lambda) {
    double d = lambda + den;
    return d == 0.0 ? 0.0 : num / d;
}

/* Objective of eq. 1 during the update of feature t, with (u, v) in place of
 * (wbar_t, hbar_t): sum (Rh - u_i v_j)^2 + lambda (||W_{-t}||^2 + ||H_{-t}||^2
 * + ||u||^2 + ||v||^2). */
static double objective_in_rank(const oracle_ccdpp *o, int32_t t) {
    double f = 0.0;
    for (int64_t i = 0; i < o->m; ++i)
        for (int64_t p = o->rp[i]; p < o->rp[i + 1]; ++p) {
            double e = o->Rh[p] - o->u[i] * o->v[o->rcol[p]];
            f += e * e;
        }
    double reg = 0.0;
    for (int64_t i = 0; i < o->m; ++i)
        for (int32_t s = 0; s < o->k; ++s) {
            double w = s == t ? o->u[i] : o->W[i * o->k + s];
            reg += w * w;
        }
    for (int64_t j = 0; j < o->n; ++j)
        for (int32_t s = 0; s < o->k; ++s) {
            double h = s == t ? o->v[j] : o->H[j * o->k + s];
            reg += h * h;
        }
    return f + o->lambda * reg;
}

int oracle_rank(oracle_ccdpp *o, int32_t t, int32_t inner, double *trace,
                double *rhat, double *u_hist, double *v_hist) {
    if (t < 0 || t >= o->k || inner < 1) return -1;
    const int64_t m = o->m, n = o->n, k = o->k;
    const double lam = o->lambda;
    const int nt = nthreads(o);

    /* R-hat_ij = R_ij + wbar_ti hbar_tj on Omega (eq. 13), or, in the
     * from-scratch mode, A_ij minus the other k-1 rank-one terms (eq. 4). */
    #pragma omp parallel for schedule(dynamic, 256) num_threads(nt)
    for (int64_t i = 0; i < m; ++i)
        for (int64_t p = o->rp[i]; p < o->rp[i + 1]; ++p) {
            int64_t j = o->rcol[p];
            if (o->from_scratch) {
                double s = 0.0;
                for (int64_t q = 0; q < k; ++q)
                    if (q != t) s += o->W[i * k + q] * o->H[j * k + q];
                o->Rh[p] = o->A[p] - s;
            } else {
                o->Rh[p] = o->R[p] + o->W[i * k + t] * o->H[j * k + t];
            }
        }
    if (rhat)
        for (int64_t p = 0; p < o->nnz; ++p) rhat[o->src[p]] = o->Rh[p];

    /* Start from the current feature pair: u = wbar_t, v = hbar_t (Algorithm 7). */
    for (int64_t i = 0; i < m; ++i) o->u[i] = o->W[i * k + t];
    for (int64_t j = 0; j < n; ++j) o->v[j] = o->H[j * k + t];
    if (trace) trace[0] = objective_in_rank(o, t);

    for (int32_t s = 0; s < inner; ++s) {
        /* u_i = sum_{j in Omega_i} Rh_ij v_j / (lambda + sum_{j in Omega_i} v_j^2)  (eq. 15) */
        #pragma omp parallel for schedule(dynamic, 256) num_threads(nt)
        for (int64_t i = 0; i < m; ++i) {
            double num = 0.0, den = 0.0;
            for (int64_t p = o->rp[i]; p < o->rp[i + 1]; ++p) {
                double vj = o->v[o->rcol[p]];
                num += o->Rh[p] * vj;
                den += vj * vj;
            }
            o->u[i] = coord(num, den, lam);
        }
        if (trace) trace[1 + 2 * s] = objective_in_rank(o, t);
        if (u_hist) memcpy(u_hist + (int64_t)s * m, o->u, (size_t)m * sizeof(double));

        /* v_j = sum_{i in Omega-bar_j} Rh_ij u_i / (lambda + sum_{i in Omega-bar_j} u_i^2)
         * (eq. 16; the paper prints u_j in the numerator, which is read as u_i:
         * only u_i makes this the minimiser of eq. 14 in v_j). */
        #pragma omp parallel for schedule(dynamic, 64) num_threads(nt)
        for (int64_t j = 0; j < n; ++j) {
            double num = 0.0, den = 0.0;
            for (int64_t q = o->cp[j]; q < o->cp[j + 1]; ++q) {
                double ui = o->u[o->crow[q]];
                num += o->Rh[o->cpos[q]] * ui;
                den += ui * ui;
            }
            o->v[j] = coord(num, den, lam);
        }
        if (trace) trace[2 + 2 * s] = objective_in_rank(o, t);
        if (v_hist) memcpy(v_hist + (int64_t)s * n, o->v, (size_t)n * sizeof(double));
    }

    /* (wbar_t, hbar_t) = (u, v)  (eq. 17) */
    for (int64_t i = 0; i < m; ++i) o->W[i * k + t] = o->u[i];
    for (int64_t j = 0; j < n; ++j) o->H[j * k + t] = o->v[j];

    /* R_ij = R-hat_ij - u_i v_j on Omega  (eq. 18) */
    #pragma omp parallel for schedule(dynamic, 256) num_threads(nt)
    for (int64_t i = 0; i < m; ++i)
        for (int64_t p = o->rp[i]; p < o->rp[i + 1]; ++p)
            o->R[p] = o->Rh[p] - o->u[i] * o->v[o->rcol[p]];
    return 0;
}

int oracle_run(oracle_ccdpp *o, int32_t outer, int32_t inner, double *trace) {
    if (outer < 0 || inner < 1) return -1;
    const int64_t per = 1 + 2 * (int64_t)inner;
    for (int32_t it = 0; it < outer; ++it)
        for (int32_t t = 0; t < o->k; ++t) {
            double *tr = trace ? trace + ((int64_t)it * o->k + t) * per : NULL;
            int rc = oracle_rank(o, t, inner, tr, NULL, NULL, NULL);
            if (rc) return rc;
        }
    return 0;
}

int oracle_run_until(oracle_ccdpp *o, int32_t max_outer, int32_t inner, double rel_tol,
                     int64_t test_nnz, const int32_t *test_row, const int32_t *test_col,
                     const double *test_a, double *history) {
    if (max_outer < 0 || inner < 1 || test_nnz < 0) return -1;
    if (test_nnz > 0 && (!test_row || !test_col || !test_a)) return -1;
    double prev = 0.0;
    int32_t done = 0;
    for (int32_t it = 0; it < max_outer; ++it) {
        int rc = oracle_run(o, 1, inner, NULL);
        if (rc) return rc;
        const double f = oracle_objective(o);
        if (history) {
            history[3 * (int64_t)it] = f;
            history[3 * (int64_t)it + 1] = o->nnz > 0 ? oracle_train_rmse(o) : 0.0;
            history[3 * (int64_t)it + 2] =
                test_nnz > 0 ? oracle_test_rmse(o, test_nnz, test_row, test_col, test_a) : NAN;
        }
        done = it + 1;
        if (it >= 1 && rel_tol >= 0.0 && prev - f <= rel_tol * prev) break;
        prev = f;
    }
    return done;
}

int oracle_ccd_run(oracle_ccdpp *o, int32_t outer) {
    if (outer < 0) return -1;
    const int64_t m = o->m, n = o->n, k = o->k;
    const double lam = o->lambda;
    const int nt = nthreads(o);
    for (int32_t it = 0; it < outer; ++it) {
        /* Update W: rows touch disjoint residual entries, so rows may run in parallel. */
        #pragma omp parallel for schedule(dynamic, 64) num_threads(nt)
        for (int64_t i = 0; i < m; ++i)
            for (int64_t t = 0; t < k; ++t) {
                double w = o->W[i * k + t], num = 0.0, den = 0.0;
                for (int64_t p = o->rp[i]; p < o->rp[i + 1]; ++p) {
                    double h = o->H[(int64_t)o->rcol[p] * k + t];
                    num += (o->R[p] + w * h) * h;          /* eq. 5 */
                    den += h * h;
                }
                double z = coord(num, den, lam);
                for (int64_t p = o->rp[i]; p < o->rp[i + 1]; ++p) {
                    double h = o->H[(int64_t)o->rcol[p] * k + t];
                    o->R[p] -= (z - w) * h;                /* eq. 6 */
                }
                o->W[i * k + t] = z;                       /* eq. 7 */
            }
        /* Update H. */
        #pragma omp parallel for schedule(dynamic, 16) num_threads(nt)
        for (int64_t j = 0; j < n; ++j)
            for (int64_t t = 0; t < k; ++t) {
                double h = o->H[j * k + t], num = 0.0, den = 0.0;
                for (int64_t q = o->cp[j]; q < o->cp[j + 1]; ++q) {
                    double w = o->W[(int64_t)o->crow[q] * k + t];
                    num += (o->R[o->cpos[q]] + w * h) * w; /* eq. 8 */
                    den += w * w;
                }
                double s = coord(num, den, lam);
                for (int64_t q = o->cp[j]; q < o->cp[j + 1]; ++q) {
                    double w = o->W[(int64_t)o->crow[q] * k + t];
                    o->R[o->cpos[q]] -= (s - h) * w;       /* eq. 9 */
                }
                o->H[j * k + t] = s;                       /* eq. 10 */
            }
    }
    return 0;
}

int oracle_get_factors(const oracle_ccdpp *o, double *W, double *H) {
    if (W) memcpy(W, o->W, (size_t)o->m * o->k * sizeof(double));
    if (H) memcpy(H, o->H, (size_t)o->n * o->k * sizeof(double));
    return 0;
}

int oracle_get_residual(const oracle_ccdpp *o, double *R) {
    if (!R && o->nnz) return -1;
    for (int64_t p = 0; p < o->nnz; ++p) R[o->src[p]] = o->R[p];
    return 0;
}

double oracle_objective(const oracle_ccdpp *o) {
    double f = 0.0, reg = 0.0;
    for (int64_t p = 0; p < o->nnz; ++p) f += o->R[p] * o->R[p];
    for (int64_t e = 0; e < o->m * o->k; ++e) reg += o->W[e] * o->W[e];
    for (int64_t e = 0; e < o->n * o->k; ++e) reg += o->H[e] * o->H[e];
    return f + o->lambda * reg;
}

double oracle_train_rmse(const oracle_ccdpp *o) {
    if (o->nnz == 0) return -1.0;
    double s = 0.0;
    for (int64_t p = 0; p < o->nnz; ++p) s += o->R[p] * o->R[p];
    return sqrt(s / (double)o->nnz);
}

double oracle_test_rmse(const oracle_ccdpp *o, int64_t nnz, const int32_t *row,
                        const int32_t *col, const double *a) {
    if (nnz <= 0 || !row || !col || !a) return -1.0;
    double s = 0.0;
    for (int64_t e = 0; e < nnz; ++e) {
        if (row[e] < 0 || row[e] >= o->m || col[e] < 0 || col[e] >= o->n) return -1.0;
        double err = a[e] - dot_wh(o, row[e], col[e]);
        s += err * err;
    }
    return sqrt(s / (double)nnz);
}
