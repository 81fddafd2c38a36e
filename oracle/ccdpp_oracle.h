/*
 * CPU oracle for CCD++ (Rodrigues, Jorge, Dutra: "Accelerating Recommender
 * Systems using GPUs", SAC'15; Section 3.2.2, Algorithm 3).
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, double-precision
 * reference that the GPU library is checked against.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg may load it.  It shares
 * no code, header, table or helper with the GPU library, and the GPU library
 * never calls it.
 *
 * Problem (Section 3, eq. 1): A is m x n, observed on the index set Omega
 * (triplets i, j, a_ij, 0-based).  Find W (m x k) and H (n x k) minimising
 *   sum_{(i,j) in Omega} (A_ij - w_i^T h_j)^2 + lambda (||W||_F^2 + ||H||_F^2).
 * W and H are held row-major here (row i of W is the paper's omega_i).
 *
 * All functions return 0 on success and a negative value on invalid input.
 */
#ifndef CCDPP_ORACLE_H
#define CCDPP_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct oracle_ccdpp oracle_ccdpp;

/* Copies every input.  W0 may be NULL (then W = 0, as Algorithms 2 and 3
 * initialise it); H0 must be given (n*k row-major).  The residual starts as
 * R_ij = A_ij - w_i^T h_j on Omega (Section 3.2; equal to A when W = 0).
 * Duplicate (i, j) pairs or out-of-range indices make it return NULL. */
oracle_ccdpp *oracle_create(int64_t m, int64_t n, int32_t k, double lambda,
                            int64_t nnz, const int32_t *row, const int32_t *col,
                            const double *a, const double *W0, const double *H0);
void oracle_destroy(oracle_ccdpp *o);

/* Number of OpenMP threads for the row and column loops (<= 0: all).  Every
 * output is reduced by one thread in ascending index order, so the results do
 * not depend on this setting. */
void oracle_set_threads(oracle_ccdpp *o, int32_t threads);

/* 1: build R-hat from A and the other k-1 rank-one terms (the eq. 4 form,
 * O(|Omega| k) per rank) instead of from the stored residual (eq. 13). */
void oracle_set_from_scratch(oracle_ccdpp *o, int32_t on);

/* Algorithm 3: for each of `outer` iterations, ranks t = 0..k-1 in order,
 * each one an oracle_rank(t, inner) call.  trace (optional) receives
 * outer*k*(1+2*inner) objective values, see oracle_rank. */
int oracle_run(oracle_ccdpp *o, int32_t outer, int32_t inner, double *trace);

/* The body of Algorithm 3 for feature t:
 *   R-hat = R + wbar_t hbar_t^T on Omega                      (eq. 13)
 *   u = wbar_t, v = hbar_t                                    (Algorithm 7)
 *   inner times: u_i from eq. 15 for every i, then v_j from eq. 16 for every j
 *   (wbar_t, hbar_t) = (u, v)                                 (eq. 17)
 *   R = R-hat - u v^T on Omega                                (eq. 18)
 * Optional outputs: trace[1+2*inner] = objective of eq. 1 with (u, v) in
 * place of feature t, before the first update and after every u- and
 * v-block; rhat[nnz] = R-hat in input order; u_hist[inner*m], v_hist[inner*n]
 * = u and v after each inner iteration. */
int oracle_rank(oracle_ccdpp *o, int32_t t, int32_t inner, double *trace,
                double *rhat, double *u_hist, double *v_hist);

/* Algorithm 3 with its outer loop left open ("until convergence", Section
 * 3.2.2): outer iterations of oracle_run(o, 1, inner), each followed by the
 * objective f of eq. 1; stop after iteration o >= 2 when f_(o-1) - f_o <=
 * rel_tol * f_(o-1), or after max_outer iterations (rel_tol < 0: never early).
 * history (optional, 3 per iteration run): f, the training RMSE and the RMSE
 * on the held-out triplets (NaN when test_nnz == 0).  Returns the number of
 * iterations run, or a negative value on invalid input. */
int oracle_run_until(oracle_ccdpp *o, int32_t max_outer, int32_t inner, double rel_tol,
                     int64_t test_nnz, const int32_t *test_row, const int32_t *test_col,
                     const double *test_a, double *history);

/* Algorithm 2 (element-wise CCD): `outer` iterations of, for every row i and
 * feature t, eq. 5 then eq. 6-7, followed by, for every column j and feature
 * t, eq. 8 then eq. 9-10. */
int oracle_ccd_run(oracle_ccdpp *o, int32_t outer);

/* Current factors, row-major (either pointer may be NULL). */
int oracle_get_factors(const oracle_ccdpp *o, double *W, double *H);
/* Current residual R in input (triplet) order. */
int oracle_get_residual(const oracle_ccdpp *o, double *R);
/* Objective of eq. 1 at the current W, H (computed from the residual). */
double oracle_objective(const oracle_ccdpp *o);
/* sqrt(sum_Omega R^2 / |Omega|); -1 if Omega is empty. */
double oracle_train_rmse(const oracle_ccdpp *o);
/* sqrt(mean (a - w_i^T h_j)^2) over the given triplets; -1 on bad input. */
double oracle_test_rmse(const oracle_ccdpp *o, int64_t nnz, const int32_t *row,
                        const int32_t *col, const double *a);

#ifdef __cplusplus
}
#endif
#endif
