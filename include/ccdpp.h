/*
 * ccdpp.h -- C ABI of the MI355X (gfx950) CCD++ library.
 *
 * CCD++ is the feature-wise cyclic coordinate descent for matrix
 * factorization of Rodrigues, Jorge and Dutra, "Accelerating Recommender
 * Systems using GPUs" (SAC'15), Section 3.2.2 (eq. 11-18, Algorithm 3), with
 * the row/column data parallelism of Section 6 (eq. 19-23) and the device
 * residency of Section 7 (Algorithm 7).
 *
 * Problem (Section 3, eq. 1): a sparse m x n rating matrix A is given as
 * triplets (i, j, a_ij) on the observed set Omega.  The library finds
 * W (m x k) and H (n x k) that minimise
 *     sum_{(i,j) in Omega} (A_ij - w_i^T h_j)^2 + lambda (||W||_F^2 + ||H||_F^2)
 * by sweeping the k features in order; for feature t it builds
 * R-hat = R + wbar_t hbar_t^T on Omega (eq. 13), alternates the closed-form
 * updates u_i = sum_j R-hat_ij v_j / (lambda + sum_j v_j^2) (eq. 15) and
 * v_j = sum_i R-hat_ij u_i / (lambda + sum_i u_i^2) (eq. 16) inner_iters
 * times, commits (wbar_t, hbar_t) = (u, v) (eq. 17) and updates the residual
 * R = R-hat - u v^T (eq. 18).
 *
 * Conventions for every call:
 *  - Indices are 0-based int32; m and n must be below 2^28 (the passes
 *    address gathered records of up to 16 bytes with 32-bit byte offsets) and
 *    nnz at most 2^31 - 1.
 *  - Every array argument is HOST memory owned by the caller.  The library
 *    copies what it needs during the call and keeps no pointer to it.
 *  - Factor matrices at the boundary are row-major float32: W is m x k
 *    (row i = w_i), H is n x k (row j = h_j).
 *  - The handle owns all device memory (on the device that was current at
 *    ccdpp_create) and is not thread-safe.  Every call on a handle makes
 *    that device current while it runs and restores the caller's afterwards.
 *  - Calls return CCDPP_OK (0) or a negative status.  Out-parameters are left
 *    untouched on error.  After a device error the handle answers every
 *    later call with CCDPP_ESTATE until it is destroyed.  A failed device
 *    allocation (ENOMEM) is reported before the call changes any state, so
 *    the handle stays usable.
 *  - Calls that compute are blocking: they synchronise the handle's stream
 *    before returning.
 */
#ifndef CCDPP_H
#define CCDPP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ccdpp ccdpp_t;

enum ccdpp_status {
    CCDPP_OK = 0,
    CCDPP_EINVAL = -1,   /* bad argument: size, range, NULL pointer, non-finite value */
    CCDPP_EDUP = -2,     /* a position (i, j) occurs twice; Omega is a set (Section 3) */
    CCDPP_ENOMEM = -3,   /* device or host allocation failed */
    CCDPP_EDEVICE = -4,  /* HIP runtime error, or no usable gfx950 device */
    CCDPP_ESTATE = -5    /* handle poisoned by an earlier device error, or NULL handle */
};

/*
 * Create a factorization problem from training triplets (Section 3: A as
 * triplets i, j, a_ij; Algorithms 3 and 7: W = 0, R = A).
 *   m, n    : rows (users) and columns (items), 1 <= m, n < 2^28
 *   k       : number of features, >= 1
 *   lambda  : regularisation of eq. 1, finite and >= 0
 *   nnz     : number of observed entries, 0 <= nnz <= 2^31 - 1
 *   row,col : int32[nnz] positions (may be NULL when nnz == 0)
 *   val     : float32[nnz] ratings, finite
 *   seed    : seed of the initial H, drawn N(0, 0.01) (standard deviation
 *             0.1) from a counter-based generator; ccdpp_set_factors
 *             replaces it with caller-supplied values
 *   out     : receives the handle
 * Validation of sizes, ranges and values happens on the host before any HIP
 * call.  Returns EDUP if a position repeats, ENOMEM or EDEVICE on device
 * failure.  The device layout (user-major and item-major copies of the
 * residual, tiled so that the gathered vectors fit in LDS, the map between
 * them and the equal-work schedule of persistent workgroups) is built on the
 * device during this call.
 */
int ccdpp_create(int64_t m, int64_t n, int32_t k, double lambda, int64_t nnz,
                 const int32_t *row, const int32_t *col, const float *val,
                 uint64_t seed, ccdpp_t **out);

/*
 * Tuning and testing knobs of the device layout (all zero = automatic, which
 * is what ccdpp_create uses).  Index 0 is the user-major copy read by the
 * u-passes of eq. 15, index 1 the item-major copy read by the v-passes of
 * eq. 16.
 *   gather_mode : 0 automatic; 1 gather the other side's coordinates from
 *                 global memory; 2 stage them in LDS, cut into tiles of
 *                 tile_width columns when they do not fit; 3 (hot) stage
 *                 the leading tile_width columns, the most frequent ones,
 *                 and gather the others from global memory (automatic
 *                 mode takes it when tiles would hold too few entries per
 *                 row)
 *   tile_width  : columns per LDS tile (0: as wide as LDS allows); at most
 *                 (163840 - 512) / (b * v) - 64, rounded down to a multiple of 64,
 *                 where b is the bytes per value (4, or 8 with precision 1)
 *                 and v = 2 for index 0 and 3 for index 1 (the vectors the
 *                 first pass of a feature stages).  With gather_mode 3, the
 *                 hot width: a multiple of 32, at most (163840 - 512) / b - 64
 *                 rounded down to a multiple of 64 (0: that maximum); each
 *                 pass stages as much of it as its vectors leave room for
 *   workgroups  : persistent workgroups per pass (0: two per compute unit,
 *                 one for copies of fewer than about 33.5M entries, four for
 *                 copies of more than about 252M, padding included)
 *   seg_weight  : work of one row segment, in entries, when the entries are
 *                 shared out among workgroups and waves (0: the default, 4;
 *                 -1: shares by entries alone)
 *   precision   : 0 float32 residual, factors and sweep arithmetic (the
 *                 paper's float version, Section 8); 1 float64 throughout
 *                 (its double version).  Partial sums across windows and the
 *                 coordinate division are float64 in both.
 *   cache       : how the passes access the copy's residual: 0 automatic;
 *                 1 streaming (non-temporal loads and stores); 2 streaming
 *                 loads and write-back stores of the updated residual;
 *                 3 cached loads and write-back stores.  2 and 3 need a
 *                 copy staged in LDS (gather_mode 2) with precision 0, else
 *                 create fails with EINVAL.  Automatic: 3 on both copies
 *                 when their residual streams (values and indices) total at
 *                 most 160 MB, so that they stay in the memory-side cache;
 *                 otherwise 2 on one copy and 1 on the other: the item-major
 *                 copy takes the 2 when it is staged in LDS and not split,
 *                 else a user-major copy staged with one tile does (neither
 *                 does when the other copy's policy is given as 2 or 3); an
 *                 automatic 2 applies to ccdpp_run and ccdpp_run_until with
 *                 inner_iters >= 2 only (elsewhere the copy streams).
 *   index_coding: 0 automatic: in a copy staged in LDS with 16-bit indices
 *                 (gather_mode 2 and fewer than 32,768 tile columns) whose
 *                 cache policy is not 3, every window of 512 entries whose
 *                 lanes' sorted columns climb by at most 2047 from one entry
 *                 to the next stores its indices delta-coded, 12 bytes per 8
 *                 entries instead of 16; 1 plain 16-bit indices everywhere.
 *   split_rows  : the item-major copy only.  0 automatic: when tiles of the
 *                 whole copy would hold too few entries per row segment (where
 *                 it would otherwise become hot), its leading items (the ones
 *                 with the most ratings) may be tiled and the others kept hot,
 *                 if their segments cost less than the gathers from global
 *                 memory they save; -1 never split; n1 > 0 (needs
 *                 gather_mode[1] = 0 and n1 < n) tile the n1 items with the most
 *                 ratings, the others hot.  The two parts are passed over one
 *                 after the other, as one pass of the copy.
 * Results differ between layouts only by floating-point summation order; the
 * cache policy and the index coding do not change them.
 */
typedef struct ccdpp_options {
    int32_t gather_mode[2];
    int32_t tile_width[2];
    int32_t workgroups;
    int32_t seg_weight;
    int32_t precision;
    int32_t cache[2];
    int32_t index_coding[2];
    int32_t split_rows;
} ccdpp_options_t;

/* ccdpp_create with explicit layout options (opts may be NULL). */
int ccdpp_create_ex(int64_t m, int64_t n, int32_t k, double lambda, int64_t nnz,
                    const int32_t *row, const int32_t *col, const float *val,
                    uint64_t seed, const ccdpp_options_t *opts, ccdpp_t **out);

/*
 * Run outer_iters iterations of Algorithm 3 (each sweeps features t = 0..k-1
 * in order), each feature with inner_iters alternations of eq. 15 then
 * eq. 16.  outer_iters >= 0, inner_iters >= 1.  State (W, H, residual)
 * persists across calls: two calls of 1 outer iteration give bitwise the
 * same result as one call of 2.  Blocking.  W and H are final on return; the
 * residual update of the last feature (eq. 18) is left pending and applied by
 * the first passes of the next ccdpp_run, or before any call that reads the
 * residual (ccdpp_train_rmse, ccdpp_get_residual, ccdpp_check_consistency,
 * ccdpp_ccd_run), so a run split into calls costs what one call does.
 */
int ccdpp_run(ccdpp_t *h, int32_t outer_iters, int32_t inner_iters);

/* Algorithm 2, element-wise CCD (Section 3.2.1): outer_iters iterations of,
 * for every row i and feature t in order, w_it from eq. 5 with the residual
 * update of eq. 6-7, then for every column j and feature t, h_jt from eq. 8
 * with eq. 9-10.  Same state as ccdpp_run (the two may be mixed), the same
 * float or double arithmetic.  outer_iters >= 0.  Blocking. */
int ccdpp_ccd_run(ccdpp_t *h, int32_t outer_iters);

/* Algorithm 3 with its outer loop left open (Section 3.2.2: iterate until
 * convergence or a bound on the iterations): outer iterations of
 * ccdpp_run(h, 1, inner_iters), each followed by the objective f of eq. 1
 * (float64: the training sum of squares plus lambda (||W||^2 + ||H||^2)).
 * Stops after iteration o >= 2 when f_(o-1) - f_o <= rel_tol * f_(o-1), or
 * after max_outer iterations; rel_tol < 0 never stops early.
 *   test_nnz, test_row/col/val : held-out triplets (host memory, copied once),
 *                                or test_nnz = 0 and NULL pointers
 *   history    : NULL, or 3 * max_outer doubles; iteration o writes f, the
 *                training RMSE and the held-out RMSE (NaN without a test set)
 *                at history[3 o .. 3 o + 2]
 *   outer_done : receives the number of outer iterations run (not NULL)
 * Arguments are checked before any iteration runs (EINVAL).  Blocking. */
int ccdpp_run_until(ccdpp_t *h, int32_t max_outer, int32_t inner_iters, double rel_tol,
                    int64_t test_nnz, const int32_t *test_row, const int32_t *test_col,
                    const float *test_val, double *history, int32_t *outer_done);

/* Copy the factors out (Section 3: W in R^(m x k) profiles the users, row i
 * being w_i; H in R^(n x k) profiles the items, row j being h_j; together they
 * minimise eq. 1.  Algorithm 7 ends with them on the host, its columns
 * wbar_t, hbar_t having been committed by eq. 17).
 *   W : NULL, or m * k floats, written row-major (W[i * k + t] = w_it)
 *   H : NULL, or n * k floats, written row-major (H[j * k + t] = h_jt)
 * Host memory owned by the caller.  Either pointer may be NULL to skip it.
 * A float64 handle rounds its factors to float32 here.  Returns ESTATE on a
 * NULL or poisoned handle.  Blocking. */
int ccdpp_get_factors(ccdpp_t *h, float *W, float *H);
/* The same in float64 (exact for a float64 handle). */
int ccdpp_get_factors_f64(ccdpp_t *h, double *W, double *H);

/* Replace the factors (row-major m x k and n x k, finite; either may be NULL
 * to keep the current one) and rebuild the residual R = A - W H^T on Omega
 * (Section 3.2) on the device.  Blocking. */
int ccdpp_set_factors(ccdpp_t *h, const float *W, const float *H);
/* The same from float64 arrays (rounded to float on a float32 handle). */
int ccdpp_set_factors_f64(ccdpp_t *h, const double *W, const double *H);

/* Root mean squared error of the predictions w_i^T h_j against held-out
 * triplets (Section 8: RMSE on the probe set; predictions are not clipped):
 * sqrt(sum (a - w_i^T h_j)^2 / nnz), accumulated in float64 on the device in
 * a fixed order.  nnz >= 1; indices must be in range.  Blocking. */
int ccdpp_rmse(ccdpp_t *h, int64_t nnz, const int32_t *row, const int32_t *col,
               const float *val, double *rmse_out);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): ccdpp_rmse with the
 * held-out triplets already in DEVICE memory, on the handle's device.  It
 * allocates nothing: its partial sums live in a fixed device array of
 * 16,400 bytes (1024 partial sums, 1024 per-block counts, two totals), one per
 * device the library has run on, held until the process ends.  Every call on
 * one device shares that array, so calls that overlap on one device (two
 * handles on two streams) race; calls in sequence do not.
 *   row, col : device int32[nnz] held-out positions
 *   val      : device float32[nnz] held-out ratings
 *   nnz      : 1 <= nnz <= 2^31 - 1; the array's size does not depend on it
 *   rmse_out : receives the RMSE (host memory)
 * The triplets are checked on the device: entries out of range or not finite are
 * never used as indices, and any such entry makes the call return EINVAL.  On
 * valid triplets the result is bitwise that of ccdpp_rmse (the same kernel and
 * the same fixed order).  Blocking. */
int ccdpp_rmse_noalloc(ccdpp_t *h, int64_t nnz, const int32_t *row, const int32_t *col,
                       const float *val, double *rmse_out);

/* Training RMSE of the current factors: the RMSE of Section 8 evaluated on
 * the training set itself, from the residual of Section 3.2
 * (R_ij = A_ij - w_i^T h_j on Omega, kept up to date by eq. 18):
 * sqrt(sum_{Omega} R_ij^2 / nnz), accumulated in float64 on the device in a
 * fixed order.  A residual update left pending by ccdpp_run is applied first.
 *   rmse_out : receives the RMSE (host memory, not NULL)
 * Returns EINVAL when the handle holds no observed entries (nnz = 0) or
 * rmse_out is NULL.  Blocking. */
int ccdpp_train_rmse(ccdpp_t *h, double *rmse_out);

/* Residual R in the order of the triplets given to ccdpp_create
 * (float32[nnz]).  Diagnostic.  Blocking. */
int ccdpp_get_residual(ccdpp_t *h, float *R);
/* The same in float64 (exact for a float64 handle). */
int ccdpp_get_residual_f64(ccdpp_t *h, double *R);

/* Count the observed entries whose residual differs, bit for bit, between
 * the row-compressed and the column-compressed device copies (0 when the two
 * copies are consistent).  Diagnostic.  Blocking. */
int ccdpp_check_consistency(ccdpp_t *h, int64_t *mismatches);

/* Use this HIP stream (a hipStream_t, e.g. PyTorch's current stream) for all
 * later work; NULL selects the device's null stream, which a handle uses from
 * its creation on (the device build included).  The stream must belong to the
 * handle's device and outlive its use.  Waits for the work already enqueued on
 * the previous stream. */
int ccdpp_set_stream(ccdpp_t *h, void *hip_stream);

/* Kernel timing.  When enabled, every kernel launch of ccdpp_run is bracketed
 * by HIP events on the handle's stream and accumulated per kernel kind
 * (CCDPP_K_*) and per residual copy (layout 0: row-compressed, the u-passes of
 * eq. 15; layout 1: column-compressed, the v-passes of eq. 16; -1: both):
 * launch count, summed device time in milliseconds, and the algorithmic bytes
 * those launches had to move (index and value arrays, residual writes,
 * per-row scalars and outputs, and one read of each gathered vector).  Enabling or disabling clears the counters. */
enum ccdpp_kernel_kind {
    CCDPP_K_PASS_FUSED = 0,  /* first u- or v-pass of a feature: eq. 18 of the previous
                                feature, eq. 13, then eq. 15 or eq. 16 */
    CCDPP_K_PASS = 1,        /* later u- or v-passes: eq. 15 or eq. 16 on R-hat */
    CCDPP_K_COMBINE = 2,     /* fixed-order combine of split heavy rows */
    CCDPP_K_COMMIT = 3,      /* eq. 17 when inner_iters == 1 */
    CCDPP_K_FLUSH = 4,       /* final eq. 18 and the training sum of squares */
    CCDPP_K_COUNT = 5
};
int ccdpp_profile(ccdpp_t *h, int32_t enable);
/* Restrict kernel timing to launches of one kind (CCDPP_K_*) on one residual
 * copy (0 or 1); -1 for either means all.  Fewer events disturb the stream
 * less.  The selection persists until changed; the default is all. */
int ccdpp_profile_only(ccdpp_t *h, int32_t kind, int32_t layout);
/* Time only every `every`-th launch that the selection matches (the first, then
 * every `every`-th after it); fewer events, less disturbance, the same means.
 * every >= 1; the default is 1.  Persists until changed. */
int ccdpp_profile_every(ccdpp_t *h, int32_t every);
int ccdpp_profile_read(ccdpp_t *h, int32_t kind, int32_t layout, int64_t *launches,
                       double *total_ms, double *algo_bytes);

/* Sizes and schedule of the handle: fills up to `len` int64 values of
 *   [0] m, [1] n, [2] nnz, [3] k, [4] device build time in microseconds,
 *   [5] user-major copy gather mode (1 global memory, 2 LDS-staged, 3 hot),
 *   [6] its number of tiles P, [7] tile width T (hot: the hot width), [8] persistent workgroups per
 *   pass, [9] row segments, [10..14] the same five for the item-major copy,
 *   [15] device bytes held, [16] bytes per value (4: float, 8: double),
 *   [17] user-major rows that the workgroups of a pass finish themselves (cut
 *   between the waves of one workgroup), [18] rows the combine kernel finishes
 *   after each pass, [19..20] the same two for the item-major copy,
 *   [21..22] the cache policy of the user-major and item-major copies
 *   (numbered as ccdpp_options_t.cache: 1, 2 or 3), [23] user-major windows
 *   (512 entries) with delta-coded indices, [24] its windows, [25..26] the
 *   same two for the item-major copy, [27] the items of a split item-major copy
 *   that are tiled (0: not split; fields 10..14, 19..22 and 25..26 then describe
 *   that tiled part), [28..34] the hot part of a split copy: gather mode, hot
 *   width, workgroups, segments, rows finished in the pass, rows combined,
 *   cache policy (zeros when not split), [35..40] the device build's phases in
 *   microseconds: inputs copied and degrees counted; relabelling; the
 *   user-major copy; the item-major copy and the map between the copies;
 *   cache policies, index coding and scratch; the factors; [41] the device
 *   set-up before them (device checks, kernel attributes, scratch address).
 * Returns the number of values written. */
int ccdpp_info(ccdpp_t *h, int64_t *out, int32_t len);

/* Testing hook for the error paths, forced from the host (process-wide):
 *   what = 0 : the device allocation made by the library after `after` more
 *              successful ones fails as if the device were out of memory;
 *   what = 1 : the sweep-kernel launch after `after` more is not made and
 *              reports a device error (EDEVICE, which poisons the handle).
 * after < 0 disarms it.  Once triggered it disarms itself.  A failed
 * allocation is reported before the call changes the handle's state: ENOMEM
 * leaves factors and residual as they were and the handle usable (a failed
 * ccdpp_create frees everything and leaves *out untouched).  Returns EINVAL
 * for another `what`. */
int ccdpp_debug_inject(int32_t what, int64_t after);

/* Human-readable message of the last failure on this handle; with h == NULL,
 * of the last failed ccdpp_create on this thread.  Never NULL. */
const char *ccdpp_last_error(const ccdpp_t *h);

/* Free the handle and all its device memory.  NULL is accepted. */
void ccdpp_destroy(ccdpp_t *h);

#ifdef __cplusplus
}
#endif
#endif
