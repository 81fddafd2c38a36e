/* A plain C caller of the library, with no Python and no PyTorch in the process.
 *
 * Usage: abi_caller DIR
 * DIR/problem.txt holds "m n k lambda nnz outer inner"; DIR/row.bin, col.bin (int32),
 * val.bin (float32, nnz each) and H0.bin (float32, n x k row-major) the inputs.  The
 * program creates a handle on the current device, sets W = 0 and H = H0, runs
 * `outer` outer iterations of `inner` inner ones, and writes DIR/W.bin, DIR/H.bin
 * (float32, row-major) and DIR/out.txt ("train_rmse mismatches").  Exit status 0 on
 * success; on a library error it prints the status and message and exits with 1. */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "ccdpp.h"

static void *load(const char *dir, const char *name, size_t bytes) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE *f = fopen(path, "rb");
    if (!f) return NULL;
    void *p = malloc(bytes ? bytes : 1);
    if (p && fread(p, 1, bytes, f) != bytes) {
        free(p);
        p = NULL;
    }
    fclose(f);
    return p;
}

static int save(const char *dir, const char *name, const void *p, size_t bytes) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE *f = fopen(path, "wb");
    if (!f) return 0;
    const int ok = fwrite(p, 1, bytes, f) == bytes;
    fclose(f);
    return ok;
}

#define CHECK(call)                                                                   \
    do {                                                                              \
        int rc_ = (call);                                                             \
        if (rc_ != CCDPP_OK) {                                                        \
            fprintf(stderr, "%s: status %d: %s\n", #call, rc_, ccdpp_last_error(h)); \
            return 1;                                                                 \
        }                                                                             \
    } while (0)

int main(int argc, char **argv) {
    if (argc != 2) {
        fprintf(stderr, "usage: %s DIR\n", argv[0]);
        return 2;
    }
    const char *dir = argv[1];
    char path[4096];
    snprintf(path, sizeof path, "%s/problem.txt", dir);
    FILE *f = fopen(path, "r");
    long long m, n, nnz;
    int k, outer, inner;
    double lambda;
    if (!f || fscanf(f, "%lld %lld %d %lf %lld %d %d", &m, &n, &k, &lambda, &nnz, &outer, &inner) != 7) {
        fprintf(stderr, "cannot read %s\n", path);
        return 2;
    }
    fclose(f);
    int32_t *row = load(dir, "row.bin", (size_t)nnz * 4);
    int32_t *col = load(dir, "col.bin", (size_t)nnz * 4);
    float *val = load(dir, "val.bin", (size_t)nnz * 4);
    float *H = load(dir, "H0.bin", (size_t)(n * k) * 4);
    float *W = calloc((size_t)(m * k), sizeof(float));
    if (!row || !col || !val || !H || !W) {
        fprintf(stderr, "cannot read the inputs\n");
        return 2;
    }
    ccdpp_t *h = NULL;
    CHECK(ccdpp_create(m, n, k, lambda, nnz, row, col, val, 7, &h));
    CHECK(ccdpp_set_factors(h, W, H));
    CHECK(ccdpp_run(h, outer, inner));
    CHECK(ccdpp_get_factors(h, W, H));
    double rmse = 0.0;
    int64_t mism = -1;
    CHECK(ccdpp_train_rmse(h, &rmse));
    CHECK(ccdpp_check_consistency(h, &mism));
    ccdpp_destroy(h);
    if (!save(dir, "W.bin", W, (size_t)(m * k) * 4) || !save(dir, "H.bin", H, (size_t)(n * k) * 4))
        return 2;
    snprintf(path, sizeof path, "%s/out.txt", dir);
    f = fopen(path, "w");
    if (!f) return 2;
    fprintf(f, "%.17g %lld\n", rmse, (long long)mism);
    fclose(f);
    free(row);
    free(col);
    free(val);
    free(H);
    free(W);
    return 0;
}
