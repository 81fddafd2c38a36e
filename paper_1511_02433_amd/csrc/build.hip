// Device-side construction of the two compressed residual copies and the
// utility kernels of the CCD++ library (gfx950).
//
// Construction (done once per handle): the observed set Omega of Section 3 is
// given as triplets.  Rows and columns are relabelled by decreasing degree
// (the per-row work of Section 6 is proportional to the row length), then
//   key = new_row * n + new_col   -> radix sort -> row-compressed copy,
//   key = new_col * m + new_row   -> radix sort -> column-compressed copy,
// with the map from every row-ordered position to its column-ordered
// position.  Adjacent equal keys after the first sort are repeated positions.
#include <hipcub/hipcub.hpp>

#include "ccdpp_internal.hpp"

namespace ccdk {
namespace {

constexpr int kT = 256;

inline dim3 grid_for(int64_t n, int64_t cap = 1 << 20) {
    int64_t g = (n + kT - 1) / kT;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return dim3((unsigned)g);
}

__global__ void k_histogram(const int32_t* __restrict__ key, int64_t n, int32_t* count) {
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < n; e += (int64_t)gridDim.x * kT)
        atomicAdd(&count[key[e]], 1);
}

__global__ void k_make_keys(const int32_t* __restrict__ row, const int32_t* __restrict__ col,
                            const int32_t* __restrict__ rnew, const int32_t* __restrict__ cnew,
                            int64_t nnz, int64_t ncols, uint64_t* __restrict__ keys,
                            int32_t* __restrict__ ids) {
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < nnz;
         e += (int64_t)gridDim.x * kT) {
        keys[e] = (uint64_t)rnew[row[e]] * (uint64_t)ncols + (uint64_t)cnew[col[e]];
        ids[e] = (int32_t)e;
    }
}

__global__ void k_dup_check(const uint64_t* __restrict__ keys, int64_t nnz, int32_t* flag) {
    for (int64_t p = (int64_t)blockIdx.x * kT + threadIdx.x; p + 1 < nnz;
         p += (int64_t)gridDim.x * kT)
        if (keys[p] == keys[p + 1]) *flag = 1;
}

__global__ void k_csr_fill(const uint64_t* __restrict__ keys, const int32_t* __restrict__ src,
                           const float* __restrict__ val_in, int64_t nnz, int64_t ncols,
                           int64_t nrows, int32_t* __restrict__ idx, float* __restrict__ val,
                           float* __restrict__ A, uint64_t* __restrict__ keys_csc,
                           int32_t* __restrict__ ids_csc) {
    for (int64_t p = (int64_t)blockIdx.x * kT + threadIdx.x; p < nnz;
         p += (int64_t)gridDim.x * kT) {
        const uint64_t key = keys[p];
        const uint64_t r = key / (uint64_t)ncols;
        const uint64_t c = key - r * (uint64_t)ncols;
        idx[p] = (int32_t)c;
        const float v = val_in[src[p]];
        val[p] = v;
        A[p] = v;
        keys_csc[p] = c * (uint64_t)nrows + r;
        ids_csc[p] = (int32_t)p;
    }
}

__global__ void k_csc_fill(const uint64_t* __restrict__ keys_csc, const int32_t* __restrict__ pos,
                           const float* __restrict__ csr_val, int64_t nnz, int64_t nrows,
                           int32_t* __restrict__ idx, float* __restrict__ val,
                           int32_t* __restrict__ csr2csc) {
    for (int64_t q = (int64_t)blockIdx.x * kT + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * kT) {
        const uint64_t key = keys_csc[q];
        const uint64_t c = key / (uint64_t)nrows;
        idx[q] = (int32_t)(key - c * (uint64_t)nrows);
        const int32_t p = pos[q];
        val[q] = csr_val[p];
        csr2csc[p] = (int32_t)q;
    }
}

__global__ void k_fill(float* __restrict__ dst, float value, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kT + threadIdx.x; i < n; i += (int64_t)gridDim.x * kT)
        dst[i] = value;
}

// colmajor[t * rows + i'] = rowmajor[new2old[i'] * k + t]
__global__ void k_factor_in(const float* __restrict__ rowmajor, const int32_t* __restrict__ new2old,
                            int64_t rows, int32_t k, float* __restrict__ colmajor) {
    const int64_t total = rows * k;
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * kT) {
        const int64_t t = e / rows;
        const int64_t i = e - t * rows;
        colmajor[e] = rowmajor[(int64_t)new2old[i] * k + t];
    }
}

// rowmajor[i * k + t] = colmajor[t * rows + old2new[i]]
__global__ void k_factor_out(const float* __restrict__ colmajor, const int32_t* __restrict__ old2new,
                             int64_t rows, int32_t k, float* __restrict__ rowmajor) {
    const int64_t total = rows * k;
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * kT) {
        const int64_t i = e / k;
        const int64_t t = e - i * k;
        rowmajor[e] = colmajor[t * rows + old2new[i]];
    }
}

// R = A - w_i^T h_j for every row-ordered entry (prediction summed in fp64 over
// ascending features, one rounding to fp32).
__global__ void k_rebuild(const int64_t* __restrict__ ptr, const int32_t* __restrict__ idx,
                          const float* __restrict__ A, const float* __restrict__ W,
                          const float* __restrict__ H, int64_t m, int64_t n, int32_t k,
                          int64_t nnz, float* __restrict__ csr_val) {
    for (int64_t p = (int64_t)blockIdx.x * kT + threadIdx.x; p < nnz;
         p += (int64_t)gridDim.x * kT) {
        // row of p: the last i with ptr[i] <= p
        int64_t lo = 0, hi = m;  // invariant ptr[lo] <= p < ptr[hi]
        while (hi - lo > 1) {
            const int64_t mid = (lo + hi) >> 1;
            if (ptr[mid] <= p) lo = mid; else hi = mid;
        }
        const int64_t j = idx[p];
        double pred = 0.0;
        for (int32_t t = 0; t < k; ++t)
            pred = __builtin_fma((double)W[(int64_t)t * m + lo], (double)H[(int64_t)t * n + j], pred);
        csr_val[p] = (float)((double)A[p] - pred);
    }
}

__global__ void k_scatter_csc(const float* __restrict__ csr_val, const int32_t* __restrict__ map,
                              int64_t nnz, float* __restrict__ csc_val) {
    for (int64_t p = (int64_t)blockIdx.x * kT + threadIdx.x; p < nnz;
         p += (int64_t)gridDim.x * kT)
        csc_val[map[p]] = csr_val[p];
}

__global__ void k_residual_out(const float* __restrict__ csr_val, const int32_t* __restrict__ src,
                               int64_t nnz, float* __restrict__ out) {
    for (int64_t p = (int64_t)blockIdx.x * kT + threadIdx.x; p < nnz;
         p += (int64_t)gridDim.x * kT)
        out[src[p]] = csr_val[p];
}

__global__ void k_consistency(const float* __restrict__ csr_val, const float* __restrict__ csc_val,
                              const int32_t* __restrict__ map, int64_t nnz,
                              unsigned long long* count) {
    for (int64_t p = (int64_t)blockIdx.x * kT + threadIdx.x; p < nnz;
         p += (int64_t)gridDim.x * kT)
        if (__float_as_uint(csr_val[p]) != __float_as_uint(csc_val[map[p]]))
            atomicAdd(count, 1ull);
}

// Workgroup b sums elements b*256 + t + s*(nparts*256) in order per thread, then a
// fixed tree: deterministic for a fixed nparts.
__device__ __forceinline__ void block_total(double acc, double* out) {
    __shared__ double s[kT];
    s[threadIdx.x] = acc;
    __syncthreads();
    for (int w = kT / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) s[threadIdx.x] += s[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) *out = s[0];
}

__global__ void k_sq_sum(const float* __restrict__ v, int64_t n, double* __restrict__ part) {
    double acc = 0.0;
    for (int64_t i = (int64_t)blockIdx.x * kT + threadIdx.x; i < n; i += (int64_t)gridDim.x * kT) {
        const double d = v[i];
        acc = __builtin_fma(d, d, acc);
    }
    block_total(acc, &part[blockIdx.x]);
}

__global__ void k_test_err(const int32_t* __restrict__ row, const int32_t* __restrict__ col,
                           const float* __restrict__ val, int64_t nnz,
                           const int32_t* __restrict__ rnew, const int32_t* __restrict__ cnew,
                           const float* __restrict__ W, const float* __restrict__ H, int64_t m,
                           int64_t n, int32_t k, double* __restrict__ part) {
    double acc = 0.0;
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < nnz;
         e += (int64_t)gridDim.x * kT) {
        const int64_t i = rnew[row[e]];
        const int64_t j = cnew[col[e]];
        double pred = 0.0;
        for (int32_t t = 0; t < k; ++t)
            pred = __builtin_fma((double)W[(int64_t)t * m + i], (double)H[(int64_t)t * n + j], pred);
        const double err = (double)val[e] - pred;
        acc = __builtin_fma(err, err, acc);
    }
    block_total(acc, &part[blockIdx.x]);
}

}  // namespace

hipError_t launch_histogram(const int32_t* key, int64_t n, int32_t* count, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_histogram, grid_for(n, 8192), dim3(kT), 0, s, key, n, count);
    return hipGetLastError();
}

hipError_t launch_make_keys_csr(const int32_t* row, const int32_t* col, const int32_t* rnew,
                                const int32_t* cnew, int64_t nnz, int64_t ncols, uint64_t* keys,
                                int32_t* ids, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    hipLaunchKernelGGL(k_make_keys, grid_for(nnz), dim3(kT), 0, s, row, col, rnew, cnew, nnz,
                       ncols, keys, ids);
    return hipGetLastError();
}

hipError_t launch_dup_check(const uint64_t* keys, int64_t nnz, int32_t* flag, hipStream_t s) {
    if (nnz < 2) return hipSuccess;
    hipLaunchKernelGGL(k_dup_check, grid_for(nnz), dim3(kT), 0, s, keys, nnz, flag);
    return hipGetLastError();
}

hipError_t launch_csr_fill(const uint64_t* keys, const int32_t* src, const float* val_in,
                           int64_t nnz, int64_t ncols, int64_t nrows, int32_t* idx, float* val,
                           float* A, uint64_t* keys_csc, int32_t* ids_csc, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    hipLaunchKernelGGL(k_csr_fill, grid_for(nnz), dim3(kT), 0, s, keys, src, val_in, nnz, ncols,
                       nrows, idx, val, A, keys_csc, ids_csc);
    return hipGetLastError();
}

hipError_t launch_csc_fill(const uint64_t* keys_csc, const int32_t* csr_pos, const float* csr_val,
                           int64_t nnz, int64_t nrows, int32_t* idx, float* val,
                           int32_t* csr2csc, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    hipLaunchKernelGGL(k_csc_fill, grid_for(nnz), dim3(kT), 0, s, keys_csc, csr_pos, csr_val, nnz,
                       nrows, idx, val, csr2csc);
    return hipGetLastError();
}

hipError_t launch_fill(float* dst, float value, int64_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill, grid_for(n), dim3(kT), 0, s, dst, value, n);
    return hipGetLastError();
}

hipError_t launch_scatter_factor_in(const float* rowmajor, const int32_t* new2old, int64_t rows,
                                    int32_t k, float* colmajor, hipStream_t s) {
    hipLaunchKernelGGL(k_factor_in, grid_for(rows * k), dim3(kT), 0, s, rowmajor, new2old, rows, k,
                       colmajor);
    return hipGetLastError();
}

hipError_t launch_gather_factor_out(const float* colmajor, const int32_t* old2new, int64_t rows,
                                    int32_t k, float* rowmajor, hipStream_t s) {
    hipLaunchKernelGGL(k_factor_out, grid_for(rows * k), dim3(kT), 0, s, colmajor, old2new, rows,
                       k, rowmajor);
    return hipGetLastError();
}

hipError_t launch_rebuild_residual(const int64_t* ptr, const int32_t* idx, const float* A,
                                   const float* W, const float* H, int64_t m, int64_t n,
                                   int32_t k, int64_t nnz, float* csr_val, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    hipLaunchKernelGGL(k_rebuild, grid_for(nnz), dim3(kT), 0, s, ptr, idx, A, W, H, m, n, k, nnz,
                       csr_val);
    return hipGetLastError();
}

hipError_t launch_scatter_csc(const float* csr_val, const int32_t* csr2csc, int64_t nnz,
                              float* csc_val, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    hipLaunchKernelGGL(k_scatter_csc, grid_for(nnz), dim3(kT), 0, s, csr_val, csr2csc, nnz,
                       csc_val);
    return hipGetLastError();
}

hipError_t launch_residual_out(const float* csr_val, const int32_t* csr_src, int64_t nnz,
                               float* out, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    hipLaunchKernelGGL(k_residual_out, grid_for(nnz), dim3(kT), 0, s, csr_val, csr_src, nnz, out);
    return hipGetLastError();
}

hipError_t launch_consistency(const float* csr_val, const float* csc_val, const int32_t* csr2csc,
                              int64_t nnz, unsigned long long* count, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    hipLaunchKernelGGL(k_consistency, grid_for(nnz), dim3(kT), 0, s, csr_val, csc_val, csr2csc,
                       nnz, count);
    return hipGetLastError();
}

hipError_t launch_sq_sum(const float* v, int64_t n, double* part, int32_t nparts, hipStream_t s) {
    hipLaunchKernelGGL(k_sq_sum, dim3(nparts), dim3(kT), 0, s, v, n, part);
    return hipGetLastError();
}

hipError_t launch_test_err(const int32_t* row, const int32_t* col, const float* val, int64_t nnz,
                           const int32_t* rold2new, const int32_t* cold2new, const float* W,
                           const float* H, int64_t m, int64_t n, int32_t k, double* part,
                           int32_t nparts, hipStream_t s) {
    hipLaunchKernelGGL(k_test_err, dim3(nparts), dim3(kT), 0, s, row, col, val, nnz, rold2new,
                       cold2new, W, H, m, n, k, part);
    return hipGetLastError();
}

// Radix sort of (key, id) pairs on the low `bits` bits of the key.
hipError_t sort_pairs(const uint64_t* kin, uint64_t* kout, const int32_t* vin, int32_t* vout,
                      int64_t n, int bits, hipStream_t s, void** tmp, size_t* tmp_bytes) {
    size_t need = 0;
    hipError_t e = hipcub::DeviceRadixSort::SortPairs(nullptr, need, kin, kout, vin, vout, (int)n,
                                                      0, bits, s);
    if (e != hipSuccess) return e;
    if (need > *tmp_bytes) {
        if (*tmp) hipFree(*tmp);
        *tmp = nullptr;
        e = hipMalloc(tmp, need);
        if (e != hipSuccess) return e;
        *tmp_bytes = need;
    }
    return hipcub::DeviceRadixSort::SortPairs(*tmp, need, kin, kout, vin, vout, (int)n, 0, bits, s);
}

}  // namespace ccdk
