// Internal definitions shared by the HIP sources of the CCD++ library (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "ccdpp.h"

namespace ccdk {

// ---------------------------------------------------------------------------
// Scheduling.  Rows of a layout (users for the row-compressed copy, items for
// the column-compressed copy) are relabelled in order of decreasing length, so
// every scheduling class is a contiguous range of rows and of entries.
//   class "block": rows longer than kGroupMaxLen; one 256-thread workgroup per
//                  row piece of at most kPieceMax entries, LDS reduction across
//                  the 4 waves; rows with several pieces are finished by a
//                  fixed-order combine kernel.
//   class G (1..64 lanes per row): rows of length <= G * E handled by groups
//                  of G lanes (256/G rows per workgroup), each lane taking E
//                  entries, reduced with DPP / permlane cross-lane moves.
// ---------------------------------------------------------------------------
constexpr int kBlock = 256;           // threads per workgroup, 4 waves of 64
constexpr int kBlockUnroll = 16;      // entries per thread per step in the block class
constexpr int kBlockStep = kBlock * kBlockUnroll;  // 4096 entries per workgroup step
constexpr int kPieceMax = 8 * kBlockStep;           // 32768 entries per workgroup at most
constexpr int kGroupMaxLen = 1024;    // longest row handled by a lane group
constexpr int kMaxSegs = 16;

enum SegKind : int32_t {
    kSegBlock = 0,   // workgroup per row piece
    kSegG1E8 = 1,    // 1 lane per row, <= 8 entries
    kSegG2E8 = 2,
    kSegG4E8 = 3,
    kSegG8E8 = 4,
    kSegG16E8 = 5,
    kSegG32E8 = 6,
    kSegG64E8 = 7,
    kSegG64E16 = 8,
};

struct Seg {
    int32_t kind;
    int32_t block_begin;   // first workgroup of the segment
    int32_t row_begin;     // first row (block class: first piece)
    int32_t row_end;       // one past the last row (block class: one past the last piece)
};

enum PassMode : int32_t {
    kModePlain = 0,     // R-hat read only: y = sum rhat x / (lambda + sum x^2)
    kModeAdd = 1,       // rhat = fma(p, q, val); store; then as plain with x
    kModeSubAdd = 2,    // rhat = fma(p, q, fma(-pp, qq, val)); store; then as plain
    kModeFlush = 3,     // r = fma(-pp, qq, val); store; sum of r^2 per workgroup
};

struct PassArgs {
    const int64_t* ptr;      // [rows + 1]
    const int32_t* idx;      // [nnz] other-side index of each entry
    float* val;              // [nnz] residual / R-hat
    const float* x;          // [cols] gathered vector of the update
    const float* p;          // [rows] self factor column of the current feature
    const float* pp;         // [rows] self factor column of the previous feature (committed)
    const float* q;          // [cols] other factor column of the current feature
    const float* qq;         // [cols] other factor column of the previous feature (committed)
    float* y;                // [rows] output coordinates
    double2* part;           // [npieces] partial (num, den) of split rows
    double* sse_part;        // [grid] flush: per-workgroup sum of squares
    const int32_t* piece_row;   // [npieces] row of each block-class piece
    const int64_t* piece_lo;    // [npieces + 1] first entry of each piece (last: end)
    int32_t rows;
    int32_t cols;
    double lambda;
    int32_t nseg;
    Seg seg[kMaxSegs];
};

struct CombineArgs {
    const int32_t* split_row;    // [nsplit] rows with more than one piece
    const int32_t* split_first;  // [nsplit + 1] first piece of each such row
    const double2* part;
    float* y;
    double lambda;
    int32_t nsplit;
};

// One compressed copy of the residual plus its schedule.
struct Layout {
    int64_t rows = 0, cols = 0, nnz = 0;
    int64_t* ptr = nullptr;
    int32_t* idx = nullptr;
    float* val = nullptr;
    // schedule
    std::vector<Seg> segs;
    int32_t grid = 0;              // workgroups per pass
    int32_t nblock_rows = 0;       // rows in the block class
    int32_t npieces = 0;
    int32_t nsplit = 0;            // rows with more than one piece
    int32_t* piece_row = nullptr;
    int64_t* piece_lo = nullptr;
    int32_t* split_row = nullptr;
    int32_t* split_first = nullptr;
    double2* part = nullptr;
};

// Launchers (sweep.hip).
hipError_t launch_pass(const Layout& L, PassMode mode, const float* x, const float* p,
                       const float* pp, const float* q, const float* qq, float* y, double lambda,
                       double* sse_part, hipStream_t s);
hipError_t launch_combine(const Layout& L, float* y, double lambda, hipStream_t s);
hipError_t launch_copy(const float* src, float* dst, int64_t n, hipStream_t s);
hipError_t launch_reduce_sum(const double* part, int32_t n, double* out, hipStream_t s);

// Device build and utilities (build.hip).
hipError_t launch_histogram(const int32_t* key, int64_t n, int32_t* count, hipStream_t s);
hipError_t launch_make_keys_csr(const int32_t* row, const int32_t* col, const int32_t* rnew,
                                const int32_t* cnew, int64_t nnz, int64_t ncols, uint64_t* keys,
                                int32_t* ids, hipStream_t s);
hipError_t launch_dup_check(const uint64_t* keys, int64_t nnz, int32_t* flag, hipStream_t s);
hipError_t launch_csr_fill(const uint64_t* keys, const int32_t* src, const float* val_in,
                           int64_t nnz, int64_t ncols, int64_t nrows, int32_t* idx, float* val,
                           float* A, uint64_t* keys_csc, int32_t* ids_csc, hipStream_t s);
hipError_t launch_csc_fill(const uint64_t* keys_csc, const int32_t* csr_pos, const float* csr_val,
                           int64_t nnz, int64_t nrows, int32_t* idx, float* val,
                           int32_t* csr2csc, hipStream_t s);
hipError_t launch_fill(float* dst, float value, int64_t n, hipStream_t s);
hipError_t launch_scatter_factor_in(const float* rowmajor, const int32_t* new2old, int64_t rows,
                                    int32_t k, float* colmajor, hipStream_t s);
hipError_t launch_gather_factor_out(const float* colmajor, const int32_t* old2new, int64_t rows,
                                    int32_t k, float* rowmajor, hipStream_t s);
hipError_t launch_rebuild_residual(const int64_t* ptr, const int32_t* idx, const float* A,
                                   const float* W, const float* H, int64_t m, int64_t n,
                                   int32_t k, int64_t nnz, float* csr_val, hipStream_t s);
hipError_t launch_scatter_csc(const float* csr_val, const int32_t* csr2csc, int64_t nnz,
                              float* csc_val, hipStream_t s);
hipError_t launch_residual_out(const float* csr_val, const int32_t* csr_src, int64_t nnz,
                               float* out, hipStream_t s);
hipError_t launch_consistency(const float* csr_val, const float* csc_val, const int32_t* csr2csc,
                              int64_t nnz, unsigned long long* count, hipStream_t s);
hipError_t launch_sq_sum(const float* v, int64_t n, double* part, int32_t nparts,
                         hipStream_t s);
hipError_t launch_test_err(const int32_t* row, const int32_t* col, const float* val, int64_t nnz,
                           const int32_t* rold2new, const int32_t* cold2new, const float* W,
                           const float* H, int64_t m, int64_t n, int32_t k, double* part,
                           int32_t nparts, hipStream_t s);
hipError_t sort_pairs(const uint64_t* kin, uint64_t* kout, const int32_t* vin, int32_t* vout,
                      int64_t n, int bits, hipStream_t s, void** tmp, size_t* tmp_bytes);

}  // namespace ccdk
