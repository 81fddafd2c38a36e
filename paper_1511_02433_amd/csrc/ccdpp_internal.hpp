// Internal definitions shared by the HIP sources of the CCD++ library (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "ccdpp.h"

namespace ccdk {

// ---------------------------------------------------------------------------
// Layout and schedule.
//
// A layout is one compressed copy of the residual: "rows" are the units whose
// coordinate a pass computes (users for the u-pass of eq. 15, items for the
// v-pass of eq. 16) and every entry names a "column" of the other side whose
// coordinate the pass gathers.
//
// The gathered dimension is cut into P tiles of T columns.  Entries are
// stored tile-major; inside a tile, the non-empty row segments come in order
// of decreasing length and each segment's entries in increasing column order.
// A pass stages the tile's slice of every gathered vector in LDS (160 KB per
// CU on gfx950), so each random gather is an LDS read instead of a cache line
// pulled from L2.  With P == 1 a segment is a whole row and the pass writes
// the coordinate directly; with P > 1 every segment yields a partial
// (numerator, denominator) and a combine kernel adds a row's partials in tile
// order.  A layout whose tiles would hold too few entries per segment keeps
// P == 1 and gathers from global memory instead ("global" mode).
//
// Work units are wave-sized: a long segment (more than kGroupMaxLen entries)
// is one unit walked by a whole wave; shorter segments are packed 64/G to a
// unit, G lanes per segment, E entries per lane.  Persistent workgroups of
// kWG threads are assigned to tiles in proportion to the tile's entries and
// their waves take the tile's units in a fixed stride, so the schedule and
// every reduction order are deterministic.
// ---------------------------------------------------------------------------
constexpr int kWG = 1024;                 // threads per persistent workgroup
constexpr int kWaves = kWG / 64;          // 16 waves
constexpr int kLongE = 16;                // entries per lane per step of a long segment
constexpr int kGroupMaxLen = 1024;        // longest segment packed into a lane group
constexpr int kLdsBytes = 160 * 1024;     // LDS per workgroup
constexpr int kMinTiledSeg = 32;          // mean entries per segment for tiling to pay

enum UnitKind : int32_t {
    kULong = 0,     // one segment, the whole wave, steps of 64 * kLongE entries
    kUG64E16 = 1,   // lanes-per-segment G and entries-per-lane E
    kUG64E8 = 2,
    kUG32E8 = 3,
    kUG16E8 = 4,
    kUG8E8 = 5,
    kUG4E8 = 6,
    kUG2E8 = 7,
    kUG1E8 = 8,
};

enum PassMode : int32_t {
    kModePlain = 0,     // R-hat read only: y = sum rhat x / (lambda + sum x^2)
    kModeAdd = 1,       // rhat = fma(p, q, val); store; then as plain
    kModeSubAdd = 2,    // rhat = fma(p, q, fma(-pp, qq, val)); store; then as plain
    kModeFlush = 3,     // r = fma(-pp, qq, val); store; per-wave sum of r^2
};

enum GatherMode : int32_t {
    kGatherAuto = 0,
    kGatherGlobal = 1,  // P == 1, gathers from global memory
    kGatherLds = 2,     // vectors staged in LDS (tiled when they do not fit)
};

struct PassArgs {
    const void* idx;            // [nnz] uint16 or int32 tile-local column
    float* val;                 // [nnz] residual / R-hat
    const int64_t* seg_start;   // [S + 1]
    const int32_t* seg_row;     // [S]
    const int2* units;          // [U] {first segment, kind | count << 8}
    const int32_t* wg_tile;     // [grid] tile of each workgroup
    const int32_t* wg_rank;     // [grid] rank of the workgroup inside its tile
    const int32_t* tile_unit;   // [P + 1] unit range of each tile
    const int32_t* tile_nwg;    // [P] workgroups of each tile
    const float* x;             // [cols] gathered vector of the update
    const float* p;             // [rows] own factor column, current feature
    const float* pp;            // [rows] own factor column, previous feature (committed)
    const float* q;             // [cols] other factor column, current feature
    const float* qq;            // [cols] other factor column, previous feature (committed)
    float* y;                   // [rows] coordinates (P == 1)
    double2* part;              // [S] partial (num, den) per segment (P > 1)
    double* sse_part;           // [grid * kWaves] flush: per-wave sum of squares
    int64_t nnz;
    int32_t rows, cols, T, P;
    int32_t nseg;
    int32_t x_is_q;             // x and q are the same vector (staged once)
    double lambda;
};

struct CombineArgs {
    const int32_t* row_seg_ptr;  // [rows + 1]
    const int32_t* row_segs;     // [S] segments of each row in tile order
    const double2* part;
    float* y;
    int32_t rows;
    double lambda;
};

// One compressed copy of the residual plus its schedule.
struct Layout {
    int64_t rows = 0, cols = 0, nnz = 0;
    int32_t gather = kGatherGlobal;
    int32_t T = 0, P = 1;
    bool idx16 = false;
    void* idx = nullptr;
    float* val = nullptr;
    int64_t* seg_start = nullptr;
    int32_t* seg_row = nullptr;
    int32_t* tile_seg = nullptr;     // [P + 1] first segment of each tile
    int2* units = nullptr;
    int32_t* wg_tile = nullptr;
    int32_t* wg_rank = nullptr;
    int32_t* tile_unit = nullptr;
    int32_t* tile_nwg = nullptr;
    int32_t* row_seg_ptr = nullptr;  // P > 1
    int32_t* row_segs = nullptr;     // P > 1
    double2* part = nullptr;         // P > 1
    int64_t nseg = 0;
    int32_t nunits = 0;
    int32_t grid = 0;                // persistent workgroups per pass
    int32_t nlong = 0;               // units of the long kind
};

// Launchers (sweep.hip).
hipError_t sweep_init();  // raise the dynamic-LDS limit of the staged kernels
hipError_t launch_pass(const Layout& L, PassMode mode, const float* x, const float* p,
                       const float* pp, const float* q, const float* qq, float* y, double lambda,
                       double* sse_part, hipStream_t s);
hipError_t launch_combine(const Layout& L, float* y, double lambda, hipStream_t s);
hipError_t launch_copy(const float* src, float* dst, int64_t n, hipStream_t s);
hipError_t launch_reduce_sum(const double* part, int32_t n, double* out, hipStream_t s);
int staged_vectors(PassMode mode, bool x_is_q);

// Device build and utilities (build.hip).
hipError_t launch_histogram(const int32_t* key, int64_t n, int32_t* count, hipStream_t s);
hipError_t launch_map(const int32_t* in, const int32_t* table, int64_t n, int32_t* out,
                      hipStream_t s);
hipError_t launch_seg_histogram(const int32_t* lrow, const int32_t* lcol, int64_t nnz,
                                int32_t rows, int32_t T, int32_t* count, hipStream_t s);
hipError_t launch_seg_keys(const int32_t* lrow, const int32_t* lcol, const int32_t* segid,
                           int64_t nnz, int32_t rows, int32_t T, int cbits, uint64_t* keys,
                           int32_t* ids, hipStream_t s);
hipError_t launch_dup_check(const uint64_t* keys, int64_t nnz, int32_t* flag, hipStream_t s);
hipError_t launch_layout_fill(const uint64_t* keys, const int32_t* perm, const float* val_in,
                              int64_t nnz, int cbits, bool idx16, void* idx, float* val,
                              hipStream_t s);
hipError_t launch_invert(const int32_t* perm, int64_t n, int32_t* inv, hipStream_t s);
hipError_t launch_compose(const int32_t* a, const int32_t* b, int64_t n, int32_t* out,
                          hipStream_t s);
hipError_t launch_fill(float* dst, float value, int64_t n, hipStream_t s);
hipError_t launch_scatter_factor_in(const float* rowmajor, const int32_t* new2old, int64_t rows,
                                    int32_t k, float* colmajor, hipStream_t s);
hipError_t launch_gather_factor_out(const float* colmajor, const int32_t* old2new, int64_t rows,
                                    int32_t k, float* rowmajor, hipStream_t s);
hipError_t launch_rebuild_residual(const Layout& L, const float* A, const float* W,
                                   const float* H, int64_t m, int64_t n, int32_t k,
                                   hipStream_t s);
hipError_t launch_scatter_f32(const float* src, const int32_t* map, int64_t n, float* dst,
                              hipStream_t s);
hipError_t launch_consistency(const float* a, const float* b, const int32_t* map, int64_t n,
                              unsigned long long* count, hipStream_t s);
hipError_t launch_sq_sum(const float* v, int64_t n, double* part, int32_t nparts,
                         hipStream_t s);
hipError_t launch_test_err(const int32_t* row, const int32_t* col, const float* val, int64_t nnz,
                           const int32_t* rold2new, const int32_t* cold2new, const float* W,
                           const float* H, int64_t m, int64_t n, int32_t k, double* part,
                           int32_t nparts, hipStream_t s);
hipError_t sort_pairs(const uint64_t* kin, uint64_t* kout, const int32_t* vin, int32_t* vout,
                      int64_t n, int bits, hipStream_t s, void** tmp, size_t* tmp_bytes);

}  // namespace ccdk
