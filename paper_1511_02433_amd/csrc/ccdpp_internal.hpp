// Internal definitions shared by the HIP sources of the CCD++ library (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <functional>

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
// stored tile-major; inside a tile, row segments (a row's entries in the tile)
// follow each other and each segment's entries come in increasing column
// order.  A pass stages the tile's slice of every gathered vector in LDS
// (160 KB per CU on gfx950), so each random gather is an LDS read instead of
// a cache line pulled from L2.  With P == 1 segment s is row s (rows are
// relabelled by decreasing length, so the empty ones come last) and the pass
// writes the coordinate directly; with P > 1 every segment yields a partial
// (numerator, denominator) and a combine kernel adds a row's partials in tile
// order.  A layout whose tiles would hold too few entries per segment keeps
// P == 1 and becomes a hot layout (below); a forced "global" layout gathers
// everything from global memory.  The item-major copy may instead be split in
// two layouts over its rows: the longest rows tiled, the others hot, their
// values in one array (api.hip).
//
// Persistent workgroups of kWG threads each own an equal, contiguous share of
// the layout's (tile-major) entries (two shares per CU when every wave still
// gets several windows, else one).  With P == 1 (float) the share bounds sit on
// row starts when that keeps the shares within an eighth of equal; rows are then
// cut only between the waves of one workgroup, which finishes them at the end of
// the pass from partials its waves leave in LDS, and no combine kernel runs.  A share that crosses tile boundaries is
// processed as one "piece" per tile, restaging LDS between pieces; inside a
// piece each of the 16 waves owns one of 16 equal contiguous chunks.  Chunk
// bounds do not follow segment bounds, so every wave streams the same number
// of entries however long the rows are: a segment cut by chunk bounds leaves
// one partial (num, den) per chunk it meets, in a slot of that chunk, and a
// combine kernel adds a row's partials in entry order.  Shares, pieces and
// chunks, and with them every reduction order, are fixed at build time, so
// results are identical run to run.
//
// Every segment starts at a multiple of kE entries, and every tile, workgroup
// share and chunk at a multiple of kAlign = kWin, so that every window a pass
// reads is one whole, aligned block of kWin entries: the build inserts padding
// entries after a segment up to the next multiple of kE (of kAlign before a new
// tile), and cuts shares and chunks at multiples of kAlign.  Inside a block the
// values are stored lane-split (val_slot): lane l's kE values sit at 4l .. 4l + 3
// and kWin/2 + 4l .. kWin/2 + 4l + 3, so that each 128-bit load or store of the
// wave covers 1 KB of contiguous memory; the indices stay in entry order (one
// 128-bit load per lane already covers 16 contiguous bytes).  A padding entry
// holds value 0 and an index that reads 0 (a zero word
// after each staged slice in LDS, or a position past the vector in global
// mode, where the bounded buffer load returns 0), so it adds exactly 0 to
// every sum and stays 0 under every residual update.
//
// Staged slices are stored XOR-swizzled: column c of the tile sits at LDS word
// lds_swizzle(c), which permutes each aligned group of 32 words by the group's
// index.  Runs of columns with a constant stride (dense rows of heavy users or
// popular items) then spread over the LDS banks instead of hitting one bank,
// and the layout stores the swizzled position as the entry's index, so the
// pass pays nothing for it.  The padding index of a staged layout is the first
// multiple of 32 at or above T, a word outside the swizzled range that staging
// sets to zero.
//
// A hot layout (P == 1, 32-bit indices) is for a gathered side too long to stage
// and too sparse to tile: its columns are relabelled by decreasing count, so the
// first ones take most of the gathers.  Each pass stages as many leading columns
// as its vectors leave room for (a multiple of 32, at most the layout's hot
// width tsw) and gathers the others from global memory.  Indices below tsw are
// swizzled positions, the rest plain columns; the padding index is cols, which
// the bounded global load turns into 0.
//
// The per-row scalars a pass reads (the own factor column of the current and
// the previous feature) are addressed by segment: with P == 1 segment s is row
// s and the factor column itself serves; with P > 1 the library keeps a copy of
// every own factor column spread over the segments (written by the combine
// kernel when the column is committed), so no pass reads through seg_row.
constexpr int kWG = 1024;                 // threads per persistent workgroup
constexpr int kWaves = kWG / 64;          // 16 waves
constexpr int kE = 8;                     // entries per lane per window
constexpr int kWin = 64 * kE;             // entries per window
constexpr int kAlign = kWin;              // tile, share and chunk starts: whole window blocks

constexpr int kLdsBytes = 160 * 1024;     // LDS per workgroup
constexpr int kCutSlotBytes = 2 * 16 * 16;  // per-wave head and tail partials (P == 1)
constexpr int kLdsVecBytes = kLdsBytes - kCutSlotBytes;  // the rest holds staged vectors
constexpr int kCutMaxSlots = 12;          // slots of a row a workgroup finishes itself
constexpr int kMinTiledSeg = 32;          // mean entries per segment for tiling to pay
constexpr int kSegWeight = 4;             // default work of one segment, in entries
constexpr int kChunkMid = 1;              // chunk flag: its first segment began in an earlier chunk
constexpr int kChunkCont = 2;             // chunk flag: its last segment goes on past its end
constexpr int kEntryPad = 64;             // entries of padding after idx and val (loads past the end)

__host__ __device__ inline uint32_t lds_swizzle(uint32_t c) { return c ^ ((c >> 5) & 31u); }

// Delta-coded index windows (copies staged in LDS with 16-bit indices).  A window
// in which every lane's valid entries climb by at most kDeltaMax columns from one
// to the next keeps its indices in the first 768 of its 1024 index bytes, 12 bytes
// per lane: lane l's 96-bit record is words 3l, 3l + 1 and 3l + 2, with
//   bits 0-15   the lane's first index as the plain format holds it (swizzled,
//               start bit included),
//   bits 16-92  seven 11-bit steps between its consecutive unswizzled columns,
//   bits 93-95  the number of valid entries less one (the others are padding).
// A bit per window (Layout::dmask) marks the windows coded this way.
constexpr uint32_t kDeltaBits = 11;
constexpr uint32_t kDeltaMax = (1u << kDeltaBits) - 1u;

// The lane's 8 indices in the plain format, from its record (d0, d1, d2).
__host__ __device__ inline void delta_decode(uint32_t d0, uint32_t d1, uint32_t d2, uint32_t pad,
                                             uint32_t out[8]) {
    const uint32_t first = d0 & 0xFFFFu;
    const uint32_t last = d2 >> 29;  // valid entries - 1
    const uint32_t st[7] = {(d0 >> 16) & kDeltaMax,         ((d0 >> 27) | (d1 << 5)) & kDeltaMax,
                            (d1 >> 6) & kDeltaMax,          (d1 >> 17) & kDeltaMax,
                            ((d1 >> 28) | (d2 << 4)) & kDeltaMax, (d2 >> 7) & kDeltaMax,
                            (d2 >> 18) & kDeltaMax};
    uint32_t c = lds_swizzle(first & 0x7FFFu);
    out[0] = first;
    for (int k = 1; k < 8; ++k) {
        c += st[k - 1];
        out[k] = (uint32_t)k <= last ? lds_swizzle(c) : pad;
    }
}

// Storage slot of the value of entry p (see above), and its inverse.  A 128-bit
// access holds E = 16 / sizeof(V) values; the block of kWin entries is stored as
// kE / E parts of 64 x E values, lane l's values k (E of them per part) at
// part k / E, position l * E + k % E.  For float: 4l .. 4l + 3 and
// kWin/2 + 4l .. kWin/2 + 4l + 3.
static_assert(kWin == 512 && kE == 8, "val_slot assumes 64 lanes of 8 entries");
template <class V>
__host__ __device__ inline int64_t val_slot(int64_t p) {
    constexpr int64_t E = 16 / sizeof(V);
    const int64_t o = p & (kWin - 1);
    const int64_t l = o >> 3, k = o & 7;
    return (p - o) + (k / E) * (64 * E) + l * E + (k % E);
}
template <class V>
__host__ __device__ inline int64_t val_entry(int64_t f) {
    constexpr int64_t E = 16 / sizeof(V);
    const int64_t o = f & (kWin - 1);
    const int64_t part = o / (64 * E), r = o % (64 * E);
    return (f - o) + ((r / E) << 3) + part * E + (r % E);
}

enum PassMode : int32_t {
    kModePlain = 0,     // R-hat read only: y = sum rhat x / (lambda + sum x^2)
    kModeAdd = 1,       // rhat = fma(p, q, val); store; then as plain
    kModeSubAdd = 2,    // rhat = fma(p, q, fma(-pp, qq, val)); store; then as plain
    kModeFlush = 3,     // r = fma(-pp, qq, val); store; per-wave sum of r^2
};

// Segments are aligned to lanes: every segment starts at a multiple of kE, the
// entries between its last entry and the next multiple of kE are padding, and
// the index of a segment's first entry carries a start bit (the top bit of the
// index word; 16-bit indices are therefore below 0x8000).  A lane's kE entries
// thus always belong to one segment, and the lane learns whether that segment
// starts with it from its own first index.
template <class I> struct IndexBits;
template <> struct IndexBits<uint16_t> {
    static constexpr uint32_t start = 0x8000u, mask = 0x7FFFu;
};
template <> struct IndexBits<int32_t> {
    static constexpr uint32_t start = 0x80000000u, mask = 0x7FFFFFFFu;
};

enum GatherMode : int32_t {
    kGatherAuto = 0,
    kGatherGlobal = 1,  // P == 1, gathers from global memory
    kGatherLds = 2,     // vectors staged in LDS (tiled when they do not fit)
    kGatherHot = 3,     // P == 1, the leading columns staged in LDS, the rest from global
};

// A segment's partial (numerator, denominator): summed in fp64 across windows and
// stored at the value type's precision (rounded once to fp32 for float values).
template <class V> struct PartOf;
template <> struct PartOf<float> { using type = float2; };
template <> struct PartOf<double> { using type = double2; };
template <class V> using part_t = typename PartOf<V>::type;

// V is the type of the residual, the factors and the in-window arithmetic:
// float (the paper's faster variant, Section 8) or double.
template <class V>
struct PassArgs {
    const void* idx;            // [npad] uint16 or int32 tile-local column
    V* val;                     // [npad] residual / R-hat, in val_slot<V> order
    const int32_t* wg_piece;    // [grid + 1] pieces of each workgroup
    const int32_t* piece_tile;  // [npieces] tile of each piece
    const int64_t* piece_chunk; // [npieces * (kWaves + 1)] chunk bounds of the waves
    const int32_t* piece_seg;   // [npieces * kWaves] segment holding each chunk's first entry
    const int32_t* chunk_flags; // [npieces * kWaves] kChunkMid | kChunkCont
    const uint64_t* dmask;      // 16-bit staged copies: bit w set when window w is
                                // delta-coded (null: none is)
    const int32_t* wg_cut;      // P == 1: [grid + 1] rows cut between the workgroup's waves,
    const int32_t* cut_row;     //   which it finishes at the end of the pass from the
    const uint64_t* cut_desc;   //   head (2w) and tail (2w + 1) partials of its waves w:
                                //   bits 0-3 the slot count - 1, then 5 bits per slot
    int32_t slot_lds;           // byte offset of those partials in LDS
    const V* x;                 // [cols] gathered vector of the update
    const V* p;                 // [S] own factor column, current feature, per segment
    const V* pp;                // [S] own factor column, previous feature (committed), per segment
    const V* q;                 // [cols] other factor column, current feature
    const V* qq;                // [cols] other factor column, previous feature (committed)
    const V* pk;                // [4 * cols] float hot or global first passes: (x, q, qq, 0)
                                // of every column, so that a gather reads one 16-byte record
    V* y;                       // [rows] coordinates (P == 1)
    part_t<V>* part;            // [S + 2 * chunks] partials: per segment (P > 1), then the
                                // head and tail slot of every chunk
    double* sse_part;           // [grid * kWaves] flush: per-wave sum of squares
    int32_t rows, cols, T, P;   // hot layouts: T is the pass's staged width
    int32_t tsw;                // hot layouts: indices below tsw are swizzled positions
    int32_t Ts;                 // LDS elements per staged vector slice
    int32_t pad;                // index held by padding entries (reads 0)
    int32_t nseg;               // S
    int32_t nseg_ne;            // segments with entries (P == 1: rows before the empty ones)
    int32_t vec_elems;          // LDS elements taken by staged vectors
    int32_t x_is_q;             // x and q are the same vector (staged once)
    double lambda;
};

// Finishes rows from partial slots: row ids[i] (or i when ids is null) adds
// part[srcs[src_ptr[i] .. src_ptr[i + 1])] in order.
template <class V>
struct CombineArgs {
    const int32_t* ids;          // [n] rows, or null
    const int32_t* src_ptr;      // [n + 1]
    const int32_t* srcs;
    const int32_t* seg_ptr;      // [n + 1] segments of each row (with yseg)
    const int32_t* segs;
    const part_t<V>* part;
    V* y;
    V* yseg;                     // optional [S]: y spread over the row's segments
    int32_t n;
    double lambda;
};

// One compressed copy of the residual plus its schedule.
// How the passes access a copy's residual stream.  Streaming (non-temporal) loads
// and stores keep a copy that is read once per pass from displacing everything
// else; a copy small enough to stay in the memory-side cache between passes
// gains from ordinary cached accesses.  The write-back policies exist for tiled
// float copies only.
enum CachePolicy : int32_t {
    kCacheStream = 0,  // non-temporal loads and stores
    kCacheStores = 1,  // non-temporal loads, write-back R-hat stores
    kCacheAll = 2,     // cached loads and write-back stores
};

struct Layout {
    int64_t rows = 0, cols = 0, nnz = 0;
    int64_t npad = 0;                // entries including alignment padding
    int32_t gather = kGatherGlobal;
    int32_t T = 0, P = 1;
    int32_t Ts = 0;                  // LDS elements per staged slice (swizzled range + zero)
    int32_t pad = 0;                 // padding index: the zero word (staged) or cols (global, hot)
    int32_t hot = 0;                 // hot layouts: the hot width tsw
    uint32_t swz_lim = 0;            // indices below it are swizzled LDS positions: all of
                                     // them (tiled), the hot width (hot), none (global)
    bool idx16 = false;
    int32_t cache = kCacheStream;    // CachePolicy of the passes over this copy
    uint64_t* dmask = nullptr;       // [ceil(npad / kWin / 64)] delta-coded windows, or null
    int64_t ndelta = 0;              // windows coded so
    void* idx = nullptr;             // [npad + kEntryPad]
    void* val = nullptr;             // [npad + kEntryPad] of the handle's value type
    int64_t* seg_start = nullptr;    // [S + 1], in padded positions
    int32_t* seg_row = nullptr;
    int32_t* tile_seg = nullptr;     // [P + 1] first segment of each tile
    int32_t* wg_piece = nullptr;
    int32_t* piece_tile = nullptr;
    int64_t* piece_chunk = nullptr;
    int32_t* piece_seg = nullptr;
    int32_t* chunk_flags = nullptr;
    int32_t npieces = 0;
    int32_t comb_lanes = 16;         // lanes per row of the combine (4 when rows have few partials)
    int32_t ncomb = 0;               // rows the combine finishes (P == 1: those cut
                                     // between workgroups)
    int32_t* comb_rows = nullptr;    // P == 1: their ids
    int32_t* src_ptr = nullptr;      // [ncomb + 1] partial slots of each combined row
    int32_t* srcs = nullptr;
    int64_t nsrc = 0;
    int32_t* wg_cut = nullptr;       // P == 1: [grid + 1] rows each workgroup finishes,
    int32_t* cut_row = nullptr;      //   those rows
    uint64_t* cut_desc = nullptr;    //   and their wave partials in entry order
    int32_t ncut = 0;
    int32_t* row_seg_ptr = nullptr;  // P > 1: segments of each row in tile order
    int32_t* row_segs = nullptr;
    void* part = nullptr;            // [nslots] part_t of the value type
    void* pk = nullptr;              // float hot or global layouts: [4 * cols] packed gathers
    int64_t nslots = 0;
    int64_t nseg = 0;
    int64_t nseg_ne = 0;
    int32_t grid = 0;                // persistent workgroups per pass
};

// Host helpers (host_copy.hip).  host_workers(): the host threads a set-up loop uses
// (at most 8).  parallel_ranges(n, w, f): f(worker, lo, hi) over w contiguous ranges of
// [0, n), the last on the calling thread; returns when all have finished.
int host_workers();
void parallel_ranges(int64_t n, int workers, const std::function<void(int, int64_t, int64_t)>& f);

// Host-to-device copies of caller memory on one stream through two pinned 32 MiB
// staging buffers (copies under 4 MiB, or without pinned memory, go straight).  The
// source may be reused once copy() returns; finish() waits until the staging
// buffers are read, and the destructor does so too before freeing them.
class Stager {
public:
    explicit Stager(hipStream_t s);
    ~Stager();
    Stager(const Stager&) = delete;
    Stager& operator=(const Stager&) = delete;
    hipError_t copy(void* dst, const void* src, size_t bytes);
    hipError_t finish();

private:
    bool ready();
    void release();
    hipStream_t s_;
    int workers_;
    void* slot_[2] = {nullptr, nullptr};
    hipEvent_t ev_[2] = {nullptr, nullptr};
    bool busy_[2] = {false, false};
    int next_ = 0;
    bool tried_ = false;
};

// Every device allocation of the library (api.hip); a host-forced failure for tests
// of the error paths returns hipErrorOutOfMemory.
hipError_t dev_malloc(void** p, size_t bytes);

// Launchers (sweep.hip), instantiated for V = float and V = double.
hipError_t sweep_init();  // raise the dynamic-LDS limit of the staged kernels
template <class V>
hipError_t launch_pass(const Layout& L, PassMode mode, const V* x, const V* p, const V* pp,
                       const V* q, const V* qq, V* y, double lambda, double* sse_part,
                       hipStream_t s);
template <class V>
hipError_t launch_combine(const Layout& L, V* y, V* yseg, double lambda, hipStream_t s);
template <class V>
hipError_t launch_copy(const V* src, V* dst, int64_t n, hipStream_t s);
hipError_t launch_reduce_sum(const double* part, int32_t n, double* out, hipStream_t s);
int staged_vectors(PassMode mode, bool x_is_q);

// Device build and utilities (build.hip); V as above, S a host-side element type.
// count[key[e]] += 1 over e < n, key[e] < bins (count zeroed by the caller); at most
// `workgroups` workgroups when the bins fit LDS.
hipError_t launch_histogram(const int32_t* key, int64_t n, int32_t bins, int32_t* count,
                           int32_t workgroups, hipStream_t s);
hipError_t launch_map(const int32_t* in, const int32_t* table, int64_t n, int32_t* out,
                      hipStream_t s);
hipError_t launch_seg_histogram(const int32_t* lrow, const int32_t* lcol, int64_t nnz,
                                int32_t rows, int32_t T, int32_t* count, hipStream_t s);
hipError_t launch_seg_keys(const int32_t* lrow, const int32_t* lcol, const int32_t* segid,
                           int64_t nnz, int32_t rows, int32_t T, int cbits, uint64_t* keys,
                           int32_t* ids, hipStream_t s);
hipError_t launch_dup_check(const uint64_t* keys, int64_t nnz, int32_t* flag, hipStream_t s);
template <class V>
hipError_t launch_layout_fill(const uint64_t* keys, const int32_t* perm, const float* val_in,
                              int64_t nnz, int cbits, const int32_t* seg_off, uint32_t swz_lim, bool idx16,
                              void* idx, V* val, int32_t* pos, hipStream_t s);
hipError_t launch_fill_idx(void* idx, bool idx16, int32_t value, int64_t n, hipStream_t s);
// Delta-codes the windows of a 16-bit index stream that allow it and marks them in
// dmask (zeroed by the caller, ceil(npad / kWin / 64) words).
hipError_t launch_delta_windows(void* idx, int64_t npad, int32_t pad, uint64_t* dmask,
                                hipStream_t s);
hipError_t launch_invert(const int32_t* perm, int64_t n, int32_t* inv, hipStream_t s);
hipError_t launch_slot_map(const int32_t* from, const int32_t* to, int64_t n, int32_t* out,
                          hipStream_t s);
template <class V>
hipError_t launch_copy_slots(const V* src, const int32_t* map, V* dst, int64_t n, hipStream_t s);
hipError_t launch_compose(const int32_t* a, const int32_t* b, int64_t n, int32_t* out,
                          hipStream_t s);
template <class V>
hipError_t launch_fill(V* dst, V value, int64_t n, hipStream_t s);
template <class S, class V>
hipError_t launch_scatter_factor_in(const S* rowmajor, const int32_t* new2old, int64_t rows,
                                    int32_t k, V* colmajor, hipStream_t s);
template <class V, class S>
hipError_t launch_gather_factor_out(const V* colmajor, const int32_t* old2new, int64_t rows,
                                    int32_t k, S* rowmajor, hipStream_t s);
template <class V>
hipError_t launch_rebuild_residual(const Layout& L, const int32_t* pos, const V* A, const V* W,
                                   const V* H, int64_t m, int64_t n, int32_t k, hipStream_t s);
// dst[dmap ? dmap[i] : i] = src[smap ? smap[i] : i] for i < n (converting between types)
template <class S, class V>
hipError_t launch_copy_mapped(const S* src, const int32_t* smap, V* dst, const int32_t* dmap,
                              int64_t n, hipStream_t s);
template <class V>
hipError_t launch_consistency(const V* a, const int32_t* amap, const V* b, const int32_t* bmap,
                              int64_t n, unsigned long long* count, hipStream_t s);
// The initial H from a seed (column-major over relabelled ids, k x n); see build.hip.
template <class V>
hipError_t launch_initial_h(uint64_t seed, const int32_t* new2old, int64_t n, int32_t k, V* H,
                            hipStream_t s);
// out[t * S + s] = F[t * rows + seg_row[s]] for t < k
template <class V>
hipError_t launch_seg_spread(const V* F, int64_t rows, const int32_t* seg_row, int64_t S,
                             int32_t k, V* out, hipStream_t s);
template <class V>
hipError_t launch_sq_sum(const V* v, int64_t n, double* part, int32_t nparts, hipStream_t s);
// Squared errors of held-out triplets into part[0 .. nparts); with `rejected`, the
// triplets are checked on the device and entries out of range or not finite are
// skipped and counted per block in rejected[0 .. nparts).
template <class V>
hipError_t launch_test_err(const int32_t* row, const int32_t* col, const float* val, int64_t nnz,
                           const int32_t* rold2new, const int32_t* cold2new, const V* W,
                           const V* H, int64_t m, int64_t n, int32_t k, double* part,
                           int32_t nparts, double* rejected, hipStream_t s);
// Device-wide primitives (rocPRIM); tmp is a temporary buffer grown as needed and
// freed by the caller.  sort_pairs: stable radix sort of (key, value) pairs on the
// low `bits` bits of the keys.  select_range: out[0 .. *count) = the indices e < n
// with lo <= key[e] < hi, in increasing order (count in device memory).
hipError_t sort_pairs(const uint64_t* kin, uint64_t* kout, const int32_t* vin, int32_t* vout,
                      int64_t n, int bits, hipStream_t s, void** tmp, size_t* tmp_bytes);
hipError_t select_range(const int32_t* key, int64_t n, int32_t lo, int32_t hi, int32_t* out,
                        int64_t* count, hipStream_t s, void** tmp, size_t* tmp_bytes);
hipError_t launch_add(int32_t* a, int64_t n, int32_t delta, hipStream_t s);

}  // namespace ccdk
