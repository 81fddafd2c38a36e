// Host runtime of the CCD++ library: the C ABI of include/ccdpp.h.
//
// The handle keeps everything on one device: the ratings A, the residual in a
// user-major and an item-major copy (each tiled and scheduled as described in
// ccdpp_internal.hpp), the map between the two copies, W and H column-major
// over relabelled ids (so the feature columns wbar_t and hbar_t of eq. 11 are
// contiguous), and the scratch vectors u and v.  Unlike the paper's
// Algorithm 7, u and v never travel to the host between features: the host
// only enqueues kernels on one stream, and ccdpp_run synchronises once at the
// end.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <mutex>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <numeric>

#include "ccdpp_internal.hpp"

using ccdk::Layout;
using ccdk::Stager;

namespace {

thread_local std::string g_create_error;

// Failures forced from the host for tests of the error paths (ccdpp_debug_inject):
// the device allocation, or the sweep-kernel launch, after this many more
// successful ones fails (-1: never).
std::atomic<int64_t> g_inject_alloc{-1};
std::atomic<int64_t> g_inject_launch{-1};

// True when the countdown c reaches this event (and disarms it).
bool injected(std::atomic<int64_t>& c) {
    int64_t v = c.load();
    while (v >= 0) {
        if (c.compare_exchange_weak(v, v - 1)) return v == 0;
    }
    return false;
}

// Gathers address records of up to 16 bytes per column with 32-bit byte offsets.
constexpr int64_t kMaxDim = int64_t(1) << 28;
constexpr int64_t kMaxNnz = INT32_MAX;
// Residual streams (values and indices of both copies) up to this size stay in
// MI355X's 256 MB memory-side cache from one pass to the next when the passes
// use cached accesses.
constexpr int64_t kCachedStreamBytes = int64_t(160) << 20;
constexpr int32_t kReduceParts = 1024;
// A row segment of a tiled layout costs about as much as this many gathers from
// global memory (its emission, partial and combine against one cache line each).
constexpr int64_t kSplitSegCost = 2;

struct ProfEvent {
    int kind;
    int layout;
    hipEvent_t a, b;
    double bytes;
};

}  // namespace

// Every device allocation of the library goes through here.
hipError_t ccdk::dev_malloc(void** p, size_t bytes) {
    if (injected(g_inject_alloc)) {
        *p = nullptr;
        return hipErrorOutOfMemory;
    }
    return hipMalloc(p, bytes);
}

// ---- scratch of the allocation-free entry point (ccdpp_rmse_noalloc) --------------
// kReduceParts partial sums of squared errors, as many per-block counts of rejected
// triplets, then the two totals: 2 * 1024 + 2 doubles, 16,400 bytes, held on every
// device the library runs on until the process ends.  Every call on a device shares
// that device's copy; each call overwrites all of it before reading it.
namespace {
constexpr int kNaPart = 0;                       // [kReduceParts] squared-error partials
constexpr int kNaRejected = kReduceParts;        // [kReduceParts] rejected-entry counts
constexpr int kNaTotals = 2 * kReduceParts;      // [2] their totals
constexpr int kNaDoubles = 2 * kReduceParts + 2;
constexpr int kMaxDevices = 64;
}  // namespace
static __device__ __align__(256) double scratch[kNaDoubles];

namespace {
std::mutex g_scratch_mu;
double* g_scratch_dev[kMaxDevices] = {};  // the device address of `scratch` per device
}  // namespace

struct ccdpp {
    int64_t m = 0, n = 0, nnz = 0;
    int32_t k = 0;
    double lambda = 0.0;
    int device = 0;
    int cus = 0;
    hipStream_t stream = nullptr;  // the device's null stream unless the caller sets one
    // 0: rows are users (eq. 15); 1: rows are items (eq. 16).  When the item-major copy
    // is split, L[1] holds its rows 0 .. split - 1 (the items with the most ratings),
    // tiled, and L[2] the others as a hot layout, its row r being item split + r; the
    // two parts' values sit in one array, L[2]'s from slot off2 on.
    Layout L[3];
    int64_t split = 0;
    int64_t off2 = 0;
    int32_t* rnew2old = nullptr;   // relabelled user id -> input user id
    int32_t* rold2new = nullptr;
    int32_t* cnew2old = nullptr;
    int32_t* cold2new = nullptr;
    // Entry e of the user-major copy in layout order, padding excluded:
    int32_t* perm0 = nullptr;      // e -> input triplet index
    int32_t* pos0 = nullptr;       // e -> value slot in the user-major copy
    int32_t* map01 = nullptr;      // e -> value slot in the item-major copy
    int32_t* slot01 = nullptr;     // element-wise CCD: user-major slot -> item-major slot (or -1)
    int32_t* slot10 = nullptr;     //   and back; built on the first ccdpp_ccd_run
    // Value type of the residual, the factors and the sweep arithmetic: float, or
    // double with options.precision = 1.  The arrays below hold that type.
    bool dbl = false;
    void* A = nullptr;             // A[e], the rating of entry e
    void* fseg[3] = {};            // P > 1: own factor columns spread over segments (k x S)
    void* W = nullptr;             // k x m: W[t*m + i]
    void* H = nullptr;             // k x n
    void* u = nullptr;
    void* v = nullptr;
    double* sse_part = nullptr;
    int32_t sse_nparts = 0;
    double* d_scalar = nullptr;
    unsigned long long* d_count = nullptr;
    double* scratch = nullptr;     // device address of this device's `scratch` array
    int32_t pending = -1;          // feature whose eq. 18 subtract is still folded into R-hat
    double train_sse = 0.0;
    bool train_sse_valid = false;
    std::string err;
    bool poisoned = false;
    int64_t build_us = 0;
    // Device build phases, microseconds: inputs and degrees; relabelling; user-major copy;
    // item-major copy and the map between the copies; cache policy, index coding and
    // scratch; factors; the device set-up before the inputs (device checks, kernel
    // attributes, scratch address).
    int64_t build_phase_us[7] = {};
    int64_t bytes_held = 0;
    std::vector<std::pair<void*, int64_t>> allocs;  // device allocations and their sizes
    // kernel timing
    bool prof = false;
    int32_t prof_kind = -1, prof_layout = -1;  // restrict timing to one kind / copy (-1: all)
    int32_t prof_every = 1;        // time every n-th launch that the selection matches
    bool cache_auto[2] = {true, true};  // the copy's cache policy was chosen automatically
    bool wb_stores = false;        // the running sweep takes automatic write-back stores
    int64_t prof_seen = 0;         // matching launches since the selection was set
    std::vector<ProfEvent> prof_pending;
    std::vector<hipEvent_t> event_pool;
    int64_t prof_launch[CCDPP_K_COUNT][2] = {};
    double prof_ms[CCDPP_K_COUNT][2] = {};
    double prof_bytes[CCDPP_K_COUNT][2] = {};
};

namespace {

int fail(ccdpp* h, int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (h) {
        h->err = buf;
        if (code == CCDPP_EDEVICE) h->poisoned = true;
    } else {
        g_create_error = buf;
    }
    return code;
}

#define HIPCK(h, expr)                                                                         \
    do {                                                                                       \
        hipError_t e_ = (expr);                                                                \
        if (e_ != hipSuccess)                                                                  \
            return fail((h), e_ == hipErrorOutOfMemory ? CCDPP_ENOMEM : CCDPP_EDEVICE,         \
                        "%s failed: %s", #expr, hipGetErrorString(e_));                       \
    } while (0)

#define RCK(expr)                      \
    do {                               \
        int r_ = (expr);               \
        if (r_ != CCDPP_OK) return r_; \
    } while (0)

// Calls f with a value of the handle's value type (float or double).
template <class F>
auto with_value_type(const ccdpp* h, F&& f) {
    return h->dbl ? f(double{}) : f(float{});
}
template <class V>
V* as(void* p) {
    return static_cast<V*>(p);
}

template <class T>
hipError_t dalloc(ccdpp* h, T** p, int64_t count) {
    size_t bytes = (size_t)std::max<int64_t>(count, 1) * sizeof(T);
    void* q = nullptr;
    hipError_t e = ccdk::dev_malloc(&q, bytes);
    if (e != hipSuccess) return e;
    h->allocs.emplace_back(q, (int64_t)bytes);
    h->bytes_held += (int64_t)bytes;
    *p = static_cast<T*>(q);
    return hipSuccess;
}

template <class T>
int upload(ccdpp* h, T** dst, const std::vector<T>& src) {
    HIPCK(h, dalloc(h, dst, (int64_t)src.size()));
    if (!src.empty())
        HIPCK(h, hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice));
    return CCDPP_OK;
}

// Frees one of the handle's device allocations before the handle goes.
void dfree(ccdpp* h, void* p) {
    for (size_t i = 0; i < h->allocs.size(); ++i)
        if (h->allocs[i].first == p) {
            h->bytes_held -= h->allocs[i].second;
            h->allocs.erase(h->allocs.begin() + (std::ptrdiff_t)i);
            (void)hipFree(p);
            return;
        }
}

// Value slots of the item-major copy: both parts when it is split.
int64_t item_slots(const ccdpp* h) {
    return h->split > 0 ? h->off2 + h->L[2].npad : h->L[1].npad;
}

// Temporary device buffer freed when it goes out of scope.
struct Tmp {
    void* p = nullptr;
    ~Tmp() {
        if (p) (void)hipFree(p);
    }
};
template <class T>
hipError_t talloc(Tmp& t, T** p, int64_t count) {
    hipError_t e = ccdk::dev_malloc(&t.p, (size_t)std::max<int64_t>(count, 1) * sizeof(T));
    *p = static_cast<T*>(t.p);
    return e;
}

bool usable(const ccdpp* h) { return h && !h->poisoned; }

int bits_for(uint64_t maxval) {
    int b = 1;
    while (b < 64 && (maxval >> b) != 0) ++b;
    return b;
}

// Order ids by decreasing count, ties by increasing id: a counting sort over the
// counts (a comparison sort when the largest count dwarfs the number of ids).
void relabel(const std::vector<int32_t>& count, std::vector<int32_t>& new2old,
             std::vector<int32_t>& old2new) {
    const int64_t N = (int64_t)count.size();
    new2old.resize(N);
    old2new.resize(N);
    const int32_t maxc = N ? *std::max_element(count.begin(), count.end()) : 0;
    if ((int64_t)maxc <= 4 * N + 1024) {
        std::vector<int64_t> start((size_t)maxc + 2, 0);  // bucket b = maxc - count
        for (int32_t c : count) ++start[(size_t)(maxc - c) + 1];
        for (size_t b = 1; b < start.size(); ++b) start[b] += start[b - 1];
        for (int64_t i = 0; i < N; ++i) new2old[(size_t)start[(size_t)(maxc - count[i])]++] = (int32_t)i;
    } else {
        std::iota(new2old.begin(), new2old.end(), 0);
        std::stable_sort(new2old.begin(), new2old.end(),
                         [&](int32_t a, int32_t b) { return count[a] > count[b]; });
    }
    for (int64_t i = 0; i < N; ++i) old2new[new2old[i]] = (int32_t)i;
}

// Rows 0 .. H - 1 of a copy (the longest: rows are relabelled by decreasing length)
// are worth tiling when their segments cost less than the gathers from global memory
// a hot layout would give them.  cnt holds the entries per (tile, row) of the tiled
// layout; a row's segments are its non-empty tiles, and its entries in tiles at or
// past `hot` columns are those a hot layout staging `hot` columns gathers from global
// memory.  H maximises the sum of (gathers - seg_cost * segments) over the rows it
// takes.
int64_t choose_split(const std::vector<int32_t>& cnt, int64_t P, int64_t rows, int64_t T,
                     int64_t hot, int64_t seg_cost) {
    // Segments and cold entries per row, gathered tile by tile (cnt is tile-major).
    std::vector<int32_t> segs((size_t)rows, 0);
    std::vector<int64_t> cold((size_t)rows, 0);
    for (int64_t p = 0; p < P; ++p) {
        const int32_t* cp = cnt.data() + p * rows;
        const bool is_cold = p * T >= hot;
        for (int64_t r = 0; r < rows; ++r) {
            segs[r] += cp[r] > 0;
            if (is_cold) cold[r] += cp[r];
        }
    }
    int64_t best = 0, H = 0, gain = 0;
    for (int64_t r = 0; r < rows; ++r) {
        if (segs[r] == 0) break;  // the empty rows come last
        gain += cold[r] - seg_cost * segs[r];
        if (gain > best) {
            best = gain;
            H = r + 1;
        }
    }
    return H;
}

// Build one layout of nnz entries.  lrow/lcol: relabelled row and gathered-column id
// of every entry (device).  side 0 is the user-major copy (its first pass stages q
// and qq, x being q), side 1 the item-major copy (first pass stages x, q, qq).  On
// return, for every entry e in layout order (padding excluded), perm[e] holds its
// index in lrow/lcol/val_in and epos[e] the slot of its value (val_slot).  With
// split_out, a copy that automatic mode would make hot may instead ask to be split:
// *split_out receives the number of leading rows to tile (0: not split), and a
// nonzero answer returns before anything is built.
int build_layout(ccdpp* h, int side, Layout& L, int64_t rows, int64_t cols, const int32_t* lrow,
                 const int32_t* lcol, const float* val_in, const ccdpp_options_t* opt,
                 int32_t* perm, int32_t* epos, hipStream_t s, int64_t nnz,
                 int64_t* split_out = nullptr, const int32_t* row_deg = nullptr) {
    using namespace ccdk;
    const int64_t N = nnz;
    L.rows = rows;
    L.cols = cols;
    L.nnz = N;
    const int nvec = side == 0 ? 2 : 3;
    // Each staged slice holds T floats rounded up to 32, then 32 more words whose first
    // is the zero the padding entries read.
    const int64_t vbytes = h->dbl ? 8 : 4;
    const int64_t tmax = ((int64_t)kLdsVecBytes / (vbytes * nvec) - 64) / 64 * 64;
    const int64_t hmax = ((int64_t)kLdsVecBytes / vbytes - 64) / 64 * 64;  // one vector
    const int forced = opt ? opt->gather_mode[side] : 0;
    const int64_t forced_T = opt ? opt->tile_width[side] : 0;
    if (forced == kGatherHot) {
        if (forced_T > hmax || forced_T % 32 != 0)
            return fail(h, CCDPP_EINVAL, "hot tile_width must be a multiple of 32, at most %lld",
                        (long long)hmax);
    } else if (forced_T > tmax) {
        return fail(h, CCDPP_EINVAL, "tile_width must be at most %lld", (long long)tmax);
    }

    // Tile width: whole vector if it fits, else balanced tiles of at most tmax.
    int64_t T = cols, P = 1;
    int mode = forced == kGatherGlobal || forced == kGatherHot ? forced : kGatherLds;
    if (forced_T > 0 && mode == kGatherLds) {
        T = forced_T;
    } else if (cols > tmax) {
        P = (cols + tmax - 1) / tmax;
        T = ((cols + P - 1) / P + 63) / 64 * 64;
    }
    if (mode != kGatherLds) T = cols;
    P = (cols + T - 1) / T;
    if ((uint64_t)P * (uint64_t)rows > (uint64_t)INT32_MAX) {
        if (forced == kGatherLds) return fail(h, CCDPP_EINVAL, "too many (tile, row) pairs");
        mode = kGatherHot;
        T = cols;
        P = 1;
    }

    // Entries per (tile, row).
    std::vector<int32_t> cnt;
    for (int attempt = 0; attempt < 2; ++attempt) {
        if (P == 1 && row_deg) {  // one tile: the entries per row are the row lengths
            cnt.assign(row_deg, row_deg + rows);
        } else {
            int32_t* d_cnt;
            Tmp tc;
            HIPCK(h, talloc(tc, &d_cnt, P * rows));
            HIPCK(h, hipMemsetAsync(d_cnt, 0, (size_t)(P * rows) * 4, s));
            HIPCK(h, launch_seg_histogram(lrow, lcol, N, (int32_t)rows, (int32_t)T, d_cnt, s));
            cnt.assign((size_t)(P * rows), 0);
            HIPCK(h, hipMemcpyAsync(cnt.data(), d_cnt, (size_t)(P * rows) * 4,
                                    hipMemcpyDeviceToHost, s));
            HIPCK(h, hipStreamSynchronize(s));
            if (std::accumulate(cnt.begin(), cnt.end(), int64_t(0)) != N)
                return fail(h, CCDPP_EDEVICE, "segment counts do not add up to nnz");
        }
        if (P == 1 || forced == kGatherLds) break;
        // Tiling pays only when segments are long enough; otherwise stage the leading
        // columns and gather the others through L2.
        int64_t nonempty = 0;
        for (int32_t c : cnt) nonempty += c > 0;
        if (nonempty > 0 && N / nonempty >= kMinTiledSeg) break;
        if (split_out && forced == 0) {
            // Stage the hot part's plain passes as wide as one vector allows.
            const int64_t H = choose_split(cnt, P, rows, T, hmax, kSplitSegCost);
            if (H > 0 && H < rows) {
                *split_out = H;
                return CCDPP_OK;
            }
        }
        mode = kGatherHot;
        T = cols;
        P = 1;
    }
    // A hot layout stages whole groups of 32 leading columns; with fewer columns than
    // that it gathers everything from global memory.
    if (mode == kGatherHot && cols < 32) mode = kGatherGlobal;
    const bool lds = mode == kGatherLds;
    L.gather = mode;
    L.T = (int32_t)T;
    L.P = (int32_t)P;
    L.pad = lds ? (int32_t)((T + 31) / 32 * 32) : (int32_t)T;
    L.Ts = lds ? L.pad + 32 : (int32_t)T + 1;
    if (mode == kGatherHot) {
        // Hot width: the widest one-vector slice, never past the last whole group of
        // 32 columns (so the padding index cols stays outside the swizzled range).
        L.hot = (int32_t)std::min<int64_t>(forced_T > 0 ? forced_T : hmax, cols / 32 * 32);
        L.swz_lim = (uint32_t)L.hot;
    } else {
        L.hot = 0;
        L.swz_lim = lds ? 0xFFFFFFFFu : 0u;
    }
    // Every index, the padding one included, fits 15 bits (the 16th is the start bit);
    // hot layouts always take 32-bit indices.
    L.idx16 = mode != kGatherHot && L.pad < (int32_t)IndexBits<uint16_t>::start;

    // Segments.  P == 1: segment r is row r (rows are relabelled by decreasing
    // length, so the empty ones come last).  P > 1: the non-empty rows of each
    // tile in increasing row order.
    std::vector<int32_t> segid((size_t)(P * rows), -1), seg_row, tile_seg(P + 1, 0);
    std::vector<int64_t> seg_start;
    int64_t pos = 0;
    for (int64_t p = 0; p < P; ++p) {
        tile_seg[p] = (int32_t)seg_row.size();
        const int32_t* cp = cnt.data() + p * rows;
        for (int64_t r = 0; r < rows; ++r) {
            if (P > 1 && cp[r] == 0) continue;
            if (P == 1 && r > 0 && cp[r] > cp[r - 1])
                return fail(h, CCDPP_EDEVICE, "internal: rows are not in decreasing length");
            segid[p * rows + r] = (int32_t)seg_row.size();
            seg_row.push_back((int32_t)r);
            seg_start.push_back(pos);
            pos += cp[r];
        }
    }
    tile_seg[P] = (int32_t)seg_row.size();
    seg_start.push_back(pos);
    const int64_t S = (int64_t)seg_row.size();
    if (pos != N) return fail(h, CCDPP_EDEVICE, "internal: segment counts do not cover nnz");
    L.nseg = S;
    int64_t S_ne = S;
    while (S_ne > 0 && seg_start[S_ne] == seg_start[S_ne - 1]) --S_ne;
    L.nseg_ne = S_ne;

    // Alignment padding: every segment starts at a multiple of kE; the first segment
    // of a tile, and a segment that begins a workgroup's share (below), at a multiple
    // of kAlign.  The entries skipped over are padding at the end of the previous
    // segment.
    const int64_t S_work = P == 1 ? S_ne : S;  // segments that hold entries
    const std::vector<int64_t> seg_start0 = seg_start;  // unpadded
    std::vector<int32_t> seg_off((size_t)S, 0);
    std::vector<char> align_first((size_t)S + 1, 0);
    for (int64_t p = 0; p < P; ++p) align_first[tile_seg[p]] = 1;
    int64_t NP = 0;
    auto pad_layout = [&]() -> int {
        int64_t off = 0;
        for (int64_t sg = 0; sg < S_work; ++sg) {
            const int64_t al = align_first[sg] ? kAlign : kE;
            off += (al - (seg_start0[sg] + off) % al) % al;
            if (seg_start0[sg] + off > (int64_t)INT32_MAX - kEntryPad)
                return fail(h, CCDPP_EINVAL, "too many entries after alignment padding");
            seg_off[sg] = (int32_t)off;
            seg_start[sg] = seg_start0[sg] + off;  // from here on, padded positions
        }
        NP = (N + off + kAlign - 1) / kAlign * kAlign;
        if (NP > (int64_t)INT32_MAX - kEntryPad)
            return fail(h, CCDPP_EINVAL, "too many entries after alignment padding");
        for (int64_t sg = S_work; sg <= S; ++sg) seg_start[sg] = NP;
        return CCDPP_OK;
    };
    RCK(pad_layout());

    // Persistent workgroups own equal shares of the work, cut at multiples of kAlign; a
    // share is processed as one piece per tile it touches, and every piece is cut
    // into kWaves chunks of equal work, one per wave.  The work of a range is its
    // entries plus seg_weight per segment starting in it (a segment's emission, and
    // the shorter windows of short segments, cost about that many entries).  Chunk
    // bounds ignore segment bounds: a segment cut by one or more chunk bounds leaves,
    // in every chunk it meets, a partial (num, den) in a slot of its own (the chunk's
    // head slot if the segment began before the chunk, else its tail slot), and the
    // partials of a row are added in entry order.
    // Two shares per compute unit when every wave still gets several windows: a
    // workgroup holds a whole CU's LDS, so the second round of workgroups goes to
    // whichever CUs finish first, which evens out the remaining differences in speed
    // between shares.  Smaller layouts take one share per compute unit, which halves
    // the per-workgroup staging and start-up; very long ones four, whose shorter last
    // round leaves less of the pass's end to the slowest shares (measured on MI355X:
    // 252.8M ratings, user-major passes 2-3% faster; with 100M ratings four rounds were
    // slower, the staging then weighing more).
    int64_t G;
    if (opt && opt->workgroups > 0) {
        G = opt->workgroups;
    } else {
        const int64_t cus = h->cus;
        const int64_t per_wave = NP / (cus * kWaves * kWin);  // windows per wave, one round
        G = per_wave >= 120 ? 4 * cus : per_wave >= 16 ? 2 * cus : cus;
        G = std::max<int64_t>(1, std::min<int64_t>(G, (NP + kWaves * kWin - 1) / (kWaves * kWin)));
    }
    const int64_t wseg = !opt || opt->seg_weight == 0 ? kSegWeight
                         : std::max<int64_t>(0, opt->seg_weight);
    auto upa = [](int64_t v) { return (v + kAlign - 1) / kAlign * kAlign; };
    // Last segment of tile p starting at or before position e.
    auto seg_of = [&](int64_t p, int64_t e) -> int64_t {
        return std::upper_bound(seg_start.begin() + tile_seg[p], seg_start.begin() + tile_seg[p + 1],
                                e) - seg_start.begin() - 1;
    };
    // Work up to position e, and the last position whose work is at most t.
    auto work_at = [&](int64_t e) -> int64_t {
        if (S_work == 0) return e;
        const int64_t sg = std::upper_bound(seg_start.begin(), seg_start.begin() + S_work, e) -
                           seg_start.begin();  // segments starting at or before e
        return e + wseg * sg;
    };
    // The largest position e <= NP with work_at(e) <= t (0 if there is none).  Segment
    // starts are strictly increasing, and inside segment s the work grows by one per
    // position from ws[s], the work at its start, so one search over the segment
    // starts finds it.
    std::vector<int64_t> ws;
    auto index_work = [&]() {
        ws.resize((size_t)S_work);
        for (int64_t sg = 0; sg < S_work; ++sg) ws[sg] = seg_start[sg] + wseg * (sg + 1);
    };
    auto pos_at = [&](int64_t t) -> int64_t {
        if (S_work == 0) return std::max<int64_t>(0, std::min(t, NP));
        const int64_t sg = std::upper_bound(ws.begin(), ws.end(), t) - ws.begin() - 1;
        if (sg < 0) return std::max<int64_t>(0, std::min(t, seg_start[0] - 1));
        const int64_t end = sg + 1 < S_work ? seg_start[sg + 1] - 1 : NP;
        return std::min(seg_start[sg] + (t - ws[sg]), std::min(end, NP));
    };
    index_work();
    auto target = [&](int64_t wt, int64_t g) { return wt / G * g + wt % G * g / G; };
    // With P == 1 (float) every share boundary moves to the start of the nearest row,
    // when none of them changes its shares by more than an eighth: rows are then
    // cut only between the waves of one workgroup, which finishes them at the end of
    // the pass, and no combine kernel runs.  Otherwise the shares stay balanced and
    // the combine kernel finishes every cut row.
    std::vector<int64_t> snap((size_t)G + 1, -1);
    bool snapped = false;
    if (P == 1 && S_work > 0 && !h->dbl) {  // (one workgroup: nothing to move)
        const int64_t wt = work_at(NP);
        snapped = true;
        for (int64_t g = 1; g < G && snapped; ++g) {
            const int64_t t = target(wt, g);
            const int64_t sg = std::min<int64_t>(seg_of(0, pos_at(t)), S_work - 1);
            int64_t best = sg;
            auto miss = [&](int64_t x) { return std::llabs(work_at(seg_start[x]) - t); };
            if (sg + 1 < S_work && miss(sg + 1) < miss(sg)) best = sg + 1;
            snap[g] = best;
            snapped = miss(best) <= wt / G / 8;
        }
        if (snapped) {
            for (int64_t g = 1; g < G; ++g) align_first[snap[g]] = 1;
            RCK(pad_layout());
            index_work();
        } else {
            std::fill(snap.begin(), snap.end(), -1);
        }
    }
    L.npad = NP;
    const int64_t work_total = work_at(NP);
    std::vector<int32_t> wg_piece(1, 0), piece_tile, piece_seg, chunk_flags;
    std::vector<int64_t> piece_chunk;
    // Partial slots of the cut segments, as (segment, slot) in the order the chunks are cut.
    std::vector<std::pair<int32_t, int32_t>> cuts;
    std::vector<int64_t> gb((size_t)G + 1);
    for (int64_t g = 0; g <= G; ++g) {
        gb[g] = g == 0 ? 0 : g == G ? NP
                : snap[g] >= 0 ? seg_start[snap[g]] : std::min(NP, upa(pos_at(target(work_total, g))));
        if (g > 0) gb[g] = std::max(gb[g], gb[g - 1]);
    }
    for (int64_t g = 0; g < G; ++g) {
        const int64_t lo = gb[g], hi = std::max(gb[g], gb[g + 1]);
        for (int64_t p = 0; p < P; ++p) {
            const int64_t a0 = std::max(lo, seg_start[tile_seg[p]]);
            const int64_t a1 = std::min(hi, seg_start[tile_seg[p + 1]]);
            if (a0 >= a1) continue;
            const int64_t pc = (int64_t)piece_tile.size();
            piece_tile.push_back((int32_t)p);
            const int64_t w0 = work_at(a0), w1 = work_at(a1);
            for (int w = 0; w <= kWaves; ++w)
                piece_chunk.push_back(w == 0 ? a0 : w == kWaves ? a1
                                      : std::min(a1, std::max(a0, upa(pos_at(w0 + (w1 - w0) * w / kWaves)))));
            for (int w = 0; w < kWaves; ++w) {
                const int64_t c0 = piece_chunk[pc * (kWaves + 1) + w];
                const int64_t c1 = piece_chunk[pc * (kWaves + 1) + w + 1];
                const int64_t gc = pc * kWaves + w;
                if (c0 >= c1) {
                    piece_seg.push_back(0);
                    chunk_flags.push_back(0);
                    continue;
                }
                const int64_t s0 = seg_of(p, c0), s1 = seg_of(p, c1 - 1);
                const bool mid = seg_start[s0] < c0;     // first segment began earlier
                const bool cont = seg_start[s1 + 1] > c1;  // last segment goes on
                piece_seg.push_back((int32_t)s0);
                chunk_flags.push_back((mid ? kChunkMid : 0) | (cont ? kChunkCont : 0));
                if (mid) cuts.emplace_back((int32_t)s0, (int32_t)(S + 2 * gc));
                if (cont && !(mid && s1 == s0)) cuts.emplace_back((int32_t)s1, (int32_t)(S + 2 * gc + 1));
            }
        }
        wg_piece.push_back((int32_t)piece_tile.size());
    }
    // Grouped by segment (a stable sort keeps each segment's slots in entry order):
    // cut_seg[c] is the c-th cut segment, its slots cut_slot[cut_off[c] .. cut_off[c + 1]).
    std::stable_sort(cuts.begin(), cuts.end(),
                     [](const std::pair<int32_t, int32_t>& a, const std::pair<int32_t, int32_t>& b) {
                         return a.first < b.first;
                     });
    std::vector<int32_t> cut_seg, cut_slot, cut_off(1, 0);
    for (const auto& c : cuts) {
        if (cut_seg.empty() || cut_seg.back() != c.first) {
            if (!cut_seg.empty()) cut_off.push_back((int32_t)cut_slot.size());
            cut_seg.push_back(c.first);
        }
        cut_slot.push_back(c.second);
    }
    if (!cut_seg.empty()) cut_off.push_back((int32_t)cut_slot.size());
    std::vector<char> cut_fin(cut_seg.size(), 0);  // finished by its workgroup in the pass
    L.grid = (int32_t)G;
    L.npieces = (int32_t)piece_tile.size();
    const int64_t nslots = S + 2 * (int64_t)L.npieces * kWaves;
    if (nslots > INT32_MAX) return fail(h, CCDPP_EINVAL, "too many partial slots");

    // Combine lists.  P == 1: only the rows whose segment was cut, each from its
    // partial slots; a row cut only between the waves of one workgroup is finished
    // by that workgroup at the end of the pass (its wg_cut list), the others by the
    // combine kernel.  P > 1: every row, from its segments in tile order (a cut
    // segment by its partial slots), plus the segment list for the per-segment
    // copy of the committed coordinate.
    if (P == 1) {
        std::vector<int32_t> piece_wg((size_t)L.npieces);
        for (int64_t g = 0; g < G; ++g)
            for (int32_t pc = wg_piece[g]; pc < wg_piece[g + 1]; ++pc) piece_wg[pc] = (int32_t)g;
        auto slot_wg = [&](int32_t slot) { return piece_wg[(slot - S) / 2 / kWaves]; };
        std::vector<int32_t> wcut(1, 0), crow;
        std::vector<uint64_t> cdesc;
        std::vector<std::vector<int64_t>> local((size_t)G);
        for (size_t c = 0; snapped && c < cut_seg.size(); ++c) {
            const int32_t* sl = cut_slot.data() + cut_off[c];
            const int32_t ns = cut_off[c + 1] - cut_off[c];
            if (ns > kCutMaxSlots) continue;
            const int32_t g0 = slot_wg(sl[0]);
            bool one = true;
            for (int32_t i = 0; i < ns; ++i) one = one && slot_wg(sl[i]) == g0;
            if (!one) continue;
            // Local slot 2w (head) or 2w + 1 (tail) of wave w: the workgroup has one piece.
            uint64_t d = (uint64_t)(ns - 1);
            for (int32_t i = 0; i < ns; ++i)
                d |= (uint64_t)((sl[i] - S) % (2 * kWaves)) << (4 + 5 * i);
            if (local[g0].size() >= 64) return fail(h, CCDPP_EDEVICE, "internal: too many cut rows");
            local[g0].push_back(cut_seg[c]);
            cdesc.push_back(d);
            cut_fin[c] = 1;
        }
        std::vector<uint64_t> cdesc_sorted;
        {
            // cdesc follows segment order, which is also workgroup order.
            size_t k = 0;
            for (int64_t g = 0; g < G; ++g) {
                for (int64_t sg : local[g]) {
                    crow.push_back((int32_t)sg);
                    cdesc_sorted.push_back(cdesc[k++]);
                }
                wcut.push_back((int32_t)crow.size());
            }
        }
        RCK(upload(h, &L.wg_cut, wcut));
        if (!crow.empty()) {
            RCK(upload(h, &L.cut_row, crow));
            RCK(upload(h, &L.cut_desc, cdesc_sorted));
        }
        L.ncut = (int32_t)crow.size();
    }
    {
        std::vector<int32_t> ids, sptr(1, 0), srcs, gptr, gsegs;
        auto add_cut = [&](size_t c) {
            srcs.insert(srcs.end(), cut_slot.begin() + cut_off[c], cut_slot.begin() + cut_off[c + 1]);
        };
        if (P == 1) {
            for (size_t c = 0; c < cut_seg.size(); ++c)
                if (!cut_fin[c]) {
                    ids.push_back(cut_seg[c]);
                    add_cut(c);
                    sptr.push_back((int32_t)srcs.size());
                }
            L.ncomb = (int32_t)ids.size();
            if (!ids.empty()) RCK(upload(h, &L.comb_rows, ids));
        } else {
            // The segments of each row in tile order: segment ids grow with the tile, so
            // bucketing them by row in id order lists each row's in tile order.
            gptr.assign((size_t)rows + 1, 0);
            for (int64_t sg = 0; sg < S; ++sg) ++gptr[seg_row[sg] + 1];
            for (int64_t r = 0; r < rows; ++r) gptr[r + 1] += gptr[r];
            gsegs.resize((size_t)S);
            {
                std::vector<int32_t> next(gptr.begin(), gptr.end() - 1);
                for (int64_t sg = 0; sg < S; ++sg) gsegs[next[seg_row[sg]]++] = (int32_t)sg;
            }
            std::vector<int32_t> cut_of((size_t)S, -1);  // index into cut_seg, or -1
            for (size_t c = 0; c < cut_seg.size(); ++c) cut_of[cut_seg[c]] = (int32_t)c;
            for (int64_t r = 0; r < rows; ++r) {
                for (int32_t i = gptr[r]; i < gptr[r + 1]; ++i) {
                    const int32_t sg = gsegs[i];
                    if (cut_of[sg] < 0)
                        srcs.push_back(sg);
                    else
                        add_cut((size_t)cut_of[sg]);
                }
                sptr.push_back((int32_t)srcs.size());
            }
            L.ncomb = (int32_t)rows;
            RCK(upload(h, &L.row_seg_ptr, gptr));
            RCK(upload(h, &L.row_segs, gsegs));
        }
        if (L.ncomb > 0) {
            RCK(upload(h, &L.src_ptr, sptr));
            RCK(upload(h, &L.srcs, srcs));
        }
        L.nsrc = (int64_t)srcs.size();
        // A quad per row when rows have fewer than 12 partials on average.
        L.comb_lanes = L.ncomb > 0 && L.nsrc < 12 * (int64_t)L.ncomb ? 4 : 16;
        RCK(with_value_type(h, [&](auto z) -> int {
            part_t<decltype(z)>* pp;
            HIPCK(h, dalloc(h, &pp, nslots));
            L.part = pp;
            return CCDPP_OK;
        }));
        L.nslots = nslots;
    }
    if (!lds && !h->dbl) {
        float* pk;
        HIPCK(h, dalloc(h, &pk, 4 * cols));
        L.pk = pk;
    }
    RCK(upload(h, &L.seg_start, seg_start));
    RCK(upload(h, &L.seg_row, seg_row));
    RCK(upload(h, &L.tile_seg, tile_seg));
    RCK(upload(h, &L.wg_piece, wg_piece));
    RCK(upload(h, &L.piece_tile, piece_tile));
    RCK(upload(h, &L.piece_chunk, piece_chunk));
    RCK(upload(h, &L.piece_seg, piece_seg));
    RCK(upload(h, &L.chunk_flags, chunk_flags));

    // Sort the entries into layout order and fill index and value arrays.
    const int cbits = bits_for((uint64_t)std::max<int64_t>(T - 1, 1));
    const int sbits = bits_for((uint64_t)std::max<int64_t>(S - 1, 1));
    if (cbits + sbits > 64) return fail(h, CCDPP_EDEVICE, "internal: sort key too wide");
    // Padding entries (and kEntryPad more after the end, for whole-lane vector loads)
    // hold value 0 and the padding index T.
    RCK(with_value_type(h, [&](auto z) -> int {
        using V = decltype(z);
        V* pv;
        HIPCK(h, dalloc(h, &pv, NP + kEntryPad));
        L.val = pv;
        HIPCK(h, launch_fill<V>(pv, V(0), NP + kEntryPad, s));
        return CCDPP_OK;
    }));
    if (L.idx16) {
        uint16_t* d;
        HIPCK(h, dalloc(h, &d, NP + kEntryPad));
        L.idx = d;
    } else {
        int32_t* d;
        HIPCK(h, dalloc(h, &d, NP + kEntryPad));
        L.idx = d;
    }
    HIPCK(h, launch_fill_idx(L.idx, L.idx16, L.pad, NP + kEntryPad, s));
    if (N > 0) {
        int32_t *d_segid, *d_off;
        uint64_t *k0, *k1;
        int32_t* i0;
        Tmp tsid, toff, tk0, tk1, ti0, ttmp;
        HIPCK(h, talloc(tsid, &d_segid, P * rows));
        HIPCK(h, hipMemcpyAsync(d_segid, segid.data(), segid.size() * 4, hipMemcpyHostToDevice, s));
        HIPCK(h, talloc(toff, &d_off, S));
        HIPCK(h, hipMemcpyAsync(d_off, seg_off.data(), seg_off.size() * 4, hipMemcpyHostToDevice, s));
        HIPCK(h, talloc(tk0, &k0, N));
        HIPCK(h, talloc(tk1, &k1, N));
        HIPCK(h, talloc(ti0, &i0, N));
        HIPCK(h, launch_seg_keys(lrow, lcol, d_segid, N, (int32_t)rows, (int32_t)T, cbits, k0, i0,
                                 s));
        void* tmp = nullptr;
        size_t tmp_bytes = 0;
        hipError_t e = sort_pairs(k0, k1, i0, perm, N, cbits + sbits, s, &tmp, &tmp_bytes);
        ttmp.p = tmp;
        HIPCK(h, e);
        if (side == 0) {
            int32_t* d_flag;
            Tmp tflag;
            HIPCK(h, talloc(tflag, &d_flag, 1));
            HIPCK(h, hipMemsetAsync(d_flag, 0, 4, s));
            HIPCK(h, launch_dup_check(k1, N, d_flag, s));
            int32_t flag = 0;
            HIPCK(h, hipMemcpyAsync(&flag, d_flag, 4, hipMemcpyDeviceToHost, s));
            HIPCK(h, hipStreamSynchronize(s));
            if (flag) return fail(h, CCDPP_EDUP, "a position (i, j) occurs more than once");
        }
        RCK(with_value_type(h, [&](auto z) -> int {
            using V = decltype(z);
            HIPCK(h, launch_layout_fill<V>(k1, perm, val_in, N, cbits, d_off, L.swz_lim, L.idx16, L.idx,
                                           as<V>(L.val), epos, s));
            return CCDPP_OK;
        }));
        HIPCK(h, hipStreamSynchronize(s));
    }
    return CCDPP_OK;
}

// Delta-coded index windows (12 index bytes per lane instead of 16 where a whole
// window allows it) for copies staged in LDS with 16-bit indices whose passes
// stream the residual.  Measured on MI355X: 3% less time per outer iteration on
// large (100M ratings), where the passes are bound by HBM; 3% more on medium (10M
// ratings), whose cached streams leave the decoding exposed.
int code_windows(ccdpp* h, int part, const ccdpp_options_t* opt) {
    using namespace ccdk;
    Layout& L = h->L[part];
    const int forced = opt ? opt->index_coding[part == 0 ? 0 : 1] : 0;
    if (forced == 1 || L.gather != kGatherLds || !L.idx16 || L.npad == 0 || L.cache == kCacheAll)
        return CCDPP_OK;
    const hipStream_t s = h->stream;
    const int64_t words = (L.npad / kWin + 63) / 64;
    HIPCK(h, dalloc(h, &L.dmask, words));
    HIPCK(h, hipMemsetAsync(L.dmask, 0, (size_t)words * 8, s));
    HIPCK(h, launch_delta_windows(L.idx, L.npad, L.pad, L.dmask, s));
    std::vector<uint64_t> bits((size_t)words);
    HIPCK(h, hipMemcpyAsync(bits.data(), L.dmask, (size_t)words * 8, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));
    L.ndelta = 0;
    for (uint64_t b : bits) L.ndelta += __builtin_popcountll(b);
    return CCDPP_OK;
}

// Refresh the per-segment copies of W (user-major copy) and H (item-major copy).
int spread_factors(ccdpp* h) {
    return with_value_type(h, [&](auto z) -> int {
        using V = decltype(z);
        for (int part = 0; part < 3; ++part)
            if (h->fseg[part]) {
                // (a tiled part's rows start at row 0 of its side)
                const Layout& L = h->L[part];
                HIPCK(h, ccdk::launch_seg_spread<V>(as<V>(part == 0 ? h->W : h->H),
                                                    part == 0 ? h->m : h->n, L.seg_row, L.nseg,
                                                    h->k, as<V>(h->fseg[part]), h->stream));
            }
        return CCDPP_OK;
    });
}

// The cache policy of each copy's residual stream (float, tiled copies; the
// others always stream).  Measured on MI355X:
// - when both streams fit in the memory-side cache (10M ratings: 123 MB), cached
//   loads and stores keep them there between passes: 7% less time per outer
//   iteration than streaming;
// - when they do not (100M ratings: 1.23 GB), cached accesses are 13% slower, but
//   write-back R-hat stores on one copy make its first pass of each feature about
//   13% faster for a slower next pass over that copy (1.7% less time per outer
//   iteration on the user-major copy of large, 1.6% on its item-major one); on both copies
//   together the gains cancel, and on a split copy they are a loss.  So the item-major
//   copy takes them when it is tiled in LDS and not split, else a user-major copy
//   tiled with P == 1.
int choose_cache(ccdpp* h, const ccdpp_options_t* opt) {
    using namespace ccdk;
    const int64_t vb = h->dbl ? 8 : 4;
    int64_t stream = 0;
    for (const Layout& L : h->L) stream += L.npad * (vb + (L.idx16 ? 2 : 4));
    auto forced_of = [&](int li) { return opt ? opt->cache[li] : 0; };
    auto eligible = [&](int part) { return !h->dbl && h->L[part].gather == kGatherLds; };
    int wb = -1;  // the part that takes automatic write-back stores
    if (stream > kCachedStreamBytes && forced_of(0) < 2 && forced_of(1) < 2) {
        if (forced_of(1) == 0 && eligible(1) && h->split == 0)
            wb = 1;
        else if (forced_of(0) == 0 && eligible(0) && h->L[0].P == 1)
            wb = 0;
    }
    for (int part = 0; part < 3; ++part) {
        Layout& L = h->L[part];
        const int li = part == 0 ? 0 : 1;
        if (L.npad == 0 && part == 2) break;  // the item-major copy is not split
        int forced = forced_of(li);
        if (part == 2 && forced > 1) forced = 1;  // a split copy's hot part always streams
        h->cache_auto[li] = forced == 0;
        if (forced > 1 && !eligible(part))
            return fail(h, CCDPP_EINVAL, "cache policy %d needs a tiled float copy", forced);
        if (forced > 0) {
            L.cache = forced - 1;
        } else if (!eligible(part)) {
            L.cache = kCacheStream;
        } else if (stream <= kCachedStreamBytes) {
            L.cache = kCacheAll;
        } else {
            L.cache = part == wb ? kCacheStores : kCacheStream;
        }
    }
    return CCDPP_OK;
}

// The item-major copy: one layout, or, when the automatic choice (or
// options.split_rows) splits it, its leading items tiled (L[1]) and the others hot
// (L[2]).  lrow: relabelled item of every triplet, lcol: relabelled user.  perm1 and
// pos1 as for build_layout, over the two parts in turn (heavy entries first), with
// the light part's slots offset by off2 into the one value array of the copy.
int build_item_major(ccdpp* h, const int32_t* lrow, const int32_t* lcol, const float* val,
                     const ccdpp_options_t* opt, int32_t* perm1, int32_t* pos1, hipStream_t s,
                     const int32_t* deg) {
    using namespace ccdk;
    const int64_t m = h->m, n = h->n, N = h->nnz;
    const int32_t forced = opt ? opt->split_rows : 0;
    int64_t H = forced > 0 ? forced : 0;
    if (forced == 0) {
        RCK(build_layout(h, 1, h->L[1], n, m, lrow, lcol, val, opt, perm1, pos1, s, N, &H, deg));
        if (H == 0) return CCDPP_OK;  // built whole
    } else if (forced < 0) {
        return build_layout(h, 1, h->L[1], n, m, lrow, lcol, val, opt, perm1, pos1, s, N, nullptr,
                            deg);
    }
    // The entries of the leading H items and of the others, each in input order.
    int32_t *ih, *il;
    int64_t* d_cnt;
    Tmp tih, til, tcnt, ttmp;
    size_t tmp_bytes = 0;
    HIPCK(h, talloc(tih, &ih, N));
    HIPCK(h, talloc(til, &il, N));
    HIPCK(h, talloc(tcnt, &d_cnt, 2));
    HIPCK(h, select_range(lrow, N, 0, (int32_t)H, ih, d_cnt, s, &ttmp.p, &tmp_bytes));
    HIPCK(h, select_range(lrow, N, (int32_t)H, (int32_t)n, il, d_cnt + 1, s, &ttmp.p, &tmp_bytes));
    int64_t cnt[2] = {0, 0};
    HIPCK(h, hipMemcpyAsync(cnt, d_cnt, sizeof cnt, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));
    const int64_t nh = cnt[0], nl = cnt[1];
    if (nh + nl != N) return fail(h, CCDPP_EDEVICE, "internal: the split does not cover nnz");
    if (nh == 0 || nl == 0) {  // one part would be empty: no split
        ccdpp_options_t o1{};
        if (opt) o1 = *opt;
        o1.split_rows = -1;
        return build_layout(h, 1, h->L[1], n, m, lrow, lcol, val, &o1, perm1, pos1, s, N, nullptr,
                            deg);
    }
    int32_t *rh, *ch, *rl, *cl, *ph, *qh, *pl, *ql;
    float *vh, *vl;
    Tmp trh, tch, tvh, trl, tcl, tvl, tph, tqh, tpl, tql;
    HIPCK(h, talloc(trh, &rh, nh));
    HIPCK(h, talloc(tch, &ch, nh));
    HIPCK(h, talloc(tvh, &vh, nh));
    HIPCK(h, talloc(trl, &rl, nl));
    HIPCK(h, talloc(tcl, &cl, nl));
    HIPCK(h, talloc(tvl, &vl, nl));
    HIPCK(h, talloc(tph, &ph, nh));
    HIPCK(h, talloc(tqh, &qh, nh));
    HIPCK(h, talloc(tpl, &pl, nl));
    HIPCK(h, talloc(tql, &ql, nl));
    HIPCK(h, launch_map(ih, lrow, nh, rh, s));
    HIPCK(h, launch_map(ih, lcol, nh, ch, s));
    HIPCK(h, (launch_copy_mapped<float, float>(val, ih, vh, nullptr, nh, s)));
    HIPCK(h, launch_map(il, lrow, nl, rl, s));
    HIPCK(h, launch_add(rl, nl, -(int32_t)H, s));  // the light part's own row ids
    HIPCK(h, launch_map(il, lcol, nl, cl, s));
    HIPCK(h, (launch_copy_mapped<float, float>(val, il, vl, nullptr, nl, s)));
    ccdpp_options_t oh{}, ol{};
    if (opt) oh = ol = *opt;
    oh.gather_mode[1] = kGatherLds;
    ol.gather_mode[1] = kGatherHot;
    ol.tile_width[1] = 0;
    RCK(build_layout(h, 1, h->L[1], H, m, rh, ch, vh, &oh, ph, qh, s, nh, nullptr, deg));
    RCK(build_layout(h, 1, h->L[2], n - H, m, rl, cl, vl, &ol, pl, ql, s, nl, nullptr, deg + H));
    const int64_t off2 = h->L[1].npad + kEntryPad;
    if (off2 + h->L[2].npad + kEntryPad > (int64_t)INT32_MAX)
        return fail(h, CCDPP_EINVAL, "the split item-major copy exceeds 2^31 value slots");
    // Triplet index of every entry, heavy part first; slots in the one value array.
    HIPCK(h, launch_map(ph, ih, nh, perm1, s));
    HIPCK(h, launch_map(pl, il, nl, perm1 + nh, s));
    HIPCK(h, hipMemcpyAsync(pos1, qh, (size_t)nh * 4, hipMemcpyDeviceToDevice, s));
    HIPCK(h, hipMemcpyAsync(pos1 + nh, ql, (size_t)nl * 4, hipMemcpyDeviceToDevice, s));
    HIPCK(h, launch_add(pos1 + nh, nl, (int32_t)off2, s));
    const size_t vb = h->dbl ? 8 : 4;
    void* both;
    HIPCK(h, dalloc(h, reinterpret_cast<char**>(&both), (int64_t)((off2 + h->L[2].npad + kEntryPad) * vb)));
    HIPCK(h, hipMemcpyAsync(both, h->L[1].val, (size_t)off2 * vb, hipMemcpyDeviceToDevice, s));
    HIPCK(h, hipMemcpyAsync(static_cast<char*>(both) + off2 * vb, h->L[2].val,
                            (size_t)(h->L[2].npad + kEntryPad) * vb, hipMemcpyDeviceToDevice, s));
    HIPCK(h, hipStreamSynchronize(s));
    dfree(h, h->L[1].val);
    dfree(h, h->L[2].val);
    h->L[1].val = both;
    h->L[2].val = static_cast<char*>(both) + off2 * vb;
    h->split = H;
    h->off2 = off2;
    return CCDPP_OK;
}

int create_device(ccdpp* h, const int32_t* row, const int32_t* col, const float* val,
                  uint64_t seed, const ccdpp_options_t* opt) {
    using namespace ccdk;
    const auto t0 = std::chrono::steady_clock::now();
    auto tprev = t0;
    auto phase = [&](int i) {
        const auto t = std::chrono::steady_clock::now();
        h->build_phase_us[i] = std::chrono::duration_cast<std::chrono::microseconds>(t - tprev).count();
        tprev = t;
    };
    const int64_t m = h->m, n = h->n, N = h->nnz;
    HIPCK(h, hipGetDevice(&h->device));
    hipDeviceProp_t prop;
    HIPCK(h, hipGetDeviceProperties(&prop, h->device));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(h, CCDPP_EDEVICE, "device %d is %s; this library is built for gfx950",
                    h->device, prop.gcnArchName);
    if (prop.sharedMemPerBlock < (size_t)kLdsBytes)
        return fail(h, CCDPP_EDEVICE, "device offers %zu bytes of LDS per workgroup, need %d",
                    prop.sharedMemPerBlock, kLdsBytes);
    h->cus = prop.multiProcessorCount;
    HIPCK(h, sweep_init());
    // The device address of the allocation-free entry point's scratch, looked up once
    // per device with that device current (host code never uses the array's name).
    if (h->device < 0 || h->device >= kMaxDevices)
        return fail(h, CCDPP_EDEVICE, "device %d: the library serves devices 0..%d", h->device,
                    kMaxDevices - 1);
    {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        if (!g_scratch_dev[h->device]) {
            void* p = nullptr;
            HIPCK(h, hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
            g_scratch_dev[h->device] = static_cast<double*>(p);
        }
        h->scratch = g_scratch_dev[h->device];
    }
    hipStream_t s = h->stream;
    phase(6);

    // Inputs and degrees.
    int32_t *d_row, *d_col, *d_cnt_r, *d_cnt_c;
    float* d_val;
    Tmp t_row, t_col, t_val, t_cr, t_cc;
    HIPCK(h, talloc(t_row, &d_row, N));
    HIPCK(h, talloc(t_col, &d_col, N));
    HIPCK(h, talloc(t_val, &d_val, N));
    HIPCK(h, talloc(t_cr, &d_cnt_r, m));
    HIPCK(h, talloc(t_cc, &d_cnt_c, n));
    Stager stage(s);
    HIPCK(h, stage.copy(d_row, row, (size_t)N * 4));
    HIPCK(h, stage.copy(d_col, col, (size_t)N * 4));
    HIPCK(h, stage.copy(d_val, val, (size_t)N * 4));
    HIPCK(h, hipMemsetAsync(d_cnt_r, 0, m * 4, s));
    HIPCK(h, hipMemsetAsync(d_cnt_c, 0, n * 4, s));
    HIPCK(h, launch_histogram(d_row, N, (int32_t)m, d_cnt_r, h->cus, s));
    HIPCK(h, launch_histogram(d_col, N, (int32_t)n, d_cnt_c, h->cus, s));
    std::vector<int32_t> cnt_r(m), cnt_c(n);
    HIPCK(h, hipMemcpyAsync(cnt_r.data(), d_cnt_r, m * 4, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipMemcpyAsync(cnt_c.data(), d_cnt_c, n * 4, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));
    // The layout places entries by these counts; they must cover every entry once.
    if (std::accumulate(cnt_r.begin(), cnt_r.end(), int64_t(0)) != N ||
        std::accumulate(cnt_c.begin(), cnt_c.end(), int64_t(0)) != N)
        return fail(h, CCDPP_EDEVICE, "degree counts do not add up to nnz");
    phase(0);

    // Relabel users and items by decreasing degree.
    std::vector<int32_t> rn2o, ro2n, cn2o, co2n;
    relabel(cnt_r, rn2o, ro2n);
    relabel(cnt_c, cn2o, co2n);
    RCK(upload(h, &h->rnew2old, rn2o));
    RCK(upload(h, &h->rold2new, ro2n));
    RCK(upload(h, &h->cnew2old, cn2o));
    RCK(upload(h, &h->cold2new, co2n));
    int32_t *d_ru, *d_ci;
    Tmp t_ru, t_ci;
    HIPCK(h, talloc(t_ru, &d_ru, N));
    HIPCK(h, talloc(t_ci, &d_ci, N));
    HIPCK(h, launch_map(d_row, h->rold2new, N, d_ru, s));
    HIPCK(h, launch_map(d_col, h->cold2new, N, d_ci, s));
    HIPCK(h, hipStreamSynchronize(s));
    phase(1);

    // The two copies, the ratings in user-major order and the map between copies.
    HIPCK(h, dalloc(h, &h->perm0, N));
    HIPCK(h, dalloc(h, &h->pos0, N));
    // Row lengths in relabelled order (rows are relabelled by decreasing length).
    std::vector<int32_t> deg_u((size_t)m), deg_i((size_t)n);
    for (int64_t r = 0; r < m; ++r) deg_u[r] = cnt_r[rn2o[r]];
    for (int64_t r = 0; r < n; ++r) deg_i[r] = cnt_c[cn2o[r]];
    RCK(build_layout(h, 0, h->L[0], m, n, d_ru, d_ci, d_val, opt, h->perm0, h->pos0, s, N, nullptr,
                     deg_u.data()));
    phase(2);
    {
        int32_t *perm1, *pos1, *inv1, *e01;
        Tmp tp1, tq1, tinv, te;
        HIPCK(h, talloc(tp1, &perm1, N));
        HIPCK(h, talloc(tq1, &pos1, N));
        RCK(build_item_major(h, d_ci, d_ru, d_val, opt, perm1, pos1, s, deg_i.data()));
        HIPCK(h, talloc(tinv, &inv1, N));
        HIPCK(h, launch_invert(perm1, N, inv1, s));
        HIPCK(h, talloc(te, &e01, N));
        HIPCK(h, launch_compose(inv1, h->perm0, N, e01, s));  // item-major entry index
        HIPCK(h, dalloc(h, &h->map01, N));
        HIPCK(h, launch_compose(pos1, e01, N, h->map01, s));
        HIPCK(h, hipStreamSynchronize(s));
    }
    phase(3);
    RCK(choose_cache(h, opt));
    for (int part = 0; part < 3; ++part) RCK(code_windows(h, part, opt));
    h->sse_nparts = std::max<int32_t>((h->L[0].grid + h->L[1].grid + h->L[2].grid) * kWaves,
                                      kReduceParts);
    HIPCK(h, dalloc(h, &h->sse_part, h->sse_nparts));
    HIPCK(h, dalloc(h, &h->d_scalar, 1));
    HIPCK(h, dalloc(h, &h->d_count, 1));
    HIPCK(h, hipStreamSynchronize(s));
    phase(4);
    for (int part = 0; part < 3; ++part)  // partials are written before they are read: start them as NaN
        if (h->L[part].part)
            HIPCK(h, launch_fill<float>(static_cast<float*>(h->L[part].part), __builtin_nanf(""),
                                        (h->dbl ? 4 : 2) * h->L[part].nslots, s));
    RCK(with_value_type(h, [&](auto z) -> int {
        using V = decltype(z);
        V *A, *W, *H, *u, *v;
        HIPCK(h, dalloc(h, &A, N));
        HIPCK(h, (launch_copy_mapped<V, V>(as<V>(h->L[0].val), h->pos0, A, nullptr, N, s)));
        // Factors: W = 0 (Algorithm 3), H from the seed; scratch.
        HIPCK(h, dalloc(h, &W, (int64_t)h->k * m));
        HIPCK(h, dalloc(h, &H, (int64_t)h->k * n));
        HIPCK(h, dalloc(h, &u, m));
        HIPCK(h, dalloc(h, &v, n));
        h->A = A;
        h->W = W;
        h->H = H;
        h->u = u;
        h->v = v;
        HIPCK(h, launch_fill<V>(W, V(0), (int64_t)h->k * m, s));
        HIPCK(h, launch_fill<V>(u, V(0), m, s));
        HIPCK(h, launch_fill<V>(v, V(0), n, s));
        for (int part = 0; part < 3; ++part)
            if (h->L[part].P > 1) {
                V* f;
                HIPCK(h, dalloc(h, &f, (int64_t)h->k * h->L[part].nseg));
                h->fseg[part] = f;
            }
        HIPCK(h, (launch_initial_h<V>(seed, h->cnew2old, n, h->k, H, s)));
        RCK(spread_factors(h));
        HIPCK(h, hipStreamSynchronize(s));
        return CCDPP_OK;
    }));
    h->pending = -1;
    phase(5);
    h->build_us = std::chrono::duration_cast<std::chrono::microseconds>(
                      std::chrono::steady_clock::now() - t0)
                      .count();
    return CCDPP_OK;
}

void destroy_all(ccdpp* h) {
    for (auto& a : h->allocs) (void)hipFree(a.first);
    h->allocs.clear();
    for (auto& pe : h->prof_pending) {
        h->event_pool.push_back(pe.a);
        h->event_pool.push_back(pe.b);
    }
    for (hipEvent_t e : h->event_pool) (void)hipEventDestroy(e);
}

// ---- kernel timing ---------------------------------------------------------------
hipEvent_t take_event(ccdpp* h) {
    if (!h->event_pool.empty()) {
        hipEvent_t e = h->event_pool.back();
        h->event_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

struct Timed {
    ccdpp* h;
    int kind;
    int layout;
    double bytes;
    hipEvent_t a = nullptr;
    Timed(ccdpp* h_, int kind_, int layout_, double bytes_)
        : h(h_), kind(kind_), layout(layout_), bytes(bytes_) {
        if (h->prof && (h->prof_kind < 0 || h->prof_kind == kind) &&
            (h->prof_layout < 0 || h->prof_layout == layout) &&
            h->prof_seen++ % h->prof_every == 0) {
            a = take_event(h);
            if (a) (void)hipEventRecord(a, h->stream);
        }
    }
    void done() {
        if (a) {
            hipEvent_t b = take_event(h);
            if (b) {
                (void)hipEventRecord(b, h->stream);
                h->prof_pending.push_back(ProfEvent{kind, layout, a, b, bytes});
            } else {
                h->event_pool.push_back(a);
            }
        }
    }
};

void collect_profile(ccdpp* h) {
    for (auto& pe : h->prof_pending) {
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, pe.a, pe.b) == hipSuccess) {
            h->prof_launch[pe.kind][pe.layout] += 1;
            h->prof_ms[pe.kind][pe.layout] += ms;
            h->prof_bytes[pe.kind][pe.layout] += pe.bytes;
        }
        h->event_pool.push_back(pe.a);
        h->event_pool.push_back(pe.b);
    }
    h->prof_pending.clear();
}

// Algorithmic bytes of one pass over layout L (see ccdpp_profile_read): index and
// value arrays, residual write-back, per-segment row scalars, outputs, and every
// gathered vector read once.  Delta-coded windows hold 1.5 index bytes per entry
// instead of 2 (counted in proportion to the windows coded).
double pass_bytes(const Layout& L, ccdk::PassMode mode, int gathered_vectors, double vb) {
    using namespace ccdk;
    const double nnz = (double)L.nnz, S = (double)L.nseg, cols = (double)L.cols;
    const double nwin = (double)(L.npad / kWin);
    const double coded = nwin > 0 ? (double)L.ndelta / nwin : 0.0;
    double b = (L.idx16 ? 2.0 - 0.5 * coded : 4.0) * nnz + vb * nnz;
    if (mode != kModePlain) b += vb * nnz;
    if (mode != kModeFlush) b += L.P == 1 ? vb * S : 2.0 * vb * S;  // coordinate or partial
    if (mode == kModeAdd || mode == kModeSubAdd) b += vb * S;
    if (mode == kModeSubAdd || mode == kModeFlush) b += vb * S;
    b += vb * cols * gathered_vectors;
    return b;
}

// Own factor column t of layout part `part` as the pass reads it: by segment, which
// with P == 1 is the column itself (from the part's first row on).
template <class V>
V* seg_col(ccdpp* h, int part, int32_t t) {
    const Layout& L = h->L[part];
    if (t < 0) return nullptr;
    if (L.P == 1)
        return as<V>(part == 0 ? h->W : h->H) + (int64_t)t * (part == 0 ? h->m : h->n) +
               (part == 2 ? h->split : 0);
    return as<V>(h->fseg[part]) + (int64_t)t * L.nseg;
}

// One pass over residual copy li (both parts of a split item-major copy, one after
// the other), then the combine of the parts that need it, which also refreshes the
// per-segment copy of column `commit` when the pass produces a committed column.
template <class V>
int pass(ccdpp* h, int li, ccdk::PassMode mode, const V* x, int32_t pcol, int32_t ppcol,
         const V* q, const V* qq, V* y, int32_t commit, int gathered) {
    const int parts[2] = {li, 2};
    const int nparts = li == 1 && h->split > 0 ? 2 : 1;
    const int kind = mode == ccdk::kModePlain ? CCDPP_K_PASS
                     : mode == ccdk::kModeFlush ? CCDPP_K_FLUSH
                                                : CCDPP_K_PASS_FUSED;
    const double vb = sizeof(V);
    if (injected(g_inject_launch))
        return fail(h, CCDPP_EDEVICE, "sweep launch failed (forced by ccdpp_debug_inject)");
    double bytes = 0.0, cbytes = 0.0;
    bool combine = false;
    for (int i = 0; i < nparts; ++i) {
        const Layout& L = h->L[parts[i]];
        bytes += pass_bytes(L, mode, gathered, vb);
        if (mode != ccdk::kModeFlush && L.ncomb > 0) {
            // Partial slots read (two values) and listed (4 B), per row a list bound, an id
            // and y; with a committed column the segment list and the per-segment copy.
            const bool yseg = commit >= 0 && L.P > 1;
            cbytes += (2.0 * vb + 4.0) * L.nsrc + (8.0 + vb) * L.ncomb +
                      (yseg ? (4.0 + vb) * L.nseg : 0.0);
            combine = true;
        }
    }
    {
        Timed tm(h, kind, li, bytes);
        for (int i = 0; i < nparts; ++i) {
            const int part = parts[i];
            const Layout& L = h->L[part];
            // Automatic write-back stores pay off only where a plain pass follows the first
            // pass over the copy (CCD++ with inner_iters >= 2); elsewhere the copy streams.
            Layout Ls;
            const Layout* Lp = &L;
            if (L.cache == ccdk::kCacheStores && h->cache_auto[li] && !h->wb_stores) {
                Ls = L;
                Ls.cache = ccdk::kCacheStream;
                Lp = &Ls;
            }
            const int64_t r0 = part == 2 ? h->split : 0;
            // The flush's per-wave sums of squares: the parts' waves in turn.
            double* sse = h->sse_part + (part == 2 ? (int64_t)h->L[1].grid * ccdk::kWaves : 0);
            HIPCK(h, ccdk::launch_pass<V>(*Lp, mode, x, seg_col<V>(h, part, pcol),
                                          seg_col<V>(h, part, ppcol), q, qq, y ? y + r0 : nullptr,
                                          h->lambda, sse, h->stream));
        }
        tm.done();
    }
    if (combine) {
        Timed tc(h, CCDPP_K_COMBINE, li, cbytes);
        for (int i = 0; i < nparts; ++i) {
            const int part = parts[i];
            const Layout& L = h->L[part];
            if (L.ncomb == 0) continue;
            V* yseg = commit >= 0 && L.P > 1 ? seg_col<V>(h, part, commit) : nullptr;
            HIPCK(h, ccdk::launch_combine<V>(L, y + (part == 2 ? h->split : 0), yseg, h->lambda,
                                             h->stream));
        }
        tc.done();
    }
    return CCDPP_OK;
}

int create_impl(int64_t m, int64_t n, int32_t k, double lambda, int64_t nnz, const int32_t* row,
                const int32_t* col, const float* val, uint64_t seed, const ccdpp_options_t* opts,
                ccdpp_t** out) {
    g_create_error.clear();
    if (!out) return fail(nullptr, CCDPP_EINVAL, "out is NULL");
    if (m < 1 || m >= kMaxDim || n < 1 || n >= kMaxDim)
        return fail(nullptr, CCDPP_EINVAL, "m and n must be in [1, 2^28)");
    if (k < 1) return fail(nullptr, CCDPP_EINVAL, "k must be >= 1");
    if (!std::isfinite(lambda) || lambda < 0.0)
        return fail(nullptr, CCDPP_EINVAL, "lambda must be finite and >= 0");
    if (nnz < 0 || nnz > kMaxNnz) return fail(nullptr, CCDPP_EINVAL, "nnz must be in [0, 2^31-1]");
    if (nnz > 0 && (!row || !col || !val))
        return fail(nullptr, CCDPP_EINVAL, "row, col and val must be non-NULL when nnz > 0");
    if (opts) {
        for (int i = 0; i < 2; ++i) {
            if (opts->gather_mode[i] < 0 || opts->gather_mode[i] > 3)
                return fail(nullptr, CCDPP_EINVAL, "gather_mode must be 0, 1, 2 or 3");
            if (opts->tile_width[i] < 0) return fail(nullptr, CCDPP_EINVAL, "tile_width < 0");
            if (opts->gather_mode[i] == ccdk::kGatherHot && opts->tile_width[i] % 32 != 0)
                return fail(nullptr, CCDPP_EINVAL, "a hot tile_width must be a multiple of 32");
            if (opts->cache[i] < 0 || opts->cache[i] > 3)
                return fail(nullptr, CCDPP_EINVAL, "cache must be 0, 1, 2 or 3");
            if (opts->index_coding[i] < 0 || opts->index_coding[i] > 1)
                return fail(nullptr, CCDPP_EINVAL, "index_coding must be 0 or 1");
        }
        if (opts->workgroups < 0) return fail(nullptr, CCDPP_EINVAL, "workgroups < 0");
        if (opts->seg_weight < -1) return fail(nullptr, CCDPP_EINVAL, "seg_weight < -1");
        if (opts->precision != 0 && opts->precision != 1)
            return fail(nullptr, CCDPP_EINVAL, "precision must be 0 (float) or 1 (double)");
        if (opts->split_rows < -1 || (opts->split_rows > 0 && opts->split_rows >= n))
            return fail(nullptr, CCDPP_EINVAL, "split_rows must be -1, 0 or in [1, n)");
        if (opts->split_rows > 0 && opts->gather_mode[1] != 0)
            return fail(nullptr, CCDPP_EINVAL, "split_rows needs gather_mode[1] = 0");
    }
    // The first bad triplet, searched by a few host threads over contiguous ranges.
    const int workers = ccdk::host_workers();
    std::vector<int64_t> first_bad(workers, nnz);
    ccdk::parallel_ranges(nnz, workers, [&](int w, int64_t lo, int64_t hi) {
        for (int64_t e = lo; e < hi; ++e) {
            if (row[e] < 0 || row[e] >= m || col[e] < 0 || col[e] >= n || !std::isfinite(val[e])) {
                first_bad[w] = e;
                return;
            }
        }
    });
    const int64_t e = *std::min_element(first_bad.begin(), first_bad.end());
    if (e < nnz) {
        if (row[e] < 0 || row[e] >= m)
            return fail(nullptr, CCDPP_EINVAL, "row[%lld] = %d out of range", (long long)e, row[e]);
        if (col[e] < 0 || col[e] >= n)
            return fail(nullptr, CCDPP_EINVAL, "col[%lld] = %d out of range", (long long)e, col[e]);
        return fail(nullptr, CCDPP_EINVAL, "val[%lld] is not finite", (long long)e);
    }
    ccdpp* h = new (std::nothrow) ccdpp();
    if (!h) return fail(nullptr, CCDPP_ENOMEM, "host allocation failed");
    h->m = m;
    h->n = n;
    h->k = k;
    h->lambda = lambda;
    h->nnz = nnz;
    h->dbl = opts && opts->precision == 1;
    int rc = create_device(h, row, col, val, seed, opts);
    if (rc != CCDPP_OK) {
        g_create_error = h->err;
        destroy_all(h);
        delete h;
        return rc;
    }
    *out = h;
    return CCDPP_OK;
}

}  // namespace

namespace {
// Fixed-order device sums into h->sse_part (kReduceParts parts) for the value type.
int launch_sq_sum_any(ccdpp* h, void* p, int64_t n) {
    return with_value_type(h, [&](auto z) -> int {
        using V = decltype(z);
        HIPCK(h, ccdk::launch_sq_sum<V>(as<V>(p), n, h->sse_part, kReduceParts, h->stream));
        return CCDPP_OK;
    });
}
int launch_test_err_any(ccdpp* h, const int32_t* dr, const int32_t* dc, const float* dv,
                        int64_t nnz, double* part = nullptr, double* rejected = nullptr) {
    return with_value_type(h, [&](auto z) -> int {
        using V = decltype(z);
        HIPCK(h, ccdk::launch_test_err<V>(dr, dc, dv, nnz, h->rold2new, h->cold2new, as<V>(h->W),
                                          as<V>(h->H), h->m, h->n, h->k,
                                          part ? part : h->sse_part, kReduceParts, rejected,
                                          h->stream));
        return CCDPP_OK;
    });
}

// Algorithm 2 (element-wise CCD): per outer iteration, every row's k coordinates
// in order (eq. 5, then the residual update of eq. 6-7), then every column's (eq.
// 8, eq. 9-10).  Rows are independent within the W phase, so the row loop and the
// feature loop are exchanged: pass t over the user-major copy computes w_.t for
// every row from R-hat = R + w_.t h_.t (the same pass as CCD++'s first u-pass), and
// the residual update of feature t is folded, as a pending subtract, into pass
// t + 1 (and a final flush).  The H phase does the same on the item-major copy.
// After each phase the other copy is refreshed from the updated one through the
// entry maps, so both copies hold the same residual again.
template <class V>
int ccd_impl(ccdpp* h, int32_t outer) {
    using namespace ccdk;
    const int64_t m = h->m, n = h->n;
    h->wb_stores = false;
    if (outer > 0 && !h->slot01) {
        // Slot-to-slot maps between the copies, for the residual refresh after each phase.
        // Both maps are allocated before the handle keeps either, so a failed
        // allocation leaves the handle as it was.
        int32_t *s01, *s10;
        Tmp t01, t10;
        HIPCK(h, talloc(t01, &s01, h->L[0].npad));
        HIPCK(h, talloc(t10, &s10, item_slots(h)));
        for (Tmp* t : {&t01, &t10}) {
            h->allocs.emplace_back(t->p, 4 * (t == &t01 ? h->L[0].npad : item_slots(h)));
            t->p = nullptr;
        }
        h->bytes_held += 4 * (h->L[0].npad + item_slots(h));
        HIPCK(h, hipMemsetAsync(s01, 0xFF, (size_t)h->L[0].npad * 4, h->stream));
        HIPCK(h, hipMemsetAsync(s10, 0xFF, (size_t)item_slots(h) * 4, h->stream));
        HIPCK(h, launch_slot_map(h->pos0, h->map01, h->nnz, s01, h->stream));
        HIPCK(h, launch_slot_map(h->map01, h->pos0, h->nnz, s10, h->stream));
        h->slot01 = s01;
        h->slot10 = s10;
    }
    for (int32_t it = 0; it < outer; ++it) {
        for (int li = 0; li < 2; ++li) {
            V* own = as<V>(li == 0 ? h->W : h->H);
            V* other = as<V>(li == 0 ? h->H : h->W);
            const int64_t rows = li == 0 ? m : n, cols = li == 0 ? n : m;
            for (int32_t t = 0; t < h->k; ++t) {
                V* ot = other + (int64_t)t * cols;
                const V* op = t > 0 ? other + (int64_t)(t - 1) * cols : nullptr;
                // R-hat = R + own_t other_t (minus the pending feature t - 1), own_t from
                // eq. 5 / eq. 8 written in place: a segment's old own_t is read before the
                // segment's new value is written, and a row cut between chunks is written
                // only after every chunk (by the workgroup at the end, or by the combine,
                // which for a tiled copy also writes own_t per segment).
                RCK(pass<V>(h, li, t > 0 ? kModeSubAdd : kModeAdd, ot, t, t - 1, ot, op,
                            own + (int64_t)t * rows, t, t > 0 ? 2 : 1));
            }
            // The pending update of feature k - 1, and for the item-major copy the
            // training sum of squares.
            RCK(pass<V>(h, li, kModeFlush, nullptr, -1, h->k - 1, nullptr,
                        other + (int64_t)(h->k - 1) * cols, nullptr, -1, 1));
            if (li == 1)
                HIPCK(h, launch_reduce_sum(h->sse_part, (h->L[1].grid + h->L[2].grid) * kWaves,
                                           h->d_scalar, h->stream));
            if (li == 0)
                HIPCK(h, (launch_copy_slots<V>(as<V>(h->L[0].val), h->slot01, as<V>(h->L[1].val),
                                               h->L[0].npad, h->stream)));
            else
                HIPCK(h, (launch_copy_slots<V>(as<V>(h->L[1].val), h->slot10, as<V>(h->L[0].val),
                                               item_slots(h), h->stream)));
        }
    }
    if (outer > 0) {
        double sse = 0.0;
        HIPCK(h, hipMemcpyAsync(&sse, h->d_scalar, 8, hipMemcpyDeviceToHost, h->stream));
        HIPCK(h, hipStreamSynchronize(h->stream));
        h->train_sse = h->L[1].grid + h->L[2].grid ? sse : 0.0;
        h->train_sse_valid = true;
    }
    HIPCK(h, hipStreamSynchronize(h->stream));
    if (h->prof) collect_profile(h);
    return CCDPP_OK;
}

template <class V>
int run_impl(ccdpp* h, int32_t outer, int32_t inner) {
    using namespace ccdk;
    const int64_t m = h->m, n = h->n;
    h->wb_stores = inner >= 2;
    V* const W = as<V>(h->W);
    V* const H = as<V>(h->H);
    V* const u = as<V>(h->u);
    V* const v = as<V>(h->v);
    for (int32_t it = 0; it < outer; ++it) {
        for (int32_t t = 0; t < h->k; ++t) {
            V* Wt = W + (int64_t)t * m;
            V* Ht = H + (int64_t)t * n;
            const bool prev = h->pending >= 0;
            const V* Wp = prev ? W + (int64_t)h->pending * m : nullptr;
            const V* Hp = prev ? H + (int64_t)h->pending * n : nullptr;
            const PassMode first = prev ? kModeSubAdd : kModeAdd;
            const int32_t pend = prev ? h->pending : -1;
            const int g1 = prev ? 2 : 1;
            const int32_t c1 = inner == 1 ? t : -1;  // with one inner pass, u and v are committed
            // First u-pass: eq. 18 of the pending feature, eq. 13, eq. 15 with v = hbar_t.
            RCK(pass<V>(h, 0, first, Ht, t, pend, Ht, Hp, u, c1, g1));
            // First v-pass: the same residual update on the item-major copy, eq. 16 with the new u.
            V* yv = inner == 1 ? Ht : v;
            RCK(pass<V>(h, 1, first, u, t, pend, Wt, Wp, yv, c1, g1 + 1));
            for (int32_t s = 2; s <= inner; ++s) {
                const bool last = s == inner;
                V* yu = last ? Wt : u;  // the last u is committed in place (eq. 17)
                RCK(pass<V>(h, 0, kModePlain, v, -1, -1, nullptr, nullptr, yu, last ? t : -1, 1));
                RCK(pass<V>(h, 1, kModePlain, yu, -1, -1, nullptr, nullptr, last ? Ht : v,
                            last ? t : -1, 1));
            }
            if (inner == 1) {
                Timed tm(h, CCDPP_K_COMMIT, 0, 2.0 * sizeof(V) * m);
                HIPCK(h, launch_copy<V>(u, Wt, m, h->stream));
                tm.done();
            }
            h->pending = t;
        }
    }
    // The last feature's eq. 18 stays pending: the next call's first passes apply it
    // (as between features), and flush_pending does when the residual is read.
    if (outer > 0 && h->pending >= 0) h->train_sse_valid = false;
    HIPCK(h, hipStreamSynchronize(h->stream));
    if (h->prof) collect_profile(h);
    return CCDPP_OK;
}

// The pending eq. 18 on both copies; the user-major flush also sums R^2 for the
// training RMSE.
template <class V>
int flush_impl(ccdpp* h) {
    using namespace ccdk;
    const V* Wp = as<V>(h->W) + (int64_t)h->pending * h->m;
    const V* Hp = as<V>(h->H) + (int64_t)h->pending * h->n;
    RCK(pass<V>(h, 0, kModeFlush, nullptr, -1, h->pending, nullptr, Hp, nullptr, -1, 1));
    HIPCK(h, launch_reduce_sum(h->sse_part, h->L[0].grid * kWaves, h->d_scalar, h->stream));
    RCK(pass<V>(h, 1, kModeFlush, nullptr, -1, h->pending, nullptr, Wp, nullptr, -1, 1));
    h->pending = -1;
    double sse = 0.0;
    HIPCK(h, hipMemcpyAsync(&sse, h->d_scalar, 8, hipMemcpyDeviceToHost, h->stream));
    HIPCK(h, hipStreamSynchronize(h->stream));
    h->train_sse = h->L[0].grid ? sse : 0.0;
    h->train_sse_valid = true;
    if (h->prof) collect_profile(h);
    return CCDPP_OK;
}

// Brings the residual up to date before anything reads it.
int flush_pending(ccdpp* h) {
    if (h->pending < 0) return CCDPP_OK;
    return h->dbl ? flush_impl<double>(h) : flush_impl<float>(h);
}

template <class S>
int get_factors_impl(ccdpp* h, S* W, S* H) {
    if (!usable(h)) return CCDPP_ESTATE;
    hipStream_t s = h->stream;
    // Both staging buffers first, so that an error leaves W and H untouched.
    S *dW = nullptr, *dH = nullptr;
    Tmp tw, th;
    if (W) HIPCK(h, talloc(tw, &dW, h->m * h->k));
    if (H) HIPCK(h, talloc(th, &dH, h->n * h->k));
    RCK(with_value_type(h, [&](auto z) -> int {
        using V = decltype(z);
        if (W) HIPCK(h, (ccdk::launch_gather_factor_out<V, S>(as<V>(h->W), h->rold2new, h->m, h->k, dW, s)));
        if (H) HIPCK(h, (ccdk::launch_gather_factor_out<V, S>(as<V>(h->H), h->cold2new, h->n, h->k, dH, s)));
        HIPCK(h, hipStreamSynchronize(s));
        return CCDPP_OK;
    }));
    if (W) HIPCK(h, hipMemcpyAsync(W, dW, h->m * h->k * sizeof(S), hipMemcpyDeviceToHost, s));
    if (H) HIPCK(h, hipMemcpyAsync(H, dH, h->n * h->k * sizeof(S), hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));
    return CCDPP_OK;
}

template <class S>
int set_factors_impl(ccdpp* h, const S* W, const S* H) {
    if (!usable(h)) return CCDPP_ESTATE;
    if (W)
        for (int64_t e = 0; e < h->m * h->k; ++e)
            if (!std::isfinite(W[e]))
                return fail(h, CCDPP_EINVAL, "W[%lld] is not finite", (long long)e);
    if (H)
        for (int64_t e = 0; e < h->n * h->k; ++e)
            if (!std::isfinite(H[e]))
                return fail(h, CCDPP_EINVAL, "H[%lld] is not finite", (long long)e);
    hipStream_t s = h->stream;
    // Staging buffers first: a failed allocation leaves the factors and the residual
    // as they were.
    S *dW = nullptr, *dH = nullptr;
    Tmp tw, th;
    if (W) HIPCK(h, talloc(tw, &dW, h->m * h->k));
    if (H) HIPCK(h, talloc(th, &dH, h->n * h->k));
    if (W) HIPCK(h, hipMemcpyAsync(dW, W, h->m * h->k * sizeof(S), hipMemcpyHostToDevice, s));
    if (H) HIPCK(h, hipMemcpyAsync(dH, H, h->n * h->k * sizeof(S), hipMemcpyHostToDevice, s));
    RCK(with_value_type(h, [&](auto z) -> int {
        using V = decltype(z);
        if (W) HIPCK(h, (ccdk::launch_scatter_factor_in<S, V>(dW, h->rnew2old, h->m, h->k, as<V>(h->W), s)));
        if (H) HIPCK(h, (ccdk::launch_scatter_factor_in<S, V>(dH, h->cnew2old, h->n, h->k, as<V>(h->H), s)));
        RCK(spread_factors(h));
        HIPCK(h, ccdk::launch_rebuild_residual<V>(h->L[0], h->pos0, as<V>(h->A), as<V>(h->W),
                                                  as<V>(h->H), h->m, h->n, h->k, s));
        HIPCK(h, (ccdk::launch_copy_mapped<V, V>(as<V>(h->L[0].val), h->pos0, as<V>(h->L[1].val),
                                                h->map01, h->nnz, s)));
        HIPCK(h, hipStreamSynchronize(s));
        return CCDPP_OK;
    }));
    h->pending = -1;
    h->train_sse_valid = false;
    return CCDPP_OK;
}

template <class S>
int get_residual_impl(ccdpp* h, S* R) {
    if (!usable(h)) return CCDPP_ESTATE;
    if (!R && h->nnz) return fail(h, CCDPP_EINVAL, "R is NULL");
    if (h->nnz == 0) return CCDPP_OK;
    hipStream_t s = h->stream;
    S* d;
    Tmp t;
    HIPCK(h, talloc(t, &d, h->nnz));
    RCK(flush_pending(h));
    RCK(with_value_type(h, [&](auto z) -> int {
        using V = decltype(z);
        HIPCK(h, (ccdk::launch_copy_mapped<V, S>(as<V>(h->L[0].val), h->pos0, d, h->perm0, h->nnz, s)));
        return CCDPP_OK;
    }));
    HIPCK(h, hipMemcpyAsync(R, d, h->nnz * sizeof(S), hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));
    return CCDPP_OK;
}
}  // namespace

// Makes the handle's device current for one call and restores the caller's after it:
// the handle's memory, kernels and null stream all belong to that device.
struct DeviceScope {
    int prev = -1;
    bool changed = false;
    explicit DeviceScope(const ccdpp* h) {
        if (h && hipGetDevice(&prev) == hipSuccess && prev != h->device)
            changed = hipSetDevice(h->device) == hipSuccess;
    }
    ~DeviceScope() {
        if (changed) (void)hipSetDevice(prev);
    }
    DeviceScope(const DeviceScope&) = delete;
    DeviceScope& operator=(const DeviceScope&) = delete;
};

extern "C" {

int ccdpp_create(int64_t m, int64_t n, int32_t k, double lambda, int64_t nnz, const int32_t* row,
                 const int32_t* col, const float* val, uint64_t seed, ccdpp_t** out) {
    return create_impl(m, n, k, lambda, nnz, row, col, val, seed, nullptr, out);
}

int ccdpp_create_ex(int64_t m, int64_t n, int32_t k, double lambda, int64_t nnz,
                    const int32_t* row, const int32_t* col, const float* val, uint64_t seed,
                    const ccdpp_options_t* opts, ccdpp_t** out) {
    return create_impl(m, n, k, lambda, nnz, row, col, val, seed, opts, out);
}


int ccdpp_run(ccdpp_t* h, int32_t outer, int32_t inner) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    if (outer < 0 || inner < 1)
        return fail(h, CCDPP_EINVAL, "outer_iters must be >= 0 and inner_iters >= 1");
    return h->dbl ? run_impl<double>(h, outer, inner) : run_impl<float>(h, outer, inner);
}

int ccdpp_ccd_run(ccdpp_t* h, int32_t outer) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    if (outer < 0) return fail(h, CCDPP_EINVAL, "outer_iters must be >= 0");
    RCK(flush_pending(h));
    return h->dbl ? ccd_impl<double>(h, outer) : ccd_impl<float>(h, outer);
}

int ccdpp_run_until(ccdpp_t* h, int32_t max_outer, int32_t inner, double rel_tol,
                    int64_t test_nnz, const int32_t* test_row, const int32_t* test_col,
                    const float* test_val, double* history, int32_t* outer_done) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    if (!outer_done) return fail(h, CCDPP_EINVAL, "outer_done is NULL");
    if (max_outer < 0 || inner < 1)
        return fail(h, CCDPP_EINVAL, "max_outer must be >= 0 and inner_iters >= 1");
    if (std::isnan(rel_tol)) return fail(h, CCDPP_EINVAL, "rel_tol is NaN");
    if (test_nnz < 0 || test_nnz > kMaxNnz)
        return fail(h, CCDPP_EINVAL, "test_nnz must be in [0, 2^31-1]");
    if (test_nnz > 0) {
        if (!test_row || !test_col || !test_val)
            return fail(h, CCDPP_EINVAL, "test arrays must be non-NULL when test_nnz > 0");
        for (int64_t e = 0; e < test_nnz; ++e) {
            if (test_row[e] < 0 || test_row[e] >= h->m || test_col[e] < 0 || test_col[e] >= h->n)
                return fail(h, CCDPP_EINVAL, "test entry %lld out of range", (long long)e);
            if (!std::isfinite(test_val[e]))
                return fail(h, CCDPP_EINVAL, "test value %lld is not finite", (long long)e);
        }
    }
    hipStream_t s = h->stream;
    int32_t *dr = nullptr, *dc = nullptr;
    float* dv = nullptr;
    Tmp tr, tc, tv;
    if (test_nnz > 0) {
        HIPCK(h, talloc(tr, &dr, test_nnz));
        HIPCK(h, talloc(tc, &dc, test_nnz));
        HIPCK(h, talloc(tv, &dv, test_nnz));
        HIPCK(h, hipMemcpyAsync(dr, test_row, test_nnz * 4, hipMemcpyHostToDevice, s));
        HIPCK(h, hipMemcpyAsync(dc, test_col, test_nnz * 4, hipMemcpyHostToDevice, s));
        HIPCK(h, hipMemcpyAsync(dv, test_val, test_nnz * 4, hipMemcpyHostToDevice, s));
    }
    // A fixed-order float64 sum on the device, read back.
    auto reduce = [&](double* out) -> int {
        HIPCK(h, ccdk::launch_reduce_sum(h->sse_part, kReduceParts, h->d_scalar, s));
        HIPCK(h, hipMemcpyAsync(out, h->d_scalar, 8, hipMemcpyDeviceToHost, s));
        HIPCK(h, hipStreamSynchronize(s));
        return CCDPP_OK;
    };
    double prev = 0.0;
    int32_t done = 0;
    for (int32_t it = 0; it < max_outer; ++it) {
        RCK(ccdpp_run(h, 1, inner));
        RCK(flush_pending(h));  // the training sum of squares
        double w2 = 0.0, h2 = 0.0, te = std::nan("");
        RCK(launch_sq_sum_any(h, h->W, h->m * h->k));
        RCK(reduce(&w2));
        RCK(launch_sq_sum_any(h, h->H, h->n * h->k));
        RCK(reduce(&h2));
        if (test_nnz > 0) {
            RCK(launch_test_err_any(h, dr, dc, dv, test_nnz));
            double sum = 0.0;
            RCK(reduce(&sum));
            te = std::sqrt(sum / (double)test_nnz);
        }
        const double f = h->train_sse + h->lambda * (w2 + h2);
        if (history) {
            history[3 * (int64_t)it] = f;
            history[3 * (int64_t)it + 1] = h->nnz > 0 ? std::sqrt(h->train_sse / (double)h->nnz) : 0.0;
            history[3 * (int64_t)it + 2] = te;
        }
        done = it + 1;
        if (it >= 1 && rel_tol >= 0.0 && prev - f <= rel_tol * prev) break;
        prev = f;
    }
    *outer_done = done;
    return CCDPP_OK;
}


int ccdpp_get_factors(ccdpp_t* h, float* W, float* H) {
    DeviceScope dev(h);
    return get_factors_impl<float>(h, W, H);
}
int ccdpp_get_factors_f64(ccdpp_t* h, double* W, double* H) {
    DeviceScope dev(h);
    return get_factors_impl<double>(h, W, H);
}
int ccdpp_set_factors(ccdpp_t* h, const float* W, const float* H) {
    DeviceScope dev(h);
    return set_factors_impl<float>(h, W, H);
}
int ccdpp_set_factors_f64(ccdpp_t* h, const double* W, const double* H) {
    DeviceScope dev(h);
    return set_factors_impl<double>(h, W, H);
}

int ccdpp_rmse(ccdpp_t* h, int64_t nnz, const int32_t* row, const int32_t* col, const float* val,
               double* rmse_out) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    if (!rmse_out) return fail(h, CCDPP_EINVAL, "rmse_out is NULL");
    if (nnz < 1 || nnz > kMaxNnz) return fail(h, CCDPP_EINVAL, "nnz must be in [1, 2^31-1]");
    if (!row || !col || !val) return fail(h, CCDPP_EINVAL, "row, col and val must be non-NULL");
    for (int64_t e = 0; e < nnz; ++e) {
        if (row[e] < 0 || row[e] >= h->m || col[e] < 0 || col[e] >= h->n)
            return fail(h, CCDPP_EINVAL, "test entry %lld out of range", (long long)e);
        if (!std::isfinite(val[e]))
            return fail(h, CCDPP_EINVAL, "test value %lld is not finite", (long long)e);
    }
    hipStream_t s = h->stream;
    int32_t *dr, *dc;
    float* dv;
    Tmp tr, tc, tv;
    HIPCK(h, talloc(tr, &dr, nnz));
    HIPCK(h, talloc(tc, &dc, nnz));
    HIPCK(h, talloc(tv, &dv, nnz));
    HIPCK(h, hipMemcpyAsync(dr, row, nnz * 4, hipMemcpyHostToDevice, s));
    HIPCK(h, hipMemcpyAsync(dc, col, nnz * 4, hipMemcpyHostToDevice, s));
    HIPCK(h, hipMemcpyAsync(dv, val, nnz * 4, hipMemcpyHostToDevice, s));
    RCK(launch_test_err_any(h, dr, dc, dv, nnz));
    HIPCK(h, ccdk::launch_reduce_sum(h->sse_part, kReduceParts, h->d_scalar, s));
    double sum = 0.0;
    HIPCK(h, hipMemcpyAsync(&sum, h->d_scalar, 8, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));
    *rmse_out = std::sqrt(sum / (double)nnz);
    return CCDPP_OK;
}

int ccdpp_rmse_noalloc(ccdpp_t* h, int64_t nnz, const int32_t* row, const int32_t* col,
                       const float* val, double* rmse_out) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    if (!rmse_out) return fail(h, CCDPP_EINVAL, "rmse_out is NULL");
    if (nnz < 1 || nnz > kMaxNnz) return fail(h, CCDPP_EINVAL, "nnz must be in [1, 2^31-1]");
    if (!row || !col || !val) return fail(h, CCDPP_EINVAL, "row, col and val must be non-NULL");
    if (!h->scratch) return fail(h, CCDPP_ESTATE, "no scratch address on this device");
    hipStream_t s = h->stream;
    double* sc = h->scratch;
    // The same kernel as ccdpp_rmse with the triplets checked on the device (they
    // cannot be checked on the host), partials and counts in the scratch array.
    RCK(launch_test_err_any(h, row, col, val, nnz, sc + kNaPart, sc + kNaRejected));
    HIPCK(h, ccdk::launch_reduce_sum(sc + kNaPart, kReduceParts, sc + kNaTotals, s));
    HIPCK(h, ccdk::launch_reduce_sum(sc + kNaRejected, kReduceParts, sc + kNaTotals + 1, s));
    double tot[2] = {0.0, 0.0};
    HIPCK(h, hipMemcpyAsync(tot, sc + kNaTotals, sizeof tot, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));
    if (tot[1] != 0.0)
        return fail(h, CCDPP_EINVAL, "%.0f held-out entries are out of range or not finite", tot[1]);
    *rmse_out = std::sqrt(tot[0] / (double)nnz);
    return CCDPP_OK;
}

int ccdpp_train_rmse(ccdpp_t* h, double* rmse_out) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    if (!rmse_out) return fail(h, CCDPP_EINVAL, "rmse_out is NULL");
    if (h->nnz < 1) return fail(h, CCDPP_EINVAL, "no observed entries");
    RCK(flush_pending(h));
    if (!h->train_sse_valid) {
        hipStream_t s = h->stream;
        RCK(launch_sq_sum_any(h, h->L[0].val, h->L[0].npad));
        HIPCK(h, ccdk::launch_reduce_sum(h->sse_part, kReduceParts, h->d_scalar, s));
        double sum = 0.0;
        HIPCK(h, hipMemcpyAsync(&sum, h->d_scalar, 8, hipMemcpyDeviceToHost, s));
        HIPCK(h, hipStreamSynchronize(s));
        h->train_sse = sum;
        h->train_sse_valid = true;
    }
    *rmse_out = std::sqrt(h->train_sse / (double)h->nnz);
    return CCDPP_OK;
}


int ccdpp_get_residual(ccdpp_t* h, float* R) {
    DeviceScope dev(h);
    return get_residual_impl<float>(h, R);
}
int ccdpp_get_residual_f64(ccdpp_t* h, double* R) {
    DeviceScope dev(h);
    return get_residual_impl<double>(h, R);
}

int ccdpp_check_consistency(ccdpp_t* h, int64_t* mismatches) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    if (!mismatches) return fail(h, CCDPP_EINVAL, "mismatches is NULL");
    RCK(flush_pending(h));
    hipStream_t s = h->stream;
    HIPCK(h, hipMemsetAsync(h->d_count, 0, 8, s));
    RCK(with_value_type(h, [&](auto z) -> int {
        using V = decltype(z);
        HIPCK(h, ccdk::launch_consistency<V>(as<V>(h->L[0].val), h->pos0, as<V>(h->L[1].val),
                                             h->map01, h->nnz, h->d_count, s));
        return CCDPP_OK;
    }));
    unsigned long long c = 0;
    HIPCK(h, hipMemcpyAsync(&c, h->d_count, 8, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));
    *mismatches = (int64_t)c;
    return CCDPP_OK;
}

int ccdpp_set_stream(ccdpp_t* h, void* hip_stream) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    HIPCK(h, hipStreamSynchronize(h->stream));
    h->stream = static_cast<hipStream_t>(hip_stream);
    return CCDPP_OK;
}

int ccdpp_profile(ccdpp_t* h, int32_t enable) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    HIPCK(h, hipStreamSynchronize(h->stream));
    collect_profile(h);
    h->prof = enable != 0;
    for (int i = 0; i < CCDPP_K_COUNT; ++i)
        for (int l = 0; l < 2; ++l) {
            h->prof_launch[i][l] = 0;
            h->prof_ms[i][l] = 0.0;
            h->prof_bytes[i][l] = 0.0;
        }
    return CCDPP_OK;
}

int ccdpp_profile_only(ccdpp_t* h, int32_t kind, int32_t layout) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    if (kind < -1 || kind >= CCDPP_K_COUNT) return fail(h, CCDPP_EINVAL, "bad kernel kind");
    if (layout < -1 || layout > 1) return fail(h, CCDPP_EINVAL, "bad layout");
    h->prof_kind = kind;
    h->prof_layout = layout;
    h->prof_seen = 0;
    return CCDPP_OK;
}

int ccdpp_profile_every(ccdpp_t* h, int32_t every) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    if (every < 1) return fail(h, CCDPP_EINVAL, "every must be >= 1");
    h->prof_every = every;
    h->prof_seen = 0;
    return CCDPP_OK;
}

int ccdpp_profile_read(ccdpp_t* h, int32_t kind, int32_t layout, int64_t* launches,
                       double* total_ms, double* algo_bytes) {
    DeviceScope dev(h);
    if (!usable(h)) return CCDPP_ESTATE;
    if (kind < 0 || kind >= CCDPP_K_COUNT) return fail(h, CCDPP_EINVAL, "bad kernel kind");
    if (layout < -1 || layout > 1) return fail(h, CCDPP_EINVAL, "bad layout");
    int64_t cnt = 0;
    double ms = 0.0, b = 0.0;
    for (int l = 0; l < 2; ++l)
        if (layout < 0 || layout == l) {
            cnt += h->prof_launch[kind][l];
            ms += h->prof_ms[kind][l];
            b += h->prof_bytes[kind][l];
        }
    if (launches) *launches = cnt;
    if (total_ms) *total_ms = ms;
    if (algo_bytes) *algo_bytes = b;
    return CCDPP_OK;
}

int ccdpp_info(ccdpp_t* h, int64_t* out, int32_t len) {
    if (!h) return CCDPP_ESTATE;
    if (!out || len < 0) return fail(h, CCDPP_EINVAL, "bad output buffer");
    auto width = [](const ccdk::Layout& L) -> int64_t {
        return L.gather == ccdk::kGatherHot ? L.hot : L.T;
    };
    const ccdk::Layout& L2 = h->L[2];
    const bool sp = h->split > 0;
    const int64_t v[42] = {h->m,         h->n,         h->nnz,       h->k,
                           h->build_us,  h->L[0].gather, h->L[0].P,  width(h->L[0]),
                           h->L[0].grid, h->L[0].nseg, h->L[1].gather, h->L[1].P,
                           width(h->L[1]), h->L[1].grid, h->L[1].nseg, h->bytes_held,
                           h->dbl ? 8 : 4, h->L[0].ncut, h->L[0].ncomb, h->L[1].ncut,
                           h->L[1].ncomb, h->L[0].cache + 1, h->L[1].cache + 1,
                           h->L[0].ndelta, h->L[0].npad / ccdk::kWin, h->L[1].ndelta,
                           h->L[1].npad / ccdk::kWin, h->split,
                           sp ? L2.gather : 0, sp ? width(L2) : 0, sp ? L2.grid : 0,
                           sp ? L2.nseg : 0, sp ? L2.ncut : 0, sp ? L2.ncomb : 0,
                           sp ? L2.cache + 1 : 0, h->build_phase_us[0], h->build_phase_us[1],
                           h->build_phase_us[2], h->build_phase_us[3], h->build_phase_us[4],
                           h->build_phase_us[5], h->build_phase_us[6]};
    int32_t w = std::min<int32_t>(len, 42);
    for (int32_t i = 0; i < w; ++i) out[i] = v[i];
    return w;
}

int ccdpp_debug_inject(int32_t what, int64_t after) {
    if (what == 0)
        g_inject_alloc.store(after < 0 ? -1 : after);
    else if (what == 1)
        g_inject_launch.store(after < 0 ? -1 : after);
    else
        return CCDPP_EINVAL;
    return CCDPP_OK;
}

const char* ccdpp_last_error(const ccdpp_t* h) {
    if (!h) return g_create_error.c_str();
    return h->err.c_str();
}

void ccdpp_destroy(ccdpp_t* h) {
    DeviceScope dev(h);
    if (!h) return;
    (void)hipStreamSynchronize(h->stream);
    destroy_all(h);
    delete h;
}

}  // extern "C"
