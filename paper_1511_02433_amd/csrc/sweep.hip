// CCD++ sweep passes for gfx950 (MI355X).
//
// One launch is one pass over one compressed copy of the residual:
//   - a u-pass over the user-major copy evaluates eq. 15 for every row i,
//   - a v-pass over the item-major copy evaluates eq. 16 for every column j
//     (read with u_i, the minimiser of eq. 14 in v_j),
// in the data-parallel form of Section 6 (eq. 20, 21): every row or column is
// an independent unit of work.  The first pass of a feature over each copy
// also folds in the residual bookkeeping of Algorithm 3: the pending eq. 18
// subtract of the previous feature and the eq. 13 add-back of the current one,
// evaluated as fma(p, q, fma(-pp, qq, val)).  Both copies evaluate that same
// expression on the same operands, so they stay bitwise identical.
//
// Memory: index and value arrays are streamed with non-temporal 128-bit loads
// (each entry is touched once per pass), the next window's loads in flight
// while the current window is reduced.  The vectors a pass gathers from are
// staged tile by tile in LDS by persistent workgroups (see ccdpp_internal.hpp),
// so a random gather costs an LDS read; layouts too sparse for tiling stage
// only their leading (most frequent) columns and gather the others through L2
// with bounded buffer loads, issued before the next windows' data so that
// waiting for them does not wait for that data too.
//
// Kernel variants: STAGED with 16-bit indices is a tiled layout, STAGED with
// 32-bit indices a hot layout (P == 1, the leading columns staged), !STAGED a
// layout that gathers everything from global memory.
//
// Arithmetic: R-hat in fp32 FMA.  Inside a window (at most 512 entries) the
// sums of R-hat*x and x^2 are fp32 segmented scans; a segment's window sums are
// added in fp64, across windows too, in a fixed order, so results are
// identical run to run.  A tiled copy stores each segment's sums as a partial
// of the value type (one fp32 rounding for float values), which the combine
// adds in fp64.  The coordinate num / (lambda + den) is an IEEE fp64
// division rounded once to fp32; a coordinate whose denominator is exactly zero
// (lambda = 0 and an empty row) is set to zero.
#include <algorithm>
#include <type_traits>

#include "ccdpp_internal.hpp"

namespace ccdk {
namespace {

using rsrc_t = __amdgpu_buffer_rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, gfx9 family
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef double f64x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 128 bits of the value type: four floats or two doubles.
template <class V> struct Vec16;
template <> struct Vec16<float> { using type = f32x4; };
template <> struct Vec16<double> { using type = f64x2; };

__device__ __forceinline__ float fmav(float a, float b, float c) { return __builtin_fmaf(a, b, c); }
__device__ __forceinline__ double fmav(double a, double b, double c) { return __builtin_fma(a, b, c); }

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint64_t bytes) {
    uint32_t lim = bytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)lim,
                                            kRsrcWord3);
}
// Bounded load: offsets past the descriptor's limit read 0.
__device__ __forceinline__ float ld_f32(rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ f32x4 ld_f32x4(rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
// Two 32-bit bounded loads (a 64-bit buffer load is not used, see the toolchain notes).
__device__ __forceinline__ double ld_f64(rsrc_t r, uint32_t off) {
    int2 v;
    v.x = __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
    v.y = __builtin_amdgcn_raw_buffer_load_b32(r, off + 4u, 0, 0);
    return __builtin_bit_cast(double, v);
}

// ---- cross-lane operations ---------------------------------------------------
// DPP controls of the gfx9 family.
constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
constexpr int kBcast15 = 0x142;   // lane 15 of each row to the next row
constexpr int kBcast31 = 0x143;   // lane 31 to rows 2 and 3
constexpr int kWaveShr1 = 0x138;  // lane l reads lane l - 1

// Lanes whose source is out of range, or whose row is masked off, get `old`
// (with BC, out-of-range sources read 0 instead).
template <int CTRL, int ROWS = 0xF, bool BC = false>
__device__ __forceinline__ int dpp_i(int old, int v) {
    return __builtin_amdgcn_update_dpp(old, v, CTRL, ROWS, 0xF, BC);
}
template <int CTRL, int ROWS = 0xF, bool BC = false>
__device__ __forceinline__ float dpp_f(float old, float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old),
                                                                 __builtin_bit_cast(int, v), CTRL,
                                                                 ROWS, 0xF, BC));
}

template <int CTRL, int ROWS = 0xF, bool BC = false>
__device__ __forceinline__ double dpp_d(double old, double v) {
    const int2 o = __builtin_bit_cast(int2, old), x = __builtin_bit_cast(int2, v);
    int2 r;
    r.x = __builtin_amdgcn_update_dpp(o.x, x.x, CTRL, ROWS, 0xF, BC);
    r.y = __builtin_amdgcn_update_dpp(o.y, x.y, CTRL, ROWS, 0xF, BC);
    return __builtin_bit_cast(double, r);
}
template <int CTRL, int ROWS = 0xF, bool BC = false>
__device__ __forceinline__ float dpp_v(float old, float v) { return dpp_f<CTRL, ROWS, BC>(old, v); }
template <int CTRL, int ROWS = 0xF, bool BC = false>
__device__ __forceinline__ double dpp_v(double old, double v) { return dpp_d<CTRL, ROWS, BC>(old, v); }

// 1.0 on the lanes whose bit is set in the wave-uniform mask m, else 0.0.
__device__ __forceinline__ float lane_factor(uint64_t m) {
    return __builtin_amdgcn_inverse_ballot_w64(m) ? 1.0f : 0.0f;
}

// One step of an inclusive segmented scan over lanes: the lanes set in m add
// the value of the lane CTRL reads (sources out of range, or in rows outside
// ROWS, contribute 0).  Every lane takes part, so every source is well defined.
template <int CTRL, int ROWS = 0xF, class V>
__device__ __forceinline__ void seg_step(uint64_t m, V& n, V& d) {
    const V f = (V)lane_factor(m);
    n = fmav(dpp_v<CTRL, ROWS, true>(V(0), n), f, n);
    d = fmav(dpp_v<CTRL, ROWS, true>(V(0), d), f, d);
}

// Lanes below the first set bit of a 16- or 32-lane group (all of them if none).
__device__ __forceinline__ uint64_t before_first16(uint64_t bits, int lo) {
    const uint32_t g = (uint32_t)(bits >> lo) & 0xFFFFu;
    return (uint64_t)((1u << __builtin_ctz(g | 0x10000u)) - 1u) << lo;
}
__device__ __forceinline__ uint64_t before_first32(uint64_t bits) {
    const uint32_t g = (uint32_t)(bits >> 32);
    return g ? ((uint64_t)((1u << __builtin_ctz(g)) - 1u) << 32) : 0xFFFFFFFF00000000ull;
}

// Inclusive segmented scan of (n, d) over the 64 lanes, restarting at the lanes
// set in `starts`.  In the step that adds the value from s lanes back, lane l
// takes it when none of lanes l - s + 1 .. l starts a segment; the row
// broadcasts extend a lane's sum into the previous row (lanes 15 and 47) and the
// previous half (lane 31) when no segment starts between that row's (or half's)
// first lane and the lane itself.  The masks are wave-uniform bit arithmetic.
template <class V>
__device__ __forceinline__ void seg_scan(uint64_t starts, V& n, V& d) {
    uint64_t m = ~starts;
    seg_step<kRowShr1>(m, n, d);
    m &= m << 1;
    seg_step<kRowShr2>(m, n, d);
    m &= m << 2;
    seg_step<kRowShr4>(m, n, d);
    m &= m << 4;
    seg_step<kRowShr8>(m, n, d);
    seg_step<kBcast15, 0xA>(before_first16(starts, 16) | before_first16(starts, 48), n, d);
    seg_step<kBcast31, 0xC>(before_first32(starts), n, d);
}

template <int CTRL>
__device__ __forceinline__ double dppq_d(double x) {
    int2 v = __builtin_bit_cast(int2, x);
    v.x = __builtin_amdgcn_update_dpp(0, v.x, CTRL, 0xF, 0xF, false);
    v.y = __builtin_amdgcn_update_dpp(0, v.y, CTRL, 0xF, 0xF, false);
    return __builtin_bit_cast(double, v);
}
// x_r + x_(r^1) over 16-lane rows: the swap leaves each row's own value in one
// output and its partner row's value in the other, in the same order for both
// rows of a pair, so both rows obtain the same bits.
__device__ __forceinline__ double xor16_sum(double x) {
    int2 v = __builtin_bit_cast(int2, x);
    auto a = __builtin_amdgcn_permlane16_swap(v.x, v.x, false, false);
    auto b = __builtin_amdgcn_permlane16_swap(v.y, v.y, false, false);
    int2 lo, hi;
    lo.x = (int)a[0]; lo.y = (int)b[0];
    hi.x = (int)a[1]; hi.y = (int)b[1];
    return __builtin_bit_cast(double, lo) + __builtin_bit_cast(double, hi);
}
// Same with the two 32-lane halves of the wave.
__device__ __forceinline__ double xor32_sum(double x) {
    int2 v = __builtin_bit_cast(int2, x);
    auto a = __builtin_amdgcn_permlane32_swap(v.x, v.x, false, false);
    auto b = __builtin_amdgcn_permlane32_swap(v.y, v.y, false, false);
    int2 lo, hi;
    lo.x = (int)a[0]; lo.y = (int)b[0];
    hi.x = (int)a[1]; hi.y = (int)b[1];
    return __builtin_bit_cast(double, lo) + __builtin_bit_cast(double, hi);
}
// Sum over the 64 lanes; every lane gets the same bits.
__device__ __forceinline__ double wave_sum(double x) {
    x += dppq_d<0xB1>(x);   // quad_perm [1,0,3,2]: lane ^ 1
    x += dppq_d<0x4E>(x);   // quad_perm [2,3,0,1]: lane ^ 2
    x += dppq_d<0x141>(x);  // row_half_mirror: the other quad of 8
    x += dppq_d<0x140>(x);  // row_mirror: the other half of 16
    x = xor16_sum(x);
    return xor32_sum(x);
}

__device__ __forceinline__ double lane_f64(double v, int src) {
    const int2 p = __builtin_bit_cast(int2, v);
    int2 r;
    r.x = __builtin_amdgcn_readlane(p.x, src);
    r.y = __builtin_amdgcn_readlane(p.y, src);
    return __builtin_bit_cast(double, r);
}

template <class V>
__device__ __forceinline__ V coordinate(double num, double den, double lambda) {
    const double d = lambda + den;
    return d == 0.0 ? V(0) : (V)(num / d);
}

template <int MODE> struct Needs {
    static constexpr bool x = MODE != kModeFlush;
    static constexpr bool q = MODE == kModeAdd || MODE == kModeSubAdd;
    static constexpr bool qq = MODE == kModeSubAdd || MODE == kModeFlush;
    static constexpr bool p = MODE == kModeAdd || MODE == kModeSubAdd;
    static constexpr bool pp = MODE == kModeSubAdd || MODE == kModeFlush;
    static constexpr bool store = MODE != kModePlain;
};

// Where a pass reads its gathered vectors: LDS slices of the tile, or global.
template <class V>
struct Gather {
    const V* lx;
    const V* lq;
    const V* lqq;
    rsrc_t gx, gq, gqq;
    rsrc_t gpk;    // packed (x, q, qq, 0) records (float first passes)
    uint32_t th;   // hot layouts: indices below th are staged
    uint32_t tsw;  // hot layouts: indices below tsw are swizzled positions
    uint32_t gpad; // a column past the vectors (reads 0)
};

template <class V>
__device__ __forceinline__ V gload(rsrc_t g, uint32_t c) {
    if constexpr (sizeof(V) == 4)
        return ld_f32(g, c * 4u);
    else
        return ld_f64(g, c * 8u);
}

// Residual bookkeeping of a mode applied to one stored value.
template <int MODE, class V>
__device__ __forceinline__ V rhat(V v, V qv, V qqv, V pr, V ppr) {
    if constexpr (MODE == kModeAdd) return fmav(pr, qv, v);
    if constexpr (MODE == kModeSubAdd) return fmav(pr, qv, fmav(-ppr, qqv, v));
    if constexpr (MODE == kModeFlush) return fmav(-ppr, qqv, v);
    return v;
}


// Copy the tile's slice of every gathered vector into LDS at the swizzled
// positions, with a zero at the padding index.  Slots come in the order x, q,
// qq; x shares q's slot when they are the same vector.  A hot layout stages its
// leading T columns as tile 0.
template <int MODE, bool HOT, class V>
__device__ __forceinline__ void stage_tile(const PassArgs<V>& a, int tile, V* lds, Gather<V>& gx) {
    using N = Needs<MODE>;
    const int T = a.T, Ts = a.Ts;
    const int c0 = tile * T;
    const int len = min(T, a.cols - c0);
    const bool alias = N::x && N::q && a.x_is_q;
    int slot = 0;
    V* sx = nullptr;
    V* sq = nullptr;
    V* sqq = nullptr;
    if (N::x && !alias) sx = lds + (slot++) * Ts;
    if (N::q) sq = lds + (slot++) * Ts;
    if (alias) sx = sq;
    if (N::qq) sqq = lds + (slot++) * Ts;
    // Strided elements per thread per step, loads first, so that a step costs one
    // memory latency: sixteen floats (one or two steps cover a tile), or four
    // doubles, which keeps the fused double kernels within their registers.
    if constexpr (sizeof(V) == 4) {
        // Float slices go straight from memory into LDS: wave w fills the 64-word blocks
        // w, w + 16, ... of every slot, lane l loading the column whose swizzled position
        // is the block's word l (the swizzle stays inside 32-word groups, so the loads
        // stay coalesced).  Columns at or past len read 0 through the bounded descriptor;
        // a slot holds at least len rounded up to 64 words (Ts).
        const int wave = (int)(threadIdx.x >> 6), lane = (int)(threadIdx.x & 63u);
        const int words = (len + 63) / 64 * 64;
        auto fill = [&](const V* src, V* dst) {
            const rsrc_t r = make_rsrc(src + c0, (uint64_t)len * sizeof(V));
            for (int b = wave * 64; b < words; b += kWG) {
                const uint32_t c = lds_swizzle((uint32_t)(b + lane));
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    r, (__attribute__((address_space(3))) void*)(dst + b), 4, c * 4u, 0, 0, 0);
            }
        };
        if (N::x && !alias) fill(a.x, sx);
        if (N::q) fill(a.q, sq);
        if (N::qq) fill(a.qq, sqq);
        __builtin_amdgcn_s_waitcnt(0);  // the loads into LDS are done
    } else {
    constexpr int kU = 4;
    for (int i0 = (int)threadIdx.x; i0 < len; i0 += kU * kWG) {
        V vx[kU], vq[kU], vqq[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int i = min(i0 + u * kWG, len - 1);
            if (N::x && !alias) vx[u] = a.x[c0 + i];
            if (N::q) vq[u] = a.q[c0 + i];
            if (N::qq) vqq[u] = a.qq[c0 + i];
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int i = i0 + u * kWG;
            if (i < len) {
                const uint32_t li = lds_swizzle((uint32_t)i);
                if (N::x && !alias) sx[li] = vx[u];
                if (N::q) sq[li] = vq[u];
                if (N::qq) sqq[li] = vqq[u];
            }
        }
    }
    }
    if (!HOT && threadIdx.x == 0) {  // hot layouts pad with a global column
        if (N::x && !alias) sx[a.pad] = V(0);
        if (N::q) sq[a.pad] = V(0);
        if (N::qq) sqq[a.pad] = V(0);
    }
    gx.lx = sx;
    gx.lq = sq;
    gx.lqq = sqq;
}

// What a window needs from memory before its arithmetic: the lane's kE values
// and indices, and the row scalars of segment sb + lane (the window's segments
// are sb .. sb + 64, sb being the one open before its first entry).
template <class V>
struct Win {
    static constexpr int E = 16 / sizeof(V);  // values per 128-bit access
    typename Vec16<V>::type vv[kE / E];
    u32x4 c0, c1;  // IDX16: c0 holds the 8 indices packed in pairs (or, with dz,
                   // the lane's delta-coded record in its first three words)
    V pr, ppr;
    bool dz;       // IDX16: the window is delta-coded (uniform)
};

// Loads and stores of the residual stream under a copy's cache policy.
template <int CA, class T>
__device__ __forceinline__ T load_res(const T* p) {
    if constexpr (CA == kCacheAll)
        return *p;
    else
        return __builtin_nontemporal_load(p);
}
template <int CA, class T>
__device__ __forceinline__ void store_res(T v, T* p) {
    if constexpr (CA == kCacheStream)
        __builtin_nontemporal_store(v, p);
    else
        *p = v;
}

// The delta-coded window bits of 64 consecutive windows, kept while a wave walks
// them (wave-uniform).
struct DMask {
    uint64_t w;
    int32_t i;  // word index, -1 before the first load
};
typedef uint32_t u32x3a __attribute__((ext_vector_type(3), aligned(4)));
// The 12-byte index record of a lane in a delta-coded window, aligned to 4 bytes
// only: loaded through its own type, since deducing load_res's parameter type would
// drop that alignment.
template <int CA>
__device__ __forceinline__ u32x3a load_rec12(const u32x3a* p) {
    if constexpr (CA == kCacheAll)
        return *p;
    else
        return __builtin_nontemporal_load(p);
}

// Data loads of the window block at b (a multiple of kWin): lane l's values from
// the two halves of the block (val_slot order), its indices in entry order (or,
// in a delta-coded window, its 12-byte record, decoded when the window is used).
// Chunks start and end at multiples of kWin, so every block a chunk reads lies
// whole inside the arrays.  A window past the chunk's end (own == false) rereads
// lane 0's part of block b on every lane: one line, never used.  Positions fit
// 31 bits (the layout build checks), so they are 32-bit here.  CA: the copy's
// cache policy (streaming loads, unless the copy stays cached).
template <bool IDX16, int CA, class V>
__device__ __forceinline__ void load_data(const PassArgs<V>& a, int32_t b, bool own, uint32_t le,
                                          Win<V>& w, DMask& dm) {
    using VV = typename Vec16<V>::type;
    const uint32_t lo = own ? le : 0u;
    const VV* vp = reinterpret_cast<const VV*>(a.val + b) + (int)(lo / kE);
#pragma unroll
    for (int q = 0; q < kE / Win<V>::E; ++q) w.vv[q] = load_res<CA>(vp + 64 * q);
    if constexpr (IDX16) {
        bool dz = false;
        if (a.dmask) {
            const int32_t wi = b / kWin;
            if ((wi >> 6) != dm.i) {  // once per 64 windows
                dm.i = wi >> 6;
                dm.w = a.dmask[dm.i];
            }
            dz = ((dm.w >> (wi & 63)) & 1u) != 0;
        }
        w.dz = dz;
        if (dz) {
            // 12 bytes per lane: the window's indices take its first 768 bytes.
            const u32x3a* rp = reinterpret_cast<const u32x3a*>(static_cast<const uint32_t*>(a.idx) +
                                                              b / 2 + 3 * (int)(lo / kE));
            const u32x3a r = load_rec12<CA>(rp);
            w.c0.x = r.x;
            w.c0.y = r.y;
            w.c0.z = r.z;
        } else {
            w.c0 = load_res<CA>(
                reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.idx) + b + lo));
        }
    } else {
        const u32x4* ip = reinterpret_cast<const u32x4*>(static_cast<const int32_t*>(a.idx) + b + lo);
        w.c0 = load_res<CA>(ip);
        w.c1 = load_res<CA>(ip + 1);
    }
}
// Row scalars of segments sb .. sb + 63, one per lane.
template <int MODE, class V>
__device__ __forceinline__ void load_slots(const PassArgs<V>& a, int sb, int lane, Win<V>& w) {
    using N = Needs<MODE>;
    if constexpr (N::p || N::pp) {
        const int sj = min(max(sb + lane, 0), a.nseg - 1);
        if constexpr (N::p) w.pr = a.p[sj];
        if constexpr (N::pp) w.ppr = a.pp[sj];
    }
}

// Index of entry k of the lane, without the segment start bit.
template <bool IDX16, class V>
__device__ __forceinline__ uint32_t col_of(const Win<V>& w, int k) {
    using B = IndexBits<typename std::conditional<IDX16, uint16_t, int32_t>::type>;
    uint32_t c;
    if constexpr (IDX16) {
        const uint32_t d = w.c0[k >> 1];
        c = (k & 1) ? (d >> 16) : (d & 0xFFFFu);
    } else {
        c = k < 4 ? w.c0[k] : w.c1[k - 4];
    }
    return k == 0 ? (c & B::mask) : c;  // only a lane's first entry carries the bit
}
template <bool IDX16, class V>
__device__ __forceinline__ bool starts_segment(const Win<V>& w) {
    using B = IndexBits<typename std::conditional<IDX16, uint16_t, int32_t>::type>;
    return (w.c0[0] & B::start) != 0u;
}
template <class V>
__device__ __forceinline__ V val_of(const Win<V>& w, int k) {
    return w.vv[k / Win<V>::E][k % Win<V>::E];
}

__device__ __forceinline__ float lane_pick(float v, uint32_t src) {
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute((int)(src << 2),
                                                                  __builtin_bit_cast(int, v)));
}
__device__ __forceinline__ double lane_pick(double v, uint32_t src) {
    const int2 x = __builtin_bit_cast(int2, v);
    int2 r;
    r.x = __builtin_amdgcn_ds_bpermute((int)(src << 2), x.x);
    r.y = __builtin_amdgcn_ds_bpermute((int)(src << 2), x.y);
    return __builtin_bit_cast(double, r);
}
__device__ __forceinline__ double lane_read(float v, int src) {
    return (double)__builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), src));
}
__device__ __forceinline__ double lane_read(double v, int src) { return lane_f64(v, src); }

// State a wave carries from window to window of its chunk.
struct Walk {
    int32_t elo;  // first entry of the next window (a multiple of kWin)
    int32_t c1;   // end of the chunk (a multiple of kWin)
    int sb;       // segment of the entry before elo (the open one, when `open`)
    bool open;    // a segment is open: it has entries before elo in this chunk
    double cn, cd;  // sums of the open segment so far
    double sse;
    int mid;      // the chunk's first segment when it began in an earlier chunk, else -1
    int head;     // the chunk's head partial slot (its tail slot follows)
};

extern __shared__ f32x4 lds_raw[];  // dynamic LDS, 16-byte aligned

// P == 1: the head (2w) and tail (2w + 1) partials of every wave w in LDS, after the
// staged vectors, from which the workgroup finishes the rows cut between its waves.
template <class V>
__device__ __forceinline__ double2* cut_slots(const PassArgs<V>& a) {
    return reinterpret_cast<double2*>(reinterpret_cast<char*>(lds_raw) + a.slot_lds);
}
template <class V>
__device__ __forceinline__ double2* wave_slots(const PassArgs<V>& a) {
    return cut_slots(a) + 2 * __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}

__device__ __forceinline__ float2 make_part(float, double n, double d) {
    return make_float2((float)n, (float)d);
}
__device__ __forceinline__ double2 make_part(double, double n, double d) { return make_double2(n, d); }

// A segment's sums over this chunk: its coordinate (P == 1: segment s is row s)
// or partial, or, for a segment that began in an earlier chunk, the chunk's
// head partial.
template <bool P1, class V>
__device__ __forceinline__ void emit(const PassArgs<V>& a, const Walk& wk, int s, double num,
                                     double den) {
    if (s == wk.mid) {
        a.part[wk.head] = make_part(V(0), num, den);
        if constexpr (P1 && sizeof(V) == 4) wave_slots(a)[0] = make_double2(num, den);
    } else if constexpr (P1)
        a.y[s] = coordinate<V>(num, den, a.lambda);
    else
        a.part[s] = make_part(V(0), num, den);
}

// One window [elo, we) of a wave's chunk: up to 64 lanes of kE entries, lane l
// holding entries elo + l*kE .. elo + l*kE + kE - 1, all of one segment.  A lane
// whose first index carries the start bit begins a new segment, so the lanes'
// segments follow from a ballot of those bits and a masked bit count.  Each lane
// sums R-hat*x and x^2 over its entries; a segmented scan over the lanes then
// gives every segment's window sum at its last lane, and the lane that starts
// the next segment emits it.  The data of the window after next is requested
// first, so two windows' loads are in flight while this one is reduced.
template <int MODE, bool STAGED, bool IDX16, bool P1, int CA, bool XQ, class V>
__device__ __forceinline__ void window(const PassArgs<V>& a, const Gather<V>& gx, Walk& wk,
                                       Win<V>& cur, Win<V>& nxt, Win<V>& nn, int lane,
                                       uint32_t le, DMask& dm) {
    using N = Needs<MODE>;
    if constexpr (IDX16) {
        if (cur.dz) {  // back to the plain format: 8 indices packed in pairs
            uint32_t c[8];
            delta_decode(cur.c0.x, cur.c0.y, cur.c0.z, (uint32_t)a.pad, c);
            cur.c0.x = c[0] | (c[1] << 16);
            cur.c0.y = c[2] | (c[3] << 16);
            cur.c0.z = c[4] | (c[5] << 16);
            cur.c0.w = c[6] | (c[7] << 16);
        }
    }
    constexpr bool HOT = STAGED && !IDX16;
    constexpr bool GLOBAL = !STAGED || HOT;  // some gathers read global memory
    // Float gathers are issued before the loads of the window after next; double
    // ones after them, inside the entry loop, where the registers allow.
    constexpr bool EARLY = GLOBAL && sizeof(V) == 4;
    // A float first pass gathers its two or three vectors as one 16-byte record.
    constexpr bool PACK = EARLY && N::q && (N::qq || (N::x && !XQ));
    const int32_t b = wk.elo;
    const int32_t we = min(b + kWin, wk.c1);
    // Gathers from global memory: in a hot layout, the entries past the staged
    // columns (the others read the padding column, which costs no memory access).
    V gq[kE], gqq[kE], gxx[kE];
    auto fetch = [&](int k, uint32_t c) {
        uint32_t g = c;
        if constexpr (HOT) g = c < gx.th ? gx.gpad : (c < gx.tsw ? lds_swizzle(c) : c);
        if constexpr (PACK) {
            const f32x4 w = ld_f32x4(gx.gpk, g * 16u);
            gxx[k] = w.x;
            gq[k] = w.y;
            gqq[k] = w.z;
        } else {
            if constexpr (N::q) gq[k] = gload<V>(gx.gq, g);
            if constexpr (N::qq) gqq[k] = gload<V>(gx.gqq, g);
            if constexpr (N::x && !XQ) gxx[k] = gload<V>(gx.gx, g);
        }
    };
    if constexpr (EARLY) {
#pragma unroll
        for (int k = 0; k < kE; ++k) fetch(k, col_of<IDX16, V>(cur, k));
        __builtin_amdgcn_sched_barrier(0);
    }
    // Data of the window after next, before anything waits on this one (past the
    // chunk's end, a reload of lane 0's part of block b that nothing reads).
    {
        const int32_t b2 = we + kWin;
        const bool more = b2 < wk.c1;
        load_data<IDX16, CA, V>(a, more ? b2 : b, more, le, nn, dm);
    }
    const int nl = (int)((we - b) / kE);  // lanes holding entries of this window
    const bool lv = lane < nl;
    const bool fl = lv && starts_segment<IDX16, V>(cur);
    const uint64_t starts = __ballot(fl);
    const int sb_n = wk.sb + __builtin_popcountll(starts);
    load_slots<MODE, V>(a, sb_n, lane, nxt);  // the next window's row scalars

    // Segments started at lanes 0 .. lane: the lane's segment is sb + cl.
    const uint64_t sh = starts >> 1;
    const uint32_t cl = __builtin_amdgcn_mbcnt_hi(
        (uint32_t)(sh >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)sh, (uint32_t)(starts & 1u)));

    // Row scalars of the lane's segment, from the window's slots; with 64 starts the
    // last lane's segment is sb + 64, past the slots.
    V pr = V(0), ppr = V(0);
    if constexpr (N::p) pr = lane_pick(cur.pr, cl);
    if constexpr (N::pp) ppr = lane_pick(cur.ppr, cl);
    if constexpr (N::p || N::pp) {
        if (starts == ~0ull && lane == 63) {
            if constexpr (N::p) pr = a.p[wk.sb + 64];
            if constexpr (N::pp) ppr = a.pp[wk.sb + 64];
        }
    }

    // Gathers, residual bookkeeping, and the lane's sums.
    V r[kE];
    V an = V(0), ad = V(0);
#pragma unroll
    for (int k = 0; k < kE; ++k) {
        const uint32_t c = col_of<IDX16, V>(cur, k);
        if constexpr (GLOBAL && !EARLY) fetch(k, c);
        V qv = V(0), qqv = V(0), xg = V(0);
        if constexpr (!STAGED) {
            if constexpr (N::q) qv = gq[k];
            if constexpr (N::qq) qqv = gqq[k];
            if constexpr (N::x && !XQ) xg = gxx[k];
        } else {
            const bool hot = !HOT || c < gx.th;
            const uint32_t lc = hot ? c : 0u;
            if constexpr (N::q) qv = gx.lq[lc];
            if constexpr (N::qq) qqv = gx.lqq[lc];
            if constexpr (N::x && !XQ) xg = gx.lx[lc];
            if constexpr (HOT) {
                if constexpr (N::q) qv = hot ? qv : gq[k];
                if constexpr (N::qq) qqv = hot ? qqv : gqq[k];
                if constexpr (N::x && !XQ) xg = hot ? xg : gxx[k];
            }
        }
        r[k] = rhat<MODE, V>(val_of<V>(cur, k), qv, qqv, pr, ppr);
        if constexpr (N::x) {
            const V xv = XQ ? qv : xg;
            an = fmav(r[k], xv, an);
            ad = fmav(xv, xv, ad);
        }
    }
    if constexpr (N::store) {
        // R-hat back to the lane's two value groups: each store instruction of the
        // wave covers 1 KB of contiguous memory.
        if (lv) {
            using VV = typename Vec16<V>::type;
            constexpr int E = Win<V>::E;
            VV* wp = reinterpret_cast<VV*>(a.val + b) + (int)(le / kE);
#pragma unroll
            for (int q = 0; q < kE / E; ++q) {
                VV w;
#pragma unroll
                for (int e = 0; e < E; ++e) w[e] = r[q * E + e];
                store_res<CA>(w, wp + 64 * q);
            }
        }
    }
    if constexpr (MODE == kModeFlush) {
        V s2 = V(0);
#pragma unroll
        for (int k = 0; k < kE; ++k) s2 = fmav(r[k], r[k], s2);
        if (lv) wk.sse += (double)s2;
    } else {
        if (!lv) {
            an = V(0);
            ad = V(0);
        }
        seg_scan(starts, an, ad);
        // A lane that starts a segment emits the previous one: its sum over the
        // earlier lanes of the window (the scan at the lane before), plus the sums
        // from earlier windows when it is the window's first segment.
        const V pn = dpp_v<kWaveShr1, 0xF, true>(V(0), an);
        const V pd = dpp_v<kWaveShr1, 0xF, true>(V(0), ad);
        if (fl) {
            const bool first = lane == (int)__builtin_ctzll(starts);
            double en = (double)pn, ed = (double)pd;
            if (first) {
                en += wk.cn;
                ed += wk.cd;
            }
            if (wk.open || lane > 0) emit<P1, V>(a, wk, wk.sb + (int)cl - 1, en, ed);
        }
        // The segment of the window's last lane stays open.
        const int ll = nl - 1;
        const double ln = lane_read(an, ll);
        const double ld = lane_read(ad, ll);
        if (starts == 0ull) {
            wk.cn += ln;
            wk.cd += ld;
        } else {
            wk.cn = ln;
            wk.cd = ld;
        }
        wk.open = true;
    }
    wk.sb = sb_n;
    wk.elo = we;
}

// One wave's chunk [c0, c1), three windows per loop turn so that the current
// window and the two whose data is in flight rotate over three register sets.
// begin_chunk requests the first two windows, so that a caller can overlap them
// with the staging of the tile.  s0 is the segment holding entry
// c0; it began in an earlier chunk when the chunk's first lane does not start it
// (flag kChunkMid).
template <int MODE, bool IDX16, int CA, class V>
__device__ __forceinline__ void begin_chunk(const PassArgs<V>& a, int32_t c0, int32_t c1, int s0,
                                            int flags, int lane, Win<V>& wa, Win<V>& wb,
                                            DMask& dm) {
    const uint32_t le = (uint32_t)lane * kE;
    load_data<IDX16, CA, V>(a, c0, true, le, wa, dm);
    load_slots<MODE, V>(a, (flags & kChunkMid) ? s0 : s0 - 1, lane, wa);
    const bool more = c0 + kWin < c1;
    load_data<IDX16, CA, V>(a, more ? c0 + kWin : c0, more, le, wb, dm);
}

// wa and wb hold the requests of begin_chunk.
template <int MODE, bool STAGED, bool IDX16, bool P1, int CA, bool XQ, class V>
__device__ __forceinline__ void run_chunk(const PassArgs<V>& a, const Gather<V>& gx, int32_t c0,
                                          int32_t c1, int s0, int flags, int gc, int lane,
                                          Win<V>& wa, Win<V>& wb, double& sse, DMask& dm) {
    const uint32_t le = (uint32_t)lane * kE;
    const bool mid = flags & kChunkMid;
    Walk wk{c0, c1, mid ? s0 : s0 - 1, mid, 0.0, 0.0, sse, mid ? s0 : -1, a.nseg + 2 * gc};
    Win<V> wc;
    while (true) {
        window<MODE, STAGED, IDX16, P1, CA, XQ, V>(a, gx, wk, wa, wb, wc, lane, le, dm);
        if (wk.elo >= c1) break;
        window<MODE, STAGED, IDX16, P1, CA, XQ, V>(a, gx, wk, wb, wc, wa, lane, le, dm);
        if (wk.elo >= c1) break;
        window<MODE, STAGED, IDX16, P1, CA, XQ, V>(a, gx, wk, wc, wa, wb, lane, le, dm);
        if (wk.elo >= c1) break;
    }
    if constexpr (MODE != kModeFlush) {
        // The last segment: finished, or going on past the chunk (a partial in the head
        // slot when it is also the segment that began earlier, else in the tail slot).
        if (lane == 0) {
            if (flags & kChunkCont) {
                const int t = wk.sb == wk.mid ? 0 : 1;
                a.part[wk.head + t] = make_part(V(0), wk.cn, wk.cd);
                if constexpr (P1 && sizeof(V) == 4) wave_slots(a)[t] = make_double2(wk.cn, wk.cd);
            } else
                emit<P1, V>(a, wk, wk.sb, wk.cn, wk.cd);
        }
    }
    sse = wk.sse;
}

// One pass: the workgroup's pieces in order, each staging its tile (when it
// differs from the one staged) and then giving every wave its chunk.  XQ: the
// update gathers the same vector as the add-back (x == q), read once per entry.
template <int MODE, bool STAGED, bool IDX16, bool P1, int CA, bool XQ, class V>
__device__ __forceinline__ void pass_main(const PassArgs<V>& a) {
    using N = Needs<MODE>;
    V* lds = reinterpret_cast<V*>(lds_raw);
    const int wg = blockIdx.x;

    constexpr bool HOT = STAGED && !IDX16;
    Gather<V> gx{};
    if constexpr (!STAGED || HOT) {
        const uint64_t vb = (uint64_t)a.cols * sizeof(V);
        if (N::x) gx.gx = make_rsrc(a.x, vb);
        if (N::q) gx.gq = make_rsrc(a.q, vb);
        if (N::qq) gx.gqq = make_rsrc(a.qq, vb);
        gx.gpk = make_rsrc(a.pk, a.pk ? (uint64_t)a.cols * 16u : 0u);
        gx.th = (uint32_t)a.T;
        gx.tsw = (uint32_t)a.tsw;
        gx.gpad = (uint32_t)a.cols;
    }
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = (int)(threadIdx.x & 63u);

    // P == 1, float: the rows cut between this workgroup's waves (at most 15), one per
    // lane of wave 0, requested now and finished at the end from the waves' LDS
    // partials.  (The double kernels are short of registers for it: their layouts
    // leave every cut row to the combine kernel.)
    constexpr bool CUT = MODE != kModeFlush && P1 && sizeof(V) == 4;
    constexpr bool CUT_EARLY = CUT;
    int cut0 = 0, ncut = 0, crow = 0;
    uint64_t cdesc = 0;
    if constexpr (CUT) {
        cut0 = a.wg_cut[wg];
        ncut = a.wg_cut[wg + 1] - cut0;
    }
    if constexpr (CUT_EARLY) {
        if (wave == 0 && lane < ncut) {
            crow = a.cut_row[cut0 + lane];
            cdesc = a.cut_desc[cut0 + lane];
        }
    }
    if constexpr (MODE != kModeFlush && P1) {
        // The rows after the last non-empty one have no entries: coordinate 0.
        for (int i = wg * kWG + (int)threadIdx.x; i < a.rows - a.nseg_ne; i += gridDim.x * kWG)
            a.y[a.nseg_ne + i] = coordinate<V>(0.0, 0.0, a.lambda);
    }

    double sse = 0.0;
    int staged = -1;
    DMask dm{0, -1};
    for (int pc = a.wg_piece[wg]; pc < a.wg_piece[wg + 1]; ++pc) {
        const int32_t c0 = (int32_t)a.piece_chunk[pc * (kWaves + 1) + wave];
        const int32_t c1 = (int32_t)a.piece_chunk[pc * (kWaves + 1) + wave + 1];
        const int gc = pc * kWaves + wave;
        const int s0 = a.piece_seg[gc], flags = a.chunk_flags[gc];
        // The chunk's first windows are requested before the staging, which they do
        // not depend on.
        Win<V> wa, wb;
        if (c0 < c1) begin_chunk<MODE, IDX16, CA, V>(a, c0, c1, s0, flags, lane, wa, wb, dm);
        if constexpr (STAGED) {
            const int tile = a.piece_tile[pc];
            if (tile != staged) {
                if (staged >= 0) __syncthreads();  // every wave is done with the old slice
                stage_tile<MODE, HOT, V>(a, tile, lds, gx);
                __syncthreads();
                staged = tile;
            }
        }
        if (c0 < c1)
            run_chunk<MODE, STAGED, IDX16, P1, CA, XQ, V>(a, gx, c0, c1, s0, flags, gc, lane, wa, wb, sse,
                                                           dm);
    }
    if constexpr (MODE == kModeFlush) {
        const double t = wave_sum(sse);
        if (lane == 0) a.sse_part[wg * kWaves + wave] = t;
    } else if constexpr (P1) {
        // Rows cut between this workgroup's waves: their partials, in entry order.
        if (ncut > 0) {       // the same for every thread of the workgroup
            __syncthreads();  // every wave's partials are in LDS
            if (wave == 0 && lane < ncut) {
                if constexpr (!CUT_EARLY) {
                    crow = a.cut_row[cut0 + lane];
                    cdesc = a.cut_desc[cut0 + lane];
                }
                const int n = (int)(cdesc & 15u) + 1;
                double num = 0.0, den = 0.0;
                for (int i = 0; i < n; ++i) {
                    const double2 pv = cut_slots(a)[(int)((cdesc >> (4 + 5 * i)) & 31u)];
                    num += pv.x;
                    den += pv.y;
                }
                a.y[crow] = coordinate<V>(num, den, a.lambda);
            }
        }
    }
}

}  // namespace

// Distinct kernel names per pass kind, so that profiles separate them.  The
// template arguments select LDS staging, the index width, whether segments are
// rows (P == 1), the copy's cache policy and the value type.
template <bool STAGED, bool IDX16, bool P1, int CA, class V>
__global__ __launch_bounds__(kWG) void ccd_pass(PassArgs<V> a) {
    pass_main<kModePlain, STAGED, IDX16, P1, CA, false, V>(a);
}
template <bool STAGED, bool IDX16, bool P1, int CA, class V>
__global__ __launch_bounds__(kWG) void ccd_pass_fused_first(PassArgs<V> a) {
    if (a.x_is_q)
        pass_main<kModeAdd, STAGED, IDX16, P1, CA, true, V>(a);
    else
        pass_main<kModeAdd, STAGED, IDX16, P1, CA, false, V>(a);
}
template <bool STAGED, bool IDX16, bool P1, int CA, class V>
__global__ __launch_bounds__(kWG) void ccd_pass_fused(PassArgs<V> a) {
    if (a.x_is_q)
        pass_main<kModeSubAdd, STAGED, IDX16, P1, CA, true, V>(a);
    else
        pass_main<kModeSubAdd, STAGED, IDX16, P1, CA, false, V>(a);
}
template <bool STAGED, bool IDX16, bool P1, int CA, class V>
__global__ __launch_bounds__(kWG) void ccd_flush(PassArgs<V> a) {
    pass_main<kModeFlush, STAGED, IDX16, P1, CA, false, V>(a);
}

// x summed over the 16 lanes of a DPP row; every lane of the row gets the same
// bits (each step adds two values that the partner lane adds in swapped order).
__device__ __forceinline__ double row16_sum(double x) {
    x += dppq_d<0xB1>(x);   // quad_perm [1,0,3,2]: lane ^ 1
    x += dppq_d<0x4E>(x);   // quad_perm [2,3,0,1]: lane ^ 2
    x += dppq_d<0x141>(x);  // row_half_mirror: the other quad of 8
    x += dppq_d<0x140>(x);  // row_mirror: the other half of 16
    return x;
}

// x summed over the 4 lanes of a quad, every lane getting the same bits.
__device__ __forceinline__ double quad_sum(double x) {
    x += dppq_d<0xB1>(x);  // lane ^ 1
    x += dppq_d<0x4E>(x);  // lane ^ 2
    return x;
}

// Fixed-order combine of a row's partials: L lanes per row (16, one DPP row, or
// 4, a quad, for layouts whose rows have few partials); lane l adds the row's
// partial slots l, l + L, ... in entry order, then a fixed tree over the L
// lanes.  With yseg, the coordinate is also written to every segment of the row.
template <int L, class V>
__global__ __launch_bounds__(256) void ccd_combine(CombineArgs<V> c) {
    const int l = (int)(threadIdx.x & (L - 1));
    const int i = blockIdx.x * (256 / L) + (int)(threadIdx.x / L);
    if (i >= c.n) return;  // whole rows of lanes leave together
    const int b = c.src_ptr[i];
    const int e = c.src_ptr[i + 1];
    int sb = 0, se = 0;
    if (c.yseg) {  // requested now, used after the sums
        sb = c.seg_ptr[i];
        se = c.seg_ptr[i + 1];
    }
    // Four of the lane's slots at a time: their list entries, then their partials, so
    // that a row of many partials waits for two loads per four slots, not per slot.
    // Positions past the row's end reload its last slot and are not added; the sums
    // still run over the lane's slots in entry order.
    constexpr int U = 4;
    double num = 0.0, den = 0.0;
    for (int k0 = b + l; k0 < e; k0 += U * L) {
        int32_t sl[U];
#pragma unroll
        for (int u = 0; u < U; ++u) sl[u] = c.srcs[min(k0 + u * L, e - 1)];
        part_t<V> pv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) pv[u] = c.part[sl[u]];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (k0 + u * L < e) {
                num += (double)pv[u].x;
                den += (double)pv[u].y;
            }
    }
    if constexpr (L == 16) {
        num = row16_sum(num);
        den = row16_sum(den);
    } else {
        num = quad_sum(num);
        den = quad_sum(den);
    }
    const V yr = coordinate<V>(num, den, c.lambda);
    if (l == 0) c.y[c.ids ? c.ids[i] : i] = yr;
    if (c.yseg)
        for (int k = sb + l; k < se; k += L) c.yseg[c.segs[k]] = yr;
}

template <class V>
__global__ __launch_bounds__(256) void ccd_copy(const V* __restrict__ src, V* __restrict__ dst,
                                                int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) dst[i] = src[i];
}

// The packed gather records of a float first pass: (x, q, qq, 0) per column,
// a null vector giving zeros.
__global__ __launch_bounds__(256) void ccd_pack(const float* __restrict__ x,
                                                const float* __restrict__ q,
                                                const float* __restrict__ qq,
                                                f32x4* __restrict__ pk, int32_t n) {
    const int32_t i = (int32_t)blockIdx.x * 256 + (int32_t)threadIdx.x;
    if (i >= n) return;
    f32x4 w;
    w.x = x ? x[i] : 0.0f;
    w.y = q ? q[i] : 0.0f;
    w.z = qq ? qq[i] : 0.0f;
    w.w = 0.0f;
    pk[i] = w;
}

// Single-workgroup fixed-order sum: thread t sums part[t], part[t+256], ... in
// order, then a fixed tree over the 256 thread sums.
__global__ __launch_bounds__(256) void ccd_reduce_sum(const double* __restrict__ part, int32_t n,
                                                      double* __restrict__ out) {
    __shared__ double s[256];
    double acc = 0.0;
    for (int32_t i = threadIdx.x; i < n; i += 256) acc += part[i];
    s[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) s[threadIdx.x] += s[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[0] = s[0];
}

int staged_vectors(PassMode mode, bool x_is_q) {
    switch (mode) {
        case kModePlain: return 1;
        case kModeAdd: return x_is_q ? 1 : 2;
        case kModeSubAdd: return x_is_q ? 2 : 3;
        case kModeFlush: return 1;
    }
    return 3;
}

namespace {
// The plain pass stores no residual: with write-back stores it is the streaming kernel.
constexpr int plain_cache(int ca) { return ca == kCacheStores ? kCacheStream : ca; }

template <bool S, bool I, bool P1, int CA, class V>
hipError_t raise_lds() {
    constexpr int CP = plain_cache(CA);
    const void* ks[] = {(const void*)ccd_pass<S, I, P1, CP, V>, (const void*)ccd_pass_fused_first<S, I, P1, CA, V>,
                        (const void*)ccd_pass_fused<S, I, P1, CA, V>, (const void*)ccd_flush<S, I, P1, CA, V>};
    for (const void* k : ks) {
        hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <bool S, bool I, bool P1, int CA, class V>
void launch_mode(PassMode mode, dim3 grid, size_t lds, hipStream_t s, const PassArgs<V>& a) {
    constexpr int CP = plain_cache(CA);
    switch (mode) {
        case kModePlain:
            hipLaunchKernelGGL((ccd_pass<S, I, P1, CP, V>), grid, dim3(kWG), lds, s, a);
            break;
        case kModeAdd:
            hipLaunchKernelGGL((ccd_pass_fused_first<S, I, P1, CA, V>), grid, dim3(kWG), lds, s, a);
            break;
        case kModeSubAdd:
            hipLaunchKernelGGL((ccd_pass_fused<S, I, P1, CA, V>), grid, dim3(kWG), lds, s, a);
            break;
        case kModeFlush:
            hipLaunchKernelGGL((ccd_flush<S, I, P1, CA, V>), grid, dim3(kWG), lds, s, a);
            break;
    }
}

// Tiled float copies also come with the write-back policies.
template <bool P1, class V>
void launch_tiled(int cache, PassMode mode, dim3 grid, size_t lds, hipStream_t s, const PassArgs<V>& a) {
    if constexpr (sizeof(V) == 4) {
        if (cache == kCacheStores) return launch_mode<true, true, P1, kCacheStores, V>(mode, grid, lds, s, a);
        if (cache == kCacheAll) return launch_mode<true, true, P1, kCacheAll, V>(mode, grid, lds, s, a);
    }
    launch_mode<true, true, P1, kCacheStream, V>(mode, grid, lds, s, a);
}

template <class V>
hipError_t raise_lds_all() {
    hipError_t e = raise_lds<true, true, true, kCacheStream, V>();
    if (e == hipSuccess) e = raise_lds<true, true, false, kCacheStream, V>();
    if (e == hipSuccess) e = raise_lds<true, false, true, kCacheStream, V>();
    if (e == hipSuccess) e = raise_lds<false, true, true, kCacheStream, V>();
    if (e == hipSuccess) e = raise_lds<false, false, true, kCacheStream, V>();
    if constexpr (sizeof(V) == 4) {
        if (e == hipSuccess) e = raise_lds<true, true, true, kCacheStores, V>();
        if (e == hipSuccess) e = raise_lds<true, true, false, kCacheStores, V>();
        if (e == hipSuccess) e = raise_lds<true, true, true, kCacheAll, V>();
        if (e == hipSuccess) e = raise_lds<true, true, false, kCacheAll, V>();
    }
    return e;
}
}  // namespace

hipError_t sweep_init() {
    hipError_t e = raise_lds_all<float>();
    if (e == hipSuccess) e = raise_lds_all<double>();
    return e;
}

template <class V>
hipError_t launch_pass(const Layout& L, PassMode mode, const V* x, const V* p, const V* pp,
                       const V* q, const V* qq, V* y, double lambda, double* sse_part,
                       hipStream_t s) {
    if (L.grid == 0) return hipSuccess;
    const bool staged = L.gather == kGatherLds;
    const bool hot = L.gather == kGatherHot;
    // Kernel variants: tiles use 16-bit indices, hot layouts 32-bit ones; global
    // gathers and hot layouts have P == 1.
    if (staged ? !L.idx16 : L.P != 1) return hipErrorInvalidValue;
    if (hot && L.idx16) return hipErrorInvalidValue;
    // Write-back cache policies: tiled float copies only.
    if (L.cache != kCacheStream && (!staged || sizeof(V) != 4)) return hipErrorInvalidValue;
    PassArgs<V> a{};
    a.idx = L.idx;
    a.val = static_cast<V*>(L.val);
    a.wg_piece = L.wg_piece;
    a.piece_tile = L.piece_tile;
    a.piece_chunk = L.piece_chunk;
    a.piece_seg = L.piece_seg;
    a.chunk_flags = L.chunk_flags;
    a.dmask = L.dmask;
    a.wg_cut = L.wg_cut;
    a.cut_row = L.cut_row;
    a.cut_desc = L.cut_desc;
    if (L.P == 1 && !L.wg_cut) return hipErrorInvalidValue;
    a.x = x;
    a.p = p;
    a.pp = pp;
    a.q = q;
    a.qq = qq;
    a.y = y;
    a.part = static_cast<part_t<V>*>(L.part);
    a.sse_part = sse_part;
    a.rows = (int32_t)L.rows;
    a.cols = (int32_t)L.cols;
    a.T = L.T;
    a.P = L.P;
    a.Ts = L.Ts;
    a.pad = L.pad;
    a.nseg = (int32_t)L.nseg;
    a.nseg_ne = (int32_t)L.nseg_ne;
    a.x_is_q = (x != nullptr && x == q) ? 1 : 0;
    a.lambda = lambda;
    const int nv = staged_vectors(mode, a.x_is_q);
    a.tsw = 0;
    a.vec_elems = staged ? nv * a.Ts : 0;
    if (hot) {
        // As many leading columns as the pass's vectors leave room for.
        const int64_t fit = ((int64_t)kLdsVecBytes / ((int64_t)sizeof(V) * nv) - 64) / 64 * 64;
        a.T = (int32_t)std::min<int64_t>(L.hot, fit);
        a.Ts = (a.T + 63) / 64 * 64;  // whole 64-word blocks (at most fit)
        a.tsw = L.hot;
        a.vec_elems = nv * a.Ts;
    }
    a.slot_lds = (int32_t)(((size_t)a.vec_elems * sizeof(V) + 15) / 16 * 16);
    const size_t lds = (size_t)a.slot_lds + (L.P == 1 ? (size_t)kCutSlotBytes : 0);
    if (lds > (size_t)kLdsBytes) return hipErrorInvalidValue;
    if (!staged && sizeof(V) == 4 && nv >= 2) {
        // Float first passes that gather two or three vectors from global memory read
        // them as packed records.
        if (!L.pk) return hipErrorInvalidValue;
        hipLaunchKernelGGL(ccd_pack, dim3((unsigned)((L.cols + 255) / 256)), dim3(256), 0, s,
                           reinterpret_cast<const float*>(x), reinterpret_cast<const float*>(q),
                           reinterpret_cast<const float*>(qq), static_cast<f32x4*>(L.pk),
                           (int32_t)L.cols);
        a.pk = static_cast<const V*>(L.pk);
    }
    const dim3 grid(L.grid);
    if (staged) {
        if (L.P == 1)
            launch_tiled<true, V>(L.cache, mode, grid, lds, s, a);
        else
            launch_tiled<false, V>(L.cache, mode, grid, lds, s, a);
    } else if (hot) {
        launch_mode<true, false, true, kCacheStream, V>(mode, grid, lds, s, a);
    } else if (L.idx16) {
        launch_mode<false, true, true, kCacheStream, V>(mode, grid, lds, s, a);
    } else {
        launch_mode<false, false, true, kCacheStream, V>(mode, grid, lds, s, a);
    }
    return hipGetLastError();
}

template <class V>
hipError_t launch_combine(const Layout& L, V* y, V* yseg, double lambda, hipStream_t s) {
    if (L.ncomb == 0) return hipSuccess;
    if (yseg && !L.row_seg_ptr) return hipErrorInvalidValue;
    CombineArgs<V> c{};
    c.ids = L.comb_rows;
    c.src_ptr = L.src_ptr;
    c.srcs = L.srcs;
    c.seg_ptr = L.row_seg_ptr;
    c.segs = L.row_segs;
    c.part = static_cast<const part_t<V>*>(L.part);
    c.y = y;
    c.yseg = yseg;
    c.n = L.ncomb;
    c.lambda = lambda;
    if (L.comb_lanes == 4)
        hipLaunchKernelGGL((ccd_combine<4, V>), dim3((unsigned)((L.ncomb + 63) / 64)), dim3(256), 0, s, c);
    else
        hipLaunchKernelGGL((ccd_combine<16, V>), dim3((unsigned)((L.ncomb + 15) / 16)), dim3(256), 0, s, c);
    return hipGetLastError();
}

template <class V>
hipError_t launch_copy(const V* src, V* dst, int64_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(ccd_copy<V>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, dst, n);
    return hipGetLastError();
}

hipError_t launch_reduce_sum(const double* part, int32_t n, double* out, hipStream_t s) {
    hipLaunchKernelGGL(ccd_reduce_sum, dim3(1), dim3(256), 0, s, part, n, out);
    return hipGetLastError();
}

#define CCDK_SWEEP_INSTANTIATE(V)                                                              \
    template hipError_t launch_pass<V>(const Layout&, PassMode, const V*, const V*, const V*,  \
                                       const V*, const V*, V*, double, double*, hipStream_t); \
    template hipError_t launch_combine<V>(const Layout&, V*, V*, double, hipStream_t);        \
    template hipError_t launch_copy<V>(const V*, V*, int64_t, hipStream_t);
CCDK_SWEEP_INSTANTIATE(float)
CCDK_SWEEP_INSTANTIATE(double)
#undef CCDK_SWEEP_INSTANTIATE

}  // namespace ccdk
