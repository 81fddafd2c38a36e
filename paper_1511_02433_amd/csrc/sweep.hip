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
// so a random gather costs an LDS read; layouts too sparse for tiling gather
// through L2 with bounded buffer loads instead.
//
// Arithmetic: R-hat in fp32 FMA.  Inside a window (at most 512 entries) the
// sums of R-hat*x and x^2 are fp32 segmented scans; a segment's window sums are
// added in fp64, across windows too, in a fixed order, so results are
// identical run to run.  The coordinate num / (lambda + den) is an IEEE fp64
// division rounded once to fp32; a coordinate whose denominator is exactly zero
// (lambda = 0 and an empty row) is set to zero.
#include "ccdpp_internal.hpp"

namespace ccdk {
namespace {

using rsrc_t = __amdgpu_buffer_rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, gfx9 family
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint64_t bytes) {
    uint32_t lim = bytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)lim,
                                            kRsrcWord3);
}
// Bounded load: offsets past the descriptor's limit read 0.
__device__ __forceinline__ float ld_f32(rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

// ---- cross-lane operations ---------------------------------------------------
// DPP controls of the gfx9 family.
constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
constexpr int kBcast15 = 0x142;   // lane 15 of each row to the next row
constexpr int kBcast31 = 0x143;   // lane 31 to rows 2 and 3
constexpr int kWaveShr1 = 0x138;  // lane l reads lane l - 1
constexpr int kWaveShl1 = 0x130;  // lane l reads lane l + 1

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

// Inclusive prefix sum over the 64 lanes.
__device__ __forceinline__ int scan_i(int v) {
    v += dpp_i<kRowShr1, 0xF, true>(0, v);
    v += dpp_i<kRowShr2, 0xF, true>(0, v);
    v += dpp_i<kRowShr4, 0xF, true>(0, v);
    v += dpp_i<kRowShr8, 0xF, true>(0, v);
    v += dpp_i<kBcast15, 0xA>(0, v);
    v += dpp_i<kBcast31, 0xC>(0, v);
    return v;
}

// One step of an inclusive segmented scan keyed by segment: add the values of
// the lane CTRL reads when it holds the same key.  Keys are segment id + 1 on
// lanes that carry data and 0 elsewhere; they never decrease over the lanes
// that carry data, so equal keys are contiguous and the steps below compose to
// the full segmented scan.  A source out of range or masked off contributes 0.
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ void seg_step(int key, float& n, float& d) {
    const int pk = dpp_i<CTRL, ROWS, true>(0, key);
    const float f = pk == key ? 1.0f : 0.0f;
    n = __builtin_fmaf(dpp_f<CTRL, ROWS, true>(0.0f, n), f, n);
    d = __builtin_fmaf(dpp_f<CTRL, ROWS, true>(0.0f, d), f, d);
}
__device__ __forceinline__ void seg_scan(int key, float& n, float& d) {
    seg_step<kRowShr1>(key, n, d);
    seg_step<kRowShr2>(key, n, d);
    seg_step<kRowShr4>(key, n, d);
    seg_step<kRowShr8>(key, n, d);
    seg_step<kBcast15, 0xA>(key, n, d);
    seg_step<kBcast31, 0xC>(key, n, d);
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

__device__ __forceinline__ int64_t lane_i64(int64_t v, int src) {
    const int2 p = __builtin_bit_cast(int2, v);
    int2 r;
    r.x = __builtin_amdgcn_readlane(p.x, src);
    r.y = __builtin_amdgcn_readlane(p.y, src);
    return __builtin_bit_cast(int64_t, r);
}
__device__ __forceinline__ double lane_f64(double v, int src) {
    const int2 p = __builtin_bit_cast(int2, v);
    int2 r;
    r.x = __builtin_amdgcn_readlane(p.x, src);
    r.y = __builtin_amdgcn_readlane(p.y, src);
    return __builtin_bit_cast(double, r);
}

__device__ __forceinline__ float coordinate(double num, double den, double lambda) {
    double d = lambda + den;
    return d == 0.0 ? 0.0f : (float)(num / d);
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
struct Gather {
    const float* lx;
    const float* lq;
    const float* lqq;
    rsrc_t gx, gq, gqq;
};

template <bool STAGED>
__device__ __forceinline__ float gat(const float* lds, rsrc_t g, uint32_t c) {
    if constexpr (STAGED)
        return lds[c];
    else
        return ld_f32(g, c * 4u);
}

// Residual bookkeeping of a mode applied to one stored value.
template <int MODE>
__device__ __forceinline__ float rhat(float v, float qv, float qqv, float pr, float ppr) {
    if constexpr (MODE == kModeAdd) return __builtin_fmaf(pr, qv, v);
    if constexpr (MODE == kModeSubAdd) return __builtin_fmaf(pr, qv, __builtin_fmaf(-ppr, qqv, v));
    if constexpr (MODE == kModeFlush) return __builtin_fmaf(-ppr, qqv, v);
    return v;
}


// Copy the tile's slice of every gathered vector into LDS at the swizzled
// positions, with a zero at the padding index.  Slots come in the order x, q,
// qq; x shares q's slot when they are the same vector.
template <int MODE>
__device__ __forceinline__ void stage_tile(const PassArgs& a, int tile, float* lds, Gather& gx) {
    using N = Needs<MODE>;
    const int T = a.T, Ts = a.Ts;
    const int c0 = tile * T;
    const int len = min(T, a.cols - c0);
    const bool alias = N::x && N::q && a.x_is_q;
    int slot = 0;
    float* sx = nullptr;
    float* sq = nullptr;
    float* sqq = nullptr;
    if (N::x && !alias) sx = lds + (slot++) * Ts;
    if (N::q) sq = lds + (slot++) * Ts;
    if (alias) sx = sq;
    if (N::qq) sqq = lds + (slot++) * Ts;
    // Four strided elements per thread per step, loads first, so that a step costs
    // one memory latency rather than four.
    constexpr int kU = 4;
    for (int i0 = (int)threadIdx.x; i0 < len; i0 += kU * kWG) {
        float vx[kU], vq[kU], vqq[kU];
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
    if (threadIdx.x == 0) {
        if (N::x && !alias) sx[a.pad] = 0.0f;
        if (N::q) sq[a.pad] = 0.0f;
        if (N::qq) sqq[a.pad] = 0.0f;
    }
    gx.lx = sx;
    gx.lq = sq;
    gx.lqq = sqq;
}

// What a window needs from memory before its arithmetic: the lane's kE values
// and indices, the start of segment scur + 1 + lane and the row scalars of
// segment scur + lane.
struct Win {
    f32x4 v0, v1;
    u32x4 c0, c1;  // IDX16: c0 holds the 8 indices packed in pairs
    int64_t st;
    float pr, ppr;
};

// Loads of the window at b (a multiple of kE).  Lanes at or past `lim` all read
// entry b instead, so every address stays inside the arrays (whose padding
// covers the last window) and a window past the chunk costs one cache line.
template <int MODE, bool IDX16>
__device__ __forceinline__ void load_window(const PassArgs& a, int64_t b, int64_t lim, uint32_t le,
                                            int scur, int lane, Win& w) {
    using N = Needs<MODE>;
    const int64_t eb = b + (b + (int64_t)le < lim ? (int64_t)le : 0);
    const f32x4* vp = reinterpret_cast<const f32x4*>(a.val + eb);
    w.v0 = __builtin_nontemporal_load(vp);
    w.v1 = __builtin_nontemporal_load(vp + 1);
    if constexpr (IDX16) {
        w.c0 = __builtin_nontemporal_load(
            reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.idx) + eb));
    } else {
        const u32x4* ip = reinterpret_cast<const u32x4*>(static_cast<const int32_t*>(a.idx) + eb);
        w.c0 = __builtin_nontemporal_load(ip);
        w.c1 = __builtin_nontemporal_load(ip + 1);
    }
    w.st = a.seg_start[min(scur + 1 + lane, a.nseg)];
    const int sj = min(scur + lane, a.nseg - 1);
    if constexpr (N::p) w.pr = a.p[sj];
    if constexpr (N::pp) w.ppr = a.pp[sj];
}

template <bool IDX16>
__device__ __forceinline__ uint32_t col_of(const Win& w, int k) {
    if constexpr (IDX16) {
        const uint32_t d = w.c0[k >> 1];
        return (k & 1) ? (d >> 16) : (d & 0xFFFFu);
    } else {
        return k < 4 ? w.c0[k] : w.c1[k - 4];
    }
}
__device__ __forceinline__ float val_of(const Win& w, int k) { return k < 4 ? w.v0[k] : w.v1[k - 4]; }

// State a wave carries from window to window of its chunk.
struct Walk {
    int64_t elo;  // first entry of the next window (a multiple of kE)
    int64_t c1;   // end of the chunk (a multiple of kE)
    int scur;     // segment holding entry elo
    int cid;      // segment left open by the previous window (-1: none), and its sums
    double cn, cd;
    double sse;
    int mid;      // the chunk's first segment when it began in an earlier chunk, else -1
    int head;     // the chunk's head partial slot (its tail slot follows)
};

// A segment's sums over this chunk: its coordinate (P == 1: segment s is row s)
// or partial, or, for a segment that began in an earlier chunk, the chunk's
// head partial.
template <bool P1>
__device__ __forceinline__ void emit(const PassArgs& a, const Walk& wk, int s, double num,
                                     double den) {
    if (s == wk.mid)
        a.part[wk.head] = make_double2(num, den);
    else if constexpr (P1)
        a.y[s] = coordinate(num, den, a.lambda);
    else
        a.part[s] = make_double2(num, den);
}

// One window [elo, we) of a wave's chunk.  Lane l holds entries elo + l*kE ..
// elo + l*kE + kE - 1; every window starts and ends on a multiple of kE, so a
// lane's entries are either all inside the window or all outside.  The window
// ends at the chunk end, after 64 lanes, or at the last multiple of kE not past
// the start of segment scur + 64, so it meets at most 64 segments and their row
// scalars fit one LDS slot per lane.  The segment of each entry comes from a
// bitmap of the segment starts inside the window (built in the wave's LDS
// scratch from one coalesced read of the segment table) and a prefix count over
// lanes.  The loads of the next window are issued before the arithmetic.
template <int MODE, bool STAGED, bool IDX16, bool P1>
__device__ __forceinline__ void window(const PassArgs& a, const Gather& gx, Walk& wk,
                                       const Win& cur, Win& nxt, int lane, uint32_t le, float* spr,
                                       float* sppr, uint32_t* bm) {
    using N = Needs<MODE>;
    const int64_t b = wk.elo;
    const int64_t st = cur.st;
    int64_t we = min(b + (int64_t)kWin, wk.c1);
    const int64_t st63 = lane_i64(st, 63);
    if (st63 < we) we = st63 & ~(int64_t)(kE - 1);
    const int adv = __builtin_popcountll(__ballot(st <= we));
    // Row scalars of the window's segments, one LDS slot per lane.
    if constexpr (N::p) spr[lane] = cur.pr;
    if constexpr (N::pp) sppr[lane] = cur.ppr;
    // Bitmap of the segment starts inside (b, we); this lane's kE bits.
    if (lane < kWin / 32) bm[lane] = 0u;
    __builtin_amdgcn_wave_barrier();
    if (st < we) {
        const uint32_t off = (uint32_t)(st - b);
        atomicOr(&bm[off >> 5], 1u << (off & 31u));
    }
    __builtin_amdgcn_wave_barrier();
    const uint32_t bits = (bm[le >> 5] >> (le & 31u)) & ((1u << kE) - 1u);

    // Next window's loads (a harmless reload of b when this window is the last).
    const int scur_n = wk.scur + adv;
    {
        const bool more = we < wk.c1;
        load_window<MODE, IDX16>(a, more ? we : b, more ? wk.c1 : b, le, scur_n, lane, nxt);
    }

    const int nl = (int)((we - b) / kE);  // lanes holding entries of this window
    const bool lv = lane < nl;
    const int nb = __builtin_popcount(bits);
    const int idb = wk.scur + scan_i(nb) - nb;  // segment of this lane's first entry

    // Gathers, residual bookkeeping, and running sums restarted at segment starts.
    float r[kE], sn[kE], sd[kE];
    float an = 0.0f, ad = 0.0f;
    int slot = idb - wk.scur;
#pragma unroll
    for (int k = 0; k < kE; ++k) {
        const bool fk = (bits >> k) & 1u;
        if constexpr (N::p || N::pp) slot += fk ? 1 : 0;
        const uint32_t c = col_of<IDX16>(cur, k);
        const float pr = N::p ? spr[slot] : 0.0f;
        const float ppr = N::pp ? sppr[slot] : 0.0f;
        const float qv = N::q ? gat<STAGED>(gx.lq, gx.gq, c) : 0.0f;
        const float qqv = N::qq ? gat<STAGED>(gx.lqq, gx.gqq, c) : 0.0f;
        r[k] = rhat<MODE>(val_of(cur, k), qv, qqv, pr, ppr);
        if constexpr (N::x) {
            const float xv = gat<STAGED>(gx.lx, gx.gx, c);
            an = __builtin_fmaf(r[k], xv, fk ? 0.0f : an);
            ad = __builtin_fmaf(xv, xv, fk ? 0.0f : ad);
            sn[k] = an;
            sd[k] = ad;
        }
    }
    if constexpr (N::store) {
        // Write R-hat back so that each store instruction covers contiguous memory:
        // lane l writes entries 4l .. 4l + 3 of the window, then 256 + 4l .. 256 + 4l + 3,
        // which are half (l & 1) of lane l / 2 and of lane 32 + l / 2.  Stores of half
        // lines from strided lanes cost far more HBM time than whole lines.
        const int srcA = (lane >> 1) << 2, srcB = (32 + (lane >> 1)) << 2;
        const bool odd = lane & 1;
        f32x4 w0, w1;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int lo = __builtin_bit_cast(int, r[k]), hi = __builtin_bit_cast(int, r[4 + k]);
            const int a0 = __builtin_amdgcn_ds_bpermute(srcA, lo), a1 = __builtin_amdgcn_ds_bpermute(srcA, hi);
            const int b0 = __builtin_amdgcn_ds_bpermute(srcB, lo), b1 = __builtin_amdgcn_ds_bpermute(srcB, hi);
            w0[k] = __builtin_bit_cast(float, odd ? a1 : a0);
            w1[k] = __builtin_bit_cast(float, odd ? b1 : b0);
        }
        const int pieces = 2 * nl;  // 4-entry pieces in this window
        float* wp = a.val + b + 4 * lane;
        if (lane < pieces) __builtin_nontemporal_store(w0, reinterpret_cast<f32x4*>(wp));
        if (lane + 64 < pieces) __builtin_nontemporal_store(w1, reinterpret_cast<f32x4*>(wp + 256));
    }
    if constexpr (MODE == kModeFlush) {
        float s2 = 0.0f;
#pragma unroll
        for (int k = 0; k < kE; ++k) s2 = __builtin_fmaf(r[k], r[k], s2);
        if (lv) wk.sse += (double)s2;
    } else {
        // A segment left open by the previous window that ended where this one starts.
        if (wk.cid >= 0 && wk.cid != wk.scur) {
            if (lane == 0) emit<P1>(a, wk, wk.cid, wk.cn, wk.cd);
            wk.cid = -1;
        }
        // Scan keys: segment + 1 of the lane's first (hk) and last (tk) entry, 0 on
        // lanes without entries.
        const int hk = lv ? idb + (int)(bits & 1u) + 1 : 0;
        const int tk = lv ? idb + nb + 1 : 0;
        float scn = an, scd = ad;
        seg_scan(tk, scn, scd);
        // Sums of this lane's first segment over earlier lanes, and from earlier windows.
        const int pk1 = dpp_i<kWaveShr1, 0xF, true>(0, tk);
        const float pn1 = dpp_f<kWaveShr1, 0xF, true>(0.0f, scn);
        const float pd1 = dpp_f<kWaveShr1, 0xF, true>(0.0f, scd);
        double hn = 0.0, hd = 0.0;
        if (pk1 == hk) {
            hn = (double)pn1;
            hd = (double)pd1;
        }
        if (hk == wk.cid + 1) {
            hn += wk.cn;
            hd += wk.cd;
        }
        // Entry k ends a segment when entry k + 1 starts one; the lane's last entry
        // when the next lane's first does.  The window's last entry stays open.
        const uint32_t nb0 = (uint32_t)dpp_i<kWaveShl1, 0xF, true>(0, (int)(bits & 1u));
        uint32_t ends = (bits >> 1) | ((lane + 1 < nl ? nb0 : 0u) << (kE - 1));
        if (!lv) ends = 0u;
        const uint32_t ff = bits ? (uint32_t)__builtin_ctz(bits) : (uint32_t)kE;  // head: k < ff
        // Emit one end per lane per round; most windows need one round.
        uint32_t rem = ends;
        while (__ballot(rem != 0u)) {
            if (rem != 0u) {
                const uint32_t k = (uint32_t)__builtin_ctz(rem);
                float vn = sn[0], vd = sd[0];
#pragma unroll
                for (int j = 1; j < kE; ++j)
                    if (k == (uint32_t)j) {
                        vn = sn[j];
                        vd = sd[j];
                    }
                double en = (double)vn, ed = (double)vd;
                if (k < ff) {
                    en += hn;
                    ed += hd;
                }
                const int s = idb + __builtin_popcount(bits & ((2u << k) - 1u));
                emit<P1>(a, wk, s, en, ed);
                rem &= rem - 1u;
            }
        }
        // The segment of the window's last entry stays open; one that started in that
        // lane has no earlier sums.
        const int ll = nl - 1;
        const double ln = (double)an + (bits == 0u ? hn : 0.0);
        const double ld = (double)ad + (bits == 0u ? hd : 0.0);
        wk.cid = __builtin_amdgcn_readlane(tk, ll) - 1;
        wk.cn = lane_f64(ln, ll);
        wk.cd = lane_f64(ld, ll);
    }
    wk.scur = scur_n;
    wk.elo = we;
}

// One wave's chunk [c0, c1) (whole segments, the first one scur), two windows per
// loop turn so the current and next window alternate between two register sets.
template <int MODE, bool STAGED, bool IDX16, bool P1>
__device__ __forceinline__ void run_chunk(const PassArgs& a, const Gather& gx, int64_t c0,
                                          int64_t c1, int scur, int flags, int gc, int lane,
                                          float* spr, float* sppr, uint32_t* bm, double& sse) {
    const uint32_t le = (uint32_t)lane * kE;
    Walk wk{c0, c1, scur, -1, 0.0, 0.0, sse, (flags & kChunkMid) ? scur : -1, a.nseg + 2 * gc};
    Win wa, wb;
    load_window<MODE, IDX16>(a, c0, c1, le, scur, lane, wa);
    while (true) {
        window<MODE, STAGED, IDX16, P1>(a, gx, wk, wa, wb, lane, le, spr, sppr, bm);
        if (wk.elo >= c1) break;
        window<MODE, STAGED, IDX16, P1>(a, gx, wk, wb, wa, lane, le, spr, sppr, bm);
        if (wk.elo >= c1) break;
    }
    if constexpr (MODE != kModeFlush) {
        // The last segment: finished, or going on past the chunk (a partial in the head
        // slot when it is also the segment that began earlier, else in the tail slot).
        if (wk.cid >= 0 && lane == 0) {
            if (flags & kChunkCont)
                a.part[wk.head + (wk.cid == wk.mid ? 0 : 1)] = make_double2(wk.cn, wk.cd);
            else
                emit<P1>(a, wk, wk.cid, wk.cn, wk.cd);
        }
    }
    sse = wk.sse;
}

// One pass: the workgroup's pieces in order, each staging its tile (when it
// differs from the one staged) and then giving every wave its chunk.
template <int MODE, bool STAGED, bool IDX16, bool P1>
__device__ __forceinline__ void pass_main(const PassArgs& a) {
    using N = Needs<MODE>;
    extern __shared__ float lds[];
    const int wg = blockIdx.x;

    Gather gx{};
    if constexpr (!STAGED) {
        const uint64_t vb = (uint64_t)a.cols * 4u;
        if (N::x) gx.gx = make_rsrc(a.x, vb);
        if (N::q) gx.gq = make_rsrc(a.q, vb);
        if (N::qq) gx.gqq = make_rsrc(a.qq, vb);
    }
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = (int)(threadIdx.x & 63u);
    uint32_t* scr = reinterpret_cast<uint32_t*>(lds + a.vec_floats) + wave * scratch_words(MODE);
    // Scratch layout (scratch_words): the bitmap, then the slots of p, then of pp.
    uint32_t* bm = scr;                                              // kWin / 32 words
    float* spr = reinterpret_cast<float*>(scr + kWin / 32);         // 64 row scalars p
    float* sppr = reinterpret_cast<float*>(scr + kWin / 32 + (N::p ? 64 : 0));  // 64 pp

    if constexpr (MODE != kModeFlush && P1) {
        // The rows after the last non-empty one have no entries: coordinate 0.
        for (int i = wg * kWG + (int)threadIdx.x; i < a.rows - a.nseg_ne; i += gridDim.x * kWG)
            a.y[a.nseg_ne + i] = coordinate(0.0, 0.0, a.lambda);
    }

    double sse = 0.0;
    int staged = -1;
    for (int pc = a.wg_piece[wg]; pc < a.wg_piece[wg + 1]; ++pc) {
        if constexpr (STAGED) {
            const int tile = a.piece_tile[pc];
            if (tile != staged) {
                if (staged >= 0) __syncthreads();  // every wave is done with the old slice
                stage_tile<MODE>(a, tile, lds, gx);
                __syncthreads();
                staged = tile;
            }
        }
        const int64_t c0 = a.piece_chunk[pc * (kWaves + 1) + wave];
        const int64_t c1 = a.piece_chunk[pc * (kWaves + 1) + wave + 1];
        const int gc = pc * kWaves + wave;
        if (c0 < c1)
            run_chunk<MODE, STAGED, IDX16, P1>(a, gx, c0, c1, a.piece_seg[gc], a.chunk_flags[gc],
                                               gc, lane, spr, sppr, bm, sse);
    }
    if constexpr (MODE == kModeFlush) {
        const double t = wave_sum(sse);
        if (lane == 0) a.sse_part[wg * kWaves + wave] = t;
    }
}

}  // namespace

// Distinct kernel names per pass kind, so that profiles separate them.  The
// template arguments select LDS staging, the index width and whether segments
// are rows (P == 1).
template <bool STAGED, bool IDX16, bool P1>
__global__ __launch_bounds__(kWG) void ccd_pass(PassArgs a) {
    pass_main<kModePlain, STAGED, IDX16, P1>(a);
}
template <bool STAGED, bool IDX16, bool P1>
__global__ __launch_bounds__(kWG) void ccd_pass_fused_first(PassArgs a) {
    pass_main<kModeAdd, STAGED, IDX16, P1>(a);
}
template <bool STAGED, bool IDX16, bool P1>
__global__ __launch_bounds__(kWG) void ccd_pass_fused(PassArgs a) {
    pass_main<kModeSubAdd, STAGED, IDX16, P1>(a);
}
template <bool STAGED, bool IDX16, bool P1>
__global__ __launch_bounds__(kWG) void ccd_flush(PassArgs a) {
    pass_main<kModeFlush, STAGED, IDX16, P1>(a);
}

// Fixed-order combine of a row's partials: one wave per row, lane k takes the
// row's partial slots k, k + 64, ... in entry order, then a fixed tree.  With
// yseg, the coordinate is also written to every segment of the row.
__global__ __launch_bounds__(256) void ccd_combine(CombineArgs c) {
    const int wave = (int)(threadIdx.x >> 6);
    const int lane = (int)(threadIdx.x & 63u);
    const int i = blockIdx.x * 4 + wave;
    if (i >= c.n) return;
    const int b = c.src_ptr[i];
    const int e = c.src_ptr[i + 1];
    double num = 0.0, den = 0.0;
    for (int k = b + lane; k < e; k += 64) {
        const double2 pv = c.part[c.srcs[k]];
        num += pv.x;
        den += pv.y;
    }
    num = wave_sum(num);
    den = wave_sum(den);
    const float yr = coordinate(num, den, c.lambda);
    if (lane == 0) c.y[c.ids ? c.ids[i] : i] = yr;
    if (c.yseg)
        for (int k = c.seg_ptr[i] + lane; k < c.seg_ptr[i + 1]; k += 64) c.yseg[c.segs[k]] = yr;
}

__global__ __launch_bounds__(256) void ccd_copy(const float* __restrict__ src,
                                                float* __restrict__ dst, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) dst[i] = src[i];
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
template <bool S, bool I, bool P1>
hipError_t raise_lds() {
    const void* ks[] = {(const void*)ccd_pass<S, I, P1>, (const void*)ccd_pass_fused_first<S, I, P1>,
                        (const void*)ccd_pass_fused<S, I, P1>, (const void*)ccd_flush<S, I, P1>};
    for (const void* k : ks) {
        hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <bool S, bool I, bool P1>
void launch_mode(PassMode mode, dim3 grid, size_t lds, hipStream_t s, const PassArgs& a) {
    switch (mode) {
        case kModePlain:
            hipLaunchKernelGGL((ccd_pass<S, I, P1>), grid, dim3(kWG), lds, s, a);
            break;
        case kModeAdd:
            hipLaunchKernelGGL((ccd_pass_fused_first<S, I, P1>), grid, dim3(kWG), lds, s, a);
            break;
        case kModeSubAdd:
            hipLaunchKernelGGL((ccd_pass_fused<S, I, P1>), grid, dim3(kWG), lds, s, a);
            break;
        case kModeFlush:
            hipLaunchKernelGGL((ccd_flush<S, I, P1>), grid, dim3(kWG), lds, s, a);
            break;
    }
}
}  // namespace

hipError_t sweep_init() {
    hipError_t e = raise_lds<true, true, true>();
    if (e == hipSuccess) e = raise_lds<true, true, false>();
    if (e == hipSuccess) e = raise_lds<false, true, true>();
    if (e == hipSuccess) e = raise_lds<false, false, true>();
    return e;
}

hipError_t launch_pass(const Layout& L, PassMode mode, const float* x, const float* p,
                       const float* pp, const float* q, const float* qq, float* y, double lambda,
                       double* sse_part, hipStream_t s) {
    if (L.grid == 0) return hipSuccess;
    const bool staged = L.gather == kGatherLds;
    // Kernel variants: LDS staging uses 16-bit indices; global gathers have P == 1.
    if (staged ? !L.idx16 : L.P != 1) return hipErrorInvalidValue;
    PassArgs a{};
    a.idx = L.idx;
    a.val = L.val;
    a.seg_start = L.seg_start;
    a.wg_piece = L.wg_piece;
    a.piece_tile = L.piece_tile;
    a.piece_chunk = L.piece_chunk;
    a.piece_seg = L.piece_seg;
    a.chunk_flags = L.chunk_flags;
    a.x = x;
    a.p = p;
    a.pp = pp;
    a.q = q;
    a.qq = qq;
    a.y = y;
    a.part = L.part;
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
    a.vec_floats = staged ? staged_vectors(mode, a.x_is_q) * a.Ts : 0;
    const size_t lds = (size_t)a.vec_floats * sizeof(float) + (size_t)kWaves * scratch_words(mode) * 4;
    if (lds > (size_t)kLdsBytes) return hipErrorInvalidValue;
    const dim3 grid(L.grid);
    if (staged) {
        if (L.P == 1)
            launch_mode<true, true, true>(mode, grid, lds, s, a);
        else
            launch_mode<true, true, false>(mode, grid, lds, s, a);
    } else if (L.idx16) {
        launch_mode<false, true, true>(mode, grid, lds, s, a);
    } else {
        launch_mode<false, false, true>(mode, grid, lds, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_combine(const Layout& L, float* y, float* yseg, double lambda, hipStream_t s) {
    if (L.ncomb == 0) return hipSuccess;
    if (yseg && !L.row_seg_ptr) return hipErrorInvalidValue;
    CombineArgs c{};
    c.ids = L.comb_rows;
    c.src_ptr = L.src_ptr;
    c.srcs = L.srcs;
    c.seg_ptr = L.row_seg_ptr;
    c.segs = L.row_segs;
    c.part = L.part;
    c.y = y;
    c.yseg = yseg;
    c.n = L.ncomb;
    c.lambda = lambda;
    hipLaunchKernelGGL(ccd_combine, dim3((unsigned)((L.ncomb + 3) / 4)), dim3(256), 0, s, c);
    return hipGetLastError();
}

hipError_t launch_copy(const float* src, float* dst, int64_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(ccd_copy, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, dst, n);
    return hipGetLastError();
}

hipError_t launch_reduce_sum(const double* part, int32_t n, double* out, hipStream_t s) {
    hipLaunchKernelGGL(ccd_reduce_sum, dim3(1), dim3(256), 0, s, part, n, out);
    return hipGetLastError();
}

}  // namespace ccdk
