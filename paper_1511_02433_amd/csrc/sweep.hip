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
// Memory: index and value arrays are streamed with non-temporal buffer loads
// (each entry is touched once per pass).  The vectors a pass gathers from are
// staged tile by tile in LDS by persistent workgroups (see ccdpp_internal.hpp),
// so a random gather costs an LDS read; layouts too sparse for tiling gather
// through L2 instead.  Buffer descriptors are rebased to each wave's own entry
// range with an exact byte limit, and masked lanes use an out-of-range offset,
// which the hardware turns into a zero load or a dropped store.
//
// Arithmetic: R-hat in fp32 FMA; sums of R-hat*x and x^2 in fp64 with a fixed
// reduction tree, so results are identical run to run; the coordinate
// num / (lambda + den) is an IEEE fp64 division rounded once to fp32.  A
// coordinate whose denominator is exactly zero (lambda = 0 and an empty row)
// is set to zero.
#include "ccdpp_internal.hpp"

namespace ccdk {
namespace {

using rsrc_t = __amdgpu_buffer_rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, gfx9 family
constexpr uint32_t kOOB = 0xFFFFFFFFu;  // offset past any limit: load 0 / drop store
constexpr int kNT = 2;                  // non-temporal cache policy (streamed once)

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint64_t bytes) {
    uint32_t lim = bytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)lim,
                                            kRsrcWord3);
}
template <int AUX>
__device__ __forceinline__ float ld_f32(rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, AUX));
}
template <bool IDX16>
__device__ __forceinline__ uint32_t ld_idx(rsrc_t r, uint32_t off) {
    if constexpr (IDX16)
        return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, kNT);
    else
        return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kNT);
}
template <int AUX>
__device__ __forceinline__ void st_f32(float v, rsrc_t r, uint32_t off) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int32_t, v), r, off, 0, AUX);
}

// ---- cross-lane sums -------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ double dpp_d(double x) {
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
// Sum over aligned groups of G lanes; every lane of a group gets the same bits.
template <int G>
__device__ __forceinline__ double group_sum(double x) {
    if constexpr (G >= 2) x += dpp_d<0xB1>(x);    // quad_perm [1,0,3,2]: lane ^ 1
    if constexpr (G >= 4) x += dpp_d<0x4E>(x);    // quad_perm [2,3,0,1]: lane ^ 2
    if constexpr (G >= 8) x += dpp_d<0x141>(x);   // row_half_mirror: the other quad of 8
    if constexpr (G >= 16) x += dpp_d<0x140>(x);  // row_mirror: the other half of 16
    if constexpr (G >= 32) x = xor16_sum(x);
    if constexpr (G >= 64) x = xor32_sum(x);
    return x;
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
        return ld_f32<0>(g, c * 4u);
}

// One entry: apply the residual bookkeeping of the mode, store it, accumulate.
template <int MODE>
__device__ __forceinline__ void entry(bool ok, float rv, float xv, float qv, float qqv, float pr,
                                      float ppr, rsrc_t rval, uint32_t voff, double& num,
                                      double& den) {
    float r = rv;
    if constexpr (MODE == kModeAdd) r = __builtin_fmaf(pr, qv, rv);
    if constexpr (MODE == kModeSubAdd) r = __builtin_fmaf(pr, qv, __builtin_fmaf(-ppr, qqv, rv));
    if constexpr (MODE == kModeFlush) r = __builtin_fmaf(-ppr, qqv, rv);
    if constexpr (MODE != kModePlain) st_f32<kNT>(r, rval, voff);  // masked lanes: kOOB, dropped
    if constexpr (MODE == kModeFlush) {
        double d = ok ? (double)r : 0.0;
        num = __builtin_fma(d, d, num);
    } else {
        double dx = ok ? (double)xv : 0.0;
        num = __builtin_fma((double)r, dx, num);
        den = __builtin_fma(dx, dx, den);
    }
}

// E entries per lane at positions first + e * STRIDE (relative to the wave's
// rebased descriptors, valid below `end`); every load is issued before any use.
template <int MODE, bool STAGED, bool IDX16, int E, int STRIDE>
__device__ __forceinline__ void run_entries(rsrc_t ridx, rsrc_t rval, const Gather& gx,
                                            uint32_t first, uint32_t end, float pr, float ppr,
                                            double& num, double& den) {
    using N = Needs<MODE>;
    constexpr uint32_t kIB = IDX16 ? 2u : 4u;
    bool ok[E];
    uint32_t voff[E];
    uint32_t c[E];
    float rv[E], xv[E], qv[E], qqv[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const uint32_t pos = first + (uint32_t)(e * STRIDE);
        ok[e] = pos < end;
        voff[e] = ok[e] ? pos * 4u : kOOB;
        c[e] = ld_idx<IDX16>(ridx, ok[e] ? pos * kIB : kOOB);
    }
#pragma unroll
    for (int e = 0; e < E; ++e) rv[e] = ld_f32<kNT>(rval, voff[e]);
#pragma unroll
    for (int e = 0; e < E; ++e) {
        xv[e] = N::x ? gat<STAGED>(gx.lx, gx.gx, c[e]) : 0.0f;
        qv[e] = N::q ? gat<STAGED>(gx.lq, gx.gq, c[e]) : 0.0f;
        qqv[e] = N::qq ? gat<STAGED>(gx.lqq, gx.gqq, c[e]) : 0.0f;
    }
#pragma unroll
    for (int e = 0; e < E; ++e)
        entry<MODE>(ok[e], rv[e], xv[e], qv[e], qqv[e], pr, ppr, rval, voff[e], num, den);
}

template <int MODE>
__device__ __forceinline__ void emit(const PassArgs& a, int s, int row, double num, double den) {
    if (a.P == 1)
        a.y[row] = coordinate(num, den, a.lambda);
    else
        a.part[s] = make_double2(num, den);
}

// A unit of up to 64/G short segments, G lanes each, E entries per lane.
template <int MODE, bool STAGED, bool IDX16, int G, int E>
__device__ __forceinline__ void unit_groups(const PassArgs& a, const Gather& gx, int s0, int cnt,
                                            int lane, double& sse) {
    using N = Needs<MODE>;
    constexpr uint32_t kIB = IDX16 ? 2u : 4u;
    const int g = lane / G;
    const int l = lane % G;
    const bool valid = g < cnt;
    const int s = s0 + (valid ? g : cnt - 1);
    const int64_t wlo = a.seg_start[s0];
    const int64_t whi = a.seg_start[s0 + cnt];
    const uint64_t wlen = (uint64_t)(whi - wlo);
    const rsrc_t ridx = make_rsrc(static_cast<const char*>(a.idx) + wlo * kIB, wlen * kIB);
    const rsrc_t rval = make_rsrc(a.val + wlo, wlen * 4u);
    const int64_t lo = a.seg_start[s];
    const int64_t hi = a.seg_start[s + 1];
    const uint32_t first = valid ? (uint32_t)(lo - wlo) + (uint32_t)l : 0u;
    const uint32_t end = valid ? (uint32_t)(hi - wlo) : 0u;
    const int row = a.seg_row[s];
    float pr = 0.0f, ppr = 0.0f;
    if constexpr (N::p) pr = a.p[row];
    if constexpr (N::pp) ppr = a.pp[row];
    double num = 0.0, den = 0.0;
    run_entries<MODE, STAGED, IDX16, E, G>(ridx, rval, gx, first, end, pr, ppr, num, den);
    if constexpr (MODE == kModeFlush) {
        sse += num;
    } else {
        num = group_sum<G>(num);
        den = group_sum<G>(den);
        if (valid && l == 0) emit<MODE>(a, s, row, num, den);
    }
}

// One long segment walked by the whole wave.
template <int MODE, bool STAGED, bool IDX16>
__device__ __forceinline__ void unit_long(const PassArgs& a, const Gather& gx, int s, int lane,
                                          double& sse) {
    using N = Needs<MODE>;
    constexpr uint32_t kIB = IDX16 ? 2u : 4u;
    constexpr int E = (MODE == kModeAdd || MODE == kModeSubAdd) ? kLongE / 2 : kLongE;
    const int64_t lo = a.seg_start[s];
    const int64_t hi = a.seg_start[s + 1];
    const uint32_t len = (uint32_t)(hi - lo);
    const rsrc_t ridx = make_rsrc(static_cast<const char*>(a.idx) + lo * kIB, (uint64_t)len * kIB);
    const rsrc_t rval = make_rsrc(a.val + lo, (uint64_t)len * 4u);
    const int row = a.seg_row[s];
    float pr = 0.0f, ppr = 0.0f;
    if constexpr (N::p) pr = a.p[row];
    if constexpr (N::pp) ppr = a.pp[row];
    double num = 0.0, den = 0.0;
    for (uint32_t base = 0; base < len; base += 64u * E)
        run_entries<MODE, STAGED, IDX16, E, 64>(ridx, rval, gx, base + (uint32_t)lane, len, pr, ppr,
                                                num, den);
    if constexpr (MODE == kModeFlush) {
        sse += num;
    } else {
        num = group_sum<64>(num);
        den = group_sum<64>(den);
        if (lane == 0) emit<MODE>(a, s, row, num, den);
    }
}

template <int MODE, bool STAGED, bool IDX16>
__device__ __forceinline__ void pass_main(const PassArgs& a) {
    using N = Needs<MODE>;
    extern __shared__ float lds[];
    const int wg = blockIdx.x;
    const int tile = a.wg_tile[wg];
    const int rank = a.wg_rank[wg];
    const int nwg = a.tile_nwg[tile];
    const int ub = a.tile_unit[tile];
    const int ue = a.tile_unit[tile + 1];

    Gather gx{};
    if constexpr (STAGED) {
        // Slots in the order x, q, qq; x shares q's slot when they are the same vector.
        const int T = a.T;
        const int c0 = tile * T;
        const int len = min(T, a.cols - c0);
        const bool alias = N::x && N::q && a.x_is_q;
        int slot = 0;
        float* sx = nullptr;
        float* sq = nullptr;
        float* sqq = nullptr;
        if (N::x && !alias) sx = lds + (slot++) * T;
        if (N::q) sq = lds + (slot++) * T;
        if (alias) sx = sq;
        if (N::qq) sqq = lds + (slot++) * T;
        for (int i = threadIdx.x; i < len; i += kWG) {
            if (N::x && !alias) sx[i] = a.x[c0 + i];
            if (N::q) sq[i] = a.q[c0 + i];
            if (N::qq) sqq[i] = a.qq[c0 + i];
        }
        __syncthreads();
        gx.lx = sx;
        gx.lq = sq;
        gx.lqq = sqq;
    } else {
        const uint64_t vb = (uint64_t)a.cols * 4u;
        if (N::x) gx.gx = make_rsrc(a.x, vb);
        if (N::q) gx.gq = make_rsrc(a.q, vb);
        if (N::qq) gx.gqq = make_rsrc(a.qq, vb);
    }

    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = (int)(threadIdx.x & 63u);
    double sse = 0.0;
    for (int u = ub + rank * kWaves + wave; u < ue; u += nwg * kWaves) {
        const int2 ud = a.units[u];
        const int kind = ud.y & 0xFF;
        const int cnt = ud.y >> 8;
        switch (kind) {
            case kULong: unit_long<MODE, STAGED, IDX16>(a, gx, ud.x, lane, sse); break;
            case kUG64E16: unit_groups<MODE, STAGED, IDX16, 64, 16>(a, gx, ud.x, cnt, lane, sse); break;
            case kUG64E8: unit_groups<MODE, STAGED, IDX16, 64, 8>(a, gx, ud.x, cnt, lane, sse); break;
            case kUG32E8: unit_groups<MODE, STAGED, IDX16, 32, 8>(a, gx, ud.x, cnt, lane, sse); break;
            case kUG16E8: unit_groups<MODE, STAGED, IDX16, 16, 8>(a, gx, ud.x, cnt, lane, sse); break;
            case kUG8E8: unit_groups<MODE, STAGED, IDX16, 8, 8>(a, gx, ud.x, cnt, lane, sse); break;
            case kUG4E8: unit_groups<MODE, STAGED, IDX16, 4, 8>(a, gx, ud.x, cnt, lane, sse); break;
            case kUG2E8: unit_groups<MODE, STAGED, IDX16, 2, 8>(a, gx, ud.x, cnt, lane, sse); break;
            default: unit_groups<MODE, STAGED, IDX16, 1, 8>(a, gx, ud.x, cnt, lane, sse); break;
        }
    }
    if constexpr (MODE == kModeFlush) {
        const double t = group_sum<64>(sse);
        if (lane == 0) a.sse_part[wg * kWaves + wave] = t;
    }
}

}  // namespace

// Distinct kernel names per pass kind, so that profiles separate them.  The
// template arguments select LDS staging and the index width.
template <bool STAGED, bool IDX16>
__global__ __launch_bounds__(kWG) void ccd_pass(PassArgs a) {
    pass_main<kModePlain, STAGED, IDX16>(a);
}
template <bool STAGED, bool IDX16>
__global__ __launch_bounds__(kWG) void ccd_pass_fused_first(PassArgs a) {
    pass_main<kModeAdd, STAGED, IDX16>(a);
}
template <bool STAGED, bool IDX16>
__global__ __launch_bounds__(kWG) void ccd_pass_fused(PassArgs a) {
    pass_main<kModeSubAdd, STAGED, IDX16>(a);
}
template <bool STAGED, bool IDX16>
__global__ __launch_bounds__(kWG) void ccd_flush(PassArgs a) {
    pass_main<kModeFlush, STAGED, IDX16>(a);
}

// Fixed-order combine of the per-tile partials of each row: one wave per row,
// lane k takes the row's segments k, k + 64, ... in tile order, then a fixed tree.
__global__ __launch_bounds__(256) void ccd_combine(CombineArgs c) {
    const int wave = (int)(threadIdx.x >> 6);
    const int lane = (int)(threadIdx.x & 63u);
    const int r = blockIdx.x * 4 + wave;
    if (r >= c.rows) return;
    const int b = c.row_seg_ptr[r];
    const int e = c.row_seg_ptr[r + 1];
    double num = 0.0, den = 0.0;
    for (int k = b + lane; k < e; k += 64) {
        const double2 pv = c.part[c.row_segs[k]];
        num += pv.x;
        den += pv.y;
    }
    num = group_sum<64>(num);
    den = group_sum<64>(den);
    if (lane == 0) c.y[r] = coordinate(num, den, c.lambda);
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
template <bool S, bool I>
hipError_t raise_lds() {
    const void* ks[] = {(const void*)ccd_pass<S, I>, (const void*)ccd_pass_fused_first<S, I>,
                        (const void*)ccd_pass_fused<S, I>, (const void*)ccd_flush<S, I>};
    for (const void* k : ks) {
        hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <bool S, bool I>
void launch_mode(PassMode mode, dim3 grid, size_t lds, hipStream_t s, const PassArgs& a) {
    switch (mode) {
        case kModePlain: hipLaunchKernelGGL((ccd_pass<S, I>), grid, dim3(kWG), lds, s, a); break;
        case kModeAdd: hipLaunchKernelGGL((ccd_pass_fused_first<S, I>), grid, dim3(kWG), lds, s, a); break;
        case kModeSubAdd: hipLaunchKernelGGL((ccd_pass_fused<S, I>), grid, dim3(kWG), lds, s, a); break;
        case kModeFlush: hipLaunchKernelGGL((ccd_flush<S, I>), grid, dim3(kWG), lds, s, a); break;
    }
}
}  // namespace

hipError_t sweep_init() {
    hipError_t e = raise_lds<true, true>();
    if (e != hipSuccess) return e;
    e = raise_lds<false, true>();
    if (e != hipSuccess) return e;
    return raise_lds<false, false>();
}

hipError_t launch_pass(const Layout& L, PassMode mode, const float* x, const float* p,
                       const float* pp, const float* q, const float* qq, float* y, double lambda,
                       double* sse_part, hipStream_t s) {
    if (L.grid == 0) return hipSuccess;
    PassArgs a{};
    a.idx = L.idx;
    a.val = L.val;
    a.seg_start = L.seg_start;
    a.seg_row = L.seg_row;
    a.units = L.units;
    a.wg_tile = L.wg_tile;
    a.wg_rank = L.wg_rank;
    a.tile_unit = L.tile_unit;
    a.tile_nwg = L.tile_nwg;
    a.x = x;
    a.p = p;
    a.pp = pp;
    a.q = q;
    a.qq = qq;
    a.y = y;
    a.part = L.part;
    a.sse_part = sse_part;
    a.nnz = L.nnz;
    a.rows = (int32_t)L.rows;
    a.cols = (int32_t)L.cols;
    a.T = L.T;
    a.P = L.P;
    a.nseg = (int32_t)L.nseg;
    a.x_is_q = (x != nullptr && x == q) ? 1 : 0;
    a.lambda = lambda;
    const dim3 grid(L.grid);
    if (L.gather == kGatherLds) {
        const size_t lds = (size_t)staged_vectors(mode, a.x_is_q) * L.T * sizeof(float);
        if (lds > (size_t)kLdsBytes) return hipErrorInvalidValue;
        launch_mode<true, true>(mode, grid, lds, s, a);
    } else if (L.idx16) {
        launch_mode<false, true>(mode, grid, 0, s, a);
    } else {
        launch_mode<false, false>(mode, grid, 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_combine(const Layout& L, float* y, double lambda, hipStream_t s) {
    if (L.P <= 1 || L.rows == 0) return hipSuccess;
    CombineArgs c{};
    c.row_seg_ptr = L.row_seg_ptr;
    c.row_segs = L.row_segs;
    c.part = L.part;
    c.y = y;
    c.rows = (int32_t)L.rows;
    c.lambda = lambda;
    hipLaunchKernelGGL(ccd_combine, dim3((unsigned)((L.rows + 3) / 4)), dim3(256), 0, s, c);
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
