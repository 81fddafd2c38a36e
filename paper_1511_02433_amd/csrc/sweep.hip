// CCD++ sweep passes for gfx950 (MI355X).
//
// One launch is one pass over one compressed copy of the residual:
//   - a u-pass over the row-compressed copy evaluates eq. 15 for every row i,
//   - a v-pass over the column-compressed copy evaluates eq. 16 for every
//     column j (read with u_i, the minimiser of eq. 14 in v_j),
// in the data-parallel form of Section 6 (eq. 20, 21): every row or column is
// an independent unit of work.  The first pass of a feature over each copy
// also folds in the residual bookkeeping of Algorithm 3: the pending eq. 18
// subtract of the previous feature and the eq. 13 add-back of the current one,
// evaluated as fma(p, q, fma(-pp, qq, val)).  Both copies evaluate that same
// expression on the same operands, so they stay bitwise identical.
//
// Memory: index and value arrays are streamed with non-temporal buffer loads
// (each entry is touched once per pass) so that the gathered vectors stay in
// L2.  Every buffer descriptor is rebased to the workgroup's own entry range
// with an exact byte limit: a lane can never touch memory outside its rows,
// and masked lanes use an out-of-range offset, which the hardware turns into a
// zero load or a dropped store.
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
constexpr int kRsrcWord3 = 0x00020000;  // raw 32-bit dword buffer, gfx9 family
constexpr uint32_t kOOB = 0xFFFFFFFFu;  // offset past any limit: load 0 / drop store
constexpr int kNT = 2;                  // non-temporal cache policy (streamed once)

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint64_t bytes) {
    uint32_t lim = bytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)lim,
                                            kRsrcWord3);
}
template <int AUX>
__device__ __forceinline__ int32_t ld_i32(rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, AUX);
}
template <int AUX>
__device__ __forceinline__ float ld_f32(rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, AUX));
}
__device__ __forceinline__ int64_t ld_i64(rsrc_t r, uint32_t off) {
    auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
    return __builtin_bit_cast(int64_t, v);
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

// ---- per-entry step ----------------------------------------------------------
// One entry: apply the residual bookkeeping of the mode, store it, accumulate.
template <int MODE>
__device__ __forceinline__ void entry(bool ok, float rv, float xv, float qv, float qqv, float pr,
                                      float ppr, rsrc_t rval, uint32_t off, double& num,
                                      double& den) {
    float r = rv;
    if constexpr (MODE == kModeAdd) r = __builtin_fmaf(pr, qv, rv);
    if constexpr (MODE == kModeSubAdd) r = __builtin_fmaf(pr, qv, __builtin_fmaf(-ppr, qqv, rv));
    if constexpr (MODE == kModeFlush) r = __builtin_fmaf(-ppr, qqv, rv);
    if constexpr (MODE != kModePlain) st_f32<kNT>(r, rval, off);  // masked lanes: kOOB, dropped
    if constexpr (MODE == kModeFlush) {
        double d = ok ? (double)r : 0.0;
        num = __builtin_fma(d, d, num);
    } else {
        double dx = ok ? (double)xv : 0.0;
        num = __builtin_fma((double)r, dx, num);
        den = __builtin_fma(dx, dx, den);
    }
}

// E entries per lane at positions base + lane + e*STRIDE (relative to the
// workgroup's rebased descriptors), all loads issued before any use.
template <int MODE, int E, int STRIDE>
__device__ __forceinline__ void run_entries(const PassArgs& a, rsrc_t ridx, rsrc_t rval,
                                            rsrc_t rx, rsrc_t rq, rsrc_t rqq, uint32_t first,
                                            uint32_t end, float pr, float ppr, double& num,
                                            double& den) {
    constexpr bool kFused = MODE != kModePlain;
    constexpr bool kGatherX = MODE != kModeFlush;
    constexpr bool kNeedQ = MODE == kModeAdd || MODE == kModeSubAdd;
    constexpr bool kNeedQQ = MODE == kModeSubAdd || MODE == kModeFlush;
    uint32_t off[E];
    int32_t c[E];
    float rv[E], xv[E], qv[E], qqv[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        uint32_t pos = first + (uint32_t)(e * STRIDE);
        off[e] = pos < end ? pos * 4u : kOOB;
    }
#pragma unroll
    for (int e = 0; e < E; ++e) c[e] = ld_i32<kNT>(ridx, off[e]);
#pragma unroll
    for (int e = 0; e < E; ++e) rv[e] = ld_f32<kNT>(rval, off[e]);
#pragma unroll
    for (int e = 0; e < E; ++e) {
        uint32_t g = (uint32_t)c[e] * 4u;
        xv[e] = kGatherX ? ld_f32<0>(rx, g) : 0.0f;
        qv[e] = kNeedQ ? ld_f32<0>(rq, g) : 0.0f;
        qqv[e] = kNeedQQ ? ld_f32<0>(rqq, g) : 0.0f;
    }
#pragma unroll
    for (int e = 0; e < E; ++e)
        entry<MODE>(off[e] != kOOB, rv[e], xv[e], qv[e], qqv[e], pr, ppr, rval, off[e], num, den);
    (void)kFused;
}

// ---- lane-group classes: G lanes per row, E entries per lane ---------------------
template <int MODE, int G, int E>
__device__ __forceinline__ void group_rows(const PassArgs& a, const Seg& sg, int blk,
                                           double* lds) {
    constexpr int kRowsPerBlock = kBlock / G;
    const int tid = threadIdx.x;
    const int lane = tid % G;
    const int grp = tid / G;
    const int r0 = sg.row_begin + (blk - sg.block_begin) * kRowsPerBlock;
    const int r1 = min(r0 + kRowsPerBlock, sg.row_end);
    const int r = r0 + grp;
    const bool valid = r < r1;

    const rsrc_t rptr = make_rsrc(a.ptr, (uint64_t)(a.rows + 1) * 8u);
    const int64_t blo = a.ptr[r0];
    const int64_t bhi = a.ptr[r1];
    const rsrc_t ridx = make_rsrc(a.idx + blo, (uint64_t)(bhi - blo) * 4u);
    const rsrc_t rval = make_rsrc(a.val + blo, (uint64_t)(bhi - blo) * 4u);
    const rsrc_t rx = make_rsrc(a.x, (uint64_t)a.cols * 4u);
    const rsrc_t rq = make_rsrc(a.q, (uint64_t)a.cols * 4u);
    const rsrc_t rqq = make_rsrc(a.qq, (uint64_t)a.cols * 4u);
    const rsrc_t rrow = make_rsrc(a.p, (uint64_t)a.rows * 4u);
    const rsrc_t rrow2 = make_rsrc(a.pp, (uint64_t)a.rows * 4u);

    const uint32_t roff8 = valid ? (uint32_t)r * 8u : kOOB;
    const int64_t lo = ld_i64(rptr, roff8);
    const int64_t hi = valid ? ld_i64(rptr, roff8 + 8u) : lo;
    // Invalid groups get an empty range, so every one of their entries is masked.
    const uint32_t first = valid ? (uint32_t)(lo - blo) + (uint32_t)lane : 0u;
    const uint32_t end = valid ? (uint32_t)(hi - blo) : 0u;
    const uint32_t roff4 = valid ? (uint32_t)r * 4u : kOOB;
    float pr = 0.0f, ppr = 0.0f;
    if constexpr (MODE == kModeAdd || MODE == kModeSubAdd) pr = ld_f32<0>(rrow, roff4);
    if constexpr (MODE == kModeSubAdd || MODE == kModeFlush) ppr = ld_f32<0>(rrow2, roff4);

    double num = 0.0, den = 0.0;
    run_entries<MODE, E, G>(a, ridx, rval, rx, rq, rqq, first, end, pr, ppr, num, den);

    if constexpr (MODE == kModeFlush) {
        // Workgroup sum of squares: wave sums, then the 4 waves in order.
        double s = group_sum<64>(num);
        if ((tid & 63) == 0) lds[tid >> 6] = s;
        __syncthreads();
        if (tid == 0) a.sse_part[blockIdx.x] = ((lds[0] + lds[1]) + lds[2]) + lds[3];
    } else {
        num = group_sum<G>(num);
        den = group_sum<G>(den);
        if (valid && lane == 0) {
            const rsrc_t ry = make_rsrc(a.y, (uint64_t)a.rows * 4u);
            st_f32<0>(coordinate(num, den, a.lambda), ry, (uint32_t)r * 4u);
        }
    }
}

// ---- workgroup class: one 256-thread workgroup per row piece ----------------------
template <int MODE>
__device__ __forceinline__ void block_piece(const PassArgs& a, const Seg& sg, int blk,
                                            double* lds) {
    const int tid = threadIdx.x;
    const int piece = sg.row_begin + (blk - sg.block_begin);
    const int r = a.piece_row[piece];
    const int64_t lo = a.piece_lo[piece];
    const int64_t hi = a.piece_lo[piece + 1];
    const int64_t rlo = a.ptr[r];
    const int64_t rhi = a.ptr[r + 1];
    const bool whole = (lo == rlo) && (hi == rhi);
    const uint32_t len = (uint32_t)(hi - lo);

    const rsrc_t ridx = make_rsrc(a.idx + lo, (uint64_t)len * 4u);
    const rsrc_t rval = make_rsrc(a.val + lo, (uint64_t)len * 4u);
    const rsrc_t rx = make_rsrc(a.x, (uint64_t)a.cols * 4u);
    const rsrc_t rq = make_rsrc(a.q, (uint64_t)a.cols * 4u);
    const rsrc_t rqq = make_rsrc(a.qq, (uint64_t)a.cols * 4u);
    float pr = 0.0f, ppr = 0.0f;
    if constexpr (MODE == kModeAdd || MODE == kModeSubAdd) pr = a.p[r];
    if constexpr (MODE == kModeSubAdd || MODE == kModeFlush) ppr = a.pp[r];

    double num = 0.0, den = 0.0;
    for (uint32_t base = 0; base < len; base += kBlockStep)
        run_entries<MODE, kBlockUnroll, kBlock>(a, ridx, rval, rx, rq, rqq, base + tid, len, pr,
                                                ppr, num, den);

    double s0 = group_sum<64>(num);
    double s1 = MODE == kModeFlush ? 0.0 : group_sum<64>(den);
    if ((tid & 63) == 0) {
        lds[tid >> 6] = s0;
        lds[4 + (tid >> 6)] = s1;
    }
    __syncthreads();
    if (tid == 0) {
        double tn = ((lds[0] + lds[1]) + lds[2]) + lds[3];
        double td = ((lds[4] + lds[5]) + lds[6]) + lds[7];
        if constexpr (MODE == kModeFlush) {
            a.sse_part[blockIdx.x] = tn;
        } else if (whole) {
            a.y[r] = coordinate(tn, td, a.lambda);
        } else {
            a.part[piece] = make_double2(tn, td);
        }
    }
}

template <int MODE>
__device__ __forceinline__ void pass_body(const PassArgs& a) {
    __shared__ double lds[8];
    const int blk = blockIdx.x;
    int s = 0;
#pragma unroll
    for (int i = 1; i < kMaxSegs; ++i)
        if (i < a.nseg && blk >= a.seg[i].block_begin) s = i;
    const Seg sg = a.seg[s];
    switch (sg.kind) {
        case kSegBlock: block_piece<MODE>(a, sg, blk, lds); break;
        case kSegG1E8: group_rows<MODE, 1, 8>(a, sg, blk, lds); break;
        case kSegG2E8: group_rows<MODE, 2, 8>(a, sg, blk, lds); break;
        case kSegG4E8: group_rows<MODE, 4, 8>(a, sg, blk, lds); break;
        case kSegG8E8: group_rows<MODE, 8, 8>(a, sg, blk, lds); break;
        case kSegG16E8: group_rows<MODE, 16, 8>(a, sg, blk, lds); break;
        case kSegG32E8: group_rows<MODE, 32, 8>(a, sg, blk, lds); break;
        case kSegG64E8: group_rows<MODE, 64, 8>(a, sg, blk, lds); break;
        case kSegG64E16: group_rows<MODE, 64, 16>(a, sg, blk, lds); break;
        default: break;
    }
}

}  // namespace

// Distinct kernel names so that profiles separate the pass kinds.
__global__ __launch_bounds__(kBlock) void ccd_pass(PassArgs a) { pass_body<kModePlain>(a); }
__global__ __launch_bounds__(kBlock) void ccd_pass_fused_first(PassArgs a) {
    pass_body<kModeAdd>(a);
}
__global__ __launch_bounds__(kBlock) void ccd_pass_fused(PassArgs a) {
    pass_body<kModeSubAdd>(a);
}
__global__ __launch_bounds__(kBlock) void ccd_flush(PassArgs a) { pass_body<kModeFlush>(a); }

// Fixed-order combine of the pieces of split rows (one thread per row).
__global__ __launch_bounds__(kBlock) void ccd_combine(CombineArgs c) {
    const int s = blockIdx.x * kBlock + threadIdx.x;
    if (s >= c.nsplit) return;
    const int r = c.split_row[s];
    double num = 0.0, den = 0.0;
    for (int p = c.split_first[s]; p < c.split_first[s + 1]; ++p) {
        num += c.part[p].x;
        den += c.part[p].y;
    }
    c.y[r] = coordinate(num, den, c.lambda);
}

__global__ __launch_bounds__(kBlock) void ccd_copy(const float* __restrict__ src,
                                                   float* __restrict__ dst, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i < n) dst[i] = src[i];
}

// Single-workgroup fixed-order sum: thread t sums part[t], part[t+256], ... in
// order, then a fixed tree over the 256 thread sums.
__global__ __launch_bounds__(kBlock) void ccd_reduce_sum(const double* __restrict__ part,
                                                         int32_t n, double* __restrict__ out) {
    __shared__ double s[kBlock];
    double acc = 0.0;
    for (int32_t i = threadIdx.x; i < n; i += kBlock) acc += part[i];
    s[threadIdx.x] = acc;
    __syncthreads();
    for (int w = kBlock / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) s[threadIdx.x] += s[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[0] = s[0];
}

hipError_t launch_pass(const Layout& L, PassMode mode, const float* x, const float* p,
                       const float* pp, const float* q, const float* qq, float* y, double lambda,
                       double* sse_part, hipStream_t s) {
    if (L.grid == 0) return hipSuccess;
    PassArgs a{};
    a.ptr = L.ptr;
    a.idx = L.idx;
    a.val = L.val;
    a.x = x;
    a.p = p;
    a.pp = pp;
    a.q = q;
    a.qq = qq;
    a.y = y;
    a.part = L.part;
    a.sse_part = sse_part;
    a.piece_row = L.piece_row;
    a.piece_lo = L.piece_lo;
    a.rows = (int32_t)L.rows;
    a.cols = (int32_t)L.cols;
    a.lambda = lambda;
    a.nseg = (int32_t)L.segs.size();
    for (size_t i = 0; i < L.segs.size(); ++i) a.seg[i] = L.segs[i];
    dim3 grid(L.grid), block(kBlock);
    switch (mode) {
        case kModePlain: hipLaunchKernelGGL(ccd_pass, grid, block, 0, s, a); break;
        case kModeAdd: hipLaunchKernelGGL(ccd_pass_fused_first, grid, block, 0, s, a); break;
        case kModeSubAdd: hipLaunchKernelGGL(ccd_pass_fused, grid, block, 0, s, a); break;
        case kModeFlush: hipLaunchKernelGGL(ccd_flush, grid, block, 0, s, a); break;
    }
    return hipGetLastError();
}

hipError_t launch_combine(const Layout& L, float* y, double lambda, hipStream_t s) {
    if (L.nsplit == 0) return hipSuccess;
    CombineArgs c{};
    c.split_row = L.split_row;
    c.split_first = L.split_first;
    c.part = L.part;
    c.y = y;
    c.lambda = lambda;
    c.nsplit = L.nsplit;
    hipLaunchKernelGGL(ccd_combine, dim3((L.nsplit + kBlock - 1) / kBlock), dim3(kBlock), 0, s, c);
    return hipGetLastError();
}

hipError_t launch_copy(const float* src, float* dst, int64_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(ccd_copy, dim3((unsigned)((n + kBlock - 1) / kBlock)), dim3(kBlock), 0, s,
                       src, dst, n);
    return hipGetLastError();
}

hipError_t launch_reduce_sum(const double* part, int32_t n, double* out, hipStream_t s) {
    hipLaunchKernelGGL(ccd_reduce_sum, dim3(1), dim3(kBlock), 0, s, part, n, out);
    return hipGetLastError();
}

}  // namespace ccdk
