// Device-side construction of the compressed residual copies and the utility
// kernels of the CCD++ library (gfx950).
//
// Construction (once per handle): the observed set Omega of Section 3 is given
// as triplets.  For each copy, every entry gets a key (segment id, column inside
// its tile) -- the segment order is decided on the host from per-(tile, row)
// counts -- and a radix sort brings the entries into layout order, carrying the
// triplet index along so values and the map between the two copies follow.
// Adjacent equal keys after the user-major sort are repeated positions.
#include <rocprim/device/device_radix_sort.hpp>
#include <rocprim/device/device_select.hpp>
#include <rocprim/iterator/counting_iterator.hpp>

#include <algorithm>
#include <type_traits>

#include "ccdpp_internal.hpp"

namespace ccdk {
namespace {

constexpr int kT = 256;
// Histograms with at most this many bins count in LDS (128 KB per workgroup).
constexpr int32_t kHistLdsBins = 32768;

inline dim3 grid_for(int64_t n, int64_t cap = 1 << 20) {
    int64_t g = (n + kT - 1) / kT;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return dim3((unsigned)g);
}

// Adds one to count[key] for every valid lane of the wave.  A lane whose key equals
// the previous lane's (a run, as in triplets grouped by row) adds through the run's
// first lane, so a run costs one atomic.  The valid lanes are a prefix of the wave,
// and every lane of the wave calls this.
__device__ inline void count_runs(int32_t key, bool valid, int32_t* count) {
    const int lane = (int)(threadIdx.x & 63);
    const int32_t prev = __shfl_up(key, 1);
    const bool head = valid && (lane == 0 || prev != key);
    const uint64_t heads = __ballot(head);
    const int nvalid = __popcll(__ballot(valid));
    if (head) {
        const uint64_t later = lane == 63 ? 0 : heads >> (lane + 1);
        const int next = later ? lane + __ffsll((unsigned long long)later) : nvalid;
        atomicAdd(&count[key], next - lane);
    }
}

// Range [lo, hi) of entries of workgroup blockIdx.x: contiguous, so that runs stay in
// one wave.
__device__ inline void block_range(int64_t n, int64_t* lo, int64_t* hi) {
    const int64_t per = ((n + gridDim.x - 1) / gridDim.x + 63) / 64 * 64;
    *lo = min(n, (int64_t)blockIdx.x * per);
    *hi = min(n, *lo + per);
}

// count[key[e]] += 1 for every e < n.  bins <= kHistLdsBins: the workgroup counts in
// LDS and adds its non-zero counts at the end; else straight into global memory.
template <bool kLds>
__global__ void __launch_bounds__(1024) k_histogram(const int32_t* __restrict__ key, int64_t n,
                                                    int32_t bins, int32_t* count) {
    extern __shared__ int32_t lds_count[];
    int32_t* c = count;
    if constexpr (kLds) {
        for (int32_t b = threadIdx.x; b < bins; b += blockDim.x) lds_count[b] = 0;
        __syncthreads();
        c = lds_count;
    }
    int64_t lo, hi;
    block_range(n, &lo, &hi);
    for (int64_t base = lo + (threadIdx.x & ~63); base < hi; base += blockDim.x) {
        const int64_t e = base + (threadIdx.x & 63);
        const bool valid = e < hi;
        count_runs(valid ? key[e] : 0, valid, c);
    }
    if constexpr (kLds) {
        __syncthreads();
        for (int32_t b = threadIdx.x; b < bins; b += blockDim.x)
            if (lds_count[b]) atomicAdd(&count[b], lds_count[b]);
    }
}

__global__ void k_add(int32_t* __restrict__ a, int64_t n, int32_t delta) {
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < n; e += (int64_t)gridDim.x * kT)
        a[e] += delta;
}

// Entries whose key lies in [lo, hi).
struct KeyInRange {
    const int32_t* key;
    int32_t lo, hi;
    __device__ bool operator()(int32_t e) const { return key[e] >= lo && key[e] < hi; }
};

__global__ void k_map(const int32_t* __restrict__ in, const int32_t* __restrict__ table,
                      int64_t n, int32_t* __restrict__ out) {
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < n; e += (int64_t)gridDim.x * kT)
        out[e] = table[in[e]];
}

// Entries per (tile, row) segment: count[(col / T) * rows + row].
__global__ void __launch_bounds__(kT) k_seg_histogram(const int32_t* __restrict__ lrow,
                                                      const int32_t* __restrict__ lcol, int64_t nnz,
                                                      int32_t rows, int32_t T, int32_t* count) {
    int64_t lo, hi;
    block_range(nnz, &lo, &hi);
    for (int64_t base = lo + (threadIdx.x & ~63); base < hi; base += blockDim.x) {
        const int64_t e = base + (threadIdx.x & 63);
        const bool valid = e < hi;
        const int32_t key = valid ? (lcol[e] / T) * rows + lrow[e] : 0;
        count_runs(key, valid, count);
    }
}

// Sort key of an entry: its segment id, then its column inside the tile.
__global__ void k_seg_keys(const int32_t* __restrict__ lrow, const int32_t* __restrict__ lcol,
                           const int32_t* __restrict__ segid, int64_t nnz, int32_t rows, int32_t T,
                           int cbits, uint64_t* __restrict__ keys, int32_t* __restrict__ ids) {
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < nnz;
         e += (int64_t)gridDim.x * kT) {
        const int64_t c = lcol[e];
        const int64_t p = c / T;
        const uint64_t s = (uint64_t)segid[p * rows + lrow[e]];
        keys[e] = (s << cbits) | (uint64_t)(c - p * T);
        ids[e] = (int32_t)e;
    }
}

__global__ void k_dup_check(const uint64_t* __restrict__ keys, int64_t nnz, int32_t* flag) {
    for (int64_t p = (int64_t)blockIdx.x * kT + threadIdx.x; p + 1 < nnz;
         p += (int64_t)gridDim.x * kT)
        if (keys[p] == keys[p + 1]) *flag = 1;
}

// Entry q of the sorted order goes to padded position p = q + seg_off[segment]:
// its index to idx[p], its value to val[val_slot(p)]; pos[q] is the value slot.
template <class I, class V>
__global__ void k_layout_fill(const uint64_t* __restrict__ keys, const int32_t* __restrict__ perm,
                              const float* __restrict__ val_in, int64_t nnz, int cbits,
                              uint64_t mask, const int32_t* __restrict__ seg_off, uint32_t swz_lim,
                              I* __restrict__ idx, V* __restrict__ val,
                              int32_t* __restrict__ pos) {
    for (int64_t q = (int64_t)blockIdx.x * kT + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * kT) {
        const uint64_t key = keys[q];
        const int64_t p = q + seg_off[key >> cbits];
        const uint32_t c = (uint32_t)(key & mask);
        const bool first = q == 0 || (keys[q - 1] >> cbits) != (key >> cbits);
        idx[p] = (I)((c < swz_lim ? lds_swizzle(c) : c) | (first ? IndexBits<I>::start : 0u));
        const int64_t f = val_slot<V>(p);
        val[f] = (V)val_in[perm[q]];
        pos[q] = (int32_t)f;
    }
}

template <class I>
__global__ void k_fill_idx(I* __restrict__ idx, I value, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kT + threadIdx.x; i < n; i += (int64_t)gridDim.x * kT)
        idx[i] = value;
}

__global__ void k_invert(const int32_t* __restrict__ perm, int64_t n, int32_t* __restrict__ inv) {
    for (int64_t q = (int64_t)blockIdx.x * kT + threadIdx.x; q < n; q += (int64_t)gridDim.x * kT)
        inv[perm[q]] = (int32_t)q;
}

__global__ void k_compose(const int32_t* __restrict__ a, const int32_t* __restrict__ b, int64_t n,
                          int32_t* __restrict__ out) {
    for (int64_t q = (int64_t)blockIdx.x * kT + threadIdx.x; q < n; q += (int64_t)gridDim.x * kT)
        out[q] = a[b[q]];
}

// out[from[e]] = to[e]: a map between value slots of the two copies.
__global__ void k_slot_map(const int32_t* __restrict__ from, const int32_t* __restrict__ to,
                           int64_t n, int32_t* __restrict__ out) {
    for (int64_t q = (int64_t)blockIdx.x * kT + threadIdx.x; q < n; q += (int64_t)gridDim.x * kT)
        out[from[q]] = to[q];
}

// dst[map[f]] = src[f] over the source copy's value slots in order (slots of
// padding entries map to -1): sequential reads, one scattered write per entry.
template <class V>
__global__ void k_copy_slots(const V* __restrict__ src, const int32_t* __restrict__ map,
                             V* __restrict__ dst, int64_t n) {
    for (int64_t f = (int64_t)blockIdx.x * kT + threadIdx.x; f < n; f += (int64_t)gridDim.x * kT) {
        const int32_t g = map[f];
        if (g >= 0) dst[g] = src[f];
    }
}

template <class V>
__global__ void k_fill(V* __restrict__ dst, V value, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kT + threadIdx.x; i < n; i += (int64_t)gridDim.x * kT)
        dst[i] = value;
}

// colmajor[t * rows + i'] = rowmajor[new2old[i'] * k + t]
template <class S, class V>
__global__ void k_factor_in(const S* __restrict__ rowmajor, const int32_t* __restrict__ new2old,
                            int64_t rows, int32_t k, V* __restrict__ colmajor) {
    const int64_t total = rows * k;
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * kT) {
        const int64_t t = e / rows;
        const int64_t i = e - t * rows;
        colmajor[e] = (V)rowmajor[(int64_t)new2old[i] * k + t];
    }
}

// rowmajor[i * k + t] = colmajor[t * rows + old2new[i]]
template <class V, class S>
__global__ void k_factor_out(const V* __restrict__ colmajor, const int32_t* __restrict__ old2new,
                             int64_t rows, int32_t k, S* __restrict__ rowmajor) {
    const int64_t total = rows * k;
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * kT) {
        const int64_t i = e / k;
        const int64_t t = e - i * k;
        rowmajor[e] = (S)colmajor[t * rows + old2new[i]];
    }
}

// Rewrites, one wave per window, every window whose lanes' valid entries each climb
// by at most kDeltaMax unswizzled columns into the delta-coded format, and sets its
// bit.  Valid entries come first in a lane (padding only ends a segment); a lane
// of padding alone is coded as its first index with one valid entry.  Every lane
// reads its 16 bytes before the vote, so the window is rewritten in place.
__global__ __launch_bounds__(kT) void k_delta_windows(uint16_t* __restrict__ idx, int64_t nwin,
                                                       uint32_t pad, uint64_t* __restrict__ dmask) {
    const int lane = (int)(threadIdx.x & 63u);
    const int64_t w = (int64_t)blockIdx.x * (kT / 64) + (threadIdx.x >> 6);
    if (w >= nwin) return;  // whole waves leave together
    uint16_t* blk = idx + w * kWin;
    const uint4 v = *reinterpret_cast<const uint4*>(blk + lane * kE);
    const uint32_t wd[4] = {v.x, v.y, v.z, v.w};
    uint32_t c[8];
    for (int k = 0; k < 8; ++k) c[k] = (wd[k >> 1] >> (16 * (k & 1))) & 0xFFFFu;
    int cnt = 0;
    while (cnt < 8 && c[cnt] != pad) ++cnt;
    bool ok = true;
    for (int k = cnt; k < 8; ++k) ok = ok && c[k] == pad;  // padding only after the valid entries
    uint32_t st[7] = {0, 0, 0, 0, 0, 0, 0};
    if (cnt > 0) {
        uint32_t prev = lds_swizzle(c[0] & 0x7FFFu);
        for (int k = 1; k < cnt; ++k) {
            const uint32_t cur = lds_swizzle(c[k]);
            ok = ok && cur >= prev && cur - prev <= kDeltaMax;
            st[k - 1] = (cur - prev) & kDeltaMax;
            prev = cur;
        }
    }
    if (!__all(ok)) return;
    const uint32_t last = (uint32_t)(cnt > 0 ? cnt - 1 : 0);
    uint32_t* words = reinterpret_cast<uint32_t*>(blk);
    words[3 * lane] = c[0] | (st[0] << 16) | (st[1] << 27);
    words[3 * lane + 1] = (st[1] >> 5) | (st[2] << 6) | (st[3] << 17) | (st[4] << 28);
    words[3 * lane + 2] = (st[4] >> 4) | (st[5] << 7) | (st[6] << 18) | (last << 29);
    if (lane == 0) atomicOr(reinterpret_cast<unsigned long long*>(dmask + (w >> 6)),
                            1ull << (w & 63));
}

// Index of entry q as the plain format holds it, from a delta-coded window when
// its bit is set.
template <class I>
__device__ __forceinline__ uint32_t index_at(const I* idx, const uint64_t* dmask, uint32_t pad,
                                             int64_t q) {
    const int64_t w = q / kWin;
    if (dmask && ((dmask[w >> 6] >> (w & 63)) & 1u)) {
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(idx + w * kWin) + 3 * ((q % kWin) / kE);
        uint32_t c[8];
        delta_decode(rec[0], rec[1], rec[2], pad, c);
        return c[q % kE];
    }
    return (uint32_t)idx[q];
}

// R = A - w_i^T h_j for every entry of the user-major layout (prediction summed
// in fp64 over ascending features, one rounding to fp32).  Entry e (A[e], in the
// unpadded layout order) has its value in slot pos[e]; its segment, and from it the
// row and the tile, are found by binary search.
template <class I, class V>
__global__ void k_rebuild(const int64_t* __restrict__ seg_start, int64_t nseg,
                          const int32_t* __restrict__ seg_row, const int32_t* __restrict__ tile_seg,
                          int32_t P, int32_t T, uint32_t swz_lim, const I* __restrict__ idx,
                          const uint64_t* __restrict__ dmask, uint32_t pad,
                          const int32_t* __restrict__ pos, const V* __restrict__ A,
                          const V* __restrict__ W, const V* __restrict__ H, int64_t m,
                          int64_t n, int32_t k, int64_t nnz, V* __restrict__ val) {
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < nnz;
         e += (int64_t)gridDim.x * kT) {
        const int64_t f = pos[e];         // value slot
        const int64_t q = val_entry<V>(f);   // entry position
        int64_t lo = 0, hi = nseg;  // last s with seg_start[s] <= q
        while (hi - lo > 1) {
            const int64_t mid = (lo + hi) >> 1;
            if (seg_start[mid] <= q) lo = mid; else hi = mid;
        }
        int32_t plo = 0, phi = P;  // last tile p with tile_seg[p] <= s
        while (phi - plo > 1) {
            const int32_t mid = (plo + phi) >> 1;
            if (tile_seg[mid] <= lo) plo = mid; else phi = mid;
        }
        const int64_t i = seg_row[lo];
        const uint32_t c = index_at<I>(idx, dmask, pad, q) & IndexBits<I>::mask;
        const int64_t j = (int64_t)plo * T + (int64_t)(c < swz_lim ? lds_swizzle(c) : c);
        double pred = 0.0;
        for (int32_t t = 0; t < k; ++t)
            pred = __builtin_fma((double)W[(int64_t)t * m + i], (double)H[(int64_t)t * n + j], pred);
        val[f] = (V)((double)A[e] - pred);
    }
}

template <class S, class V>
__global__ void k_copy_mapped(const S* __restrict__ src, const int32_t* __restrict__ smap,
                              V* __restrict__ dst, const int32_t* __restrict__ dmap,
                              int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kT + threadIdx.x; i < n; i += (int64_t)gridDim.x * kT)
        dst[dmap ? dmap[i] : i] = (V)src[smap ? smap[i] : i];
}

// Bitwise comparison of the two copies (as unsigned words of the value's size).
template <class V>
__global__ void k_consistency(const V* __restrict__ a, const int32_t* __restrict__ amap,
                              const V* __restrict__ b, const int32_t* __restrict__ bmap,
                              int64_t n, unsigned long long* count) {
    using U = typename std::conditional<sizeof(V) == 4, uint32_t, uint64_t>::type;
    for (int64_t i = (int64_t)blockIdx.x * kT + threadIdx.x; i < n; i += (int64_t)gridDim.x * kT)
        if (__builtin_bit_cast(U, a[amap[i]]) != __builtin_bit_cast(U, b[bmap[i]]))
            atomicAdd(count, 1ull);
}

// splitmix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
// generators", OOPSLA 2014): a counter-based 64-bit generator.
__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

// The initial H: entry (j, t) of the row-major n x k matrix over input ids, e = j k + t,
// is 0.1 z, z ~ N(0, 1) by the Box-Muller transform of the counter draws 2e and 2e + 1
// of a stream keyed by the seed, rounded to float; written column-major over
// relabelled ids (H[t n + j'] for j' = old2new[j]).
template <class V>
__global__ void k_initial_h(uint64_t seed, const int32_t* __restrict__ new2old, int64_t n,
                            int32_t k, V* __restrict__ H) {
    const uint64_t key = splitmix64(seed);
    const int64_t total = n * k;
    for (int64_t q = (int64_t)blockIdx.x * kT + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * kT) {
        const int64_t t = q / n;
        const int64_t jn = q - t * n;
        const uint64_t e = (uint64_t)new2old[jn] * (uint64_t)k + (uint64_t)t;
        const double u1 = (double)(splitmix64(key + 2 * e) >> 11) * 0x1.0p-53;
        const double u2 = (double)(splitmix64(key + 2 * e + 1) >> 11) * 0x1.0p-53;
        const double z = __builtin_sqrt(-2.0 * log1p(-u1)) * cos(6.283185307179586 * u2);
        H[q] = (V)(float)(0.1 * z);
    }
}

template <class V>
__global__ void k_seg_spread(const V* __restrict__ F, int64_t rows,
                             const int32_t* __restrict__ seg_row, int64_t S, int32_t k,
                             V* __restrict__ out) {
    const int64_t total = S * k;
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * kT) {
        const int64_t t = e / S;
        const int64_t sg = e - t * S;
        out[e] = F[t * rows + seg_row[sg]];
    }
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

template <class V>
__global__ void k_sq_sum(const V* __restrict__ v, int64_t n, double* __restrict__ part) {
    double acc = 0.0;
    for (int64_t i = (int64_t)blockIdx.x * kT + threadIdx.x; i < n; i += (int64_t)gridDim.x * kT) {
        const double d = v[i];
        acc = __builtin_fma(d, d, acc);
    }
    block_total(acc, &part[blockIdx.x]);
}

// Squared prediction errors of held-out triplets, one fixed-order partial per block.
// CHECK: the triplets were not validated on the host; an entry whose indices are out
// of range or whose value is not finite is skipped (never used as an index) and
// counted in rejected[blockIdx.x].  Valid entries take the same arithmetic in the
// same order either way.
template <class V, bool CHECK>
__global__ void k_test_err(const int32_t* __restrict__ row, const int32_t* __restrict__ col,
                           const float* __restrict__ val, int64_t nnz,
                           const int32_t* __restrict__ rnew, const int32_t* __restrict__ cnew,
                           const V* __restrict__ W, const V* __restrict__ H, int64_t m,
                           int64_t n, int32_t k, double* __restrict__ part,
                           double* __restrict__ rejected) {
    double acc = 0.0;
    double bad = 0.0;
    for (int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x; e < nnz;
         e += (int64_t)gridDim.x * kT) {
        const int32_t r = row[e], c = col[e];
        const float a = val[e];
        if constexpr (CHECK) {
            if (r < 0 || (int64_t)r >= m || c < 0 || (int64_t)c >= n || !__builtin_isfinite(a)) {
                bad += 1.0;
                continue;
            }
        }
        const int64_t i = rnew[r];
        const int64_t j = cnew[c];
        double pred = 0.0;
        for (int32_t t = 0; t < k; ++t)
            pred = __builtin_fma((double)W[(int64_t)t * m + i], (double)H[(int64_t)t * n + j], pred);
        const double err = (double)a - pred;
        acc = __builtin_fma(err, err, acc);
    }
    block_total(acc, &part[blockIdx.x]);
    if constexpr (CHECK) {
        __syncthreads();  // block_total's LDS is reused
        block_total(bad, &rejected[blockIdx.x]);
    }
}

}  // namespace

hipError_t launch_histogram(const int32_t* key, int64_t n, int32_t bins, int32_t* count,
                           int32_t workgroups, hipStream_t s) {
    if (n == 0) return hipSuccess;
    if (bins <= kHistLdsBins) {
        const size_t lds = (size_t)bins * 4;
        hipError_t e = hipFuncSetAttribute((const void*)k_histogram<true>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        const int64_t g = std::min<int64_t>(workgroups, (n + 1023) / 1024);
        hipLaunchKernelGGL(k_histogram<true>, dim3((unsigned)g), dim3(1024), lds, s, key, n, bins,
                           count);
    } else {
        hipLaunchKernelGGL(k_histogram<false>, grid_for(n, 8192), dim3(kT), 0, s, key, n, bins,
                           count);
    }
    return hipGetLastError();
}

hipError_t launch_map(const int32_t* in, const int32_t* table, int64_t n, int32_t* out,
                      hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_map, grid_for(n), dim3(kT), 0, s, in, table, n, out);
    return hipGetLastError();
}

hipError_t launch_seg_histogram(const int32_t* lrow, const int32_t* lcol, int64_t nnz,
                                int32_t rows, int32_t T, int32_t* count, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    hipLaunchKernelGGL(k_seg_histogram, grid_for(nnz, 8192), dim3(kT), 0, s, lrow, lcol, nnz, rows,
                       T, count);
    return hipGetLastError();
}

hipError_t launch_seg_keys(const int32_t* lrow, const int32_t* lcol, const int32_t* segid,
                           int64_t nnz, int32_t rows, int32_t T, int cbits, uint64_t* keys,
                           int32_t* ids, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    hipLaunchKernelGGL(k_seg_keys, grid_for(nnz), dim3(kT), 0, s, lrow, lcol, segid, nnz, rows, T,
                       cbits, keys, ids);
    return hipGetLastError();
}

hipError_t launch_dup_check(const uint64_t* keys, int64_t nnz, int32_t* flag, hipStream_t s) {
    if (nnz < 2) return hipSuccess;
    hipLaunchKernelGGL(k_dup_check, grid_for(nnz), dim3(kT), 0, s, keys, nnz, flag);
    return hipGetLastError();
}

template <class V>
hipError_t launch_layout_fill(const uint64_t* keys, const int32_t* perm, const float* val_in,
                              int64_t nnz, int cbits, const int32_t* seg_off, uint32_t swz_lim, bool idx16,
                              void* idx, V* val, int32_t* pos, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    const uint64_t mask = cbits >= 64 ? ~0ull : ((1ull << cbits) - 1);
    if (idx16)
        hipLaunchKernelGGL((k_layout_fill<uint16_t, V>), grid_for(nnz), dim3(kT), 0, s, keys, perm,
                           val_in, nnz, cbits, mask, seg_off, swz_lim, static_cast<uint16_t*>(idx), val,
                           pos);
    else
        hipLaunchKernelGGL((k_layout_fill<int32_t, V>), grid_for(nnz), dim3(kT), 0, s, keys, perm,
                           val_in, nnz, cbits, mask, seg_off, swz_lim, static_cast<int32_t*>(idx), val,
                           pos);
    return hipGetLastError();
}

hipError_t launch_fill_idx(void* idx, bool idx16, int32_t value, int64_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    if (idx16)
        hipLaunchKernelGGL(k_fill_idx<uint16_t>, grid_for(n), dim3(kT), 0, s,
                           static_cast<uint16_t*>(idx), (uint16_t)value, n);
    else
        hipLaunchKernelGGL(k_fill_idx<int32_t>, grid_for(n), dim3(kT), 0, s,
                           static_cast<int32_t*>(idx), value, n);
    return hipGetLastError();
}

hipError_t launch_invert(const int32_t* perm, int64_t n, int32_t* inv, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_invert, grid_for(n), dim3(kT), 0, s, perm, n, inv);
    return hipGetLastError();
}

hipError_t launch_compose(const int32_t* a, const int32_t* b, int64_t n, int32_t* out,
                          hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_compose, grid_for(n), dim3(kT), 0, s, a, b, n, out);
    return hipGetLastError();
}

hipError_t launch_slot_map(const int32_t* from, const int32_t* to, int64_t n, int32_t* out,
                          hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_slot_map, grid_for(n), dim3(kT), 0, s, from, to, n, out);
    return hipGetLastError();
}

template <class V>
hipError_t launch_copy_slots(const V* src, const int32_t* map, V* dst, int64_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL((k_copy_slots<V>), grid_for(n), dim3(kT), 0, s, src, map, dst, n);
    return hipGetLastError();
}

template <class V>
hipError_t launch_fill(V* dst, V value, int64_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill<V>, grid_for(n), dim3(kT), 0, s, dst, value, n);
    return hipGetLastError();
}

template <class S, class V>
hipError_t launch_scatter_factor_in(const S* rowmajor, const int32_t* new2old, int64_t rows,
                                    int32_t k, V* colmajor, hipStream_t s) {
    hipLaunchKernelGGL((k_factor_in<S, V>), grid_for(rows * k), dim3(kT), 0, s, rowmajor, new2old,
                       rows, k, colmajor);
    return hipGetLastError();
}

template <class V, class S>
hipError_t launch_gather_factor_out(const V* colmajor, const int32_t* old2new, int64_t rows,
                                    int32_t k, S* rowmajor, hipStream_t s) {
    hipLaunchKernelGGL((k_factor_out<V, S>), grid_for(rows * k), dim3(kT), 0, s, colmajor, old2new,
                       rows, k, rowmajor);
    return hipGetLastError();
}

hipError_t launch_delta_windows(void* idx, int64_t npad, int32_t pad, uint64_t* dmask,
                                hipStream_t s) {
    const int64_t nwin = npad / kWin;
    if (nwin == 0) return hipSuccess;
    hipLaunchKernelGGL(k_delta_windows, dim3((unsigned)((nwin + kT / 64 - 1) / (kT / 64))), dim3(kT),
                       0, s, static_cast<uint16_t*>(idx), nwin, (uint32_t)pad, dmask);
    return hipGetLastError();
}

template <class V>
hipError_t launch_rebuild_residual(const Layout& L, const int32_t* pos, const V* A, const V* W,
                                   const V* H, int64_t m, int64_t n, int32_t k, hipStream_t s) {
    if (L.nnz == 0) return hipSuccess;
    if (L.idx16)
        hipLaunchKernelGGL((k_rebuild<uint16_t, V>), grid_for(L.nnz), dim3(kT), 0, s, L.seg_start,
                           L.nseg, L.seg_row, L.tile_seg, L.P, L.T, L.swz_lim,
                           static_cast<const uint16_t*>(L.idx), L.dmask, (uint32_t)L.pad, pos, A, W,
                           H, m, n, k, L.nnz, static_cast<V*>(L.val));
    else
        hipLaunchKernelGGL((k_rebuild<int32_t, V>), grid_for(L.nnz), dim3(kT), 0, s, L.seg_start,
                           L.nseg, L.seg_row, L.tile_seg, L.P, L.T, L.swz_lim,
                           static_cast<const int32_t*>(L.idx), nullptr, (uint32_t)L.pad, pos, A, W,
                           H, m, n, k, L.nnz, static_cast<V*>(L.val));
    return hipGetLastError();
}

template <class S, class V>
hipError_t launch_copy_mapped(const S* src, const int32_t* smap, V* dst, const int32_t* dmap,
                              int64_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL((k_copy_mapped<S, V>), grid_for(n), dim3(kT), 0, s, src, smap, dst, dmap, n);
    return hipGetLastError();
}

template <class V>
hipError_t launch_consistency(const V* a, const int32_t* amap, const V* b, const int32_t* bmap,
                              int64_t n, unsigned long long* count, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_consistency<V>, grid_for(n), dim3(kT), 0, s, a, amap, b, bmap, n, count);
    return hipGetLastError();
}

template <class V>
hipError_t launch_initial_h(uint64_t seed, const int32_t* new2old, int64_t n, int32_t k, V* H,
                            hipStream_t s) {
    if (n * k == 0) return hipSuccess;
    hipLaunchKernelGGL(k_initial_h<V>, grid_for(n * k), dim3(kT), 0, s, seed, new2old, n, k, H);
    return hipGetLastError();
}

template <class V>
hipError_t launch_seg_spread(const V* F, int64_t rows, const int32_t* seg_row, int64_t S,
                             int32_t k, V* out, hipStream_t s) {
    if (S == 0 || k == 0) return hipSuccess;
    hipLaunchKernelGGL(k_seg_spread<V>, grid_for(S * k), dim3(kT), 0, s, F, rows, seg_row, S, k,
                       out);
    return hipGetLastError();
}

template <class V>
hipError_t launch_sq_sum(const V* v, int64_t n, double* part, int32_t nparts, hipStream_t s) {
    hipLaunchKernelGGL(k_sq_sum<V>, dim3(nparts), dim3(kT), 0, s, v, n, part);
    return hipGetLastError();
}

template <class V>
hipError_t launch_test_err(const int32_t* row, const int32_t* col, const float* val, int64_t nnz,
                           const int32_t* rold2new, const int32_t* cold2new, const V* W,
                           const V* H, int64_t m, int64_t n, int32_t k, double* part,
                           int32_t nparts, double* rejected, hipStream_t s) {
    if (rejected)
        hipLaunchKernelGGL((k_test_err<V, true>), dim3(nparts), dim3(kT), 0, s, row, col, val, nnz,
                           rold2new, cold2new, W, H, m, n, k, part, rejected);
    else
        hipLaunchKernelGGL((k_test_err<V, false>), dim3(nparts), dim3(kT), 0, s, row, col, val, nnz,
                           rold2new, cold2new, W, H, m, n, k, part, nullptr);
    return hipGetLastError();
}

#define CCDK_BUILD_INSTANTIATE(V)                                                               \
    template hipError_t launch_layout_fill<V>(const uint64_t*, const int32_t*, const float*,    \
                                              int64_t, int, const int32_t*, uint32_t, bool, void*, \
                                              V*, int32_t*, hipStream_t);                       \
    template hipError_t launch_fill<V>(V*, V, int64_t, hipStream_t);                            \
    template hipError_t launch_copy_slots<V>(const V*, const int32_t*, V*, int64_t, hipStream_t); \
    template hipError_t launch_scatter_factor_in<float, V>(const float*, const int32_t*,        \
                                                           int64_t, int32_t, V*, hipStream_t);  \
    template hipError_t launch_scatter_factor_in<double, V>(const double*, const int32_t*,      \
                                                            int64_t, int32_t, V*, hipStream_t); \
    template hipError_t launch_gather_factor_out<V, float>(const V*, const int32_t*, int64_t,   \
                                                           int32_t, float*, hipStream_t);       \
    template hipError_t launch_gather_factor_out<V, double>(const V*, const int32_t*, int64_t,  \
                                                            int32_t, double*, hipStream_t);     \
    template hipError_t launch_rebuild_residual<V>(const Layout&, const int32_t*, const V*,     \
                                                   const V*, const V*, int64_t, int64_t,        \
                                                   int32_t, hipStream_t);                       \
    template hipError_t launch_copy_mapped<V, V>(const V*, const int32_t*, V*, const int32_t*,  \
                                                 int64_t, hipStream_t);                         \
    template hipError_t launch_consistency<V>(const V*, const int32_t*, const V*,               \
                                              const int32_t*, int64_t, unsigned long long*,     \
                                              hipStream_t);                                     \
    template hipError_t launch_seg_spread<V>(const V*, int64_t, const int32_t*, int64_t,        \
                                             int32_t, V*, hipStream_t);                         \
    template hipError_t launch_initial_h<V>(uint64_t, const int32_t*, int64_t, int32_t, V*,     \
                                            hipStream_t);                                       \
    template hipError_t launch_sq_sum<V>(const V*, int64_t, double*, int32_t, hipStream_t);     \
    template hipError_t launch_test_err<V>(const int32_t*, const int32_t*, const float*,        \
                                           int64_t, const int32_t*, const int32_t*, const V*,   \
                                           const V*, int64_t, int64_t, int32_t, double*,        \
                                           int32_t, double*, hipStream_t);
CCDK_BUILD_INSTANTIATE(float)
CCDK_BUILD_INSTANTIATE(double)
#undef CCDK_BUILD_INSTANTIATE
template hipError_t launch_copy_mapped<double, float>(const double*, const int32_t*, float*,
                                                      const int32_t*, int64_t, hipStream_t);
template hipError_t launch_copy_mapped<float, double>(const float*, const int32_t*, double*,
                                                      const int32_t*, int64_t, hipStream_t);

// Radix sort of (key, id) pairs on the low `bits` bits of the key.
// Grows the shared temporary buffer of the device-wide primitives when needed.
hipError_t ensure_tmp(void** tmp, size_t* tmp_bytes, size_t need) {
    if (need <= *tmp_bytes) return hipSuccess;
    if (*tmp) (void)hipFree(*tmp);
    *tmp = nullptr;
    *tmp_bytes = 0;
    hipError_t e = dev_malloc(tmp, need);
    if (e == hipSuccess) *tmp_bytes = need;
    return e;
}

hipError_t sort_pairs(const uint64_t* kin, uint64_t* kout, const int32_t* vin, int32_t* vout,
                      int64_t n, int bits, hipStream_t s, void** tmp, size_t* tmp_bytes) {
    size_t need = 0;
    hipError_t e = rocprim::radix_sort_pairs(nullptr, need, kin, kout, vin, vout, (size_t)n, 0u,
                                             (unsigned)bits, s);
    if (e == hipSuccess) e = ensure_tmp(tmp, tmp_bytes, need);
    if (e != hipSuccess) return e;
    return rocprim::radix_sort_pairs(*tmp, need, kin, kout, vin, vout, (size_t)n, 0u,
                                     (unsigned)bits, s);
}

hipError_t select_range(const int32_t* key, int64_t n, int32_t lo, int32_t hi, int32_t* out,
                        int64_t* count, hipStream_t s, void** tmp, size_t* tmp_bytes) {
    const rocprim::counting_iterator<int32_t> ids(0);
    const KeyInRange pred{key, lo, hi};
    size_t need = 0;
    hipError_t e = rocprim::select(nullptr, need, ids, out, count, (size_t)n, pred, s);
    if (e == hipSuccess) e = ensure_tmp(tmp, tmp_bytes, need);
    if (e != hipSuccess) return e;
    return rocprim::select(*tmp, need, ids, out, count, (size_t)n, pred, s);
}

hipError_t launch_add(int32_t* a, int64_t n, int32_t delta, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_add, grid_for(n), dim3(kT), 0, s, a, n, delta);
    return hipGetLastError();
}

}  // namespace ccdk
