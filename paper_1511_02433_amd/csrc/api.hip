// Host runtime of the CCD++ library: the C ABI of include/ccdpp.h.
//
// The handle keeps everything on one device: the ratings A, the residual in a
// row-compressed and a column-compressed copy, the map between the copies, W
// and H column-major over relabelled ids (so the feature columns wbar_t and
// hbar_t of eq. 11 are contiguous), and the scratch vectors u and v.  Unlike
// the paper's Algorithm 7, u and v never travel to the host between features:
// the host only enqueues kernels on one stream, and ccdpp_run synchronises
// once at the end.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <numeric>

#include "ccdpp_internal.hpp"

using ccdk::Layout;

namespace {

thread_local std::string g_create_error;

constexpr int64_t kMaxDim = int64_t(1) << 30;
constexpr int64_t kMaxNnz = INT32_MAX;
constexpr int32_t kReduceParts = 1024;

struct ProfEvent {
    int kind;
    hipEvent_t a, b;
    double bytes;
};

}  // namespace

struct ccdpp {
    int64_t m = 0, n = 0, nnz = 0;
    int32_t k = 0;
    double lambda = 0.0;
    int device = 0;
    hipStream_t own_stream = nullptr;
    hipStream_t stream = nullptr;
    Layout L[2];                   // 0: rows are users (eq. 15), 1: rows are items (eq. 16)
    int32_t* rnew2old = nullptr;   // relabelled user id -> input user id
    int32_t* rold2new = nullptr;
    int32_t* cnew2old = nullptr;
    int32_t* cold2new = nullptr;
    int32_t* csr_src = nullptr;    // row-ordered position -> input triplet index
    int32_t* csr2csc = nullptr;    // row-ordered position -> column-ordered position
    float* A = nullptr;            // ratings, row order
    float* W = nullptr;            // k x m: W[t*m + i]
    float* H = nullptr;            // k x n
    float* u = nullptr;
    float* v = nullptr;
    double* sse_part = nullptr;
    int32_t sse_nparts = 0;
    double* d_scalar = nullptr;
    unsigned long long* d_count = nullptr;
    int32_t pending = -1;          // feature whose eq. 18 subtract is still folded into R-hat
    double train_sse = 0.0;
    bool train_sse_valid = false;
    std::string err;
    bool poisoned = false;
    int64_t build_us = 0;
    int64_t bytes_held = 0;
    std::vector<void*> allocs;
    // kernel timing
    bool prof = false;
    std::vector<ProfEvent> prof_pending;
    std::vector<hipEvent_t> event_pool;
    int64_t prof_launch[CCDPP_K_COUNT] = {};
    double prof_ms[CCDPP_K_COUNT] = {};
    double prof_bytes[CCDPP_K_COUNT] = {};
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

template <class T>
hipError_t dalloc(ccdpp* h, T** p, int64_t count) {
    size_t bytes = (size_t)std::max<int64_t>(count, 1) * sizeof(T);
    void* q = nullptr;
    hipError_t e = hipMalloc(&q, bytes);
    if (e != hipSuccess) return e;
    h->allocs.push_back(q);
    h->bytes_held += (int64_t)bytes;
    *p = static_cast<T*>(q);
    return hipSuccess;
}

// Temporary device buffer freed when it goes out of scope.
struct Tmp {
    void* p = nullptr;
    ~Tmp() {
        if (p) hipFree(p);
    }
};
template <class T>
hipError_t talloc(Tmp& t, T** p, int64_t count) {
    hipError_t e = hipMalloc(&t.p, (size_t)std::max<int64_t>(count, 1) * sizeof(T));
    *p = static_cast<T*>(t.p);
    return e;
}

bool usable(const ccdpp* h) { return h && !h->poisoned; }

// splitmix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
// generators", OOPSLA 2014): a counter-based 64-bit generator.
uint64_t splitmix64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

// H0 entry e (row-major n x k): N(0, 0.01) by Box-Muller on two counter draws.
float initial_h(uint64_t seed, uint64_t e) {
    const uint64_t s = splitmix64(seed);
    const double u1 = (double)(splitmix64(s + 2 * e) >> 11) * 0x1.0p-53;
    const double u2 = (double)(splitmix64(s + 2 * e + 1) >> 11) * 0x1.0p-53;
    const double z = std::sqrt(-2.0 * std::log1p(-u1)) * std::cos(6.283185307179586 * u2);
    return (float)(0.1 * z);
}

// Schedule of one layout from its row lengths (already in decreasing order).
int build_schedule(ccdpp* h, Layout& L, const std::vector<int64_t>& len) {
    using namespace ccdk;
    const int64_t rows = (int64_t)len.size();
    int64_t nb = 0;
    while (nb < rows && len[nb] > kGroupMaxLen) ++nb;
    std::vector<int32_t> piece_row, split_row, split_first;
    std::vector<int64_t> piece_lo;
    int64_t pos = 0;
    for (int64_t r = 0; r < nb; ++r) {
        const int64_t npc = (len[r] + kPieceMax - 1) / kPieceMax;
        const int64_t base = len[r] / npc, extra = len[r] % npc;
        if (npc > 1) {
            split_row.push_back((int32_t)r);
            split_first.push_back((int32_t)piece_row.size());
        }
        for (int64_t c = 0; c < npc; ++c) {
            piece_row.push_back((int32_t)r);
            piece_lo.push_back(pos);
            pos += base + (c < extra ? 1 : 0);
        }
    }
    piece_lo.push_back(pos);
    split_first.push_back((int32_t)piece_row.size());

    L.segs.clear();
    int64_t blocks = 0;
    if (!piece_row.empty()) {
        L.segs.push_back(Seg{kSegBlock, (int32_t)blocks, 0, (int32_t)piece_row.size()});
        blocks += (int64_t)piece_row.size();
    }
    struct Cls {
        int kind;
        int64_t maxlen;
        int g;
    };
    static const Cls classes[] = {{kSegG64E16, 1024, 64}, {kSegG64E8, 512, 64},
                                  {kSegG32E8, 256, 32},   {kSegG16E8, 128, 16},
                                  {kSegG8E8, 64, 8},      {kSegG4E8, 32, 4},
                                  {kSegG2E8, 16, 2},      {kSegG1E8, 8, 1}};
    int64_t r = nb;
    for (int ci = 0; ci < 8; ++ci) {
        const int64_t minlen = ci + 1 < 8 ? classes[ci + 1].maxlen + 1 : 0;
        int64_t e = r;
        while (e < rows && len[e] >= minlen) ++e;
        if (e > r) {
            const int64_t per = kBlock / classes[ci].g;
            L.segs.push_back(Seg{classes[ci].kind, (int32_t)blocks, (int32_t)r, (int32_t)e});
            blocks += (e - r + per - 1) / per;
        }
        r = e;
    }
    if (r != rows) return fail(h, CCDPP_EDEVICE, "internal: schedule does not cover all rows");
    if ((int)L.segs.size() > kMaxSegs) return fail(h, CCDPP_EDEVICE, "internal: too many segments");
    if (blocks > INT32_MAX) return fail(h, CCDPP_EINVAL, "too many workgroups per pass");
    L.grid = (int32_t)blocks;
    L.nblock_rows = (int32_t)nb;
    L.npieces = (int32_t)piece_row.size();
    L.nsplit = (int32_t)split_row.size();
    HIPCK(h, dalloc(h, &L.piece_row, L.npieces));
    HIPCK(h, dalloc(h, &L.piece_lo, L.npieces + 1));
    HIPCK(h, dalloc(h, &L.split_row, L.nsplit));
    HIPCK(h, dalloc(h, &L.split_first, L.nsplit + 1));
    HIPCK(h, dalloc(h, &L.part, L.npieces));
    if (L.npieces) {
        HIPCK(h, hipMemcpy(L.piece_row, piece_row.data(), piece_row.size() * 4, hipMemcpyHostToDevice));
    }
    HIPCK(h, hipMemcpy(L.piece_lo, piece_lo.data(), piece_lo.size() * 8, hipMemcpyHostToDevice));
    if (L.nsplit) {
        HIPCK(h, hipMemcpy(L.split_row, split_row.data(), split_row.size() * 4, hipMemcpyHostToDevice));
    }
    HIPCK(h, hipMemcpy(L.split_first, split_first.data(), split_first.size() * 4,
                       hipMemcpyHostToDevice));
    return CCDPP_OK;
}

// Order ids by decreasing count, ties by increasing id.
void relabel(const std::vector<int32_t>& count, std::vector<int32_t>& new2old,
             std::vector<int32_t>& old2new) {
    const int64_t N = (int64_t)count.size();
    new2old.resize(N);
    std::iota(new2old.begin(), new2old.end(), 0);
    std::stable_sort(new2old.begin(), new2old.end(),
                     [&](int32_t a, int32_t b) { return count[a] > count[b]; });
    old2new.resize(N);
    for (int64_t i = 0; i < N; ++i) old2new[new2old[i]] = (int32_t)i;
}

int bits_for(uint64_t maxkey) {
    int b = 1;
    while (b < 64 && (maxkey >> b) != 0) ++b;
    return b;
}

int create_device(ccdpp* h, const int32_t* row, const int32_t* col, const float* val,
                  uint64_t seed) {
    using namespace ccdk;
    const auto t0 = std::chrono::steady_clock::now();
    const int64_t m = h->m, n = h->n, N = h->nnz;
    HIPCK(h, hipGetDevice(&h->device));
    hipDeviceProp_t prop;
    HIPCK(h, hipGetDeviceProperties(&prop, h->device));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(h, CCDPP_EDEVICE, "device %d is %s; this library is built for gfx950",
                    h->device, prop.gcnArchName);
    HIPCK(h, hipStreamCreateWithFlags(&h->own_stream, hipStreamNonBlocking));
    h->stream = h->own_stream;
    hipStream_t s = h->stream;

    // Inputs and degrees.
    int32_t *d_row, *d_col, *d_cnt_r, *d_cnt_c;
    float* d_val;
    Tmp t_row, t_col, t_val, t_cr, t_cc;
    HIPCK(h, talloc(t_row, &d_row, N));
    HIPCK(h, talloc(t_col, &d_col, N));
    HIPCK(h, talloc(t_val, &d_val, N));
    HIPCK(h, talloc(t_cr, &d_cnt_r, m));
    HIPCK(h, talloc(t_cc, &d_cnt_c, n));
    if (N) {
        HIPCK(h, hipMemcpyAsync(d_row, row, N * 4, hipMemcpyHostToDevice, s));
        HIPCK(h, hipMemcpyAsync(d_col, col, N * 4, hipMemcpyHostToDevice, s));
        HIPCK(h, hipMemcpyAsync(d_val, val, N * 4, hipMemcpyHostToDevice, s));
    }
    HIPCK(h, hipMemsetAsync(d_cnt_r, 0, m * 4, s));
    HIPCK(h, hipMemsetAsync(d_cnt_c, 0, n * 4, s));
    HIPCK(h, launch_histogram(d_row, N, d_cnt_r, s));
    HIPCK(h, launch_histogram(d_col, N, d_cnt_c, s));
    std::vector<int32_t> cnt_r(m), cnt_c(n);
    HIPCK(h, hipMemcpyAsync(cnt_r.data(), d_cnt_r, m * 4, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipMemcpyAsync(cnt_c.data(), d_cnt_c, n * 4, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));

    // Relabel by decreasing degree.
    std::vector<int32_t> rn2o, ro2n, cn2o, co2n;
    relabel(cnt_r, rn2o, ro2n);
    relabel(cnt_c, cn2o, co2n);
    HIPCK(h, dalloc(h, &h->rnew2old, m));
    HIPCK(h, dalloc(h, &h->rold2new, m));
    HIPCK(h, dalloc(h, &h->cnew2old, n));
    HIPCK(h, dalloc(h, &h->cold2new, n));
    HIPCK(h, hipMemcpyAsync(h->rnew2old, rn2o.data(), m * 4, hipMemcpyHostToDevice, s));
    HIPCK(h, hipMemcpyAsync(h->rold2new, ro2n.data(), m * 4, hipMemcpyHostToDevice, s));
    HIPCK(h, hipMemcpyAsync(h->cnew2old, cn2o.data(), n * 4, hipMemcpyHostToDevice, s));
    HIPCK(h, hipMemcpyAsync(h->cold2new, co2n.data(), n * 4, hipMemcpyHostToDevice, s));

    // Persistent arrays.
    Layout& R = h->L[0];
    Layout& C = h->L[1];
    R.rows = m; R.cols = n; R.nnz = N;
    C.rows = n; C.cols = m; C.nnz = N;
    HIPCK(h, dalloc(h, &R.ptr, m + 1));
    HIPCK(h, dalloc(h, &R.idx, N));
    HIPCK(h, dalloc(h, &R.val, N));
    HIPCK(h, dalloc(h, &C.ptr, n + 1));
    HIPCK(h, dalloc(h, &C.idx, N));
    HIPCK(h, dalloc(h, &C.val, N));
    HIPCK(h, dalloc(h, &h->A, N));
    HIPCK(h, dalloc(h, &h->csr_src, N));
    HIPCK(h, dalloc(h, &h->csr2csc, N));

    // Sort to row order, check repeats, fill the row copy; sort to column order.
    {
        uint64_t *k0, *k1;
        int32_t *i0, *i1;
        Tmp tk0, tk1, ti0, ti1, ttmp;
        void* tmp = nullptr;
        size_t tmp_bytes = 0;
        HIPCK(h, talloc(tk0, &k0, N));
        HIPCK(h, talloc(tk1, &k1, N));
        HIPCK(h, talloc(ti0, &i0, N));
        HIPCK(h, talloc(ti1, &i1, N));
        HIPCK(h, launch_make_keys_csr(d_row, d_col, h->rold2new, h->cold2new, N, n, k0, i0, s));
        const int bits = bits_for((uint64_t)m * (uint64_t)n - 1);
        hipError_t e = N ? sort_pairs(k0, k1, i0, h->csr_src, N, bits, s, &tmp, &tmp_bytes)
                         : hipSuccess;
        ttmp.p = tmp;
        HIPCK(h, e);
        int32_t* d_flag;
        Tmp tflag;
        HIPCK(h, talloc(tflag, &d_flag, 1));
        HIPCK(h, hipMemsetAsync(d_flag, 0, 4, s));
        HIPCK(h, launch_dup_check(k1, N, d_flag, s));
        int32_t flag = 0;
        HIPCK(h, hipMemcpyAsync(&flag, d_flag, 4, hipMemcpyDeviceToHost, s));
        HIPCK(h, hipStreamSynchronize(s));
        if (flag) return fail(h, CCDPP_EDUP, "a position (i, j) occurs more than once");
        HIPCK(h, launch_csr_fill(k1, h->csr_src, d_val, N, n, m, R.idx, R.val, h->A, k0, i0, s));
        const int bits2 = bits_for((uint64_t)n * (uint64_t)m - 1);
        tmp = ttmp.p;
        e = N ? sort_pairs(k0, k1, i0, i1, N, bits2, s, &tmp, &tmp_bytes) : hipSuccess;
        ttmp.p = tmp;
        HIPCK(h, e);
        HIPCK(h, launch_csc_fill(k1, i1, R.val, N, m, C.idx, C.val, h->csr2csc, s));
        HIPCK(h, hipStreamSynchronize(s));
    }

    // Row pointers and schedules from the sorted degrees.
    std::vector<int64_t> len_r(m), len_c(n), ptr_r(m + 1), ptr_c(n + 1);
    for (int64_t i = 0; i < m; ++i) len_r[i] = cnt_r[rn2o[i]];
    for (int64_t j = 0; j < n; ++j) len_c[j] = cnt_c[cn2o[j]];
    ptr_r[0] = 0;
    for (int64_t i = 0; i < m; ++i) ptr_r[i + 1] = ptr_r[i] + len_r[i];
    ptr_c[0] = 0;
    for (int64_t j = 0; j < n; ++j) ptr_c[j + 1] = ptr_c[j] + len_c[j];
    HIPCK(h, hipMemcpy(R.ptr, ptr_r.data(), (m + 1) * 8, hipMemcpyHostToDevice));
    HIPCK(h, hipMemcpy(C.ptr, ptr_c.data(), (n + 1) * 8, hipMemcpyHostToDevice));
    int rc = build_schedule(h, R, len_r);
    if (rc) return rc;
    rc = build_schedule(h, C, len_c);
    if (rc) return rc;

    // Factors: W = 0 (Algorithm 3), H from the seed; scratch.
    HIPCK(h, dalloc(h, &h->W, (int64_t)h->k * m));
    HIPCK(h, dalloc(h, &h->H, (int64_t)h->k * n));
    HIPCK(h, dalloc(h, &h->u, m));
    HIPCK(h, dalloc(h, &h->v, n));
    h->sse_nparts = std::max<int32_t>({R.grid, C.grid, kReduceParts});
    HIPCK(h, dalloc(h, &h->sse_part, h->sse_nparts));
    HIPCK(h, dalloc(h, &h->d_scalar, 1));
    HIPCK(h, dalloc(h, &h->d_count, 1));
    HIPCK(h, launch_fill(h->W, 0.0f, (int64_t)h->k * m, s));
    HIPCK(h, launch_fill(h->u, 0.0f, m, s));
    HIPCK(h, launch_fill(h->v, 0.0f, n, s));
    {
        std::vector<float> h0((size_t)n * h->k);
        for (int64_t e = 0; e < n * h->k; ++e) h0[e] = initial_h(seed, (uint64_t)e);
        float* d_h0;
        Tmp th0;
        HIPCK(h, talloc(th0, &d_h0, n * h->k));
        HIPCK(h, hipMemcpyAsync(d_h0, h0.data(), h0.size() * 4, hipMemcpyHostToDevice, s));
        HIPCK(h, launch_scatter_factor_in(d_h0, h->cnew2old, n, h->k, h->H, s));
        HIPCK(h, hipStreamSynchronize(s));
    }
    h->pending = -1;
    h->build_us = std::chrono::duration_cast<std::chrono::microseconds>(
                      std::chrono::steady_clock::now() - t0)
                      .count();
    return CCDPP_OK;
}

void destroy_all(ccdpp* h) {
    for (void* p : h->allocs) hipFree(p);
    h->allocs.clear();
    for (auto& pe : h->prof_pending) {
        h->event_pool.push_back(pe.a);
        h->event_pool.push_back(pe.b);
    }
    for (hipEvent_t e : h->event_pool) hipEventDestroy(e);
    if (h->own_stream) hipStreamDestroy(h->own_stream);
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
    double bytes;
    hipEvent_t a = nullptr;
    Timed(ccdpp* h_, int kind_, double bytes_) : h(h_), kind(kind_), bytes(bytes_) {
        if (h->prof) {
            a = take_event(h);
            if (a) hipEventRecord(a, h->stream);
        }
    }
    void done() {
        if (h->prof && a) {
            hipEvent_t b = take_event(h);
            if (b) {
                hipEventRecord(b, h->stream);
                h->prof_pending.push_back(ProfEvent{kind, a, b, bytes});
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
            h->prof_launch[pe.kind] += 1;
            h->prof_ms[pe.kind] += ms;
            h->prof_bytes[pe.kind] += pe.bytes;
        }
        h->event_pool.push_back(pe.a);
        h->event_pool.push_back(pe.b);
    }
    h->prof_pending.clear();
}

// Algorithmic bytes of one pass over layout L (see ccdpp_profile_read).
double pass_bytes(const Layout& L, ccdk::PassMode mode, int gathered_vectors) {
    const double nnz = (double)L.nnz, rows = (double)L.rows, cols = (double)L.cols;
    double b = 8.0 * nnz + 8.0 * (rows + 1);             // index + value reads, row pointers
    if (mode != ccdk::kModePlain) b += 4.0 * nnz;      // residual write-back
    if (mode != ccdk::kModeFlush) b += 4.0 * rows;     // output coordinates
    if (mode == ccdk::kModeAdd || mode == ccdk::kModeSubAdd) b += 4.0 * rows;  // p
    if (mode == ccdk::kModeSubAdd || mode == ccdk::kModeFlush) b += 4.0 * rows;  // pp
    b += 4.0 * cols * gathered_vectors;
    return b;
}

int pass(ccdpp* h, int li, ccdk::PassMode mode, const float* x, const float* p, const float* pp,
         const float* q, const float* qq, float* y, int gathered) {
    const Layout& L = h->L[li];
    const int kind = mode == ccdk::kModePlain ? CCDPP_K_PASS
                     : mode == ccdk::kModeFlush ? CCDPP_K_FLUSH
                                                 : CCDPP_K_PASS_FUSED;
    {
        Timed tm(h, kind, pass_bytes(L, mode, gathered));
        HIPCK(h, ccdk::launch_pass(L, mode, x, p, pp, q, qq, y, h->lambda, h->sse_part, h->stream));
        tm.done();
    }
    if (mode != ccdk::kModeFlush && L.nsplit > 0) {
        Timed tc(h, CCDPP_K_COMBINE, 16.0 * L.npieces + 12.0 * L.nsplit);
        HIPCK(h, ccdk::launch_combine(L, y, h->lambda, h->stream));
        tc.done();
    }
    return CCDPP_OK;
}

}  // namespace

extern "C" {

int ccdpp_create(int64_t m, int64_t n, int32_t k, double lambda, int64_t nnz, const int32_t* row,
                 const int32_t* col, const float* val, uint64_t seed, ccdpp_t** out) {
    g_create_error.clear();
    if (!out) return fail(nullptr, CCDPP_EINVAL, "out is NULL");
    if (m < 1 || m >= kMaxDim || n < 1 || n >= kMaxDim)
        return fail(nullptr, CCDPP_EINVAL, "m and n must be in [1, 2^30)");
    if (k < 1) return fail(nullptr, CCDPP_EINVAL, "k must be >= 1");
    if (!std::isfinite(lambda) || lambda < 0.0)
        return fail(nullptr, CCDPP_EINVAL, "lambda must be finite and >= 0");
    if (nnz < 0 || nnz > kMaxNnz) return fail(nullptr, CCDPP_EINVAL, "nnz must be in [0, 2^31-1]");
    if (nnz > 0 && (!row || !col || !val))
        return fail(nullptr, CCDPP_EINVAL, "row, col and val must be non-NULL when nnz > 0");
    for (int64_t e = 0; e < nnz; ++e) {
        if (row[e] < 0 || row[e] >= m)
            return fail(nullptr, CCDPP_EINVAL, "row[%lld] = %d out of range", (long long)e, row[e]);
        if (col[e] < 0 || col[e] >= n)
            return fail(nullptr, CCDPP_EINVAL, "col[%lld] = %d out of range", (long long)e, col[e]);
        if (!std::isfinite(val[e]))
            return fail(nullptr, CCDPP_EINVAL, "val[%lld] is not finite", (long long)e);
    }
    ccdpp* h = new (std::nothrow) ccdpp();
    if (!h) return fail(nullptr, CCDPP_ENOMEM, "host allocation failed");
    h->m = m;
    h->n = n;
    h->k = k;
    h->lambda = lambda;
    h->nnz = nnz;
    int rc = create_device(h, row, col, val, seed);
    if (rc != CCDPP_OK) {
        g_create_error = h->err;
        destroy_all(h);
        delete h;
        return rc;
    }
    *out = h;
    return CCDPP_OK;
}

int ccdpp_run(ccdpp_t* h, int32_t outer, int32_t inner) {
    using namespace ccdk;
    if (!usable(h)) return CCDPP_ESTATE;
    if (outer < 0 || inner < 1)
        return fail(h, CCDPP_EINVAL, "outer_iters must be >= 0 and inner_iters >= 1");
    const int64_t m = h->m, n = h->n;
    int rc;
    for (int32_t it = 0; it < outer; ++it) {
        for (int32_t t = 0; t < h->k; ++t) {
            float* Wt = h->W + (int64_t)t * m;
            float* Ht = h->H + (int64_t)t * n;
            const bool prev = h->pending >= 0;
            const float* Wp = prev ? h->W + (int64_t)h->pending * m : nullptr;
            const float* Hp = prev ? h->H + (int64_t)h->pending * n : nullptr;
            const PassMode first = prev ? kModeSubAdd : kModeAdd;
            const int g1 = prev ? 2 : 1;
            // First u-pass: eq. 18 of the pending feature, eq. 13, eq. 15 with v = hbar_t.
            rc = pass(h, 0, first, Ht, Wt, Wp, Ht, Hp, h->u, g1);
            if (rc) return rc;
            // First v-pass: the same residual update on the column copy, eq. 16 with the new u.
            float* yv = inner == 1 ? Ht : h->v;
            rc = pass(h, 1, first, h->u, Ht, Hp, Wt, Wp, yv, g1 + 1);
            if (rc) return rc;
            for (int32_t s = 2; s <= inner; ++s) {
                const bool last = s == inner;
                float* yu = last ? Wt : h->u;  // the last u is committed in place (eq. 17)
                rc = pass(h, 0, kModePlain, h->v, nullptr, nullptr, nullptr, nullptr, yu, 1);
                if (rc) return rc;
                rc = pass(h, 1, kModePlain, yu, nullptr, nullptr, nullptr, nullptr,
                          last ? Ht : h->v, 1);
                if (rc) return rc;
            }
            if (inner == 1) {
                Timed tm(h, CCDPP_K_COMMIT, 8.0 * m);
                HIPCK(h, launch_copy(h->u, Wt, m, h->stream));
                tm.done();
            }
            h->pending = t;
        }
    }
    if (h->pending >= 0) {
        // Final eq. 18 on both copies; the row copy also sums R^2 for the training RMSE.
        const float* Wp = h->W + (int64_t)h->pending * m;
        const float* Hp = h->H + (int64_t)h->pending * n;
        rc = pass(h, 0, kModeFlush, nullptr, nullptr, Wp, nullptr, Hp, nullptr, 1);
        if (rc) return rc;
        HIPCK(h, launch_reduce_sum(h->sse_part, h->L[0].grid, h->d_scalar, h->stream));
        rc = pass(h, 1, kModeFlush, nullptr, nullptr, Hp, nullptr, Wp, nullptr, 1);
        if (rc) return rc;
        h->pending = -1;
        double sse = 0.0;
        HIPCK(h, hipMemcpyAsync(&sse, h->d_scalar, 8, hipMemcpyDeviceToHost, h->stream));
        HIPCK(h, hipStreamSynchronize(h->stream));
        h->train_sse = h->L[0].grid ? sse : 0.0;
        h->train_sse_valid = true;
    } else {
        HIPCK(h, hipStreamSynchronize(h->stream));
    }
    if (h->prof) collect_profile(h);
    return CCDPP_OK;
}

int ccdpp_get_factors(ccdpp_t* h, float* W, float* H) {
    if (!usable(h)) return CCDPP_ESTATE;
    hipStream_t s = h->stream;
    if (W) {
        float* d;
        Tmp t;
        HIPCK(h, talloc(t, &d, h->m * h->k));
        HIPCK(h, ccdk::launch_gather_factor_out(h->W, h->rold2new, h->m, h->k, d, s));
        HIPCK(h, hipMemcpyAsync(W, d, h->m * h->k * 4, hipMemcpyDeviceToHost, s));
        HIPCK(h, hipStreamSynchronize(s));
    }
    if (H) {
        float* d;
        Tmp t;
        HIPCK(h, talloc(t, &d, h->n * h->k));
        HIPCK(h, ccdk::launch_gather_factor_out(h->H, h->cold2new, h->n, h->k, d, s));
        HIPCK(h, hipMemcpyAsync(H, d, h->n * h->k * 4, hipMemcpyDeviceToHost, s));
        HIPCK(h, hipStreamSynchronize(s));
    }
    return CCDPP_OK;
}

int ccdpp_set_factors(ccdpp_t* h, const float* W, const float* H) {
    if (!usable(h)) return CCDPP_ESTATE;
    if (W)
        for (int64_t e = 0; e < h->m * h->k; ++e)
            if (!std::isfinite(W[e])) return fail(h, CCDPP_EINVAL, "W[%lld] is not finite", (long long)e);
    if (H)
        for (int64_t e = 0; e < h->n * h->k; ++e)
            if (!std::isfinite(H[e])) return fail(h, CCDPP_EINVAL, "H[%lld] is not finite", (long long)e);
    hipStream_t s = h->stream;
    if (W) {
        float* d;
        Tmp t;
        HIPCK(h, talloc(t, &d, h->m * h->k));
        HIPCK(h, hipMemcpyAsync(d, W, h->m * h->k * 4, hipMemcpyHostToDevice, s));
        HIPCK(h, ccdk::launch_scatter_factor_in(d, h->rnew2old, h->m, h->k, h->W, s));
        HIPCK(h, hipStreamSynchronize(s));
    }
    if (H) {
        float* d;
        Tmp t;
        HIPCK(h, talloc(t, &d, h->n * h->k));
        HIPCK(h, hipMemcpyAsync(d, H, h->n * h->k * 4, hipMemcpyHostToDevice, s));
        HIPCK(h, ccdk::launch_scatter_factor_in(d, h->cnew2old, h->n, h->k, h->H, s));
        HIPCK(h, hipStreamSynchronize(s));
    }
    HIPCK(h, ccdk::launch_rebuild_residual(h->L[0].ptr, h->L[0].idx, h->A, h->W, h->H, h->m,
                                            h->n, h->k, h->nnz, h->L[0].val, s));
    HIPCK(h, ccdk::launch_scatter_csc(h->L[0].val, h->csr2csc, h->nnz, h->L[1].val, s));
    HIPCK(h, hipStreamSynchronize(s));
    h->pending = -1;
    h->train_sse_valid = false;
    return CCDPP_OK;
}

int ccdpp_rmse(ccdpp_t* h, int64_t nnz, const int32_t* row, const int32_t* col, const float* val,
               double* rmse_out) {
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
    HIPCK(h, ccdk::launch_test_err(dr, dc, dv, nnz, h->rold2new, h->cold2new, h->W, h->H, h->m,
                                    h->n, h->k, h->sse_part, kReduceParts, s));
    HIPCK(h, ccdk::launch_reduce_sum(h->sse_part, kReduceParts, h->d_scalar, s));
    double sum = 0.0;
    HIPCK(h, hipMemcpyAsync(&sum, h->d_scalar, 8, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));
    *rmse_out = std::sqrt(sum / (double)nnz);
    return CCDPP_OK;
}

int ccdpp_train_rmse(ccdpp_t* h, double* rmse_out) {
    if (!usable(h)) return CCDPP_ESTATE;
    if (!rmse_out) return fail(h, CCDPP_EINVAL, "rmse_out is NULL");
    if (h->nnz < 1) return fail(h, CCDPP_EINVAL, "no observed entries");
    if (!h->train_sse_valid) {
        hipStream_t s = h->stream;
        HIPCK(h, ccdk::launch_sq_sum(h->L[0].val, h->nnz, h->sse_part, kReduceParts, s));
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
    if (!usable(h)) return CCDPP_ESTATE;
    if (!R && h->nnz) return fail(h, CCDPP_EINVAL, "R is NULL");
    if (h->nnz == 0) return CCDPP_OK;
    hipStream_t s = h->stream;
    float* d;
    Tmp t;
    HIPCK(h, talloc(t, &d, h->nnz));
    HIPCK(h, ccdk::launch_residual_out(h->L[0].val, h->csr_src, h->nnz, d, s));
    HIPCK(h, hipMemcpyAsync(R, d, h->nnz * 4, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));
    return CCDPP_OK;
}

int ccdpp_check_consistency(ccdpp_t* h, int64_t* mismatches) {
    if (!usable(h)) return CCDPP_ESTATE;
    if (!mismatches) return fail(h, CCDPP_EINVAL, "mismatches is NULL");
    hipStream_t s = h->stream;
    HIPCK(h, hipMemsetAsync(h->d_count, 0, 8, s));
    HIPCK(h, ccdk::launch_consistency(h->L[0].val, h->L[1].val, h->csr2csc, h->nnz, h->d_count, s));
    unsigned long long c = 0;
    HIPCK(h, hipMemcpyAsync(&c, h->d_count, 8, hipMemcpyDeviceToHost, s));
    HIPCK(h, hipStreamSynchronize(s));
    *mismatches = (int64_t)c;
    return CCDPP_OK;
}

int ccdpp_set_stream(ccdpp_t* h, void* hip_stream) {
    if (!usable(h)) return CCDPP_ESTATE;
    HIPCK(h, hipStreamSynchronize(h->stream));
    h->stream = hip_stream ? static_cast<hipStream_t>(hip_stream) : h->own_stream;
    return CCDPP_OK;
}

int ccdpp_profile(ccdpp_t* h, int32_t enable) {
    if (!usable(h)) return CCDPP_ESTATE;
    HIPCK(h, hipStreamSynchronize(h->stream));
    collect_profile(h);
    h->prof = enable != 0;
    for (int i = 0; i < CCDPP_K_COUNT; ++i) {
        h->prof_launch[i] = 0;
        h->prof_ms[i] = 0.0;
        h->prof_bytes[i] = 0.0;
    }
    return CCDPP_OK;
}

int ccdpp_profile_read(ccdpp_t* h, int32_t kind, int64_t* launches, double* total_ms,
                       double* algo_bytes) {
    if (!usable(h)) return CCDPP_ESTATE;
    if (kind < 0 || kind >= CCDPP_K_COUNT) return fail(h, CCDPP_EINVAL, "bad kernel kind");
    if (launches) *launches = h->prof_launch[kind];
    if (total_ms) *total_ms = h->prof_ms[kind];
    if (algo_bytes) *algo_bytes = h->prof_bytes[kind];
    return CCDPP_OK;
}

int ccdpp_info(ccdpp_t* h, int64_t* out, int32_t len) {
    if (!h) return CCDPP_ESTATE;
    if (!out || len < 0) return fail(h, CCDPP_EINVAL, "bad output buffer");
    const int64_t v[12] = {h->m,
                           h->n,
                           h->nnz,
                           h->k,
                           h->build_us,
                           h->L[0].nblock_rows,
                           h->L[0].nsplit,
                           h->L[0].grid,
                           h->L[1].nblock_rows,
                           h->L[1].nsplit,
                           h->L[1].grid,
                           h->bytes_held};
    int32_t w = std::min<int32_t>(len, 12);
    for (int32_t i = 0; i < w; ++i) out[i] = v[i];
    return w;
}

const char* ccdpp_last_error(const ccdpp_t* h) {
    if (!h) return g_create_error.c_str();
    return h->err.c_str();
}

void ccdpp_destroy(ccdpp_t* h) {
    if (!h) return;
    if (h->stream) hipStreamSynchronize(h->stream);
    destroy_all(h);
    delete h;
}

}  // extern "C"
