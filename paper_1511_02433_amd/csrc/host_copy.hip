// Host-side helpers of the library's set-up: a loop split over a few host threads,
// and the copy of caller (pageable) host memory to the device through two pinned
// staging buffers, host threads filling one while the DMA engine drains the other.
#include <algorithm>
#include <cstring>
#include <system_error>
#include <thread>
#include <vector>

#include "ccdpp_internal.hpp"

namespace ccdk {

int host_workers() {
    const unsigned hc = std::thread::hardware_concurrency();
    return (int)std::max(1u, std::min(hc == 0 ? 1u : hc, 8u));
}

void parallel_ranges(int64_t n, int workers, const std::function<void(int, int64_t, int64_t)>& f) {
    workers = (int)std::max<int64_t>(1, std::min<int64_t>(workers, n));
    const int64_t per = (n + workers - 1) / workers;
    std::vector<std::thread> pool;
    pool.reserve(workers - 1);
    int w = 0;
    for (; w + 1 < workers; ++w) {
        const int64_t lo = std::min(n, w * per), hi = std::min(n, lo + per);
        try {
            pool.emplace_back(f, w, lo, hi);
        } catch (const std::system_error&) {
            break;  // no more threads: the calling thread does the rest
        }
    }
    f(w, std::min(n, w * per), n);
    for (auto& t : pool) t.join();
}

namespace {
constexpr size_t kStageBytes = size_t(32) << 20;  // per staging buffer
constexpr size_t kStageMin = size_t(4) << 20;     // smaller copies go straight through
}  // namespace

Stager::Stager(hipStream_t s) : s_(s), workers_(host_workers()) {}

Stager::~Stager() { release(); }

void Stager::release() {
    for (int b = 0; b < 2; ++b) {
        if (ev_[b]) {
            if (busy_[b]) (void)hipEventSynchronize(ev_[b]);
            (void)hipEventDestroy(ev_[b]);
            ev_[b] = nullptr;
        }
        busy_[b] = false;
        if (slot_[b]) {
            (void)hipHostFree(slot_[b]);
            slot_[b] = nullptr;
        }
    }
}

// The pinned buffers, on first use.  Without them (no pinned memory to be had) every
// copy goes straight from the caller's memory.
bool Stager::ready() {
    if (tried_) return slot_[0] != nullptr;
    tried_ = true;
    for (int b = 0; b < 2; ++b) {
        if (hipHostMalloc(&slot_[b], kStageBytes, hipHostMallocDefault) != hipSuccess ||
            hipEventCreateWithFlags(&ev_[b], hipEventDisableTiming) != hipSuccess) {
            (void)hipGetLastError();
            release();
            return false;
        }
    }
    return true;
}

hipError_t Stager::copy(void* dst, const void* src, size_t bytes) {
    if (bytes == 0) return hipSuccess;
    if (bytes < kStageMin || !ready())
        return hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s_);
    const char* from = static_cast<const char*>(src);
    char* to = static_cast<char*>(dst);
    for (size_t off = 0; off < bytes; off += kStageBytes) {
        const size_t len = std::min(kStageBytes, bytes - off);
        const int b = next_;
        next_ ^= 1;
        if (busy_[b]) {
            hipError_t e = hipEventSynchronize(ev_[b]);  // its last copy has read it
            if (e != hipSuccess) return e;
            busy_[b] = false;
        }
        char* slot = static_cast<char*>(slot_[b]);
        const int64_t lines = (int64_t)((len + 63) / 64);
        parallel_ranges(lines, workers_, [&](int, int64_t lo, int64_t hi) {
            const size_t a = (size_t)lo * 64, z = std::min(len, (size_t)hi * 64);
            if (z > a) std::memcpy(slot + a, from + off + a, z - a);
        });
        hipError_t e = hipMemcpyAsync(to + off, slot, len, hipMemcpyHostToDevice, s_);
        if (e != hipSuccess) return e;
        e = hipEventRecord(ev_[b], s_);
        if (e != hipSuccess) return e;
        busy_[b] = true;
    }
    return hipSuccess;
}

hipError_t Stager::finish() {
    for (int b = 0; b < 2; ++b) {
        if (busy_[b]) {
            hipError_t e = hipEventSynchronize(ev_[b]);
            if (e != hipSuccess) return e;
            busy_[b] = false;
        }
    }
    return hipSuccess;
}

}  // namespace ccdk
