// api.cpp -- the C ABI of include/krex.h: argument validation, counter-and-
// gate around every launch, device-completion tracking of counted work,
// region entry and exit, and the timed loop.
//
// Completion tracking follows the AMD variant of the paper (Section 5): a
// launch raises the process's in-flight count when it is admitted, and the
// count drops when the HIP event recorded right after the launch completes,
// observed by one tracking thread per process that blocks on such events. A failed launch releases its count at once (Section
// 4.2: decrement on error returns too).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <chrono>
#include <condition_variable>
#include <deque>
#include <map>
#include <mutex>
#include <thread>
#include <vector>

#include "gate.hpp"
#include "krex.h"
#include "launch.hpp"

namespace {

thread_local int32_t g_last_hip = 0;
thread_local hipError_t g_fn_error = hipSuccess;   // set by the ready-made launch functions

krex_status hip_fail(hipError_t e)
{
    g_last_hip = (int32_t)e;
    return KREX_EHIP;
}

size_t elem_size(int32_t dt)
{
    switch (dt) {
    case KREX_F32: return 4;
    case KREX_BF16: return 2;
    case KREX_F16: return 2;
    case KREX_F8E4M3: return 1;
    case KREX_U32: return 4;
    default: return 0;
    }
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

int current_device()
{
    int d = 0;
    if (hipGetDevice(&d) != hipSuccess) return 0;
    return d;
}

// ------------------------------------------------------------ completion tracking

class Tracker {
public:
    // Records a completion event for counted work on `s` and hands it to the
    // tracking thread. On failure the count is released here. may_create =
    // false (the entry point that allocates nothing): only a pooled event is
    // used; with the pool empty the call waits for `s` and releases the
    // count itself.
    krex_status track(hipStream_t s, bool may_create = true)
    {
        const int dev = current_device();
        hipEvent_t ev = take_event(dev, may_create);
        if (!ev && !may_create) {
            const hipError_t w = hipStreamSynchronize(s);
            if (w != hipSuccess) krexg::mark_failed();
            krexg::release(1);
            return w == hipSuccess ? KREX_OK : hip_fail(w);
        }
        hipError_t e = ev ? hipEventRecord(ev, s) : hipErrorOutOfMemory;
        if (e != hipSuccess) {
            if (ev) give_event(dev, ev);
            krexg::release(1);
            return hip_fail(e);
        }
        {
            std::lock_guard<std::mutex> g(mu_);
            q_.push_back({ev, dev});
            pending_.fetch_add(1);
            if (!started_) {
                started_ = true;
                th_ = std::thread([this] { run(); });
                atexit([] { Tracker::instance().shutdown(); });
            }
        }
        cv_.notify_one();
        return KREX_OK;
    }

    // Waits (up to timeout_ms) until every tracked operation was released.
    bool drain(uint32_t timeout_ms)
    {
        const auto end = std::chrono::steady_clock::now() + std::chrono::milliseconds(timeout_ms);
        while (pending_.load() != 0) {
            if (std::chrono::steady_clock::now() > end) return false;
            std::this_thread::sleep_for(std::chrono::microseconds(50));
        }
        return true;
    }

    // Creates up to n pooled events for device dev (made current meanwhile),
    // so that counted launches on it need not create any.
    void prefill(int dev, size_t n)
    {
        if (dev < 0 || dev >= 64) return;
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) return;
        if (cur != dev && hipSetDevice(dev) != hipSuccess) return;
        {
            std::lock_guard<std::mutex> g(pool_mu_);
            while (pool_[dev].size() < n) {
                hipEvent_t ev = nullptr;
                if (hipEventCreateWithFlags(&ev, hipEventDisableTiming | hipEventBlockingSync) != hipSuccess) break;
                pool_[dev].push_back(ev);
            }
        }
        if (cur != dev) (void)hipSetDevice(cur);
    }

    static Tracker &instance()
    {
        static Tracker *t = new Tracker();   // never destroyed; the thread is joined at exit
        return *t;
    }

private:
    struct Item {
        hipEvent_t ev;
        int dev;
    };

    hipEvent_t take_event(int dev, bool may_create)
    {
        std::lock_guard<std::mutex> g(pool_mu_);
        if (dev >= 0 && dev < 64 && !pool_[dev].empty()) {
            hipEvent_t ev = pool_[dev].back();
            pool_[dev].pop_back();
            return ev;
        }
        if (!may_create) return nullptr;
        hipEvent_t ev = nullptr;
        if (hipEventCreateWithFlags(&ev, hipEventDisableTiming | hipEventBlockingSync) != hipSuccess) return nullptr;
        return ev;
    }

    void give_event(int dev, hipEvent_t ev)
    {
        std::lock_guard<std::mutex> g(pool_mu_);
        if (dev >= 0 && dev < 64) pool_[dev].push_back(ev);
        else (void)hipEventDestroy(ev);   // a pool beyond 64 devices is not kept
    }

    void run()
    {
        int cur = -1;
        for (;;) {
            Item it;
            {
                std::unique_lock<std::mutex> g(mu_);
                cv_.wait(g, [this] { return !q_.empty() || stop_; });
                if (q_.empty()) return;   // stop requested and nothing left
                it = q_.front();
                q_.pop_front();
            }
            if (it.dev != cur) {
                // a failure shows in the event wait below, which marks the slot failed
                (void)hipSetDevice(it.dev);
                cur = it.dev;
            }
            // A failed wait means the context hit a device error: the count is
            // released and the slot marked failed (no sibling waits on it).
            if (hipEventSynchronize(it.ev) != hipSuccess) krexg::mark_failed();
            krexg::release(1);
            give_event(it.dev, it.ev);
            pending_.fetch_sub(1);
        }
    }

    void shutdown()
    {
        {
            std::lock_guard<std::mutex> g(mu_);
            stop_ = true;
        }
        cv_.notify_all();
        if (th_.joinable()) th_.join();
    }

    std::mutex mu_;
    std::condition_variable cv_;
    std::deque<Item> q_;
    std::thread th_;
    bool started_ = false;
    bool stop_ = false;
    std::atomic<int64_t> pending_{0};
    std::mutex pool_mu_;
    std::vector<hipEvent_t> pool_[64];
};

uint64_t gate_timeout_ns()
{
    static uint64_t t = [] {
        const char *e = getenv("KREX_GATE_TIMEOUT_MS");
        return e ? (uint64_t)strtoull(e, nullptr, 10) * 1000000ull : 0ull;
    }();
    return t;
}

// True when `s` is capturing into a HIP graph: its launches are recorded,
// not run.
bool capturing(hipStream_t s)
{
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    return hipStreamIsCapturing(s, &cs) == hipSuccess && cs != hipStreamCaptureStatusNone;
}

// Counter-and-gate around one submission: admit, launch, then either track
// its completion or release it at once on failure. may_create: see
// Tracker::track.
template <typename F>
krex_status submit(hipStream_t s, F &&launch_fn, bool may_create = true)
{
    // With the dispatch interceptor active every kernel is counted at its
    // queue; counting here too could hold a count while the same launch
    // waits at the gate. A launch recorded into a graph runs only when the
    // graph is launched, which this library does not see: nothing is in
    // flight to count now, and a completion event recorded during capture
    // would never be reached.
    if (krexg::intercepted() || capturing(s)) {
        const hipError_t e = launch_fn();
        return e == hipSuccess ? KREX_OK : hip_fail(e);
    }
    bool counted = false;
    const int rc = krexg::admit(gate_timeout_ns(), &counted);
    if (rc != KREX_OK) return rc;
    const hipError_t e = launch_fn();
    if (e != hipSuccess) {
        if (counted) krexg::release(1);
        return hip_fail(e);
    }
    if (counted) return Tracker::instance().track(s, may_create);
    return KREX_OK;
}

// Chunked submission (KREX_CHUNK_BYTES, off when unset or 0): a gated
// process splits a large generation, injection or flush into launches of at
// most that many output bytes, each admitted through counter-and-gate on its
// own, and keeps at most KREX_CHUNK_DEPTH (default 2) of them in flight,
// waiting for the oldest before it submits the next. A region entered by
// another process then waits for at most that many chunks of this call
// (Section 4.2 step 3: the drain), not for the whole tensor, and the rest
// parks at the closed gate. Generation and injection are counter-based, so
// a chunk [j0, j0 + m) is the same call on the shifted pointers and offsets
// and writes the same values. Chunk lengths are multiples of 64 elements,
// which keeps aligned calls on their vector paths.
uint64_t chunk_bytes()
{
    static const uint64_t v = [] {
        const char *e = getenv("KREX_CHUNK_BYTES");
        return e ? (uint64_t)strtoull(e, nullptr, 10) : 0ull;
    }();
    return v;
}

uint32_t chunk_depth()
{
    static const uint32_t v = [] {
        const char *e = getenv("KREX_CHUNK_DEPTH");
        const unsigned long d = e ? strtoul(e, nullptr, 10) : 2ul;
        return (uint32_t)(d == 0 ? 1 : (d > 16 ? 16 : d));
    }();
    return v;
}

// Events marking the chunks in flight, per thread and device (created with
// that device current, kept for the thread's life).
hipEvent_t *chunk_events(int dev, uint32_t count)
{
    thread_local std::vector<hipEvent_t> by_dev[krex::kMaxDevices];
    if (dev < 0 || dev >= krex::kMaxDevices) return nullptr;
    std::vector<hipEvent_t> &ev = by_dev[dev];
    while (ev.size() < count) {
        hipEvent_t e = nullptr;
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return nullptr;
        ev.push_back(e);
    }
    return ev.data();
}

// launch(j0, m) enqueues elements [j0, j0 + m) of an n-element call whose
// elements are `elem_bytes` each.
template <typename F>
krex_status submit_chunked(hipStream_t s, uint64_t n, uint64_t elem_bytes, F &&launch)
{
    const uint64_t cb = chunk_bytes();
    const bool chunk = cb != 0 && krexg::attached() && krexg::gated() && !krexg::intercepted() &&
                       !krexg::in_region() && !capturing(s);
    uint64_t per = chunk ? cb / elem_bytes : n;
    per -= per % 64;
    if (!chunk || per == 0 || n <= per) return submit(s, [&] { return launch(0, n); });
    const uint32_t depth = chunk_depth();
    hipEvent_t *ev = chunk_events(current_device(), depth);
    if (!ev) return hip_fail(hipErrorOutOfMemory);
    uint64_t k = 0;
    for (uint64_t j0 = 0; j0 < n; j0 += per, ++k) {
        if (k >= depth) {
            const hipError_t e = hipEventSynchronize(ev[k % depth]);
            if (e != hipSuccess) return hip_fail(e);
        }
        const uint64_t m = (n - j0) < per ? (n - j0) : per;
        const krex_status st = submit(s, [&] { return launch(j0, m); });
        if (st != KREX_OK) return st;
        const hipError_t e = hipEventRecord(ev[k % depth], s);
        if (e != hipSuccess) return hip_fail(e);
    }
    return KREX_OK;
}

// Cached timing events for the timed loop, per device.
std::mutex g_ev_mu;
std::vector<hipEvent_t> g_timing_events[64];

krex_status timing_events(int dev, size_t count, hipEvent_t **out)
{
    if (dev < 0 || dev >= 64) return KREX_EINVAL;
    std::vector<hipEvent_t> &v = g_timing_events[dev];
    while (v.size() < count) {
        hipEvent_t ev;
        hipError_t e = hipEventCreate(&ev);
        if (e != hipSuccess) return hip_fail(e);
        v.push_back(ev);
    }
    *out = v.data();
    return KREX_OK;
}

// Per-(device, stream) scratch of the check's block partials, allocated on
// first use and kept: calls on one stream are ordered by the stream, calls
// on different streams use different buffers.
std::mutex g_scratch_mu;
std::map<std::pair<int, hipStream_t>, void *> g_scratch;

krex_status check_scratch(hipStream_t s, void **out)
{
    const int dev = current_device();
    std::lock_guard<std::mutex> g(g_scratch_mu);
    auto it = g_scratch.find({dev, s});
    if (it != g_scratch.end()) {
        *out = it->second;
        return KREX_OK;
    }
    void *p = nullptr;
    const hipError_t e = hipMalloc(&p, krex::check_scratch_bytes());
    if (e != hipSuccess) return hip_fail(e);
    g_scratch[{dev, s}] = p;
    *out = p;
    return KREX_OK;
}

bool finite_f(float x) { return isfinite(x) != 0; }

bool gen_params_ok(int32_t dist, float p0, float p1)
{
    if (dist == KREX_UNIFORM) return finite_f(p0) && finite_f(p1) && p0 <= p1 && finite_f(p1 - p0);
    if (dist == KREX_NORMAL) return finite_f(p0) && finite_f(p1) && p1 >= 0.0f;
    return dist == KREX_BITCAST;
}

int32_t g_device_attached = -1;

}  // namespace

namespace krex {

int device_cus()
{
    static std::atomic<int> cache[64];
    const int dev = current_device();
    if (dev < 0 || dev >= 64) return 256;
    int v = cache[dev].load();
    if (v == 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
        cache[dev].store(v);
    }
    return v;
}

}  // namespace krex

extern "C" {

// Completion events created per device at attach, so that counted launches
// (among them those of the entry point that allocates nothing) take pooled
// ones.
static constexpr size_t kEventPrefill = 64;

krex_status krex_attach(int32_t device, const char *shm_name, uint32_t flags)
{
    if (flags & ~(KREX_ATTACH_NO_GATE | KREX_ATTACH_CPU_EXCLUSIVE)) return KREX_EINVAL;
    if (krexg::intercepted() && krexg::attached()) {
        // Registered by the dispatch interceptor: reuse that registration.
        if (((flags & KREX_ATTACH_NO_GATE) != 0) != ((krexg::flags() & krexg::kNoGate) != 0)) return KREX_ESTATE;
        krexg::set_cpu_exclusive((flags & KREX_ATTACH_CPU_EXCLUSIVE) != 0);
        g_device_attached = device;
        return KREX_OK;
    }
    char name[256];
    if (shm_name) {
        if (strlen(shm_name) >= sizeof name) return KREX_EINVAL;
        strcpy(name, shm_name);
    } else {
        char bus[64];
        hipError_t e = hipDeviceGetPCIBusId(bus, (int)sizeof bus, device);
        if (e != hipSuccess) return hip_fail(e);
        for (char *p = bus; *p; ++p)
            if (*p == ':' || *p == '.') *p = '_';
        snprintf(name, sizeof name, "/krex-%s", bus);
    }
    const uint32_t gf = ((flags & KREX_ATTACH_NO_GATE) ? krexg::kNoGate : 0u) |
                        ((flags & KREX_ATTACH_CPU_EXCLUSIVE) ? krexg::kCpuExclusive : 0u);
    const int rc = krexg::attach(name, gf);
    if (rc == KREX_OK) {
        g_device_attached = device;
        if (!(flags & KREX_ATTACH_NO_GATE)) Tracker::instance().prefill(device, kEventPrefill);
    }
    return rc;
}

krex_status krex_detach(void)
{
    if (!krexg::attached()) return KREX_ESTATE;
    if (krexg::in_region()) return KREX_ESTATE;
    if (krexg::intercepted()) return KREX_OK;   // the interceptor's registration stays
    if (!Tracker::instance().drain(60000)) return KREX_ETIMEDOUT;
    const int rc = krexg::detach();
    if (rc == KREX_OK) g_device_attached = -1;
    return rc;
}

krex_status krex_gen(void *dst, int32_t dtype, uint64_t n, uint64_t seed, uint64_t offset, int32_t dist, float p0,
                     float p1, void *stream)
{
    const size_t es = elem_size(dtype);
    if (es == 0) return KREX_EINVAL;
    if (dtype != KREX_U32 && !gen_params_ok(dist, p0, p1)) return KREX_EINVAL;
    if (n > 0 && offset > UINT64_MAX - (n - 1)) return KREX_EINVAL;
    if (n > 0 && !dst) return KREX_EINVAL;
    if (!aligned(dst, es)) return KREX_EALIGN;
    if (n == 0) return KREX_OK;
    hipStream_t s = (hipStream_t)stream;
    return submit_chunked(s, n, es, [&](uint64_t j0, uint64_t m) {
        return krex::launch_gen((uint8_t *)dst + j0 * es, dtype, m, seed, offset + j0, dist, p0, p1, s);
    });
}

krex_status krex_gen_packed(void *dst, int32_t dtype, uint64_t n, uint64_t seed, uint64_t offset, int32_t dist,
                            float p0, float p1, void *stream)
{
    if (dtype != KREX_BF16 && dtype != KREX_F16 && dtype != KREX_F8E4M3) return KREX_EINVAL;
    const size_t es = elem_size(dtype);
    if (!gen_params_ok(dist, p0, p1)) return KREX_EINVAL;
    if (n > 0 && offset > UINT64_MAX - (n - 1)) return KREX_EINVAL;
    if (n > 0 && !dst) return KREX_EINVAL;
    if (!aligned(dst, es)) return KREX_EALIGN;
    if (n == 0) return KREX_OK;
    hipStream_t s = (hipStream_t)stream;
    return submit_chunked(s, n, es, [&](uint64_t j0, uint64_t m) {
        return krex::launch_gen_packed((uint8_t *)dst + j0 * es, dtype, m, seed, offset + j0, dist, p0, p1, s);
    });
}

krex_status krex_transform_words(void *dst, int32_t dtype, uint64_t n, const uint32_t *words, int32_t dist, float p0,
                                 float p1, void *stream)
{
    const size_t es = elem_size(dtype);
    if (es == 0) return KREX_EINVAL;
    if (dtype != KREX_U32 && !gen_params_ok(dist, p0, p1)) return KREX_EINVAL;
    if (dtype != KREX_U32 && dist == KREX_NORMAL && (n & 1u)) return KREX_EINVAL;
    if (n > 0 && (!dst || !words)) return KREX_EINVAL;
    if (!aligned(dst, es) || !aligned(words, 4)) return KREX_EALIGN;
    if (n == 0) return KREX_OK;
    hipStream_t s = (hipStream_t)stream;
    return submit(s, [&] { return krex::launch_xform(dst, dtype, n, words, dist, p0, p1, s); });
}

krex_status krex_inject(void *y, const void *x, int32_t dtype, uint64_t n, uint64_t mask_seed, uint64_t mask_offset,
                        double rate, float delta, int32_t mode, void *stream)
{
    const size_t es = elem_size(dtype);
    if (es == 0 || dtype == KREX_U32) return KREX_EINVAL;
    if (!(rate >= 0.0 && rate <= 1.0)) return KREX_EINVAL;
    if (!finite_f(delta)) return KREX_EINVAL;
    if (mode != KREX_INJ_ROUND && mode != KREX_INJ_EXACT) return KREX_EINVAL;
    if (n > 0 && mask_offset > UINT64_MAX - (n - 1)) return KREX_EINVAL;
    if (n > 0 && (!x || !y)) return KREX_EINVAL;
    if (!aligned(x, es) || !aligned(y, es)) return KREX_EALIGN;
    if (n == 0) return KREX_OK;
    if (x != y) {
        const uintptr_t xa = (uintptr_t)x, ya = (uintptr_t)y, len = (uintptr_t)(n * es);
        if (xa < ya + len && ya < xa + len) return KREX_EINVAL;   // partial overlap
    }
    double t = floor(rate * 4294967296.0);
    const uint64_t T = t <= 0.0 ? 0ull : (t >= 4294967296.0 ? (1ull << 32) : (uint64_t)t);
    hipStream_t s = (hipStream_t)stream;
    return submit_chunked(s, n, es, [&](uint64_t j0, uint64_t m) {
        return krex::launch_inject((uint8_t *)y + j0 * es, (const uint8_t *)x + j0 * es, dtype, m, mask_seed,
                                   mask_offset + j0, T, delta, mode, s);
    });
}

krex_status krex_gen_inject(void *x, void *y, int32_t dtype, uint64_t n, uint64_t seed, uint64_t offset,
                            int32_t dist, float p0, float p1, uint64_t mask_seed, uint64_t mask_offset, double rate,
                            float delta, int32_t mode, void *stream)
{
    const size_t es = elem_size(dtype);
    if (es == 0 || dtype == KREX_U32) return KREX_EINVAL;
    if (!gen_params_ok(dist, p0, p1)) return KREX_EINVAL;
    if (!(rate >= 0.0 && rate <= 1.0)) return KREX_EINVAL;
    if (!finite_f(delta)) return KREX_EINVAL;
    if (mode != KREX_INJ_ROUND && mode != KREX_INJ_EXACT) return KREX_EINVAL;
    if (n > 0 && (offset > UINT64_MAX - (n - 1) || mask_offset > UINT64_MAX - (n - 1))) return KREX_EINVAL;
    if (n > 0 && (!x || !y)) return KREX_EINVAL;
    if (!aligned(x, es) || !aligned(y, es)) return KREX_EALIGN;
    if (n == 0) return KREX_OK;
    const uintptr_t xa = (uintptr_t)x, ya = (uintptr_t)y, len = (uintptr_t)(n * es);
    if (xa < ya + len && ya < xa + len) return KREX_EINVAL;   // two outputs: no overlap at all
    double t = floor(rate * 4294967296.0);
    const uint64_t T = t <= 0.0 ? 0ull : (t >= 4294967296.0 ? (1ull << 32) : (uint64_t)t);
    hipStream_t s = (hipStream_t)stream;
    return submit_chunked(s, n, 2 * es, [&](uint64_t j0, uint64_t m) {
        return krex::launch_gen_inject((uint8_t *)x + j0 * es, (uint8_t *)y + j0 * es, dtype, m, seed, offset + j0,
                                       dist, p0, p1, mask_seed, mask_offset + j0, T, delta, mode, s);
    });
}

krex_status krex_check(const void *a, int32_t dta, const void *b, int32_t dtb, uint64_t n, float rtol, float atol,
                       krex_check_result *out, void *stream)
{
    const size_t sa = elem_size(dta), sb = elem_size(dtb);
    if (sa == 0 || sb == 0 || dta == KREX_U32 || dtb == KREX_U32) return KREX_EINVAL;
    if (!(rtol >= 0.0f) || !(atol >= 0.0f) || !finite_f(rtol) || !finite_f(atol)) return KREX_EINVAL;
    if (n >= (1ull << 33)) return KREX_EINVAL;
    if (!out) return KREX_EINVAL;
    if (n > 0 && (!a || !b)) return KREX_EINVAL;
    if (!aligned(a, sa) || !aligned(b, sb) || !aligned(out, 8)) return KREX_EALIGN;
    hipStream_t s = (hipStream_t)stream;
    void *scratch = nullptr;
    const krex_status rc = check_scratch(s, &scratch);
    if (rc != KREX_OK) return rc;
    return submit(s, [&] { return krex::launch_check(a, dta, b, dtb, n, rtol, atol, scratch, out, s); });
}

krex_status krex_check_noalloc(const void *a, int32_t dta, const void *b, int32_t dtb, uint64_t n, float rtol,
                               float atol, krex_check_result *out, void *stream)
{
    const size_t sa = elem_size(dta), sb = elem_size(dtb);
    if (sa == 0 || sb == 0 || dta == KREX_U32 || dtb == KREX_U32) return KREX_EINVAL;
    if (!(rtol >= 0.0f) || !(atol >= 0.0f) || !finite_f(rtol) || !finite_f(atol)) return KREX_EINVAL;
    // the fixed scratch holds the partials of every grid the check uses, so
    // the size limit is the check's own: n < 2^33
    if (n >= (1ull << 33)) return KREX_EINVAL;
    if (!out) return KREX_EINVAL;
    if (n > 0 && (!a || !b)) return KREX_EINVAL;
    if (!aligned(a, sa) || !aligned(b, sb) || !aligned(out, 8)) return KREX_EALIGN;
    hipStream_t s = (hipStream_t)stream;
    void *scratch = nullptr;
    const hipError_t e = krex::noalloc_scratch(&scratch);
    if (e != hipSuccess) return hip_fail(e);
    return submit(s, [&] { return krex::launch_check(a, dta, b, dtb, n, rtol, atol, scratch, out, s); },
                  /*may_create=*/false);
}

krex_status krex_check_gen(const void *a, int32_t dta, int32_t dtb, uint64_t n, uint64_t seed, uint64_t offset,
                           int32_t dist, float p0, float p1, float rtol, float atol, krex_check_result *out,
                           void *stream)
{
    const size_t sa = elem_size(dta), sb = elem_size(dtb);
    if (sa == 0 || sb == 0 || dta == KREX_U32 || dtb == KREX_U32) return KREX_EINVAL;
    if (!gen_params_ok(dist, p0, p1)) return KREX_EINVAL;
    if (!(rtol >= 0.0f) || !(atol >= 0.0f) || !finite_f(rtol) || !finite_f(atol)) return KREX_EINVAL;
    if (n >= (1ull << 33)) return KREX_EINVAL;
    if (n > 0 && offset > UINT64_MAX - (n - 1)) return KREX_EINVAL;
    if (!out) return KREX_EINVAL;
    if (n > 0 && !a) return KREX_EINVAL;
    if (!aligned(a, sa) || !aligned(out, 8)) return KREX_EALIGN;
    hipStream_t s = (hipStream_t)stream;
    void *scratch = nullptr;
    const krex_status rc = check_scratch(s, &scratch);
    if (rc != KREX_OK) return rc;
    return submit(s, [&] {
        return krex::launch_check_gen(a, dta, dtb, n, seed, offset, dist, p0, p1, rtol, atol, scratch, out, s);
    });
}

krex_status krex_check_gen_packed(const void *a, int32_t dta, int32_t dtb, uint64_t n, uint64_t seed,
                                  uint64_t offset, int32_t dist, float p0, float p1, float rtol, float atol,
                                  krex_check_result *out, void *stream)
{
    const size_t sa = elem_size(dta);
    if (sa == 0 || dta == KREX_U32) return KREX_EINVAL;
    if (dtb != KREX_BF16 && dtb != KREX_F16 && dtb != KREX_F8E4M3) return KREX_EINVAL;
    if (!gen_params_ok(dist, p0, p1)) return KREX_EINVAL;
    if (!(rtol >= 0.0f) || !(atol >= 0.0f) || !finite_f(rtol) || !finite_f(atol)) return KREX_EINVAL;
    if (n >= (1ull << 33)) return KREX_EINVAL;
    if (n > 0 && offset > UINT64_MAX - (n - 1)) return KREX_EINVAL;
    if (!out) return KREX_EINVAL;
    if (n > 0 && !a) return KREX_EINVAL;
    if (!aligned(a, sa) || !aligned(out, 8)) return KREX_EALIGN;
    hipStream_t s = (hipStream_t)stream;
    void *scratch = nullptr;
    const krex_status rc = check_scratch(s, &scratch);
    if (rc != KREX_OK) return rc;
    return submit(s, [&] {
        return krex::launch_check_gen_packed(a, dta, dtb, n, seed, offset, dist, p0, p1, rtol, atol, scratch, out, s);
    });
}

krex_status krex_flush(void *buf, uint64_t bytes, uint32_t pattern, void *stream)
{
    if (bytes % 16 != 0) return KREX_EINVAL;
    if (bytes > 0 && !buf) return KREX_EINVAL;
    if (!aligned(buf, 16)) return KREX_EALIGN;
    if (bytes == 0) return KREX_OK;
    hipStream_t s = (hipStream_t)stream;
    return submit_chunked(s, bytes / 16, 16, [&](uint64_t j0, uint64_t m) {
        return krex::launch_flush((uint8_t *)buf + j0 * 16, m * 16, pattern, s);
    });
}

krex_status krex_probe(uint64_t iters, float *sink, void *stream)
{
    if (!sink) return KREX_EINVAL;
    if (!aligned(sink, 4)) return KREX_EALIGN;
    hipStream_t s = (hipStream_t)stream;
    return submit(s, [&] { return krex::launch_probe(iters, sink, nullptr, s); });
}

krex_status krex_probe_clocked(uint64_t iters, float *sink, uint64_t *clocks, void *stream)
{
    if (!sink || !clocks) return KREX_EINVAL;
    if (!aligned(sink, 4) || !aligned(clocks, 16)) return KREX_EALIGN;
    hipStream_t s = (hipStream_t)stream;
    return submit(s, [&] { return krex::launch_probe(iters, sink, clocks, s); });
}

krex_status krex_fixture_sgemm(uint32_t M, uint32_t N, uint32_t K, const float *A, const float *B, float *C,
                               void *stream)
{
    if ((uint64_t)M * N > 0 && (!C || (K > 0 && (!A || !B)))) return KREX_EINVAL;
    if (!aligned(A, 4) || !aligned(B, 4) || !aligned(C, 4)) return KREX_EALIGN;
    hipStream_t s = (hipStream_t)stream;
    return submit(s, [&] { return krex::launch_sgemm(M, N, K, A, B, C, s); });
}

void krex_probe_launch(void *user, void *stream)
{
    const krex_probe_args *a = (const krex_probe_args *)user;
    const hipError_t e = krex::launch_probe(a->iters, a->sink, a->clocks, (hipStream_t)stream);
    if (e != hipSuccess && g_fn_error == hipSuccess) g_fn_error = e;
}

void krex_sgemm_launch(void *user, void *stream)
{
    const krex_sgemm_args *a = (const krex_sgemm_args *)user;
    const hipError_t e = krex::launch_sgemm(a->M, a->N, a->K, a->A, a->B, a->C, (hipStream_t)stream);
    if (e != hipSuccess && g_fn_error == hipSuccess) g_fn_error = e;
}

krex_status krex_region_begin(void *stream, uint32_t timeout_ms, void *flush_buf, uint64_t flush_bytes)
{
    if (!krexg::attached()) return KREX_ENOTATTACHED;
    if (krexg::in_region()) return KREX_ESTATE;
    if (flush_buf && (flush_bytes % 16 != 0 || !aligned(flush_buf, 16))) return KREX_EINVAL;
    // This process's own earlier work finishes before the region starts.
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e);
    const int rc = krexg::region_begin(timeout_ms);
    if (rc < 0) return rc;
    if (flush_buf && flush_bytes) {
        hipStream_t s = (hipStream_t)stream;
        e = krex::launch_flush(flush_buf, flush_bytes, 0u, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) {
            krexg::region_end();
            return hip_fail(e);
        }
    }
    return rc;
}

krex_status krex_region_end(void *stream)
{
    (void)stream;
    if (!krexg::attached()) return KREX_ENOTATTACHED;
    if (!krexg::in_region()) return KREX_ESTATE;
    // The region's work (on any stream of this process) finishes before the
    // gate reopens; the region is left even if that wait reports an error.
    const hipError_t e = hipDeviceSynchronize();
    const int rc = krexg::region_end();
    if (e != hipSuccess) return hip_fail(e);
    return rc;
}

krex_status krex_time_loop(krex_launch_fn fn, void *user, uint32_t warmup, uint32_t reps, void *flush_buf,
                           uint64_t flush_bytes, uint32_t flags, uint32_t timeout_ms, void *stream, float *times_ms,
                           float *flush_ms)
{
    if (!fn || reps == 0 || !times_ms) return KREX_EINVAL;
    if (flags & ~KREX_TL_REGION) return KREX_EINVAL;
    if (flush_buf && (flush_bytes % 16 != 0 || flush_bytes == 0)) return KREX_EINVAL;
    if (flush_buf && !aligned(flush_buf, 16)) return KREX_EALIGN;
    const bool region = (flags & KREX_TL_REGION) != 0;
    if (region && !krexg::attached()) return KREX_ENOTATTACHED;
    if (region && krexg::in_region()) return KREX_ESTATE;
    hipStream_t s = (hipStream_t)stream;
    const int dev = current_device();
    std::lock_guard<std::mutex> evg(g_ev_mu);
    hipEvent_t *ev = nullptr;
    krex_status rc = timing_events(dev, (size_t)reps * 3, &ev);
    if (rc != KREX_OK) return rc;
    hipEvent_t *ev_flush = ev, *ev_start = ev + reps, *ev_end = ev + 2 * (size_t)reps;

    bool counted = false;
    krex_status entry = KREX_OK;
    if (region) {
        entry = krex_region_begin(stream, timeout_ms, nullptr, 0);
        if (entry < 0) return entry;   // a failed entry starts no measurement
    } else if (!krexg::intercepted()) {
        rc = krexg::admit(gate_timeout_ns(), &counted);
        if (rc != KREX_OK) return rc;
    }
    g_fn_error = hipSuccess;
    hipError_t e = hipSuccess;
    for (uint32_t w = 0; w < warmup && e == hipSuccess; ++w) {
        fn(user, stream);
        e = g_fn_error;
    }
    for (uint32_t r = 0; r < reps && e == hipSuccess; ++r) {
        if (flush_buf) {
            e = hipEventRecord(ev_flush[r], s);
            if (e == hipSuccess) e = krex::launch_flush(flush_buf, flush_bytes, 0x9E3779B9u * (r + 1u), s);
        }
        if (e == hipSuccess) e = hipEventRecord(ev_start[r], s);
        if (e == hipSuccess) {
            fn(user, stream);
            e = g_fn_error;
        }
        if (e == hipSuccess) e = hipEventRecord(ev_end[r], s);
    }
    if (e == hipSuccess) e = hipEventSynchronize(ev_end[reps - 1]);
    for (uint32_t r = 0; r < reps && e == hipSuccess; ++r) {
        e = hipEventElapsedTime(&times_ms[r], ev_start[r], ev_end[r]);
        if (e == hipSuccess && flush_ms) e = flush_buf ? hipEventElapsedTime(&flush_ms[r], ev_flush[r], ev_start[r])
                                                       : (flush_ms[r] = 0.0f, hipSuccess);
    }
    if (region) {
        const krex_status end = krex_region_end(stream);
        if (e == hipSuccess && end < 0) return end;
    } else {
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (counted) krexg::release(1);
    }
    if (e != hipSuccess) return hip_fail(e);
    return entry;
}

krex_status krex_get_gate_stats(krex_gate_stats *out)
{
    if (!out) return KREX_EINVAL;
    krexg::Stats st;
    krexg::get_stats(&st);
    out->regions = st.regions;
    out->last_drain_ns = st.last_drain_ns;
    out->total_drain_ns = st.total_drain_ns;
    out->parks = st.parks;
    out->park_ns = st.park_ns;
    out->recoveries = st.recoveries;
    out->last_frozen = st.last_frozen;
    out->revocations = st.revocations;
    out->slot = st.slot;
    out->gated = st.gated;
    return KREX_OK;
}

krex_status krex_health_check(void *stream)
{
    hipStream_t s = (hipStream_t)stream;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) == hipSuccess && cs != hipStreamCaptureStatusNone) {
        krexg::mark_failed();
        return KREX_ESTATE;
    }
    const hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        krexg::mark_failed();
        return hip_fail(e);
    }
    return krexg::failed() ? KREX_EHIP : KREX_OK;
}

const char *krex_strerror(krex_status st)
{
    switch (st) {
    case KREX_OK: return "ok";
    case KREX_RECOVERED: return "ok (region lock recovered from a dead holder)";
    case KREX_EINVAL: return "invalid argument";
    case KREX_EALIGN: return "misaligned pointer";
    case KREX_EHIP: return "HIP runtime error";
    case KREX_ETIMEDOUT: return "timed out";
    case KREX_ESTATE: return "invalid state for this call";
    case KREX_ENOTATTACHED: return "process not attached to a region coordinator";
    case KREX_ENOMEM: return "out of host memory";
    case KREX_EPEER: return "shared segment unusable";
    case KREX_ESYS: return "system call failed";
    case KREX_EREVOKED: return "region revoked after its lease expired";
    default: return "unknown status";
    }
}

int32_t krex_last_hip_error(void) { return g_last_hip; }

const char *krex_version(void) { return "krex-mi355x 0.1 (gfx950)"; }

}  // extern "C"
