// intercept.cpp -- ROCm tools library that puts every kernel dispatch of a
// process behind the region coordinator's counter-and-gate, whether or not
// the process calls this library's C ABI (torch kernels, library GEMMs, HIP's
// own copy kernels).
//
// Paper, Section 5 (AMD): the interposer is a ROCm tools library that swaps
// queue creation in the runtime's dispatch table, so every kernel launch of
// every queue is seen on its way to the GPU. Each launch batch raises the
// process's in-flight count; a poller thread lowers it once the batch's
// completion signal reports the work done, and a region holder waits for
// every other process's count to reach zero (Section 4.2, step 3). A tenant
// joins only after its initialisation (here: at its first dispatch).
//
// Mechanism: loaded by the HSA runtime through HSA_TOOLS_LIB, OnLoad swaps
// hsa_queue_create for a wrapper that creates an intercept queue and
// registers a packet handler. The handler runs on the thread that rings the
// queue's doorbell. For a batch holding at least one kernel dispatch it
// takes one admission (blocking while another process holds the gate),
// writes the batch, then writes a barrier-AND packet with the barrier bit
// set and a signal of this library's: the packet processor decrements that
// signal once every earlier packet of the queue has completed. A poller
// thread waits on the signals in submission order and releases the count.
// Non-dispatch batches pass through untouched.
//
// Environment: KREX_INTERCEPT_SHM names the coordinator's shared-memory
// segment (unset: the library passes everything through); with
// KREX_INTERCEPT_NO_GATE=1 the process registers ungated.
#include <hsa/hsa.h>
#include <hsa/hsa_api_trace.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>

#include <atomic>
#include <condition_variable>
#include <deque>
#include <mutex>
#include <thread>
#include <vector>

#include "gate.hpp"
#include "krex.h"
#include "krex_intercept.h"

namespace {

CoreApiTable g_core;     // the runtime's own entries, saved at load
AmdExtTable g_amd;
decltype(hsa_queue_create) *g_queue_create_orig = nullptr;

std::once_flag g_attach_once;
bool g_enabled = false;  // a segment was named and the attach succeeded

std::atomic<uint64_t> g_batches{0}, g_dispatches{0}, g_passthrough{0}, g_timeouts{0}, g_errors{0};

uint64_t now_ns()
{
    timespec ts;
    clock_gettime(CLOCK_MONOTONIC, &ts);
    return (uint64_t)ts.tv_sec * 1000000000ull + (uint64_t)ts.tv_nsec;
}

// Admission/completion log of the gated batches (for tests and analysis).
constexpr uint64_t kLogCap = 1u << 16;
struct LogEntry {
    uint64_t t_admit, t_done;
};
std::mutex g_log_mu;
std::vector<LogEntry> g_log;

void do_attach()
{
    const char *name = getenv("KREX_INTERCEPT_SHM");
    if (!name || !*name) return;
    const char *ng = getenv("KREX_INTERCEPT_NO_GATE");
    const uint32_t flags = (ng && strcmp(ng, "1") == 0) ? krexg::kNoGate : 0u;
    if (krexg::attached()) {   // the process registered itself first
        krexg::set_intercepted(true);
        g_enabled = true;
        return;
    }
    if (krexg::attach(name, flags) == KREX_OK) {
        krexg::set_intercepted(true);
        g_enabled = true;
    }
}

// ---------------------------------------------------------------- poller

class Poller {
public:
    void push(hsa_signal_t sig, uint64_t t_admit)
    {
        {
            std::lock_guard<std::mutex> g(mu_);
            q_.push_back({sig, t_admit});
            if (!started_) {
                started_ = true;
                th_ = std::thread([this] { run(); });
                th_.detach();
            }
        }
        cv_.notify_one();
    }

    hsa_signal_t take()
    {
        {
            std::lock_guard<std::mutex> g(pool_mu_);
            if (!pool_.empty()) {
                hsa_signal_t s = pool_.back();
                pool_.pop_back();
                return s;
            }
        }
        hsa_signal_t s{0};
        if (g_core.hsa_signal_create_fn(1, 0, nullptr, &s) != HSA_STATUS_SUCCESS) s.handle = 0;
        return s;
    }

    static Poller &instance()
    {
        static Poller *p = new Poller();   // never destroyed: the thread may outlive static destruction
        return *p;
    }

private:
    struct Item {
        hsa_signal_t sig;
        uint64_t t_admit;
    };

    void run()
    {
        for (;;) {
            Item it;
            {
                std::unique_lock<std::mutex> g(mu_);
                cv_.wait(g, [this] { return !q_.empty(); });
                it = q_.front();
                q_.pop_front();
            }
            // Completion of the barrier packet: every packet before it in the
            // queue has finished.
            while (g_core.hsa_signal_wait_scacquire_fn(it.sig, HSA_SIGNAL_CONDITION_LT, 1, 50000000ull,
                                                       HSA_WAIT_STATE_BLOCKED) >= 1) {
            }
            const uint64_t t_done = now_ns();
            krexg::release(1);
            {
                std::lock_guard<std::mutex> g(g_log_mu);
                if (g_log.size() < kLogCap) g_log.push_back({it.t_admit, t_done});
            }
            g_core.hsa_signal_store_relaxed_fn(it.sig, 1);
            std::lock_guard<std::mutex> g(pool_mu_);
            pool_.push_back(it.sig);
        }
    }

    std::mutex mu_;
    std::condition_variable cv_;
    std::deque<Item> q_;
    std::thread th_;
    bool started_ = false;
    std::mutex pool_mu_;
    std::vector<hsa_signal_t> pool_;
};

// ---------------------------------------------------------------- handler

constexpr uint16_t kTypeMask = (1u << HSA_PACKET_HEADER_WIDTH_TYPE) - 1u;

void on_submit(const void *pkts, uint64_t count, uint64_t, void *, hsa_amd_queue_intercept_packet_writer writer)
{
    const auto *p = static_cast<const hsa_kernel_dispatch_packet_t *>(pkts);
    uint64_t dispatches = 0;
    for (uint64_t i = 0; i < count; ++i)
        if (((p[i].header >> HSA_PACKET_HEADER_TYPE) & kTypeMask) == HSA_PACKET_TYPE_KERNEL_DISPATCH) ++dispatches;
    if (dispatches == 0) {
        writer(pkts, count);
        return;
    }
    std::call_once(g_attach_once, do_attach);
    if (!g_enabled) {
        g_passthrough.fetch_add(1);
        writer(pkts, count);
        return;
    }
    bool counted = false;
    const int rc = krexg::admit(0, &counted);   // no timeout: a dispatch waits as long as the region lasts
    if (rc != KREX_OK || !counted) {
        if (rc == KREX_ETIMEDOUT) g_timeouts.fetch_add(1);
        else if (rc != KREX_OK) g_errors.fetch_add(1);
        else g_passthrough.fetch_add(1);
        writer(pkts, count);   // fail open: never drop the tenant's work
        return;
    }
    const uint64_t t_admit = now_ns();
    hsa_signal_t sig = Poller::instance().take();
    if (sig.handle == 0) {
        g_errors.fetch_add(1);
        writer(pkts, count);
        krexg::release(1);
        return;
    }
    hsa_barrier_and_packet_t b;
    memset(&b, 0, sizeof b);
    b.completion_signal = sig;
    // Barrier bit: the packet completes only after every earlier packet of
    // the queue; no cache fences (it only marks completion).
    b.header = (uint16_t)((HSA_PACKET_TYPE_BARRIER_AND << HSA_PACKET_HEADER_TYPE) | (1u << HSA_PACKET_HEADER_BARRIER) |
                          (HSA_FENCE_SCOPE_NONE << HSA_PACKET_HEADER_SCACQUIRE_FENCE_SCOPE) |
                          (HSA_FENCE_SCOPE_NONE << HSA_PACKET_HEADER_SCRELEASE_FENCE_SCOPE));
    writer(pkts, count);
    writer(&b, 1);
    g_batches.fetch_add(1);
    g_dispatches.fetch_add(dispatches);
    Poller::instance().push(sig, t_admit);
}

hsa_status_t queue_create(hsa_agent_t agent, uint32_t size, hsa_queue_type32_t type,
                          void (*callback)(hsa_status_t status, hsa_queue_t *source, void *data), void *data,
                          uint32_t private_segment_size, uint32_t group_segment_size, hsa_queue_t **queue)
{
    hsa_device_type_t dt = HSA_DEVICE_TYPE_CPU;
    if (g_core.hsa_agent_get_info_fn(agent, HSA_AGENT_INFO_DEVICE, &dt) != HSA_STATUS_SUCCESS ||
        dt != HSA_DEVICE_TYPE_GPU)
        return g_queue_create_orig(agent, size, type, callback, data, private_segment_size, group_segment_size,
                                   queue);
    hsa_status_t st = g_amd.hsa_amd_queue_intercept_create_fn(agent, size, type, callback, data,
                                                              private_segment_size, group_segment_size, queue);
    if (st != HSA_STATUS_SUCCESS) return st;
    return g_amd.hsa_amd_queue_intercept_register_fn(*queue, on_submit, nullptr);
}

}  // namespace

extern "C" {

// Called by the HSA runtime when it loads the libraries in HSA_TOOLS_LIB.
__attribute__((visibility("default"))) bool OnLoad(HsaApiTable *table, uint64_t, uint64_t, const char *const *)
{
    if (!table || !table->core_ || !table->amd_ext_) return false;
    const char *name = getenv("KREX_INTERCEPT_SHM");
    if (!name || !*name) return true;   // loaded but inactive
    memcpy(&g_core, table->core_, sizeof(CoreApiTable) < table->core_->version.minor_id
                                      ? sizeof(CoreApiTable) : table->core_->version.minor_id);
    memcpy(&g_amd, table->amd_ext_, sizeof(AmdExtTable) < table->amd_ext_->version.minor_id
                                        ? sizeof(AmdExtTable) : table->amd_ext_->version.minor_id);
    if (!g_amd.hsa_amd_queue_intercept_create_fn || !g_amd.hsa_amd_queue_intercept_register_fn ||
        !g_core.hsa_signal_create_fn || !g_core.hsa_signal_wait_scacquire_fn || !g_core.hsa_agent_get_info_fn)
        return true;
    g_queue_create_orig = table->core_->hsa_queue_create_fn;
    table->core_->hsa_queue_create_fn = queue_create;
    return true;
}

__attribute__((visibility("default"))) void OnUnload() {}

krex_status krex_intercept_stats(krex_intercept_counters *out)
{
    if (!out) return KREX_EINVAL;
    out->batches = g_batches.load();
    out->dispatches = g_dispatches.load();
    out->passthrough = g_passthrough.load();
    out->timeouts = g_timeouts.load();
    out->errors = g_errors.load();
    out->active = g_enabled ? 1 : 0;
    out->reserved = 0;
    return KREX_OK;
}

uint64_t krex_intercept_log(uint64_t *t_admit, uint64_t *t_done, uint64_t max)
{
    std::lock_guard<std::mutex> g(g_log_mu);
    const uint64_t n = g_log.size() < max ? g_log.size() : max;
    for (uint64_t i = 0; i < n; ++i) {
        if (t_admit) t_admit[i] = g_log[i].t_admit;
        if (t_done) t_done[i] = g_log[i].t_done;
    }
    return n;
}

}  // extern "C"
