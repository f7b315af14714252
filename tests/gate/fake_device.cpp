// Test harness for the region coordinator (paper_2609_30057_amd/csrc/gate.cpp)
// on the CPU: a fake in-order "device" executes each admitted operation on a
// worker thread for a given duration and releases its in-flight count when
// it finishes, as the GPU completion tracking does. Logs the execution
// interval of every operation (CLOCK_MONOTONIC ns, comparable across
// processes).
#include <stdint.h>
#include <time.h>
#include <unistd.h>

#include <atomic>
#include <condition_variable>
#include <deque>
#include <mutex>
#include <thread>
#include <vector>

#include "gate.hpp"
#include "krex.h"

namespace {

uint64_t now_ns()
{
    timespec ts;
    clock_gettime(CLOCK_MONOTONIC, &ts);
    return (uint64_t)ts.tv_sec * 1000000000ull + (uint64_t)ts.tv_nsec;
}

struct Op {
    uint64_t dur_ns;
    bool counted;
};

struct Dev {
    std::mutex mu;
    std::condition_variable cv;
    std::deque<Op> q;
    std::vector<std::pair<uint64_t, uint64_t>> log;
    std::atomic<int64_t> pending{0};
    std::thread th;
    bool started = false;

    void run()
    {
        for (;;) {
            Op op;
            {
                std::unique_lock<std::mutex> g(mu);
                cv.wait(g, [this] { return !q.empty(); });
                op = q.front();
                q.pop_front();
            }
            const uint64_t s = now_ns();
            while (now_ns() - s < op.dur_ns) {
                const uint64_t left = op.dur_ns - (now_ns() - s);
                timespec ts{0, (long)(left > 200000 ? 200000 : left)};
                nanosleep(&ts, nullptr);
            }
            const uint64_t e = now_ns();
            {
                std::lock_guard<std::mutex> g(mu);
                log.push_back({s, e});
            }
            if (op.counted) krexg::release(1);
            pending.fetch_sub(1);
        }
    }
};

Dev &dev()
{
    static Dev *d = new Dev();
    return *d;
}

bool wait_idle(uint32_t timeout_ms)
{
    const uint64_t end = now_ns() + (uint64_t)timeout_ms * 1000000ull;
    while (dev().pending.load() != 0) {
        if (now_ns() > end) return false;
        usleep(50);
    }
    return true;
}

}  // namespace

extern "C" {

int kg_attach(const char *name, uint32_t flags) { return krexg::attach(name, flags); }

int kg_detach()
{
    wait_idle(60000);
    return krexg::detach();
}

// Counter-and-gate, then enqueue a fake operation of dur_us; *t_admit gets
// the admission time.
int kg_submit(uint32_t dur_us, uint64_t timeout_ns, uint64_t *t_admit)
{
    bool counted = false;
    const int rc = krexg::admit(timeout_ns, &counted);
    if (rc != KREX_OK) return rc;
    if (t_admit) *t_admit = now_ns();
    Dev &d = dev();
    {
        std::lock_guard<std::mutex> g(d.mu);
        if (!d.started) {
            d.started = true;
            d.th = std::thread([&d] { d.run(); });
            d.th.detach();
        }
        d.q.push_back({(uint64_t)dur_us * 1000ull, counted});
        d.pending.fetch_add(1);
    }
    d.cv.notify_one();
    return KREX_OK;
}

int kg_wait_idle(uint32_t timeout_ms) { return wait_idle(timeout_ms) ? 0 : -1; }

// Region entry waits for this process's own operations first, as the
// library's entry waits for the process's own GPU work.
int kg_region_begin(uint32_t timeout_ms)
{
    if (!krexg::attached()) return KREX_ENOTATTACHED;
    if (krexg::in_region()) return KREX_ESTATE;
    wait_idle(60000);
    return krexg::region_begin(timeout_ms);
}

int kg_region_end()
{
    if (!krexg::attached()) return KREX_ENOTATTACHED;
    if (!krexg::in_region()) return KREX_ESTATE;
    wait_idle(60000);
    return krexg::region_end();
}

int64_t kg_inflight() { return krexg::inflight_self(); }

// What the library does when a context fails its health check.
void kg_fail() { krexg::mark_failed(); }

uint64_t kg_now() { return now_ns(); }

void kg_stats(krexg::Stats *out) { krexg::get_stats(out); }

int kg_log_count()
{
    std::lock_guard<std::mutex> g(dev().mu);
    return (int)dev().log.size();
}

void kg_log_get(int i, uint64_t *s, uint64_t *e)
{
    std::lock_guard<std::mutex> g(dev().mu);
    *s = dev().log[i].first;
    *e = dev().log[i].second;
}

}
