// gate.hpp -- host-side region coordinator shared by all processes that use
// one GPU: the region lock, the gate with holder and epoch, the registration
// slots with their in-flight counters, and spin-then-park waiting.
//
// Paper, Section 4.2 ("GPU exclusivity"): a tenant entering a region takes
// the GPU's region lock (step 1), atomically claims a shared-memory gate
// recording itself and a unique epoch (step 2), and waits until every other
// registered process has nothing in flight (step 3). Every submission
// increments its process's in-flight counter before it checks the gate
// (counter-and-gate); on AMD the counter is released when the device
// completes the operation (Section 5). Waiting spins briefly and then parks
// on a futex (Section 4.3, spin-park policy). A failed entry reopens the gate
// and releases the lock before returning (Section 4.2, entry failure); a
// holder that dies is recovered by the next process that takes the lock
// (Section 4.2, holder death; here the robust mutex serialises recovery with
// normal exit). With CPU exclusivity the holder also stops the siblings'
// processes after the drain and pins its own thread (Section 4.2, steps 4
// and 5), and resumes them before the gate reopens (step 7); the stop is
// SIGSTOP / SIGCONT of the registered processes, recorded in shared memory
// so that recovery from the holder's death resumes them. A region that
// outlives the segment's lease (KREX_REGION_LEASE_MS of the process that
// created the segment; 0 or unset: no lease) is revoked by a parked
// submitter: the gate reopens (bound to the region's holder and epoch) and
// the holder's exit returns KREX_EREVOKED (Section 4.3, time limits).
//
// This file is plain POSIX C++ (no HIP): the GPU-side completion tracking
// lives in the ABI layer, and the CPU tests drive the same code with a fake
// device.
#pragma once

#include <stdint.h>

namespace krexg {

struct Stats {
    uint64_t regions;
    uint64_t last_drain_ns;
    uint64_t total_drain_ns;
    uint64_t parks;
    uint64_t park_ns;
    uint64_t recoveries;
    uint64_t last_frozen;
    uint64_t revocations;
    int32_t slot;
    int32_t gated;
};

constexpr uint32_t kNoGate = 1u;          // register, never block or count
constexpr uint32_t kCpuExclusive = 2u;    // as holder: stop siblings, pin the region thread
constexpr uint32_t kFailed = 4u;          // slot state: failed health check, never waited for
constexpr int kSlots = 64;

// All functions return krex status codes (KREX_OK, KREX_E*).
int attach(const char *shm_name, uint32_t flags);
int detach();
bool attached();
bool gated();
bool in_region();

// Counter-and-gate: on KREX_OK this process's in-flight counter was
// incremented and the gate was open (or held by this process) when checked.
// Parks while another process holds the gate; KREX_ETIMEDOUT after
// timeout_ns. A no-op returning KREX_OK when not attached or ungated
// (*counted = false then).
int admit(uint64_t timeout_ns, bool *counted);
// Releases k counted submissions (device completion or launch failure).
void release(uint64_t k);
// Marks this process's slot failed (a sticky device error or an unusable
// context, Section 4.3): entries stop waiting for its work and its further
// submissions are refused with KREX_EHIP.
void mark_failed();
bool failed();
// Set by the dispatch interceptor once it registered this process: every
// kernel dispatch is then counted at the queue, so callers stop counting
// their own launches.
void set_intercepted(bool on);
bool intercepted();
// Updates the CPU-exclusivity choice of an existing registration.
void set_cpu_exclusive(bool on);
uint32_t flags();
int64_t inflight_self();

// Region entry after the caller's own work has finished (steps 1-3); exit
// after the caller's region work has finished (step 8).
int region_begin(uint32_t timeout_ms);
int region_end();

void get_stats(Stats *out);

// Spin interval before parking, in microseconds (default 50, or the
// KREX_SPIN_US environment variable read at attach).
void set_spin_us(uint32_t us);

}  // namespace krexg
