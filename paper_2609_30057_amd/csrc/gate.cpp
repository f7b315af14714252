// gate.cpp -- region coordinator over a POSIX shared-memory segment.
// See gate.hpp for the protocol and the passages of the paper it follows.
#include "gate.hpp"

#include <errno.h>
#include <fcntl.h>
#include <linux/futex.h>
#include <pthread.h>
#include <sched.h>
#include <signal.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <sys/mman.h>
#include <sys/stat.h>
#include <sys/syscall.h>
#include <time.h>
#include <unistd.h>

#include <dirent.h>

#include <atomic>
#include <climits>
#include <mutex>

#include "krex.h"

namespace krexg {
// ThreadSanitizer builds of the CPU test harness: the sanitizer has no
// interceptor for pthread_mutex_clocklock, so the acquisition is announced to
// it explicitly (otherwise the matching unlock reads as an unlock of an
// unlocked mutex). Other builds call the function directly.
#if defined(__SANITIZE_THREAD__)
#include <sanitizer/tsan_interface.h>
#endif

namespace {

int timed_lock(pthread_mutex_t *m, const timespec *abs)
{
#if defined(__SANITIZE_THREAD__)
    __tsan_mutex_pre_lock(m, 0);
    const int rc = pthread_mutex_clocklock(m, CLOCK_MONOTONIC, abs);
    if (rc == 0 || rc == EOWNERDEAD)
        __tsan_mutex_post_lock(m, 0, 0);
    else
        __tsan_mutex_post_lock(m, __tsan_mutex_try_lock_failed, 0);
    return rc;
#else
    return pthread_mutex_clocklock(m, CLOCK_MONOTONIC, abs);
#endif
}

}  // namespace

namespace {

constexpr uint64_t kMagic = 0x4b52455847415445ull;   // "KREXGATE"
constexpr uint32_t kVersion = 5;
constexpr uint64_t kEpochMask = (1ull << 48) - 1;

struct alignas(64) Slot {
    std::atomic<int32_t> pid;          // 0 = free
    std::atomic<uint32_t> flags;       // kNoGate, kCpuExclusive, kFailed
    std::atomic<uint64_t> start_time;  // /proc start time of pid, guards pid reuse
    std::atomic<int64_t> inflight;     // counted submissions not yet completed
    std::atomic<uint64_t> frozen_by;   // gate word of the region that stopped this process; 0 = running
};

struct Segment {
    std::atomic<uint64_t> magic;       // written last by the creator
    uint32_t version;
    uint32_t nslots;
    pthread_mutex_t lock;              // region lock: robust, process-shared
    alignas(64) std::atomic<uint64_t> gate;      // holder (slot + 1) << 48 | epoch; holder 0 = open
    alignas(64) std::atomic<uint32_t> gate_seq;  // futex word, bumped on every gate change
    std::atomic<uint32_t> parked;                // processes parked on gate_seq
    alignas(64) std::atomic<uint64_t> epoch;
    std::atomic<uint64_t> gate_since;  // CLOCK_MONOTONIC ns when the current gate closed
    std::atomic<uint64_t> lease_ns;    // region lease (0: none), fixed by the segment's creator
    std::atomic<uint64_t> revoked;     // gate word of the last revoked region
    Slot slots[kSlots];
};

static_assert(std::atomic<uint64_t>::is_always_lock_free, "64-bit atomics must be lock-free");
static_assert(std::atomic<int64_t>::is_always_lock_free, "64-bit atomics must be lock-free");

struct State {
    std::mutex mu;                     // attach / detach / region calls of this process
    Segment *seg = nullptr;
    int slot = -1;
    bool gated_ = false;
    std::atomic<bool> in_region{false};
    bool entering = false;             // a region_begin of this process waits for the region lock
    uint32_t flags = 0;
    uint32_t spin_us = 50;
    uint64_t region_gate = 0;          // gate word of this process's current region
    bool pinned = false;
    cpu_set_t saved_affinity;
    std::atomic<uint64_t> regions{0}, last_drain_ns{0}, total_drain_ns{0}, parks{0}, park_ns{0}, recoveries{0};
    std::atomic<uint64_t> last_frozen{0};
    std::atomic<uint64_t> revocations{0};
};

State &st()
{
    static State *s = new State();   // never destroyed: usable from atexit handlers
    return *s;
}

uint64_t now_ns()
{
    timespec ts;
    clock_gettime(CLOCK_MONOTONIC, &ts);
    return (uint64_t)ts.tv_sec * 1000000000ull + (uint64_t)ts.tv_nsec;
}

inline void cpu_relax() { __builtin_ia32_pause(); }

long futex_wait(std::atomic<uint32_t> *addr, uint32_t expected, uint64_t timeout_ns)
{
    timespec ts;
    ts.tv_sec = (time_t)(timeout_ns / 1000000000ull);
    ts.tv_nsec = (long)(timeout_ns % 1000000000ull);
    return syscall(SYS_futex, reinterpret_cast<uint32_t *>(addr), FUTEX_WAIT, expected, &ts, nullptr, 0);
}

void futex_wake_all(std::atomic<uint32_t> *addr)
{
    syscall(SYS_futex, reinterpret_cast<uint32_t *>(addr), FUTEX_WAKE, INT_MAX, nullptr, nullptr, 0);
}

// Start time of a process in clock ticks since boot (field 22 of
// /proc/<pid>/stat), 0 if unreadable.
uint64_t proc_start_time(int32_t pid)
{
    char path[64];
    snprintf(path, sizeof path, "/proc/%d/stat", (int)pid);
    FILE *f = fopen(path, "r");
    if (!f) return 0;
    char buf[1024];
    size_t n = fread(buf, 1, sizeof buf - 1, f);
    fclose(f);
    buf[n] = 0;
    const char *p = strrchr(buf, ')');   // the command name may contain spaces
    if (!p) return 0;
    int field = 2;
    unsigned long long v = 0;
    for (++p; *p; ++p) {
        if (*p == ' ') {
            ++field;
            if (field == 22) {
                v = strtoull(p + 1, nullptr, 10);
                break;
            }
        }
    }
    return v;
}

bool alive(int32_t pid, uint64_t start)
{
    if (pid <= 0) return false;
    if (kill(pid, 0) != 0 && errno == ESRCH) return false;
    const uint64_t now = proc_start_time(pid);
    return start == 0 || now == 0 || now == start;
}

inline uint32_t holder_of(uint64_t g) { return (uint32_t)(g >> 48); }

// Scheduler state letter of a process (field 3 of /proc/<pid>/stat), 0 if
// the process is gone.
char proc_state(int32_t pid)
{
    char path[64];
    snprintf(path, sizeof path, "/proc/%d/stat", (int)pid);
    FILE *f = fopen(path, "r");
    if (!f) return 0;
    char buf[512];
    size_t n = fread(buf, 1, sizeof buf - 1, f);
    fclose(f);
    buf[n] = 0;
    const char *p = strrchr(buf, ')');
    return (p && p[1] == ' ') ? p[2] : 0;
}

// Waits (bounded) until a signalled process has actually stopped, so that it
// cannot fork between the signal and the enumeration of its children.
void wait_stopped(int32_t pid, uint64_t until)
{
    while (now_ns() < until) {
        const char c = proc_state(pid);
        if (c == 'T' || c == 't' || c == 0 || c == 'Z' || c == 'X') return;
        cpu_relax();
    }
}

// Direct children of every thread of `pid` (/proc/<pid>/task/<tid>/children).
int children_of(int32_t pid, int32_t *out, int max)
{
    char path[64];
    snprintf(path, sizeof path, "/proc/%d/task", (int)pid);
    DIR *d = opendir(path);
    if (!d) return 0;
    int n = 0;
    while (dirent *e = readdir(d)) {
        if (e->d_name[0] < '0' || e->d_name[0] > '9') continue;
        char cp[sizeof "/proc//task//children" + 12 + sizeof e->d_name];
        snprintf(cp, sizeof cp, "/proc/%d/task/%s/children", (int)pid, e->d_name);
        FILE *f = fopen(cp, "r");
        if (!f) continue;
        int c;
        while (n < max && fscanf(f, "%d", &c) == 1) out[n++] = c;
        fclose(f);
    }
    closedir(d);
    return n;
}

constexpr int kMaxTree = 256;

// Stops the process tree rooted at `root` top-down, each parent stopped
// before its children are listed, never stopping `self` or anything below it
// (a holder may itself descend from a registered sibling). Returns the number
// of processes signalled.
int freeze_tree(int32_t root, int32_t self, uint64_t until)
{
    int32_t q[kMaxTree];
    int head = 0, tail = 0, count = 0;
    if (root == self) return 0;
    q[tail++] = root;
    while (head < tail) {
        const int32_t p = q[head++];
        if (kill(p, SIGSTOP) != 0) continue;
        ++count;
        wait_stopped(p, until);
        int32_t kids[kMaxTree];
        const int k = children_of(p, kids, kMaxTree);
        for (int i = 0; i < k && tail < kMaxTree; ++i)
            if (kids[i] != self) q[tail++] = kids[i];
    }
    return count;
}

// Resumes the tree rooted at `root`: descendants first (listed while the
// tree is still stopped), the root last.
void thaw_tree(int32_t root, int32_t self)
{
    int32_t q[kMaxTree];
    int head = 0, tail = 0;
    q[tail++] = root;
    while (head < tail) {
        int32_t kids[kMaxTree];
        const int k = children_of(q[head++], kids, kMaxTree);
        for (int i = 0; i < k && tail < kMaxTree; ++i)
            if (kids[i] != self) q[tail++] = kids[i];
    }
    for (int i = tail - 1; i >= 0; --i) kill(q[i], SIGCONT);
}

// Resumes every registered process tree stopped by the region whose gate
// word is `g` (Section 4.2, step 7 and holder-death cleanup: bound to the
// holder and epoch, so a late cleanup never undoes a later region's freeze).
void thaw_region(Segment *seg, uint64_t g)
{
    const int32_t self = (int32_t)getpid();
    for (int i = 0; i < kSlots; ++i) {
        Slot &sl = seg->slots[i];
        if (sl.frozen_by.load() != g) continue;
        const int32_t pid = sl.pid.load();
        if (pid > 0 && alive(pid, sl.start_time.load())) thaw_tree(pid, self);
        sl.frozen_by.store(0);
    }
}

void open_gate(Segment *seg, uint64_t epoch)
{
    seg->gate.store(epoch & kEpochMask, std::memory_order_seq_cst);
    seg->gate_seq.fetch_add(1, std::memory_order_seq_cst);
    futex_wake_all(&seg->gate_seq);
}

// Revokes the region whose gate word is g once it has outlived the lease
// (Section 4.3: a client exceeding its time limit is recovered like a dead
// one). Bound to the holder and epoch: the compare-and-swap succeeds only
// while g is still the gate, so a late revocation never reopens a later
// region. The holder keeps the region lock; its region exit reports the
// revocation.
bool revoke(Segment *seg, uint64_t g)
{
    uint64_t expect = g;
    if (!seg->gate.compare_exchange_strong(expect, g & kEpochMask, std::memory_order_seq_cst)) return false;
    thaw_region(seg, g);
    seg->revoked.store(g, std::memory_order_seq_cst);
    seg->gate_seq.fetch_add(1, std::memory_order_seq_cst);
    futex_wake_all(&seg->gate_seq);
    st().revocations.fetch_add(1);
    return true;
}

// Called with the region lock held after EOWNERDEAD: the previous holder died
// inside its region. Reopen its gate (only if it is still that holder's
// closure) and free its slot.
void recover_dead_holder(Segment *seg)
{
    const uint64_t g = seg->gate.load(std::memory_order_seq_cst);
    const uint32_t h = holder_of(g);
    if (h != 0) {
        thaw_region(seg, g);
        Slot &s = seg->slots[h - 1];
        const int32_t pid = s.pid.load();
        if (pid == 0 || !alive(pid, s.start_time.load())) {
            s.inflight.store(0);
            s.pid.store(0);
        }
        uint64_t expect = g;
        seg->gate.compare_exchange_strong(expect, g & kEpochMask, std::memory_order_seq_cst);
        seg->gate_seq.fetch_add(1, std::memory_order_seq_cst);
        futex_wake_all(&seg->gate_seq);
    }
    st().recoveries.fetch_add(1);
}

// A parked submitter found the gate holder dead: take the lock to run the
// recovery (the robust mutex serialises it with any other recovery or entry).
void try_recover(Segment *seg)
{
    int rc = pthread_mutex_trylock(&seg->lock);
    if (rc == EOWNERDEAD) {
        recover_dead_holder(seg);
        pthread_mutex_consistent(&seg->lock);
        pthread_mutex_unlock(&seg->lock);
    } else if (rc == 0) {
        // Lock free but the gate closed by a dead process that had released
        // the lock cannot happen (the gate is closed only under the lock);
        // still reopen defensively if the holder is dead.
        const uint64_t g = seg->gate.load();
        const uint32_t h = holder_of(g);
        if (h != 0) {
            Slot &s = seg->slots[h - 1];
            if (!alive(s.pid.load(), s.start_time.load())) recover_dead_holder(seg);
        }
        pthread_mutex_unlock(&seg->lock);
    }
}

int map_segment(const char *name, Segment **out)
{
    bool creator = false;
    int fd = shm_open(name, O_RDWR | O_CREAT | O_EXCL, 0600);
    if (fd >= 0) {
        creator = true;
        if (ftruncate(fd, sizeof(Segment)) != 0) {
            close(fd);
            shm_unlink(name);
            return KREX_ESYS;
        }
    } else if (errno == EEXIST) {
        fd = shm_open(name, O_RDWR, 0600);
        if (fd < 0) return KREX_ESYS;
        const uint64_t deadline = now_ns() + 5000000000ull;
        for (;;) {
            struct stat sb;
            if (fstat(fd, &sb) != 0) {
                close(fd);
                return KREX_ESYS;
            }
            if ((size_t)sb.st_size >= sizeof(Segment)) break;
            if (sb.st_size != 0 && (size_t)sb.st_size != sizeof(Segment)) {
                close(fd);
                return KREX_EPEER;
            }
            if (now_ns() > deadline) {
                close(fd);
                return KREX_EPEER;
            }
            usleep(100);
        }
    } else {
        return KREX_ESYS;
    }
    void *p = mmap(nullptr, sizeof(Segment), PROT_READ | PROT_WRITE, MAP_SHARED, fd, 0);
    close(fd);
    if (p == MAP_FAILED) return KREX_ESYS;
    Segment *seg = static_cast<Segment *>(p);
    if (creator) {
        // ftruncate zero-filled the segment, which is a valid initial state
        // for every atomic; only the mutex needs its attributes.
        pthread_mutexattr_t a;
        pthread_mutexattr_init(&a);
        pthread_mutexattr_setpshared(&a, PTHREAD_PROCESS_SHARED);
        pthread_mutexattr_setrobust(&a, PTHREAD_MUTEX_ROBUST);
        pthread_mutex_init(&seg->lock, &a);
        pthread_mutexattr_destroy(&a);
        seg->version = kVersion;
        seg->nslots = kSlots;
        if (const char *e = getenv("KREX_REGION_LEASE_MS"))
            seg->lease_ns.store((uint64_t)strtoull(e, nullptr, 10) * 1000000ull);
        seg->magic.store(kMagic, std::memory_order_release);
    } else {
        const uint64_t deadline = now_ns() + 5000000000ull;
        while (seg->magic.load(std::memory_order_acquire) != kMagic) {
            if (now_ns() > deadline) {
                munmap(p, sizeof(Segment));
                return KREX_EPEER;
            }
            usleep(100);
        }
        if (seg->version != kVersion || seg->nslots != (uint32_t)kSlots) {
            munmap(p, sizeof(Segment));
            return KREX_EPEER;
        }
    }
    *out = seg;
    return KREX_OK;
}

void at_exit_release()
{
    State &s = st();
    if (!s.seg || s.slot < 0) return;
    Segment *seg = s.seg;
    // A forked child inherits this state but not the registration: only the
    // registered process releases its slot and region.
    if (seg->slots[s.slot].pid.load() != (int32_t)getpid()) return;
    if (s.in_region) {
        thaw_region(seg, s.region_gate);
        open_gate(seg, seg->epoch.load());
        pthread_mutex_unlock(&seg->lock);
        s.in_region = false;
    }
    seg->slots[s.slot].inflight.store(0);
    seg->slots[s.slot].pid.store(0);
    s.slot = -1;
}

}  // namespace

void set_spin_us(uint32_t us) { st().spin_us = us; }

int attach(const char *shm_name, uint32_t flags)
{
    State &s = st();
    std::lock_guard<std::mutex> g(s.mu);
    if (s.seg) return KREX_ESTATE;
    if (!shm_name || shm_name[0] != '/' || strlen(shm_name) > 200) return KREX_EINVAL;
    Segment *seg = nullptr;
    int rc = map_segment(shm_name, &seg);
    if (rc != KREX_OK) return rc;
    const int32_t me = (int32_t)getpid();
    const uint64_t start = proc_start_time(me);
    int slot = -1;
    // Prefer a free slot; reuse a dead process's slot only while the gate is
    // open, so slots being drained are not reassigned mid-region.
    for (int pass = 0; pass < 2 && slot < 0; ++pass) {
        for (int i = 0; i < kSlots && slot < 0; ++i) {
            Slot &sl = seg->slots[i];
            int32_t p = sl.pid.load();
            if (p == 0) {
                if (sl.pid.compare_exchange_strong(p, me)) slot = i;
            } else if (pass == 1 && holder_of(seg->gate.load()) == 0 && !alive(p, sl.start_time.load())) {
                if (sl.pid.compare_exchange_strong(p, me)) slot = i;
            }
        }
    }
    if (slot < 0) {
        munmap(seg, sizeof(Segment));
        return KREX_ESYS;
    }
    Slot &sl = seg->slots[slot];
    sl.start_time.store(start);
    sl.flags.store(flags & (kNoGate | kCpuExclusive));
    sl.inflight.store(0);
    sl.frozen_by.store(0);
    s.seg = seg;
    s.slot = slot;
    s.gated_ = (flags & kNoGate) == 0;
    s.flags = flags;
    s.in_region = false;
    s.regions.store(0);
    s.last_drain_ns.store(0);
    s.total_drain_ns.store(0);
    s.parks.store(0);
    s.park_ns.store(0);
    s.recoveries.store(0);
    if (const char *e = getenv("KREX_SPIN_US")) s.spin_us = (uint32_t)strtoul(e, nullptr, 10);
    static bool registered = false;
    if (!registered) {
        atexit(at_exit_release);
        registered = true;
    }
    return KREX_OK;
}

int detach()
{
    State &s = st();
    std::lock_guard<std::mutex> g(s.mu);
    if (!s.seg) return KREX_ESTATE;
    if (s.in_region || s.entering) return KREX_ESTATE;
    Segment *seg = s.seg;
    seg->slots[s.slot].inflight.store(0);
    seg->slots[s.slot].pid.store(0);
    s.slot = -1;
    s.seg = nullptr;
    s.gated_ = false;
    munmap(seg, sizeof(Segment));
    return KREX_OK;
}

bool attached() { return st().seg != nullptr; }
bool gated() { return st().seg != nullptr && st().gated_; }
bool in_region() { return st().in_region; }

int64_t inflight_self()
{
    State &s = st();
    if (!s.seg) return 0;
    return s.seg->slots[s.slot].inflight.load();
}

int admit(uint64_t timeout_ns, bool *counted)
{
    State &s = st();
    *counted = false;
    Segment *seg = s.seg;
    if (!seg || !s.gated_) return KREX_OK;
    Slot &me = seg->slots[s.slot];
    if (me.flags.load() & kFailed) return KREX_EHIP;   // failed health: no further submissions
    const uint32_t mine = (uint32_t)s.slot + 1;
    uint64_t t_park = 0;
    const uint64_t start = now_ns();
    const uint64_t deadline = timeout_ns ? start + timeout_ns : UINT64_MAX;
    for (;;) {
        // Increment before checking: a racing holder either sees this count
        // (and drains it) or this check sees its closed gate.
        me.inflight.fetch_add(1, std::memory_order_seq_cst);
        const uint64_t g = seg->gate.load(std::memory_order_seq_cst);
        const uint32_t h = holder_of(g);
        if (h == 0 || h == mine) {
            if (t_park) s.park_ns.fetch_add(now_ns() - t_park);
            *counted = true;
            return KREX_OK;
        }
        me.inflight.fetch_sub(1, std::memory_order_seq_cst);
        if (!t_park) {
            t_park = now_ns();
            s.parks.fetch_add(1);
        }
        // Spin briefly, then park on the gate's futex word until it changes.
        const uint32_t seq = seg->gate_seq.load(std::memory_order_seq_cst);
        const uint64_t spin_end = now_ns() + (uint64_t)s.spin_us * 1000ull;
        bool changed = false;
        while (now_ns() < spin_end) {
            if (seg->gate.load(std::memory_order_seq_cst) != g) {
                changed = true;
                break;
            }
            cpu_relax();
        }
        if (changed) continue;
        const uint64_t now = now_ns();
        if (now >= deadline) {
            s.park_ns.fetch_add(now - t_park);
            return KREX_ETIMEDOUT;
        }
        uint64_t slice = 20000000ull;   // re-check holder liveness every 20 ms
        if (deadline - now < slice) slice = deadline - now;
        seg->parked.fetch_add(1, std::memory_order_seq_cst);
        if (seg->gate.load(std::memory_order_seq_cst) == g) futex_wait(&seg->gate_seq, seq, slice);
        seg->parked.fetch_sub(1, std::memory_order_seq_cst);
        if (seg->gate.load(std::memory_order_seq_cst) == g) {
            Slot &hs = seg->slots[h - 1];
            if (!alive(hs.pid.load(), hs.start_time.load())) {
                try_recover(seg);
            } else {
                const uint64_t lease = seg->lease_ns.load();
                if (lease && now_ns() - seg->gate_since.load() > lease) revoke(seg, g);
            }
        }
    }
}

void mark_failed()
{
    State &s = st();
    if (!s.seg || s.slot < 0) return;
    Slot &me = s.seg->slots[s.slot];
    me.flags.fetch_or(kFailed);
    me.inflight.store(0);          // a failed context's counts are not waited for
}

std::atomic<bool> g_intercepted{false};

void set_intercepted(bool on) { g_intercepted.store(on); }
bool intercepted() { return g_intercepted.load(); }

void set_cpu_exclusive(bool on)
{
    State &s = st();
    std::lock_guard<std::mutex> g(s.mu);
    s.flags = on ? (s.flags | kCpuExclusive) : (s.flags & ~kCpuExclusive);
    if (s.seg && s.slot >= 0) {
        if (on) s.seg->slots[s.slot].flags.fetch_or(kCpuExclusive);
        else s.seg->slots[s.slot].flags.fetch_and(~kCpuExclusive);
    }
}

uint32_t flags() { return st().flags; }

bool failed()
{
    State &s = st();
    return s.seg && s.slot >= 0 && (s.seg->slots[s.slot].flags.load() & kFailed);
}

void release(uint64_t k)
{
    State &s = st();
    if (!s.seg || k == 0) return;
    s.seg->slots[s.slot].inflight.fetch_sub((int64_t)k, std::memory_order_seq_cst);
}

int region_begin(uint32_t timeout_ms)
{
    State &s = st();
    Segment *seg = nullptr;
    {
        // The state is checked under the process mutex, but the wait for the
        // region lock happens without it: the region lock always comes first
        // (region_end holds it when it takes the mutex). `entering` keeps
        // the other calls of this process out meanwhile.
        std::lock_guard<std::mutex> g(s.mu);
        seg = s.seg;
        if (!seg) return KREX_ENOTATTACHED;
        if (s.in_region || s.entering) return KREX_ESTATE;
        s.entering = true;
    }
    const uint64_t t0 = now_ns();
    const uint64_t deadline = t0 + (uint64_t)timeout_ms * 1000000ull;
    timespec abs;
    clock_gettime(CLOCK_MONOTONIC, &abs);
    abs.tv_sec += timeout_ms / 1000;
    abs.tv_nsec += (long)(timeout_ms % 1000) * 1000000L;
    if (abs.tv_nsec >= 1000000000L) {
        abs.tv_sec += 1;
        abs.tv_nsec -= 1000000000L;
    }
    int status = KREX_OK;
    // Step 1: the region lock.
    int rc = timed_lock(&seg->lock, &abs);
    std::lock_guard<std::mutex> g(s.mu);
    s.entering = false;
    if (rc == EOWNERDEAD) {
        recover_dead_holder(seg);
        pthread_mutex_consistent(&seg->lock);
        status = KREX_RECOVERED;
    } else if (rc == ETIMEDOUT) {
        return KREX_ETIMEDOUT;
    } else if (rc == ENOTRECOVERABLE) {
        return KREX_EPEER;
    } else if (rc != 0) {
        return KREX_ESYS;
    }
    // Step 2: close the gate with this process as holder and a new epoch.
    const uint64_t epoch = seg->epoch.fetch_add(1, std::memory_order_seq_cst) + 1;
    seg->gate_since.store(now_ns(), std::memory_order_seq_cst);
    seg->gate.store(((uint64_t)(s.slot + 1) << 48) | (epoch & kEpochMask), std::memory_order_seq_cst);
    seg->gate_seq.fetch_add(1, std::memory_order_seq_cst);
    // Step 3: wait until every other gated process has nothing in flight.
    const uint64_t td = now_ns();
    for (int i = 0; i < kSlots; ++i) {
        if (i == s.slot) continue;
        Slot &sl = seg->slots[i];
        uint64_t spins = 0;
        uint64_t next_liveness = now_ns() + 10000000ull;
        for (;;) {
            const int32_t pid = sl.pid.load(std::memory_order_seq_cst);
            if (pid == 0 || (sl.flags.load() & (kNoGate | kFailed))) break;
            if (sl.inflight.load(std::memory_order_seq_cst) <= 0) break;
            const uint64_t now = now_ns();
            if (now >= next_liveness) {
                next_liveness = now + 10000000ull;
                if (!alive(pid, sl.start_time.load())) {
                    int32_t p = pid;
                    if (sl.pid.compare_exchange_strong(p, 0)) sl.inflight.store(0);
                    break;
                }
            }
            if (now >= deadline) {
                open_gate(seg, epoch);
                pthread_mutex_unlock(&seg->lock);
                return KREX_ETIMEDOUT;
            }
            if (++spins < 2000) {
                cpu_relax();
            } else {
                timespec ts{0, 20000};
                nanosleep(&ts, nullptr);
            }
        }
    }
    const uint64_t drain = now_ns() - td;
    s.last_drain_ns.store(drain);
    s.total_drain_ns.fetch_add(drain);
    s.regions.fetch_add(1);
    s.region_gate = seg->gate.load(std::memory_order_seq_cst);
    s.last_frozen.store(0);
    if (s.flags & kCpuExclusive) {
        // Step 4: with every sibling's in-flight count at zero, stop their
        // process trees; each stopped slot records this region's gate word,
        // so a recovery after this holder's death resumes exactly these.
        const int32_t self = (int32_t)getpid();
        const uint64_t until = now_ns() + 20000000ull;
        uint64_t frozen = 0;
        for (int i = 0; i < kSlots; ++i) {
            if (i == s.slot) continue;
            Slot &sl = seg->slots[i];
            const int32_t pid = sl.pid.load();
            if (pid <= 0 || pid == self || !alive(pid, sl.start_time.load())) continue;
            sl.frozen_by.store(s.region_gate);
            frozen += (uint64_t)freeze_tree(pid, self, until);
        }
        s.last_frozen.store(frozen);
        // Step 5 (second half): pin this thread to one core of its set
        // (KREX_REGION_CPU=none leaves it unpinned).
        const char *pin_env = getenv("KREX_REGION_CPU");
        const bool pin = !(pin_env && strcmp(pin_env, "none") == 0);
        if (pin && sched_getaffinity(0, sizeof(cpu_set_t), &s.saved_affinity) == 0) {
            int core = -1;
            if (pin_env) core = atoi(pin_env);
            if (core < 0 || !CPU_ISSET(core, &s.saved_affinity))
                for (int c = CPU_SETSIZE - 1; c >= 0; --c)
                    if (CPU_ISSET(c, &s.saved_affinity)) {
                        core = c;
                        break;
                    }
            if (core >= 0) {
                cpu_set_t one;
                CPU_ZERO(&one);
                CPU_SET(core, &one);
                s.pinned = sched_setaffinity(0, sizeof(cpu_set_t), &one) == 0;
            }
        }
    }
    s.in_region = true;
    return status;
}

int region_end()
{
    State &s = st();
    std::lock_guard<std::mutex> g(s.mu);
    Segment *seg = s.seg;
    if (!seg) return KREX_ENOTATTACHED;
    if (!s.in_region) return KREX_ESTATE;
    // Step 7: resume stopped siblings and unpin; step 8: reopen the gate,
    // wake parked siblings, release the lock. The reopening is a
    // compare-and-swap from this region's gate word, so exactly one of this
    // exit and a lease revocation reopens it; if the revocation won, the
    // region is reported as revoked (its timings are not exclusive).
    if (s.flags & kCpuExclusive) thaw_region(seg, s.region_gate);
    if (s.pinned) {
        sched_setaffinity(0, sizeof(cpu_set_t), &s.saved_affinity);
        s.pinned = false;
    }
    uint64_t expect = s.region_gate;
    const bool ours = seg->gate.compare_exchange_strong(expect, s.region_gate & kEpochMask, std::memory_order_seq_cst);
    seg->gate_seq.fetch_add(1, std::memory_order_seq_cst);
    futex_wake_all(&seg->gate_seq);
    s.in_region = false;
    pthread_mutex_unlock(&seg->lock);
    return ours ? KREX_OK : KREX_EREVOKED;
}

void get_stats(Stats *out)
{
    State &s = st();
    out->regions = s.regions.load();
    out->last_drain_ns = s.last_drain_ns.load();
    out->total_drain_ns = s.total_drain_ns.load();
    out->parks = s.parks.load();
    out->park_ns = s.park_ns.load();
    out->recoveries = s.recoveries.load();
    out->last_frozen = s.last_frozen.load();
    out->revocations = s.revocations.load();
    out->slot = s.slot;
    out->gated = s.seg && s.gated_ ? 1 : 0;
}

}  // namespace krexg
