/*
 * krex.h -- C ABI of the MI355X (gfx950) hot path of a kernel benchmarking
 * command: seeded input generation, mismatch injection, the allclose
 * correctness check, the cache flush, and the timed loop inside a critical
 * region that excludes sibling processes sharing the GPU.
 *
 * Paper: KREX, "Concurrent Kernel Benchmarking on Shared GPUs via
 * Region-Granular Exclusivity". A benchmarking command generates inputs,
 * checks the candidate against a reference and then times it (Section 1;
 * Section 2.1). Generation and checking produce values, not timings, and
 * must give the same tensors and verdict under contention (Section 2.1,
 * "Benchmarking command"). Exclusive use of the device matters for the
 * timed loop alone, which is marked as a critical region (Section 3, R1; Section 4.1), entered by
 * lock -> gate -> drain -> cache flush and left by wait -> reopen -> unlock
 * (Section 4.2, steps 1-3, 5, 6, 8), with the AMD variant's completion
 * counters (Section 5).
 *
 * Conventions for every entry point:
 *  - Status: KREX_OK (0) on success, a positive value for success with a
 *    note, a negative KREX_E* code on failure. No exception crosses the ABI.
 *    Argument errors are detected before anything is launched, so
 *    KREX_EINVAL / KREX_EALIGN have no side effects.
 *  - Memory: the caller owns every buffer. Pointers named "device" must be
 *    device memory of the current HIP device (hipMalloc, or torch CUDA
 *    tensors on ROCm). The library never allocates or frees them.
 *  - Streams: `stream` is a hipStream_t passed as void* (NULL = the legacy
 *    default stream). Kernel entry points are stream-ordered and return once
 *    the work is enqueued.
 *  - Gating: after krex_attach (gate on), every enqueueing entry point
 *    follows counter-and-gate (Section 4.2, "GPU exclusivity"): it counts
 *    itself in flight, then checks the region gate; if another process
 *    holds a region it retracts, parks (spin, then futex) until the gate
 *    reopens, and retries. The count is released when the device finishes
 *    the work (Section 5, AMD), or at once when the launch fails (Section
 *    4.2: the counter is decremented on error returns too). Without
 *    krex_attach the kernel entry points run ungated. A call on a stream
 *    that is capturing into a HIP graph is recorded, not run, so it is
 *    neither gated nor counted (nor chunked); launching the graph later is
 *    the caller's, outside the library's count.
 *  - Chunking: with KREX_CHUNK_BYTES set (bytes, 0 or unset = off) a gated
 *    process splits krex_gen, krex_gen_packed, krex_inject, krex_gen_inject
 *    and krex_flush calls larger than that into launches of at most that
 *    many output bytes (multiples of 64 elements), each admitted on its own,
 *    with at most KREX_CHUNK_DEPTH (default 2) in flight: the call then
 *    waits on the host for its oldest chunk before submitting the next. A
 *    region entered by another process drains at most that many chunks of
 *    the call (Section 4.2, step 3); the values written are the same.
 *    krex_check is never split.
 *  - Failures are explicit (Section 4.3: unsupported calls fail rather than
 *    bypass): a HIP error returns KREX_EHIP and krex_last_hip_error() gives
 *    the hipError_t of the calling thread.
 */
#ifndef KREX_H
#define KREX_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t krex_status;

#define KREX_OK 0
#define KREX_RECOVERED 1        /* region lock taken over from a dead holder */
#define KREX_EINVAL (-1)        /* bad argument value */
#define KREX_EALIGN (-2)        /* pointer not aligned to its element size */
#define KREX_EHIP (-3)          /* HIP runtime error, see krex_last_hip_error */
#define KREX_ETIMEDOUT (-4)     /* region entry or gate wait timed out */
#define KREX_ESTATE (-5)        /* call not valid in this state (nesting, ...) */
#define KREX_ENOTATTACHED (-6)  /* region call without krex_attach */
#define KREX_ENOMEM (-7)        /* host allocation failed */
#define KREX_EPEER (-8)         /* shared segment unusable (version, peer died in init) */
#define KREX_ESYS (-9)          /* POSIX call failed (shm, futex, threads) */
#define KREX_EREVOKED (-10)     /* the region outlived its lease and was revoked */

/* Element types. KREX_F8E4M3 is OCP fp8 e4m3fn (bias 7, max 448, no
 * infinity), gfx950's native fp8. KREX_U32 is the raw 32-bit word stream. */
#define KREX_F32 0
#define KREX_BF16 1
#define KREX_F16 2
#define KREX_F8E4M3 3
#define KREX_U32 4

/* Value distributions of krex_gen. */
#define KREX_UNIFORM 0   /* [p0, p1): u = (W >> 8) 2^-24, v = p0 + (p1 - p0) u */
#define KREX_NORMAL 1    /* mean p0, std p1: Box-Muller on word pairs */
#define KREX_BITCAST 2   /* the word's bits read as an fp32 value (any pattern) */

/* Injection modes of krex_inject. */
#define KREX_INJ_ROUND 0 /* y = cvt(x + delta) */
#define KREX_INJ_EXACT 1 /* x + delta if exact in the dtype, else x - delta, else x */

/* Result of krex_check; 64 bytes, must be device-accessible. */
typedef struct krex_check_result {
    uint64_t n;            /* elements compared */
    uint64_t mismatches;   /* elements not close, NaN ones included */
    uint64_t nan_count;    /* elements with a NaN on either side */
    uint64_t argmax_abs;   /* lowest index attaining max_abs; UINT64_MAX if none */
    float max_abs;         /* max |a - b| over NaN-free elements (0 if none) */
    float max_rel;         /* max |a - b| / |b| over NaN-free elements (0 if none) */
    uint64_t reserved[3];  /* reduction scratch; unspecified after the call */
} krex_check_result;

/* --- process registration ------------------------------------------------
 * Registers this process with the region coordinator of `device` (Section
 * 4.2: each process registers before it submits GPU work). shm_name names
 * the POSIX shared-memory segment shared by every process on that GPU (NULL:
 * "/krex-" + the device's PCI bus id). The first process creates and
 * initialises it. flags: KREX_ATTACH_NO_GATE registers without gating (the
 * ungated control configuration of Section 6.1); the process can still
 * enter regions. KREX_ATTACH_CPU_EXCLUSIVE adds CPU exclusivity to this
 * process's regions (Section 4.2, steps 4, 5 and 7): after the drain it
 * stops the process tree of every other registered process with SIGSTOP and
 * pins the entering thread to one core of its affinity set (the core named
 * by the KREX_REGION_CPU environment variable if it is in the set, else the
 * highest-numbered one; KREX_REGION_CPU=none disables the pinning); region exit resumes them with SIGCONT and restores
 * the affinity before the gate reopens. A holder that dies inside such a
 * region has its stopped siblings resumed by the process that recovers the
 * lock. With gating it also creates 64 completion events for `device`, the
 * pool counted launches take theirs from (more are created on demand,
 * except by krex_check_noalloc). Returns KREX_EINVAL for unknown flags,
 * KREX_ESTATE if already attached, KREX_EPEER if the segment has another
 * layout version, KREX_ESYS on a POSIX failure. */
#define KREX_ATTACH_NO_GATE 1u
#define KREX_ATTACH_CPU_EXCLUSIVE 2u
krex_status krex_attach(int32_t device, const char *shm_name, uint32_t flags);

/* Ends the registration krex_attach made (Section 4.2: each process
 * registers with the GPU's coordinator, serialised with gate closure; this
 * is the inverse step, so later drains stop looking at it). Waits for this process's
 * in-flight work so no count is left behind, then releases its slot and the
 * mapping. Returns KREX_ESTATE inside a region or when not attached,
 * KREX_ETIMEDOUT if its work has not finished within 60 s. */
krex_status krex_detach(void);

/* --- generation -----------------------------------------------------------
 * Fills dst[0..n) (device, dtype `dtype`, aligned to its element size) with
 * element j = transform(W_seed[offset + j]), where W_s[w] is output lane
 * w mod 4 of Philox4x32-10 (Salmon et al., SC'11) with key
 * (seed mod 2^32, seed >> 32) and counter (b mod 2^32, b >> 32, 0, 0),
 * b = w >> 2. This is the input generation of a benchmarking command
 * (Section 1; Section 2.1); being counter-based, it is independent of
 * launch shape, timing and colocated work (Section 2.1, "Benchmarking
 * command"). KREX_NORMAL pairs words (2p, 2p + 1), p = w >> 1, and element w
 * takes the cosine branch when w is even, the sine branch when odd.
 * Conversions to bf16 / fp16 / fp8 round to nearest even; fp8 is
 * non-saturating (NaN beyond 448). KREX_U32 stores the words and ignores
 * dist, p0, p1. Requires offset + n <= 2^64; uniform: finite p0 <= p1 with
 * finite p1 - p0; normal: finite p0, finite p1 >= 0. */
krex_status krex_gen(void *dst, int32_t dtype, uint64_t n, uint64_t seed, uint64_t offset,
                     int32_t dist, float p0, float p1, void *stream);

/* Packed stream, the narrow-dtype form of krex_gen (same Philox words,
 * fewer per element; an extension of the generation of Section 1 and
 * Section 2.1, which name no generator). The word stream is cut into W-bit
 * fields, low bits first: field q is bits [(q mod K) W, (q mod K) W + W) of
 * W_seed[q / K], K = 32 / W. W = 16 for KREX_BF16 and KREX_F16 (every
 * distribution) and for KREX_F8E4M3 with KREX_NORMAL; W = 8 for KREX_F8E4M3
 * uniform and bitcast. Element j uses field q = offset + j (offset counts
 * fields). Uniform: krex_gen's uniform transform of the word f << (32 - W),
 * i.e. u = f 2^-W. Normal: krex_gen's Box-Muller on the word pair
 * (f_{2p} << 16, f_{2p+1} << 16), p = q >> 1 (both fields in word p), cosine
 * branch for even q, sine for odd. Bitcast: the element's bits are the
 * field. Rounding and parameter rules as krex_gen. dst: device, aligned to
 * the element size; fastest when 16-byte aligned with offset a multiple of
 * 16 / element size. KREX_EINVAL for KREX_F32 or KREX_U32. */
krex_status krex_gen_packed(void *dst, int32_t dtype, uint64_t n, uint64_t seed, uint64_t offset,
                            int32_t dist, float p0, float p1, void *stream);

/* Same transforms applied to caller-supplied words: element j of dst is
 * transform(words[j]) (normal: pairs (words[2p], words[2p + 1]); n even).
 * words: device, n uint32 values. */
krex_status krex_transform_words(void *dst, int32_t dtype, uint64_t n, const uint32_t *words,
                                 int32_t dist, float p0, float p1, void *stream);

/* --- mismatch injection ---------------------------------------------------
 * y[i] = perturbed x[i] where W_mask_seed[mask_offset + i] < floor(rate 2^32)
 * (a Bernoulli mask on its own word stream), else x[i]. ROUND: cvt(x + delta).
 * EXACT: x + delta if both the fp32 sum and its conversion are exact, else
 * x - delta under the same test, else x unchanged. y may equal x (in place)
 * but must not otherwise overlap it. Stands in for a candidate's wrong
 * outputs so the check's verdict is known (Section 2.1). rate in [0, 1],
 * delta finite, dtype not KREX_U32. */
krex_status krex_inject(void *y, const void *x, int32_t dtype, uint64_t n, uint64_t mask_seed,
                        uint64_t mask_offset, double rate, float delta, int32_t mode, void *stream);

/* Generation and injection in one call: x = krex_gen(x, dtype, n, seed,
 * offset, dist, p0, p1) and y = krex_inject(y, x, dtype, n, mask_seed,
 * mask_offset, rate, delta, mode), with the same results bit for bit. A
 * benchmarking command's input and the perturbed output that stands in for
 * a wrong candidate (Section 2.1) come from one pass that writes x and y
 * without reading x back when offset and mask_offset are multiples of 4 and
 * x, y are 16-byte aligned (otherwise the two kernels run in order). x and y
 * (device, aligned to the element size) must not overlap. Arguments and
 * errors as for the two calls; dtype not KREX_U32. */
krex_status krex_gen_inject(void *x, void *y, int32_t dtype, uint64_t n, uint64_t seed, uint64_t offset,
                            int32_t dist, float p0, float p1, uint64_t mask_seed, uint64_t mask_offset, double rate,
                            float delta, int32_t mode, void *stream);

/* --- correctness check ----------------------------------------------------
 * Compares a (candidate, dtype dta) with b (reference, dtype dtb), n elements
 * each, device memory, and writes *out (device-accessible; overwritten, no
 * need to clear it). Per element, both sides are upcast to fp32 (exact):
 * NaN on either side -> mismatch, counted in nan_count, left out of the
 * maxima; a == b -> close, d = 0, rel = 0; else an infinity on either side
 * -> mismatch, d = rel = +inf; else d = |a - b|, close iff d is finite and
 * d <= atol + rtol |b| (fp32, two roundings), rel = d / |b|. The check of a
 * benchmarking command (Section 1; Section 2.1). rtol, atol finite >= 0;
 * n < 2^33; a and b aligned to their element sizes. n = 0 writes the empty
 * result. The result is ready when the stream reaches it. */
krex_status krex_check(const void *a, int32_t dta, const void *b, int32_t dtb, uint64_t n, float rtol,
                       float atol, krex_check_result *out, void *stream);

/* krex_check without allocation, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same arguments, checks and result, field for
 * field, but the block partials the check reduces live in a fixed device
 * array of the library (4096 partials, 128 KiB per GPU, held until the
 * process ends) instead of a per-stream buffer allocated on first use. It
 * calls no hipMalloc / hipFree. Every size krex_check accepts fits in the
 * array (n < 2^33; larger n returns KREX_EINVAL), and no partial needs
 * clearing: each call writes the ones it reads. All calls on one GPU share
 * the array, so two calls that may overlap on one GPU (on different
 * streams, or from different threads without ordering) race and can return
 * wrong records; calls ordered on one stream are safe. When the process is
 * attached with gating, completion is tracked, as for every entry point,
 * with a HIP event from the pool krex_attach creates (64 per device); this
 * call creates none: if every pooled event is in use it waits for the
 * stream itself and then releases its count. Under graph capture it is
 * recorded like any launch (see Gating above). */
krex_status krex_check_noalloc(const void *a, int32_t dta, const void *b, int32_t dtb, uint64_t n, float rtol,
                               float atol, krex_check_result *out, void *stream);

/* The same check against a reference that is regenerated instead of read:
 * *out equals krex_check(a, dta, b, dtb, n, rtol, atol) for the b that
 * krex_gen(b, dtb, n, seed, offset, dist, p0, p1) writes, field for field,
 * but b is never materialised: each reference element is recomputed from
 * its Philox word (the reference of a benchmarking command whose expected
 * output is itself a generated tensor, Section 1; Section 2.1), so only a is
 * read from memory. Fastest when a is 16-byte aligned and offset is a
 * multiple of 4. Arguments and errors as for krex_gen (dist, p0, p1, offset)
 * and krex_check (a, dta, rtol, atol, n, out); dtb not KREX_U32. */
krex_status krex_check_gen(const void *a, int32_t dta, int32_t dtb, uint64_t n, uint64_t seed, uint64_t offset,
                           int32_t dist, float p0, float p1, float rtol, float atol, krex_check_result *out,
                           void *stream);

/* The same for the packed stream: *out equals krex_check(a, dta, b, dtb, n,
 * rtol, atol) for the b that krex_gen_packed(b, dtb, n, seed, offset, dist,
 * p0, p1) writes (offset in fields), regenerated in registers at one Philox
 * block per 16 bytes of b (two for fp8 normal), so only a is read. Fastest
 * when a is 16-byte aligned and offset is a multiple of 16 / size(dtb).
 * Arguments and errors as for krex_gen_packed (dtb bf16, fp16 or fp8) and
 * krex_check. */
krex_status krex_check_gen_packed(const void *a, int32_t dta, int32_t dtb, uint64_t n, uint64_t seed,
                                  uint64_t offset, int32_t dist, float p0, float p1, float rtol, float atol,
                                  krex_check_result *out, void *stream);

/* --- cache flush ------------------------------------------------------------
 * Writes `pattern` to every 32-bit word of buf[0..bytes) (device, 16-byte
 * aligned, bytes a multiple of 16) with stores that allocate in the
 * Infinity Cache (written through L2 with system-scope coherence), evicting
 * its earlier contents when bytes exceeds its 256 MB (Section 2.1: flush
 * between timed iterations; Section 4.2 step 5: memset over a cache-sized
 * buffer). L2 holds nothing across kernel launches on gfx950 (the runtime
 * writes it back and invalidates it at kernel boundaries), so the Infinity
 * Cache is the cache a timed launch could otherwise inherit data from. */
krex_status krex_flush(void *buf, uint64_t bytes, uint32_t pattern, void *stream);

/* --- probe kernel -----------------------------------------------------------
 * A known-work timed kernel: 256 blocks x 256 threads, each thread runs 8
 * independent fp32 FMA chains for `iters` steps and writes their sum to
 * sink[thread] (device, 65536 floats). Used to measure timing inflation
 * (Section 6.4, Eq. 1). */
#define KREX_PROBE_THREADS 65536
krex_status krex_probe(uint64_t iters, float *sink, void *stream);

/* krex_probe that also records each wave's clocks (the per-sample evidence
 * of the device's clock state behind a timing ratio of Eq. 1): clocks
 * (device, 16-byte aligned, KREX_PROBE_WAVES x 8 uint64 words) receives for
 * wave w = 4 block + wave-in-block, at words 8w .. 8w + 7: the shader-clock
 * cycle counter at the wave's start and end, the constant 100 MHz real-time
 * counter at its start and end, the HW_ID register, 0, the XCC_ID register,
 * 0. sink as for krex_probe, with the same values. */
#define KREX_PROBE_WAVES 1024
#define KREX_PROBE_CLOCK_WORDS 8
krex_status krex_probe_clocked(uint64_t iters, float *sink, uint64_t *clocks, void *stream);

/* --- critical region --------------------------------------------------------
 * Begins a critical region on this process's GPU (Section 4.1; Section 4.2):
 * waits for this process's own earlier GPU work, takes the region lock
 * (step 1), closes the gate with this process as holder and a new epoch
 * (step 2), waits until every other registered process has no work in
 * flight (step 3, completion counters of Section 5), then, if flush_buf is
 * non-NULL, flushes flush_bytes of it on `stream` and waits for it (step 5).
 * Fails without entering (gate reopened, lock released) on timeout, on a
 * HIP error or if the lock cannot be taken within timeout_ms (Section 4.2:
 * a failed entry starts no measurement). Returns KREX_RECOVERED when the
 * lock was taken over from a holder that died inside its region.
 * KREX_ENOTATTACHED without krex_attach; KREX_ESTATE when already inside. */
krex_status krex_region_begin(void *stream, uint32_t timeout_ms, void *flush_buf, uint64_t flush_bytes);

/* Ends the region: waits for this process's region work to finish on the
 * device, reopens the gate, wakes parked siblings and releases the lock
 * (Section 4.2, step 8). KREX_ESTATE when not inside a region.
 * KREX_EREVOKED when the region outlived the segment's lease
 * (KREX_REGION_LEASE_MS in the environment of the process that created the
 * segment; unset or 0: no lease) and a parked sibling reopened the gate
 * (Section 4.3: a client over its time limit is recovered like a dead one);
 * the region is still left and the lock released, but timings taken in it
 * were not exclusive. Revocation needs a running parked submitter, so it
 * does not happen while CPU exclusivity has every sibling stopped. */
krex_status krex_region_end(void *stream);

/* --- timed loop ---------------------------------------------------------------
 * do_bench-style loop (Section 2.1; Triton's do_bench, Section 8): `warmup`
 * untimed calls of fn(user, stream), then `reps` times: flush flush_bytes of
 * flush_buf with pattern 0x9E3779B9 * (rep + 1) (if flush_buf is non-NULL),
 * record a start event, fn(user, stream), record an end event; one
 * synchronisation at the end. times_ms[rep] (host, reps entries) receives
 * each rep's start-to-end time; flush_ms (host, optional) each flush's
 * time. With KREX_TL_REGION the whole loop, warm-up included, runs inside a
 * critical region (Section 4.1: the region holds the warm-up and the timed
 * loop, not the checks), entered with timeout_ms. reps >= 1. */
typedef void (*krex_launch_fn)(void *user, void *stream);
#define KREX_TL_REGION 1u
krex_status krex_time_loop(krex_launch_fn fn, void *user, uint32_t warmup, uint32_t reps, void *flush_buf,
                           uint64_t flush_bytes, uint32_t flags, uint32_t timeout_ms, void *stream,
                           float *times_ms, float *flush_ms);

/* Ready-made launch functions for krex_time_loop. */
typedef struct krex_probe_args {
    uint64_t iters;
    float *sink;          /* device, KREX_PROBE_THREADS floats */
    uint64_t *clocks;     /* NULL, or as for krex_probe_clocked */
} krex_probe_args;
void krex_probe_launch(void *user /* krex_probe_args* */, void *stream);

/* Naive fp32 GEMM, row-major C[M x N] = A[M x K] B[K x N], each element an
 * fma chain over k ascending from +0: the candidate kernel of the tiny GEMM
 * benchmarking command (a stand-in for an agent's kernel, Section 2.1). */
typedef struct krex_sgemm_args {
    uint32_t M, N, K;
    const float *A, *B;   /* device */
    float *C;             /* device */
} krex_sgemm_args;
krex_status krex_fixture_sgemm(uint32_t M, uint32_t N, uint32_t K, const float *A, const float *B, float *C,
                               void *stream);
void krex_sgemm_launch(void *user /* krex_sgemm_args* */, void *stream);

/* --- introspection -------------------------------------------------------------
 * Counters of this process since its last krex_attach. */
typedef struct krex_gate_stats {
    uint64_t regions;          /* regions entered by this process */
    uint64_t last_drain_ns;    /* gate closed -> siblings drained, last entry */
    uint64_t total_drain_ns;
    uint64_t parks;            /* submissions of this process that waited at a closed gate */
    uint64_t park_ns;          /* time spent waiting there */
    uint64_t recoveries;       /* dead holders recovered by this process */
    uint64_t last_frozen;      /* processes stopped at the last entry (CPU exclusivity) */
    uint64_t revocations;      /* regions of other processes revoked by this one (lease) */
    int32_t slot;              /* this process's registration slot, -1 if none */
    int32_t gated;             /* 1 if submissions are gated */
} krex_gate_stats;
krex_status krex_get_gate_stats(krex_gate_stats *out /* host */);

/* --- health -----------------------------------------------------------------
 * Context health check after a command (Section 4.3, context cleanup): waits
 * for all of this process's work on its current device and reports whether
 * the context is still usable. An unhealthy context (a sticky device error,
 * or `stream` left in graph capture) marks this process's slot failed:
 * region entries stop waiting for its work and its further submissions are
 * refused with KREX_EHIP, so the caller must retire the process. Returns
 * KREX_OK, KREX_EHIP (device error; see krex_last_hip_error) or KREX_ESTATE
 * (capture in progress). The completion tracker marks the slot failed the
 * same way when waiting for a counted operation reports an error. */
krex_status krex_health_check(void *stream);

const char *krex_strerror(krex_status st);
int32_t krex_last_hip_error(void);
const char *krex_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KREX_H */
