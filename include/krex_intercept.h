/*
 * krex_intercept.h -- introspection of libkrex_intercept.so, the ROCm tools
 * library that gates every kernel dispatch of a process (torch kernels,
 * library GEMMs, HIP's copy kernels), not only this library's own launches.
 *
 * Paper, Section 5 (AMD): the interposer swaps queue creation in the
 * runtime's dispatch table, so every kernel launch of every queue passes
 * through it; a launch batch raises the process's in-flight count and a
 * poller thread lowers it when the batch's completion signal reports the
 * work done; a tenant joins only after its initialisation.
 *
 * Use: start the tenant with HSA_TOOLS_LIB=<path>/libkrex_intercept.so and
 * KREX_INTERCEPT_SHM=<segment name> (the coordinator segment of
 * krex_attach); KREX_INTERCEPT_NO_GATE=1 registers without gating. The
 * process registers at its first kernel dispatch. Each submitted batch that
 * holds a kernel dispatch takes one admission (waiting while another
 * process holds the gate) and is followed in its queue by a barrier-AND
 * packet carrying a completion signal of the library's; the count is
 * released when that signal fires. Without KREX_INTERCEPT_SHM the library
 * passes every packet through. In a process with interception active,
 * libkrex's own launches are not counted a second time, and krex_attach
 * reuses the interceptor's registration.
 *
 * Both functions are host-only, thread-safe and never block on the device.
 */
#ifndef KREX_INTERCEPT_H
#define KREX_INTERCEPT_H

#include <stdint.h>

#include "krex.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct krex_intercept_counters {
    uint64_t batches;      /* gated batches submitted */
    uint64_t dispatches;   /* kernel dispatch packets in them */
    uint64_t passthrough;  /* dispatch batches passed through ungated (no registration, or ungated) */
    uint64_t timeouts;     /* admissions that timed out (the batch was submitted anyway) */
    uint64_t errors;       /* admissions or signals that failed (the batch was submitted anyway) */
    int32_t active;        /* 1 once the process is registered through the interceptor */
    int32_t reserved;
} krex_intercept_counters;

/* Counters since the library was loaded. out: host. */
krex_status krex_intercept_stats(krex_intercept_counters *out);

/* Copies up to max (admission, completion) CLOCK_MONOTONIC nanosecond pairs
 * of gated batches, in completion order (the first 65536 of the process);
 * returns the number copied. Either array may be NULL. Every batch's
 * kernels executed inside [admission, completion]. */
uint64_t krex_intercept_log(uint64_t *t_admit, uint64_t *t_done, uint64_t max);

#ifdef __cplusplus
}
#endif

#endif
