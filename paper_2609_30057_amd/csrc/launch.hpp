// launch.hpp -- host-side launchers of the gfx950 kernels (kernels.hip),
// called by the C ABI layer (api.cpp) after argument validation and gating.
// Each returns the launch's hipError_t; none synchronises.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "krex.h"

namespace krex {

// Compute units of the current device (cached per device).
int device_cus();

// Generation's transform constant for (dist, p0, p1): c = range 2^-24 when
// the uniform range fl(p1 - p0) scales every 24-bit integer exactly (returns
// true; the transform is then one fused multiply-add), else the range
// (uniform) or p1 (normal, bitcast).
bool gen_transform_constants(int dist, float p0, float p1, float *q1);

// `p1` is the distribution's second parameter as given (upper bound or std).
hipError_t launch_gen(void *dst, int dt, uint64_t n, uint64_t seed, uint64_t offset, int dist, float p0, float p1,
                      hipStream_t s);
// The packed stream's transform constants for (dt, dist, p0, p1): *q1 the
// range fl(p1 - p0) (uniform) or p1, *rs = *q1 2^-W (uniform); returns the
// uniform mode (UM_WORD, UM_SCALED or UM_FUSED; UM_WORD otherwise).
int packed_transform_constants(int dt, int dist, float p0, float p1, float *q1, float *rs);
// Packed stream (bf16, fp16, fp8 only); offset counts fields.
hipError_t launch_gen_packed(void *dst, int dt, uint64_t n, uint64_t seed, uint64_t offset, int dist, float p0,
                             float p1, hipStream_t s);
hipError_t launch_xform(void *dst, int dt, uint64_t n, const uint32_t *words, int dist, float p0, float p1,
                        hipStream_t s);
hipError_t launch_inject(void *y, const void *x, int dt, uint64_t n, uint64_t mseed, uint64_t moff, uint64_t T,
                         float delta, int mode, hipStream_t s);
// launch_gen into x, then launch_inject from x into y, as one fused kernel
// when both offsets are multiples of 4 and x, y are 16-byte aligned.
hipError_t launch_gen_inject(void *x, void *y, int dt, uint64_t n, uint64_t seed, uint64_t offset, int dist, float p0,
                             float p1, uint64_t mseed, uint64_t moff, uint64_t T, float delta, int mode,
                             hipStream_t s);
// The check reduces per-block partials held in `scratch` (device memory of
// check_scratch_bytes()); calls that may overlap need distinct scratch.
size_t check_scratch_bytes();
// Devices the library keeps per-device state for.
static constexpr int kMaxDevices = 64;
// The device address, on the current device, of the library's fixed check
// scratch (check_scratch_bytes() bytes, a file-scope device array), looked
// up once per device and cached. Used by krex_check_noalloc in place of an
// allocated buffer; every call on one device shares it.
hipError_t noalloc_scratch(void **out);
hipError_t launch_check(const void *a, int dta, const void *b, int dtb, uint64_t n, float rtol, float atol,
                        void *scratch, krex_check_result *out, hipStream_t s);
// The check of a against the reference krex_gen would write for (dtb,
// seed, offset, dist, p0, p1), regenerated instead of read; scratch as for
// launch_check.
hipError_t launch_check_gen(const void *a, int dta, int dtb, uint64_t n, uint64_t seed, uint64_t offset, int dist,
                            float p0, float p1, float rtol, float atol, void *scratch, krex_check_result *out,
                            hipStream_t s);
// As launch_check_gen for the reference krex_gen_packed would write
// (dtb bf16, fp16 or fp8; offset counts fields).
hipError_t launch_check_gen_packed(const void *a, int dta, int dtb, uint64_t n, uint64_t seed, uint64_t offset,
                                   int dist, float p0, float p1, float rtol, float atol, void *scratch,
                                   krex_check_result *out, hipStream_t s);
hipError_t launch_flush(void *buf, uint64_t bytes, uint32_t pattern, hipStream_t s);
// The probe: kProbeBlocks blocks of 256 threads; clocks (device,
// 8 x 64-bit words per wave, kProbeBlocks x 4 waves) or null.
static constexpr int kProbeBlocks = 256;
hipError_t launch_probe(uint64_t iters, float *sink, uint64_t *clocks, hipStream_t s);
hipError_t launch_sgemm(uint32_t M, uint32_t N, uint32_t K, const float *A, const float *B, float *C,
                        hipStream_t s);

}  // namespace krex
