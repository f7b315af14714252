// check_gen_packed.hip -- the fused allclose check against a reference
// regenerated from the packed stream (Section 1; Section 2.1), the stream
// that spends 16 or 8 bits of the Philox words per narrow element: only the
// candidate is read, and the reference costs one Philox block per 16 bytes
// of it (two for fp8 normal) instead of one per four elements.
//
//   k_check_gen_packed  the check body of check_device.hpp with the
//                       reference source RefGenPacked; k_check_final
//                       reduces its partials.
//
// The vector path needs a 16-byte aligned candidate and an offset that is a
// multiple of the fields per unit (16 / size of the reference's dtype);
// anything else takes the element path, whose chunks compute one unit more
// and shift the fields into place.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "check_device.hpp"
#include "hip_launch.hpp"
#include "krex_device.hpp"
#include "launch.hpp"

namespace krex {

template <int DA, int DB, int DIST, int UM, bool VEC, int D>
__global__ __launch_bounds__(kThreads) void k_check_gen_packed(const uint8_t *a,
                                                               RefGenPacked<DB, DIST, UM, chunk_elems<DA, DB>()> ref,
                                                               uint64_t n, float rtol, float atol,
                                                               CheckPartial *partials, uint32_t U)
{
    check_body<DA, DB, VEC, D>(a, ref, n, rtol, atol, partials, U);
}

namespace {

struct PackedRefArgs {
    uint64_t seed, offset;
    float p0, p1, rs;
};

// Depth of the candidate's load ring, as for the word-stream reference.
constexpr int kPackedCheckDepth = 2;

template <int DA, int DB, int DIST, int UM>
hipError_t check_t(const void *a, const PackedRefArgs &g, uint64_t n, float rtol, float atol, void *scratch,
                   krex_check_result *out, hipStream_t s)
{
    constexpr int E = chunk_elems<DA, DB>();
    constexpr int D = kPackedCheckDepth;
    constexpr int EP = packed_of<DB, DIST>::E;
    const RefGenPacked<DB, DIST, UM, E> ref{g.offset, round_keys(g.seed), g.p0, g.p1, g.rs};
    const bool vec = ((uintptr_t)a & 15u) == 0 && (g.offset % EP) == 0;
    static uint32_t cache_vec[64] = {}, cache_el[64] = {};
    const uint64_t resident =
        vec ? resident_blocks((const void *)k_check_gen_packed<DA, DB, DIST, UM, true, D>, cache_vec)
            : resident_blocks((const void *)k_check_gen_packed<DA, DB, DIST, UM, false, 2>, cache_el);
    uint32_t U, G;
    check_grid(n / E, resident, &U, &G);
    CheckPartial *parts = (CheckPartial *)scratch;
    hipError_t e;
    if (vec)
        e = launch(k_check_gen_packed<DA, DB, DIST, UM, true, D>, dim3(G), dim3(kThreads), s, (const uint8_t *)a, ref,
                   n, rtol, atol, parts, U);
    else
        e = launch(k_check_gen_packed<DA, DB, DIST, UM, false, 2>, dim3(G), dim3(kThreads), s, (const uint8_t *)a,
                   ref, n, rtol, atol, parts, U);
    if (e != hipSuccess) return e;
    return launch_check_final(parts, G, n, out, s);
}

template <int DA, int DB>
hipError_t check_ab(const void *a, const PackedRefArgs &g, int dist, int um, uint64_t n, float rtol, float atol,
                    void *scratch, krex_check_result *out, hipStream_t s)
{
    switch (dist) {
    case UNIFORM:
        if (um == UM_FUSED) return check_t<DA, DB, UNIFORM, UM_FUSED>(a, g, n, rtol, atol, scratch, out, s);
        if (um == UM_SCALED) return check_t<DA, DB, UNIFORM, UM_SCALED>(a, g, n, rtol, atol, scratch, out, s);
        return check_t<DA, DB, UNIFORM, UM_WORD>(a, g, n, rtol, atol, scratch, out, s);
    case NORMAL: return check_t<DA, DB, NORMAL, UM_WORD>(a, g, n, rtol, atol, scratch, out, s);
    default: return check_t<DA, DB, BITCAST, UM_WORD>(a, g, n, rtol, atol, scratch, out, s);
    }
}

template <int DA>
hipError_t check_a(const void *a, int dtb, const PackedRefArgs &g, int dist, int um, uint64_t n, float rtol,
                   float atol, void *scratch, krex_check_result *out, hipStream_t s)
{
    switch (dtb) {
    case BF16: return check_ab<DA, BF16>(a, g, dist, um, n, rtol, atol, scratch, out, s);
    case F16: return check_ab<DA, F16>(a, g, dist, um, n, rtol, atol, scratch, out, s);
    default: return check_ab<DA, F8>(a, g, dist, um, n, rtol, atol, scratch, out, s);
    }
}

}  // namespace

hipError_t launch_check_gen_packed(const void *a, int dta, int dtb, uint64_t n, uint64_t seed, uint64_t offset,
                                   int dist, float p0, float p1, float rtol, float atol, void *scratch,
                                   krex_check_result *out, hipStream_t s)
{
    if (n == 0) return launch_check_final((const CheckPartial *)scratch, 0u, n, out, s);
    if (dtb != BF16 && dtb != F16 && dtb != F8) return hipErrorInvalidValue;
    PackedRefArgs g;
    g.seed = seed;
    g.offset = offset;
    g.p0 = p0;
    const int um = packed_transform_constants(dtb, dist, p0, p1, &g.p1, &g.rs);
    switch (dta) {
    case F32: return check_a<F32>(a, dtb, g, dist, um, n, rtol, atol, scratch, out, s);
    case BF16: return check_a<BF16>(a, dtb, g, dist, um, n, rtol, atol, scratch, out, s);
    case F16: return check_a<F16>(a, dtb, g, dist, um, n, rtol, atol, scratch, out, s);
    default: return check_a<F8>(a, dtb, g, dist, um, n, rtol, atol, scratch, out, s);
    }
}

}  // namespace krex
