// check_gen.hip -- the fused allclose check against a reference that is
// regenerated instead of read (Section 1; Section 2.1: a command generates
// its inputs and checks against a reference). When the reference is itself a
// generated tensor -- the expected output of a copy, cast or identity
// candidate, or a check of data that crossed a link -- its values are a pure
// function of (seed, offset + j), so the check recomputes them in registers
// and reads only the candidate: half the HBM bytes of the two-operand check
// for equal dtypes, at the cost of one Philox block per four elements.
//
//   k_check_gen  the check body of check_device.hpp with the reference
//                source RefGen; its partials are reduced by k_check_final
//                like the two-operand check's.
//
// The vector path needs a 16-byte aligned candidate and a word offset that is
// a multiple of 4 (every chunk starts on a Philox block); anything else takes
// the element path, which computes the E / 4 + 1 blocks a chunk touches.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "check_device.hpp"
#include "hip_launch.hpp"
#include "krex_device.hpp"
#include "launch.hpp"

namespace krex {

template <int DA, int DB, int DIST, bool POW2, bool VEC, int D>
__global__ __launch_bounds__(kThreads) void k_check_gen(const uint8_t *a,
                                                        RefGen<DB, DIST, POW2, chunk_elems<DA, DB>()> ref, uint64_t n,
                                                        float rtol, float atol, CheckPartial *partials, uint32_t U)
{
    check_body<DA, DB, VEC, D>(a, ref, n, rtol, atol, partials, U);
}

namespace {

// What the launchers pass down: generation's stream and transform constants.
struct GenRefArgs {
    uint64_t seed, offset;
    float p0, p1;   // p1: c when the uniform scale is exact, else the range or the std
};

// Depth of the candidate's load ring: one operand is loaded and the Philox
// arithmetic between loads hides their latency, so two buffers suffice.
constexpr int kGenCheckDepth = 2;

template <int DA, int DB, int DIST, bool POW2>
hipError_t check_gen_t(const void *a, const GenRefArgs &g, uint64_t n, float rtol, float atol, void *scratch,
                       krex_check_result *out, hipStream_t s)
{
    constexpr int E = chunk_elems<DA, DB>();
    constexpr int D = kGenCheckDepth;
    const RefGen<DB, DIST, POW2, E> ref{g.offset, round_keys(g.seed), g.p0, g.p1, (uint32_t)(g.offset & 3u)};
    const bool vec = ((uintptr_t)a & 15u) == 0 && (g.offset & 3u) == 0;
    static uint32_t cache_vec[64] = {}, cache_el[64] = {};
    const uint64_t resident = vec ? resident_blocks((const void *)k_check_gen<DA, DB, DIST, POW2, true, D>, cache_vec)
                                  : resident_blocks((const void *)k_check_gen<DA, DB, DIST, POW2, false, 2>, cache_el);
    uint32_t U, G;
    check_grid(n / E, resident, &U, &G);
    CheckPartial *parts = (CheckPartial *)scratch;
    hipError_t e;
    if (vec)
        e = launch(k_check_gen<DA, DB, DIST, POW2, true, D>, dim3(G), dim3(kThreads), s, (const uint8_t *)a, ref, n,
                   rtol, atol, parts, U);
    else
        e = launch(k_check_gen<DA, DB, DIST, POW2, false, 2>, dim3(G), dim3(kThreads), s, (const uint8_t *)a, ref, n,
                   rtol, atol, parts, U);
    if (e != hipSuccess) return e;
    return launch_check_final(parts, G, n, out, s);
}

template <int DA, int DB>
hipError_t check_gen_ab(const void *a, const GenRefArgs &g, int dist, bool pow2, uint64_t n, float rtol, float atol,
                        void *scratch, krex_check_result *out, hipStream_t s)
{
    switch (dist) {
    case UNIFORM:
        if (pow2) return check_gen_t<DA, DB, UNIFORM, true>(a, g, n, rtol, atol, scratch, out, s);
        return check_gen_t<DA, DB, UNIFORM, false>(a, g, n, rtol, atol, scratch, out, s);
    case NORMAL: return check_gen_t<DA, DB, NORMAL, false>(a, g, n, rtol, atol, scratch, out, s);
    default: return check_gen_t<DA, DB, BITCAST, false>(a, g, n, rtol, atol, scratch, out, s);
    }
}

template <int DA>
hipError_t check_gen_a(const void *a, int dtb, const GenRefArgs &g, int dist, bool pow2, uint64_t n, float rtol,
                       float atol, void *scratch, krex_check_result *out, hipStream_t s)
{
    switch (dtb) {
    case F32: return check_gen_ab<DA, F32>(a, g, dist, pow2, n, rtol, atol, scratch, out, s);
    case BF16: return check_gen_ab<DA, BF16>(a, g, dist, pow2, n, rtol, atol, scratch, out, s);
    case F16: return check_gen_ab<DA, F16>(a, g, dist, pow2, n, rtol, atol, scratch, out, s);
    default: return check_gen_ab<DA, F8>(a, g, dist, pow2, n, rtol, atol, scratch, out, s);
    }
}

}  // namespace

hipError_t launch_check_gen(const void *a, int dta, int dtb, uint64_t n, uint64_t seed, uint64_t offset, int dist,
                            float p0, float p1, float rtol, float atol, void *scratch, krex_check_result *out,
                            hipStream_t s)
{
    if (n == 0) return launch_check_final((const CheckPartial *)scratch, 0u, n, out, s);
    GenRefArgs g;
    g.seed = seed;
    g.offset = offset;
    g.p0 = p0;
    const bool pow2 = gen_transform_constants(dist, p0, p1, &g.p1);
    switch (dta) {
    case F32: return check_gen_a<F32>(a, dtb, g, dist, pow2, n, rtol, atol, scratch, out, s);
    case BF16: return check_gen_a<BF16>(a, dtb, g, dist, pow2, n, rtol, atol, scratch, out, s);
    case F16: return check_gen_a<F16>(a, dtb, g, dist, pow2, n, rtol, atol, scratch, out, s);
    default: return check_gen_a<F8>(a, dtb, g, dist, pow2, n, rtol, atol, scratch, out, s);
    }
}

}  // namespace krex
