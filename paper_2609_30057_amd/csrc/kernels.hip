// kernels.hip -- gfx950 kernels of the benchmarking-command hot path and
// their launchers.
//
//   k_gen     seeded generation (Section 1; Section 2.1): one Philox block
//             gives four consecutive elements; a thread owns G blocks so
//             that its output is one 16-byte store (G = 1 for 4-byte
//             types, 2 for 2-byte, 4 for fp8).
//   k_xform   the same transforms on caller-supplied words.
//   k_inject  Bernoulli mismatch injection on its own word stream.
//   k_check   fused allclose check (Section 2.1): 16-byte loads of both
//             operands, branch-free verdicts, wave64 ballots and shuffles,
//             LDS across the block's four waves, one partial per block;
//             k_check_final reduces the partials into the result record.
//   k_flush   16-byte allocating stores of a pattern (Section 2.1 flush
//             between iterations; Section 4.2 step 5).
//   k_probe   fixed-work FMA kernel timed by the fidelity measurement
//             (Section 6.4, Eq. 1).
//   k_sgemm   naive fp32 GEMM standing in for a candidate kernel.
//
// Work is laid out block-contiguously in address order (block b owns units
// [b 256 U, (b + 1) 256 U), thread t takes unit b 256 U + u 256 + t), which
// streams HBM faster on gfx950 than persistent grid-stride loops. The launch
// shape never changes a result: every element's value depends only on its
// index.
#include <hip/hip_runtime.h>
#include <float.h>
#include <math.h>
#include <stdlib.h>

#include <cmath>
#include <mutex>

#include "check_device.hpp"
#include "hip_launch.hpp"
#include "krex_device.hpp"
#include "launch.hpp"

namespace krex {

template <int DT> struct group_of { static constexpr int G = 4 / dtype_traits<DT>::size; };

// ------------------------------------------------------------------ generation

struct GenParams {
    uint8_t *dst;
    uint64_t n;
    uint64_t offset;
    float p0, p1;      // uniform: lo and fl(hi - lo); normal: mean and std
    float c;           // uniform with a power-of-two range: range 2^-24
    int pow2;          // uniform range is a power of two (c normal)
    uint64_t b0;       // first Philox block
    uint64_t ngroups;  // groups of G blocks
    uint32_t U;        // groups per thread, block-contiguous
    int vec;           // offset % 4 == 0 and dst 16-byte aligned
    RoundKeys rk;      // the seed's Philox key schedule
};

// POW2: uniform with a power-of-two range (the fused transform; P.c).
template <int DT, int DIST, bool POW2>
__global__ __launch_bounds__(kThreads) void k_gen(GenParams P)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int G = group_of<DT>::G;
    union Pack {
        uint4 v;
        uint32_t w[4];
        T s[4 * G];
    };
    // Group g: G Philox blocks from P.b0 + g G, transformed and packed into
    // 16 bytes.
    auto group = [&](uint64_t g, Pack &pk) {
        const uint64_t bfirst = P.b0 + g * G;
        if constexpr (DT == U32) {
            const words4 w = philox_block(bfirst, P.rk);
#pragma unroll
            for (int l = 0; l < 4; ++l) pk.w[l] = w.v[l];
        } else {
            words4 wb[G];
            philox_blocks<G>(bfirst, P.rk, wb);
            float v[4 * G];
#pragma unroll
            for (int i = 0; i < G; ++i) transform4<DIST, POW2>(wb[i], P.p0, POW2 ? P.c : P.p1, v + 4 * i);
            pack_narrow<DT, DIST == BITCAST>(v, pk.w);
        }
    };
    const uint64_t gb0 = (uint64_t)blockIdx.x * P.U * kThreads;   // the block's first group
    const uint64_t gend = gb0 + (uint64_t)P.U * kThreads;
    // vec: offset % 4 == 0, so group g's first element is 4 G g. A block whose
    // groups all lie in range takes the path without per-lane checks (a
    // block-uniform branch); only the grid's last block can miss it.
    if (P.vec && gend <= P.ngroups && 4 * G * gend <= P.n) {
        for (uint32_t u = 0; u < P.U; ++u) {
            const uint64_t gb = gb0 + (uint64_t)u * kThreads;
            Pack pk;
            group(gb + threadIdx.x, pk);
            store16_stream(P.dst + 4 * G * gb * ES, 16u * threadIdx.x, pk.v);
        }
        return;
    }
    for (uint32_t u = 0; u < P.U; ++u) {
        const uint64_t g = gb0 + (uint64_t)u * kThreads + threadIdx.x;
        if (g >= P.ngroups) break;
        const uint64_t bfirst = P.b0 + g * G;
        Pack pk;
        group(g, pk);
        const uint64_t j0 = 4 * bfirst - P.offset;
        if (P.vec && j0 + 4 * G <= P.n) {
            // the block's first group starts at element jb (uniform across
            // the block) and lane t's 16 bytes at jb + 4 G t
            const uint64_t gb = gb0 + (uint64_t)u * kThreads;
            const uint64_t jb = 4 * (P.b0 + gb * G) - P.offset;
            store16_stream(P.dst + jb * ES, 16u * threadIdx.x, pk.v);
        } else {
#pragma unroll
            for (int e = 0; e < 4 * G; ++e) {
                const uint64_t w = 4 * bfirst + (uint64_t)e;
                if (w >= P.offset && w - P.offset < P.n) reinterpret_cast<T *>(P.dst)[w - P.offset] = pk.s[e];
            }
        }
    }
}

// Units per thread and grid of the block-contiguous layout: block b owns
// units [b 256 U, (b + 1) 256 U). U grows beyond u_pref only to keep a
// dispatch within 2^31 work-items.
static void shape(uint64_t units, uint32_t u_pref, uint32_t *U, uint32_t *grid)
{
    uint64_t u = u_pref ? u_pref : 1;
    const uint64_t min_u = (units + (1ull << 31) - 1) >> 31;
    if (u < min_u) u = min_u;
    uint64_t g = (units + kThreads * u - 1) / (kThreads * u);
    *U = (uint32_t)u;
    *grid = (uint32_t)(g ? g : 1);
}

// Whether range 2^-W times every integer f in [0, 2^W) is an exact fp32
// product: range positive and finite, c = range 2^-W normal, and the odd part
// q of range's 24-bit significand small enough that f q < 2^24 for every f
// (range = q 2^s, so f c = f q 2^(s - W) is then a 24-bit integer times a
// power of two, at least c, hence a normal float). W = 24 with q = 1: a power
// of two. Then lo + fl(c f) equals the single fused multiply-add. *c = c.
static bool exact_scale(float range, int W, float *c)
{
    *c = 0.0f;
    if (!(range > 0.0f) || !std::isfinite(range)) return false;
    int e = 0;
    const float m = frexpf(range, &e);                       // m in [1/2, 1)
    const uint32_t sig = (uint32_t)ldexpf(m, 24);             // exact 24-bit significand
    const uint64_t q = sig >> __builtin_ctz(sig);
    const float cc = ldexpf(range, -W);
    if (!(cc >= FLT_MIN) || q * ((1ull << W) - 1ull) >= (1ull << 24)) return false;
    *c = cc;
    return true;
}

bool gen_transform_constants(int dist, float p0, float p1, float *q1)
{
    const float r = (dist == UNIFORM) ? (p1 - p0) : p1;
    float c = 0.0f;
    if (dist == UNIFORM && exact_scale(r, 24, &c)) {
        *q1 = c;
        return true;
    }
    *q1 = r;
    return false;
}

// Preferred units per thread, measured per kernel on gfx950 (rocprofv3
// averages at 268M narrow / 67M fp32 elements). One unit per thread, a
// one-shot grid in address order, streams HBM fastest: it wins where the
// stores bound the kernel (fp32 and packed 16-bit uniform generation, fp32
// and 16-bit injection) and, less clearly, for the normal transform. Where a
// unit's Philox work takes about as long as its store (narrow word-stream
// uniform and bitcast generation, the packed fp8 uniform stream, fp8
// injection and narrow generation with injection), four units per thread
// are 5-10% faster: a wave's store of one unit overlaps its arithmetic for
// the next, and a quarter of the waves are dispatched. The packed normal
// transform gains ~4% from two. KREX_GEN_U, KREX_PACKED_U, KREX_INJECT_U and
// KREX_GEN_INJECT_U override these.
template <int DT, int DIST>
static constexpr uint32_t gen_units()
{
    return (DIST != NORMAL && dtype_traits<DT>::size <= 2) ? 4u : 1u;
}

template <int DT, int DIST>
static constexpr uint32_t packed_units()
{
    return DIST == NORMAL ? 2u : (DT == F8 && DIST == UNIFORM) ? 4u : 1u;
}

template <int DT>
static constexpr uint32_t inject_units()
{
    return dtype_traits<DT>::size == 1 ? 4u : 1u;
}

template <int DT, int DIST>
static hipError_t gen_dt_dist(GenParams P, hipStream_t s)
{
    static const uint32_t u_env = tune_env("KREX_GEN_U", 0);
    const uint32_t u_pref = u_env ? u_env : gen_units<DT, DIST>();
    uint32_t grid;
    shape(P.ngroups, u_pref, &P.U, &grid);
    if constexpr (DIST == UNIFORM && DT != U32)
        if (P.pow2) return launch(k_gen<DT, DIST, true>, dim3(grid), dim3(kThreads), s, P);
    return launch(k_gen<DT, DIST, false>, dim3(grid), dim3(kThreads), s, P);
}

template <int DT>
static hipError_t gen_dt(const GenParams &P, int dist, hipStream_t s)
{
    if constexpr (DT == U32) return gen_dt_dist<U32, UNIFORM>(P, s);
    switch (dist) {
    case UNIFORM: return gen_dt_dist<DT, UNIFORM>(P, s);
    case NORMAL: return gen_dt_dist<DT, NORMAL>(P, s);
    default: return gen_dt_dist<DT, BITCAST>(P, s);
    }
}

// Generation parameters of krex_gen (n > 0): Philox key, first block,
// groups of G blocks, the uniform transform's constants.
static GenParams make_gen_params(void *dst, int dt, uint64_t n, uint64_t seed, uint64_t offset, int dist, float p0,
                                 float p1)
{
    GenParams P;
    P.dst = (uint8_t *)dst;
    P.n = n;
    P.offset = offset;
    P.p0 = p0;
    P.p1 = (dist == UNIFORM) ? (p1 - p0) : p1;
    P.pow2 = (dist == UNIFORM && exact_scale(P.p1, 24, &P.c)) ? 1 : 0;
    P.b0 = offset >> 2;
    const uint64_t blast = (offset + (n - 1)) >> 2;
    const uint64_t nblocks = blast - P.b0 + 1;
    int G = 1;
    switch (dt) {
    case BF16: case F16: G = 2; break;
    case F8: G = 4; break;
    default: G = 1; break;
    }
    P.ngroups = (nblocks + (uint64_t)G - 1) / (uint64_t)G;
    P.vec = ((offset & 3u) == 0 && ((uintptr_t)dst & 15u) == 0) ? 1 : 0;
    P.U = 1;
    P.rk = round_keys(seed);
    return P;
}

hipError_t launch_gen(void *dst, int dt, uint64_t n, uint64_t seed, uint64_t offset, int dist, float p0,
                      float p1, hipStream_t s)
{
    if (n == 0) return hipSuccess;
    const GenParams P = make_gen_params(dst, dt, n, seed, offset, dist, p0, p1);
    switch (dt) {
    case F32: return gen_dt<F32>(P, dist, s);
    case BF16: return gen_dt<BF16>(P, dist, s);
    case F16: return gen_dt<F16>(P, dist, s);
    case F8: return gen_dt<F8>(P, dist, s);
    default: return gen_dt<U32>(P, dist, s);
    }
}

// ------------------------------------------------------------- packed stream
//
// The generator of the packed stream (its units are built by packed_unit of
// the device header): one thread unit is one 16-byte output vector.

struct PackedParams {
    uint8_t *dst;
    uint64_t n;
    uint64_t offset;   // in fields
    float p0, p1;      // uniform: lo and fl(hi - lo); normal: mean and std
    float rs;          // uniform: fl(hi - lo) 2^-W when that is exact
    int umode;         // uniform: UM_WORD, UM_SCALED or UM_FUSED
    uint64_t u0;       // first unit (units are E fields, E-aligned)
    uint64_t nunits;
    uint32_t U;        // units per thread, block-contiguous
    int vec;           // offset % E == 0 and dst 16-byte aligned
    RoundKeys rk;      // the seed's Philox key schedule
};

template <int DT, int DIST, int UM>
__global__ __launch_bounds__(kThreads) void k_gen_packed(PackedParams P)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int E = packed_of<DT, DIST>::E;
    union Pack {
        uint4 v;
        uint32_t w[4];
        T s[E];
    };
    auto unit_values = [&](uint64_t unit, Pack &pk) {
        packed_unit<DT, DIST, UM>(unit, P.rk, P.p0, P.p1, P.rs, pk.w);
    };
    const uint64_t gb0 = (uint64_t)blockIdx.x * P.U * kThreads;   // the block's first unit (from u0)
    const uint64_t gend = gb0 + (uint64_t)P.U * kThreads;
    // vec: offset % E == 0, so unit u0 + g starts at field E g. A block whose
    // units all lie in range stores without per-lane checks (a block-uniform
    // branch); only the grid's last block can miss it.
    if (P.vec && gend <= P.nunits && E * gend <= P.n) {
        for (uint32_t u = 0; u < P.U; ++u) {
            const uint64_t gb = gb0 + (uint64_t)u * kThreads;
            Pack pk;
            unit_values(P.u0 + gb + threadIdx.x, pk);
            store16_stream(P.dst + E * gb * ES, 16u * threadIdx.x, pk.v);
        }
        return;
    }
    for (uint32_t u = 0; u < P.U; ++u) {
        const uint64_t g = gb0 + (uint64_t)u * kThreads + threadIdx.x;
        if (g >= P.nunits) break;
        const uint64_t unit = P.u0 + g;
        Pack pk;
        unit_values(unit, pk);
        const uint64_t q0 = unit * (uint64_t)E;
        if (P.vec && q0 >= P.offset && q0 - P.offset + E <= P.n) {
            const uint64_t gb = gb0 + (uint64_t)u * kThreads;
            const uint64_t qb = (P.u0 + gb) * (uint64_t)E - P.offset;
            store16_stream(P.dst + qb * ES, 16u * threadIdx.x, pk.v);
        } else {
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const uint64_t q = q0 + (uint64_t)e;
                if (q >= P.offset && q - P.offset < P.n) reinterpret_cast<T *>(P.dst)[q - P.offset] = pk.s[e];
            }
        }
    }
}

int packed_transform_constants(int dt, int dist, float p0, float p1, float *q1, float *rs)
{
    const int W = (dt == F8 && dist != NORMAL) ? 8 : 16;
    *q1 = (dist == UNIFORM) ? (p1 - p0) : p1;
    *rs = 0.0f;
    if (dist != UNIFORM) return UM_WORD;
    *rs = ldexpf(*q1, -W);
    if (ldexpf(*rs, W) != *q1) return UM_WORD;
    float c;
    return exact_scale(*q1, W, &c) ? UM_FUSED : UM_SCALED;
}

template <int DT, int DIST>
static hipError_t gen_packed_dt_dist(PackedParams P, hipStream_t s)
{
    constexpr int E = packed_of<DT, DIST>::E;
    P.u0 = P.offset / E;
    P.nunits = (P.offset + (P.n - 1)) / E - P.u0 + 1;
    P.vec = (P.offset % E == 0 && ((uintptr_t)P.dst & 15u) == 0) ? 1 : 0;
    static const uint32_t u_env = tune_env("KREX_PACKED_U", 0);
    const uint32_t u_pref = u_env ? u_env : packed_units<DT, DIST>();
    uint32_t grid;
    shape(P.nunits, u_pref, &P.U, &grid);
    if constexpr (DIST == UNIFORM) {
        if (P.umode == UM_FUSED) return launch(k_gen_packed<DT, DIST, UM_FUSED>, dim3(grid), dim3(kThreads), s, P);
        if (P.umode == UM_SCALED) return launch(k_gen_packed<DT, DIST, UM_SCALED>, dim3(grid), dim3(kThreads), s, P);
    }
    return launch(k_gen_packed<DT, DIST, UM_WORD>, dim3(grid), dim3(kThreads), s, P);
}

template <int DT>
static hipError_t gen_packed_dt(const PackedParams &P, int dist, hipStream_t s)
{
    switch (dist) {
    case UNIFORM: return gen_packed_dt_dist<DT, UNIFORM>(P, s);
    case NORMAL: return gen_packed_dt_dist<DT, NORMAL>(P, s);
    default: return gen_packed_dt_dist<DT, BITCAST>(P, s);
    }
}

hipError_t launch_gen_packed(void *dst, int dt, uint64_t n, uint64_t seed, uint64_t offset, int dist, float p0,
                             float p1, hipStream_t s)
{
    if (n == 0) return hipSuccess;
    PackedParams P;
    P.dst = (uint8_t *)dst;
    P.n = n;
    P.offset = offset;
    P.rk = round_keys(seed);
    P.p0 = p0;
    P.umode = packed_transform_constants(dt, dist, p0, p1, &P.p1, &P.rs);
    switch (dt) {
    case BF16: return gen_packed_dt<BF16>(P, dist, s);
    case F16: return gen_packed_dt<F16>(P, dist, s);
    case F8: return gen_packed_dt<F8>(P, dist, s);
    default: return hipErrorInvalidValue;
    }
}

// ------------------------------------------------------------- words transform

struct XformParams {
    uint8_t *dst;
    const uint32_t *words;
    uint64_t n;
    float p0, p1;
    float c;           // as in GenParams
    int pow2;
    uint64_t ngroups;
    uint32_t U;
    int vec;
};

template <int DT, int DIST>
__global__ __launch_bounds__(kThreads) void k_xform(XformParams P)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int G = group_of<DT>::G;
    for (uint32_t u = 0; u < P.U; ++u) {
        const uint64_t g = ((uint64_t)blockIdx.x * P.U + u) * kThreads + threadIdx.x;
        if (g >= P.ngroups) break;
        const uint64_t j0 = g * 4 * G;
        if (P.vec && j0 + 4 * G <= P.n) {
            union {
                uint4 v;
                uint32_t w[4];
                T s[4 * G];
            } pk;
            float v[4 * G];
#pragma unroll
            for (int i = 0; i < G; ++i) {
                const uint4 raw = reinterpret_cast<const uint4 *>(P.words + j0)[i];
                words4 w;
                w.v[0] = raw.x; w.v[1] = raw.y; w.v[2] = raw.z; w.v[3] = raw.w;
                if constexpr (DT == U32) {
#pragma unroll
                    for (int l = 0; l < 4; ++l) pk.w[l] = w.v[l];
                } else if (DIST == UNIFORM && P.pow2) {
                    transform4<DIST, true>(w, P.p0, P.c, v + 4 * i);
                } else {
                    transform4<DIST>(w, P.p0, P.p1, v + 4 * i);
                }
            }
            if constexpr (DT != U32) pack_narrow<DT, DIST == BITCAST>(v, pk.w);
            const uint64_t jb = ((uint64_t)blockIdx.x * P.U + u) * kThreads * 4 * G;
            store16_stream(P.dst + jb * ES, 16u * threadIdx.x, pk.v);
        } else {
            for (int e = 0; e < 4 * G; ++e) {
                const uint64_t j = j0 + (uint64_t)e;
                if (j >= P.n) break;
                T out;
                if constexpr (DT == U32) {
                    out = P.words[j];
                } else {
                    float v;
                    if constexpr (DIST == UNIFORM) {
                        v = P.pow2 ? uniform_f32_pow2(P.words[j], P.p0, P.c) : uniform_f32(P.words[j], P.p0, P.p1);
                    } else if constexpr (DIST == NORMAL) {
                        float z0, z1;
                        normal_pair(P.words[j & ~(uint64_t)1], P.words[j | 1u], z0, z1);
                        const float sz = P.p1 * ((j & 1u) ? z1 : z0);
                        v = P.p0 + sz;
                    } else {
                        v = __uint_as_float(P.words[j]);
                    }
                    out = narrow<DT, DIST == BITCAST>(v);
                }
                reinterpret_cast<T *>(P.dst)[j] = out;
            }
        }
    }
}

template <int DT>
static hipError_t xform_dt(XformParams P, int dist, hipStream_t s)
{
    uint32_t grid;
    shape(P.ngroups, 1, &P.U, &grid);
    if constexpr (DT == U32) return launch(k_xform<U32, UNIFORM>, dim3(grid), dim3(kThreads), s, P);
    switch (dist) {
    case UNIFORM: return launch(k_xform<DT, UNIFORM>, dim3(grid), dim3(kThreads), s, P);
    case NORMAL: return launch(k_xform<DT, NORMAL>, dim3(grid), dim3(kThreads), s, P);
    default: return launch(k_xform<DT, BITCAST>, dim3(grid), dim3(kThreads), s, P);
    }
}

hipError_t launch_xform(void *dst, int dt, uint64_t n, const uint32_t *words, int dist, float p0, float p1,
                        hipStream_t s)
{
    if (n == 0) return hipSuccess;
    XformParams P;
    P.dst = (uint8_t *)dst;
    P.words = words;
    P.n = n;
    P.p0 = p0;
    P.p1 = (dist == UNIFORM) ? (p1 - p0) : p1;
    P.pow2 = (dist == UNIFORM && exact_scale(P.p1, 24, &P.c)) ? 1 : 0;
    const int G = (dt == BF16 || dt == F16) ? 2 : (dt == F8 ? 4 : 1);
    P.ngroups = (n + 4u * G - 1) / (4u * G);
    P.vec = (((uintptr_t)dst & 15u) == 0 && ((uintptr_t)words & 15u) == 0) ? 1 : 0;
    switch (dt) {
    case F32: return xform_dt<F32>(P, dist, s);
    case BF16: return xform_dt<BF16>(P, dist, s);
    case F16: return xform_dt<F16>(P, dist, s);
    case F8: return xform_dt<F8>(P, dist, s);
    default: return xform_dt<U32>(P, dist, s);
    }
}

// ------------------------------------------------------------------ injection

struct InjectParams {
    uint8_t *y;
    const uint8_t *x;
    uint64_t n;
    uint64_t moff;
    uint64_t T;        // threshold in [0, 2^32]
    float delta;
    uint64_t b0;
    uint64_t ngroups;
    uint32_t U;
    int vec;
    RoundKeys rk;      // the mask seed's Philox key schedule
};

template <int DT, int MODE>
__device__ __forceinline__ typename dtype_traits<DT>::storage perturb(typename dtype_traits<DT>::storage bits,
                                                                      float delta)
{
    const float X = widen<DT>(bits);
    if constexpr (MODE == INJ_ROUND) {
        const float s = X + delta;
        return narrow<DT>(s);
    } else {
        const float sp = X + delta;
        const float dp = sp - X;
        if (dp == delta && widen<DT>(narrow<DT, false>(sp)) == sp) return narrow<DT, false>(sp);
        const float sm = X - delta;
        const float dm = X - sm;
        if (dm == delta && widen<DT>(narrow<DT, false>(sm)) == sm) return narrow<DT, false>(sm);
        return bits;
    }
}

// The 4 G elements of s perturbed where their mask words (G Philox blocks)
// are below T. At the commands' rates a perturbation is rare, so the
// branches are wave-uniform (a ballot decides): one for the whole group,
// then one per element, whose perturbation is computed for the wave and
// selected per lane. Divergent per-lane branches would cost scalar
// exec-mask instructions on every element.
// T is in [0, 2^32]: w < T is tested as w <= T - 1 in 32 bits, T = 0 (no
// element) returning at once.
template <int DT, int MODE, int G>
__device__ __forceinline__ void perturb_group(const words4 (&m)[G], uint64_t T, float delta,
                                              typename dtype_traits<DT>::storage (&s)[4 * G])
{
    if (T == 0) return;
    const uint32_t last = (uint32_t)(T - 1);
    uint32_t wmin = m[0].v[0];     // the lane's smallest mask word (three-way minima)
#pragma unroll
    for (int i = 0; i < G; ++i)
#pragma unroll
        for (int l = 0; l < 4; ++l) wmin = wmin < m[i].v[l] ? wmin : m[i].v[l];
    if (__ballot(wmin <= last) == 0) return;
#pragma unroll
    for (int i = 0; i < G; ++i)
#pragma unroll
        for (int l = 0; l < 4; ++l) {
            const bool hit = m[i].v[l] <= last;
            if (__ballot(hit) != 0) {
                const typename dtype_traits<DT>::storage p = perturb<DT, MODE>(s[4 * i + l], delta);
                s[4 * i + l] = hit ? p : s[4 * i + l];
            }
        }
}

template <int DT, int MODE>
__global__ __launch_bounds__(kThreads) void k_inject(InjectParams P)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int G = group_of<DT>::G;
    union Pack {
        uint4 v;
        T s[4 * G];
    };
    // The 4 G elements from the group starting at Philox block bfirst,
    // perturbed where their mask word is below T.
    auto mask_group = [&](uint64_t bfirst, Pack &pk) {
        words4 m[G];
#pragma unroll
        for (int i = 0; i < G; ++i) m[i] = philox_block(bfirst + i, P.rk);
        perturb_group<DT, MODE, G>(m, P.T, P.delta, pk.s);
    };
    const uint64_t gb0 = (uint64_t)blockIdx.x * P.U * kThreads;   // the block's first group
    const uint64_t gend = gb0 + (uint64_t)P.U * kThreads;
    // vec: moff % 4 == 0, so group g's first element is 4 G g. A block whose
    // groups all lie in range takes the path without per-lane checks (a
    // block-uniform branch); only the grid's last block can miss it.
    if (P.vec && gend <= P.ngroups && 4 * G * gend <= P.n) {
        for (uint32_t u = 0; u < P.U; ++u) {
            const uint64_t gb = gb0 + (uint64_t)u * kThreads;
            const uint64_t g = gb + threadIdx.x;
            Pack pk;
            pk.v = load16_stream(P.x + 4 * G * g * ES);
            mask_group(P.b0 + g * G, pk);
            store16_stream(P.y + 4 * G * gb * ES, 16u * threadIdx.x, pk.v);
        }
        return;
    }
    for (uint32_t u = 0; u < P.U; ++u) {
        const uint64_t g = gb0 + (uint64_t)u * kThreads + threadIdx.x;
        if (g >= P.ngroups) break;
        const uint64_t bfirst = P.b0 + g * G;
        const uint64_t j0 = 4 * bfirst - P.moff;
        if (P.vec && j0 + 4 * G <= P.n) {
            Pack pk;
            pk.v = load16_stream(P.x + j0 * ES);
            mask_group(bfirst, pk);
            const uint64_t gb = gb0 + (uint64_t)u * kThreads;
            const uint64_t jb = 4 * (P.b0 + gb * G) - P.moff;
            store16_stream(P.y + jb * ES, 16u * threadIdx.x, pk.v);
        } else {
            for (int i = 0; i < G; ++i) {
                const words4 w = philox_block(bfirst + i, P.rk);
                for (int l = 0; l < 4; ++l) {
                    const uint64_t wi = 4 * (bfirst + i) + (uint64_t)l;
                    if (wi < P.moff || wi - P.moff >= P.n) continue;
                    const uint64_t j = wi - P.moff;
                    T v = reinterpret_cast<const T *>(P.x)[j];
                    if ((uint64_t)w.v[l] < P.T) v = perturb<DT, MODE>(v, P.delta);
                    reinterpret_cast<T *>(P.y)[j] = v;
                }
            }
        }
    }
}

template <int DT>
static hipError_t inject_dt(InjectParams P, int mode, hipStream_t s)
{
    static const uint32_t u_env = tune_env("KREX_INJECT_U", 0);
    const uint32_t u_pref = u_env ? u_env : inject_units<DT>();
    uint32_t grid;
    shape(P.ngroups, u_pref, &P.U, &grid);
    if (mode == INJ_ROUND) return launch(k_inject<DT, INJ_ROUND>, dim3(grid), dim3(kThreads), s, P);
    return launch(k_inject<DT, INJ_EXACT>, dim3(grid), dim3(kThreads), s, P);
}

hipError_t launch_inject(void *y, const void *x, int dt, uint64_t n, uint64_t mseed, uint64_t moff,
                         uint64_t T, float delta, int mode, hipStream_t s)
{
    if (n == 0) return hipSuccess;
    InjectParams P;
    P.y = (uint8_t *)y;
    P.x = (const uint8_t *)x;
    P.n = n;
    P.moff = moff;
    P.rk = round_keys(mseed);
    P.T = T;
    P.delta = delta;
    P.b0 = moff >> 2;
    const uint64_t blast = (moff + (n - 1)) >> 2;
    const uint64_t nblocks = blast - P.b0 + 1;
    const int G = (dt == BF16 || dt == F16) ? 2 : (dt == F8 ? 4 : 1);
    P.ngroups = (nblocks + G - 1) / G;
    P.vec = ((moff & 3u) == 0 && ((uintptr_t)y & 15u) == 0 && ((uintptr_t)x & 15u) == 0) ? 1 : 0;
    switch (dt) {
    case F32: return inject_dt<F32>(P, mode, s);
    case BF16: return inject_dt<BF16>(P, mode, s);
    case F16: return inject_dt<F16>(P, mode, s);
    default: return inject_dt<F8>(P, mode, s);
    }
}

// ---------------------------------------------------- generation with injection
//
// A command's input and its perturbed copy in one pass: x = krex_gen and
// y = krex_inject(x), without writing x and reading it back. With the value
// offset and the mask offset both multiples of 4, element j's value word and
// mask word are the same lane of their Philox blocks, so a thread unit is
// G value blocks (one 16-byte vector of x), the G mask blocks of the same
// elements, and one 16-byte vector of y. The host runs the two separate
// kernels otherwise.

struct GenInjectParams {
    GenParams g;       // generation of x (offset % 4 == 0)
    uint8_t *y;
    uint64_t mb0;      // first mask block: mask offset / 4
    uint64_t T;        // threshold in [0, 2^32]
    float delta;
    RoundKeys mrk;     // the mask key's schedule
};

template <int DT, int DIST, bool POW2, int MODE>
__global__ __launch_bounds__(kThreads) void k_gen_inject(GenInjectParams Q)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int G = group_of<DT>::G;
    const GenParams &P = Q.g;
    union Pack {
        uint4 v;
        uint32_t w[4];
        T s[4 * G];
    };
    // Group g of x (G value blocks from P.b0 + g G) and of y (x perturbed
    // where the mask words from Q.mb0 + g G are below T).
    auto group = [&](uint64_t g, Pack &px, Pack &py) {
        const uint64_t bfirst = P.b0 + g * G;
        const uint64_t mfirst = Q.mb0 + g * G;
        float v[4 * G];
        words4 m[G];
        if constexpr (DIST == NORMAL) {
            words4 wb[G];
            philox_blocks<G>(bfirst, P.rk, wb);
#pragma unroll
            for (int i = 0; i < G; ++i) transform4<DIST, POW2>(wb[i], P.p0, P.p1, v + 4 * i);
            philox_blocks<G>(mfirst, Q.mrk, m);
        } else {
#pragma unroll
            for (int i = 0; i < G; ++i)
                transform4<DIST, POW2>(philox_block(bfirst + i, P.rk), P.p0, POW2 ? P.c : P.p1, v + 4 * i);
#pragma unroll
            for (int i = 0; i < G; ++i) m[i] = philox_block(mfirst + i, Q.mrk);
        }
        pack_narrow<DT, DIST == BITCAST>(v, px.w);
        py.v = px.v;
        perturb_group<DT, MODE, G>(m, Q.T, Q.delta, py.s);
    };
    // offset % 4 == 0 (the launcher guarantees it), so group g's first
    // element is 4 G g; blocks wholly in range store without per-lane checks.
    const uint64_t gb0 = (uint64_t)blockIdx.x * P.U * kThreads;
    const uint64_t gend = gb0 + (uint64_t)P.U * kThreads;
    if (gend <= P.ngroups && 4 * G * gend <= P.n) {
        for (uint32_t u = 0; u < P.U; ++u) {
            const uint64_t gb = gb0 + (uint64_t)u * kThreads;
            Pack px, py;
            group(gb + threadIdx.x, px, py);
            store16_stream(P.dst + 4 * G * gb * ES, 16u * threadIdx.x, px.v);
            store16_stream(Q.y + 4 * G * gb * ES, 16u * threadIdx.x, py.v);
        }
        return;
    }
    for (uint32_t u = 0; u < P.U; ++u) {
        const uint64_t g = gb0 + (uint64_t)u * kThreads + threadIdx.x;
        if (g >= P.ngroups) break;
        Pack px, py;
        group(g, px, py);
        const uint64_t j0 = 4 * G * g;
        if (j0 + 4 * G <= P.n) {
            const uint64_t gb = gb0 + (uint64_t)u * kThreads;
            store16_stream(P.dst + 4 * G * gb * ES, 16u * threadIdx.x, px.v);
            store16_stream(Q.y + 4 * G * gb * ES, 16u * threadIdx.x, py.v);
        } else {
            for (int e = 0; e < 4 * G; ++e) {
                const uint64_t j = j0 + (uint64_t)e;
                if (j >= P.n) break;
                reinterpret_cast<T *>(P.dst)[j] = px.s[e];
                reinterpret_cast<T *>(Q.y)[j] = py.s[e];
            }
        }
    }
}

template <int DT, int DIST, bool POW2>
static hipError_t gen_inject_mode(GenInjectParams Q, int mode, hipStream_t s)
{
    static const uint32_t u_env = tune_env("KREX_GEN_INJECT_U", 0);
    const uint32_t u_pref = u_env ? u_env : gen_units<DT, DIST>();
    uint32_t grid;
    shape(Q.g.ngroups, u_pref, &Q.g.U, &grid);
    if (mode == INJ_ROUND) return launch(k_gen_inject<DT, DIST, POW2, INJ_ROUND>, dim3(grid), dim3(kThreads), s, Q);
    return launch(k_gen_inject<DT, DIST, POW2, INJ_EXACT>, dim3(grid), dim3(kThreads), s, Q);
}

template <int DT>
static hipError_t gen_inject_dt(const GenInjectParams &Q, int dist, int mode, hipStream_t s)
{
    switch (dist) {
    case UNIFORM:
        return Q.g.pow2 ? gen_inject_mode<DT, UNIFORM, true>(Q, mode, s) : gen_inject_mode<DT, UNIFORM, false>(Q, mode, s);
    case NORMAL: return gen_inject_mode<DT, NORMAL, false>(Q, mode, s);
    default: return gen_inject_mode<DT, BITCAST, false>(Q, mode, s);
    }
}

hipError_t launch_gen_inject(void *x, void *y, int dt, uint64_t n, uint64_t seed, uint64_t offset, int dist, float p0,
                             float p1, uint64_t mseed, uint64_t moff, uint64_t T, float delta, int mode,
                             hipStream_t s)
{
    if (n == 0) return hipSuccess;
    if ((offset & 3u) != 0 || (moff & 3u) != 0 || ((uintptr_t)x & 15u) != 0 || ((uintptr_t)y & 15u) != 0) {
        const hipError_t e = launch_gen(x, dt, n, seed, offset, dist, p0, p1, s);
        if (e != hipSuccess) return e;
        return launch_inject(y, x, dt, n, mseed, moff, T, delta, mode, s);
    }
    GenInjectParams Q;
    Q.g = make_gen_params(x, dt, n, seed, offset, dist, p0, p1);
    Q.y = (uint8_t *)y;
    Q.mb0 = moff >> 2;
    Q.mrk = round_keys(mseed);
    Q.T = T;
    Q.delta = delta;
    switch (dt) {
    case F32: return gen_inject_dt<F32>(Q, dist, mode, s);
    case BF16: return gen_inject_dt<BF16>(Q, dist, mode, s);
    case F16: return gen_inject_dt<F16>(Q, dist, mode, s);
    default: return gen_inject_dt<F8>(Q, dist, mode, s);
    }
}

// ---------------------------------------------------------------------- check
//
// The kernel body, its building blocks and the reference sources live in
// check_device.hpp; k_check takes the reference from memory.

size_t check_scratch_bytes() { return (size_t)kMaxCheckBlocks * sizeof(CheckPartial); }

// The fixed partial buffer of krex_check_noalloc: one CheckPartial per check
// block, kMaxCheckBlocks of them (128 KiB), the most any check grid uses.
// Each GPU the library runs on holds its own copy until the process ends.
// Host code never passes this name to a kernel (on the host it is only a
// stand-in for the symbol); it passes the device address that
// noalloc_scratch() looks up once per device.
static __device__ __align__(256) CheckPartial scratch[kMaxCheckBlocks];

static_assert(sizeof(scratch) == (size_t)kMaxCheckBlocks * sizeof(CheckPartial), "noalloc scratch size");

hipError_t noalloc_scratch(void **out)
{
    static std::mutex mu;
    static void *addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> g(mu);
    if (!addr[dev]) {
        // with `dev` current: its own copy of the array
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *out = addr[dev];
    return hipSuccess;
}

// Reference operand in memory.
template <int DA, int DB, bool VEC, int D>
__global__ __launch_bounds__(kThreads) void k_check(const uint8_t *a, const uint8_t *b, uint64_t n, float rtol,
                                                    float atol, CheckPartial *partials, uint32_t U)
{
    check_body<DA, DB, VEC, D>(a, RefMem<DB, chunk_elems<DA, DB>()>{b}, n, rtol, atol, partials, U);
}

__global__ __launch_bounds__(kFinalThreads) void k_check_final(const CheckPartial *partials, uint32_t nblocks,
                                                               uint64_t n, krex_check_result *out)
{
    // Every thread issues all of its partial loads before using any, so the
    // kernel pays one memory latency.
    constexpr int PER = kMaxCheckBlocks / kFinalThreads;
    uint64_t m = 0, nn = 0, key = 0;
    uint32_t rb = 0;
    CheckPartial p[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const uint32_t i = threadIdx.x + (uint32_t)j * kFinalThreads;
        if (i < nblocks) p[j] = partials[i];
        else p[j] = CheckPartial{0, 0, 0, 0, 0};
    }
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        m += p[j].mism;
        nn += p[j].nan;
        key = p[j].key > key ? p[j].key : key;
        rb = p[j].rel_bits > rb ? p[j].rel_bits : rb;   // non-negative floats order as integers
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        m += __shfl_xor((unsigned long long)m, off, 64);
        nn += __shfl_xor((unsigned long long)nn, off, 64);
        const uint64_t k2 = __shfl_xor((unsigned long long)key, off, 64);
        key = k2 > key ? k2 : key;
        const uint32_t r2 = __shfl_xor(rb, off, 64);
        rb = r2 > rb ? r2 : rb;
    }
    constexpr int W = kFinalThreads / 64;
    __shared__ uint64_t s_m[W], s_n[W], s_k[W];
    __shared__ uint32_t s_r[W];
    const int w = threadIdx.x / 64;
    if ((threadIdx.x & 63) == 0) {
        s_m[w] = m;
        s_n[w] = nn;
        s_k[w] = key;
        s_r[w] = rb;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
#pragma unroll
        for (int i = 1; i < W; ++i) {
            s_m[0] += s_m[i];
            s_n[0] += s_n[i];
            s_k[0] = s_k[i] > s_k[0] ? s_k[i] : s_k[0];
            s_r[0] = s_r[i] > s_r[0] ? s_r[i] : s_r[0];
        }
        const uint64_t K = s_k[0];
        out->n = n;
        out->mismatches = s_m[0];
        out->nan_count = s_n[0];
        out->argmax_abs = K ? kIdxMask - (K & kIdxMask) : ~0ull;
        out->max_abs = K ? __uint_as_float((uint32_t)(K >> 33)) : 0.0f;
        out->max_rel = __uint_as_float(s_r[0]);
        out->reserved[0] = 0;
        out->reserved[1] = 0;
        out->reserved[2] = 0;
    }
}

hipError_t launch_check_final(const CheckPartial *partials, uint32_t nblocks, uint64_t n, krex_check_result *out,
                              hipStream_t s)
{
    return launch(k_check_final, dim3(1), dim3(kFinalThreads), s, partials, nblocks, n, out);
}

// Blocks per compute unit of the check's one resident round when both
// operands stream from memory. Every block sweeps its own region, and on
// gfx950 the fewer regions are read at once, the closer two streams come to
// the read rate of a dispatch-ordered grid: 2 blocks per CU took fp16 x fp16
// (1 GiB) from 169-170 to 164-165 us, fp32 x fp32 (512 MiB) from 86-87 to
// 82-86 us and the 16.8M-element bf16 x fp32 check from 23.7 to 22.2 us per
// call, against the 5-6 blocks occupancy allows (1 per CU: 218 us). Pairs
// with an fp8 operand (16 elements per chunk) issue more per byte and keep
// the occupancy limit (fp8 x fp8 94 us at 5 per CU, 96-102 us at 2).
template <int DA, int DB>
static constexpr uint32_t check_blocks_per_cu()
{
    return chunk_elems<DA, DB>() == 16 ? 0u : 2u;
}

template <int DA, int DB, int D>
static hipError_t check_ab_d(const void *a, const void *b, uint64_t n, float rtol, float atol, void *scratch,
                             krex_check_result *out, hipStream_t s)
{
    constexpr int E = chunk_elems<DA, DB>();
    const bool vec = (((uintptr_t)a & 15u) == 0 && ((uintptr_t)b & 15u) == 0);
    static uint32_t cache_vec[64] = {}, cache_el[64] = {};
    const uint64_t resident = vec ? resident_blocks((const void *)k_check<DA, DB, true, D>, cache_vec,
                                                    check_blocks_per_cu<DA, DB>())
                                  : resident_blocks((const void *)k_check<DA, DB, false, 2>, cache_el);
    uint32_t U, G;
    check_grid(n / E, resident, &U, &G);
    CheckPartial *parts = (CheckPartial *)scratch;
    hipError_t e;
    if (vec)
        e = launch(k_check<DA, DB, true, D>, dim3(G), dim3(kThreads), s, (const uint8_t *)a, (const uint8_t *)b, n,
                   rtol, atol, parts, U);
    else
        e = launch(k_check<DA, DB, false, 2>, dim3(G), dim3(kThreads), s, (const uint8_t *)a, (const uint8_t *)b, n,
                   rtol, atol, parts, U);
    if (e != hipSuccess) return e;
    return launch_check_final(parts, G, n, out, s);
}

// Depth of the load ring: a third buffer in flight pays for pairs of one-
// and two-byte operands (one 16-byte vector of each per chunk; measured on
// gfx950 with non-temporal loads: fp16 x fp16 -5%, fp8 x fp8 -13%), not for
// pairs with a four-byte operand, whose extra registers only lower
// occupancy.
template <int DA, int DB>
static constexpr int check_depth()
{
    return (dtype_traits<DA>::size == dtype_traits<DB>::size && dtype_traits<DA>::size <= 2) ? 3 : 2;
}

template <int DA, int DB>
static hipError_t check_ab(const void *a, const void *b, uint64_t n, float rtol, float atol, void *scratch,
                           krex_check_result *out, hipStream_t s)
{
    return check_ab_d<DA, DB, check_depth<DA, DB>()>(a, b, n, rtol, atol, scratch, out, s);
}

template <int DA>
static hipError_t check_a(const void *a, int dtb, const void *b, uint64_t n, float rtol, float atol, void *scratch,
                          krex_check_result *out, hipStream_t s)
{
    switch (dtb) {
    case F32: return check_ab<DA, F32>(a, b, n, rtol, atol, scratch, out, s);
    case BF16: return check_ab<DA, BF16>(a, b, n, rtol, atol, scratch, out, s);
    case F16: return check_ab<DA, F16>(a, b, n, rtol, atol, scratch, out, s);
    default: return check_ab<DA, F8>(a, b, n, rtol, atol, scratch, out, s);
    }
}

hipError_t launch_check(const void *a, int dta, const void *b, int dtb, uint64_t n, float rtol, float atol,
                        void *scratch, krex_check_result *out, hipStream_t s)
{
    if (n == 0)
        return launch(k_check_final, dim3(1), dim3(kFinalThreads), s, (const CheckPartial *)scratch, 0u, n, out);
    switch (dta) {
    case F32: return check_a<F32>(a, dtb, b, n, rtol, atol, scratch, out, s);
    case BF16: return check_a<BF16>(a, dtb, b, n, rtol, atol, scratch, out, s);
    case F16: return check_a<F16>(a, dtb, b, n, rtol, atol, scratch, out, s);
    default: return check_a<F8>(a, dtb, b, n, rtol, atol, scratch, out, s);
    }
}

// ---------------------------------------------------------------------- flush

// One 16-byte store per thread, blocks in address order. On gfx950 this
// dispatch-ordered shape streams writes at ~85% of HBM peak, well above
// persistent grid-stride loops (whose 2048 concurrently active blocks spread
// each wave of stores across the whole buffer).
//
// The stores (store16_alloc, raw buffer stores) carry the system-scope
// coherence bits (sc0 sc1): they write through L2 without allocating there,
// which streams ~2% faster, and still
// allocate in the Infinity Cache, whose contents the flush exists to evict
// (a 64 MiB working set re-read after a 1 GiB flush runs at HBM speed, not
// at Infinity Cache speed). L2 needs no eviction: the runtime writes back and
// invalidates L2 at kernel boundaries, so a working set read by one launch
// misses L2 in the next one with or without a flush (measured with the L2
// hit counters). Non-temporal stores would leave the Infinity Cache intact.
__global__ __launch_bounds__(kThreads) void k_flush(uint4 *buf, uint64_t nvec, uint32_t pattern)
{
    const uint64_t i = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < nvec) store16_alloc(buf + (uint64_t)blockIdx.x * kThreads, 16u * threadIdx.x,
                                make_uint4(pattern, pattern, pattern, pattern));
}

hipError_t launch_flush(void *buf, uint64_t bytes, uint32_t pattern, hipStream_t s)
{
    // A dispatch covers at most 2^32 - 1 work-items; split larger buffers.
    const uint64_t per_launch = (1ull << 31);   // vectors (32 GiB) per dispatch
    uint4 *p = (uint4 *)buf;
    uint64_t nvec = bytes / 16;
    while (nvec > 0) {
        const uint64_t m = nvec < per_launch ? nvec : per_launch;
        const uint32_t grid = (uint32_t)((m + kThreads - 1) / kThreads);
        const hipError_t e = launch(k_flush, dim3(grid), dim3(kThreads), s, p, m, pattern);
        if (e != hipSuccess) return e;
        p += m;
        nvec -= m;
    }
    return hipSuccess;
}

// ---------------------------------------------------------------------- probe

// clocks (optional): per wave w = 4 blockIdx.x + wave, eight 64-bit words
// at clocks + 8 w: the shader-clock cycle counter (s_memtime) and the
// constant-rate real-time counter (s_memrealtime, 100 MHz) read when the
// wave starts and when its chains are done, the HW_ID register (CU, SIMD,
// shader array / engine) and the XCC_ID register. The wave's
// effective shader clock is its cycle delta over its real-time delta. Only
// the wave's first lane stores, with an ordinary vector store; the sink's
// value does not depend on it.
__global__ __launch_bounds__(kThreads) void k_probe(uint64_t iters, float *sink, uint64_t *clocks)
{
    const uint32_t g = blockIdx.x * kThreads + threadIdx.x;
    uint64_t c0 = 0, r0 = 0;
    if (clocks) {
        c0 = __builtin_amdgcn_s_memtime();
        r0 = __builtin_amdgcn_s_memrealtime();
    }
    float x[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = (float)(g * 8u + (uint32_t)c) * 0x1p-19f;
    const float a = 1.0f - 0x1p-10f;
    const float bb = 0x1p-10f;
    for (uint64_t it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < 8; ++c) x[c] = __builtin_fmaf(x[c], a, bb);
    }
    float s = x[0];
#pragma unroll
    for (int c = 1; c < 8; ++c) s = s + x[c];
    if (clocks) {
        // the end stamps depend on s, so they are read after the chains
        __asm__ volatile("" ::"v"(s));
        const uint64_t c1 = __builtin_amdgcn_s_memtime();
        const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
        uint32_t hw, xcc;
        __asm__ volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
        __asm__ volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
        if ((threadIdx.x & 63u) == 0) {
            uint4 *o = reinterpret_cast<uint4 *>(clocks + 8u * (blockIdx.x * (kThreads / 64) + threadIdx.x / 64));
            o[0] = make_uint4((uint32_t)c0, (uint32_t)(c0 >> 32), (uint32_t)c1, (uint32_t)(c1 >> 32));
            o[1] = make_uint4((uint32_t)r0, (uint32_t)(r0 >> 32), (uint32_t)r1, (uint32_t)(r1 >> 32));
            o[2] = make_uint4(hw, 0u, xcc, 0u);
            o[3] = make_uint4(0u, 0u, 0u, 0u);
        }
    }
    sink[g] = s;
}

hipError_t launch_probe(uint64_t iters, float *sink, uint64_t *clocks, hipStream_t s)
{
    return launch(k_probe, dim3(kProbeBlocks), dim3(kThreads), s, iters, sink, clocks);
}

// ------------------------------------------------------------------- fixture

__global__ __launch_bounds__(kThreads) void k_sgemm(uint32_t M, uint32_t N, uint32_t K, const float *A,
                                                    const float *B, float *C)
{
    const uint64_t idx = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
    if (idx >= (uint64_t)M * N) return;
    const uint32_t i = (uint32_t)(idx / N), j = (uint32_t)(idx % N);
    float acc = 0.0f;
    for (uint32_t k = 0; k < K; ++k) acc = __builtin_fmaf(A[(uint64_t)i * K + k], B[(uint64_t)k * N + j], acc);
    C[idx] = acc;
}

hipError_t launch_sgemm(uint32_t M, uint32_t N, uint32_t K, const float *A, const float *B, float *C,
                        hipStream_t s)
{
    const uint64_t total = (uint64_t)M * N;
    if (total == 0) return hipSuccess;
    const uint32_t grid = (uint32_t)((total + kThreads - 1) / kThreads);
    return launch(k_sgemm, dim3(grid), dim3(kThreads), s, M, N, K, A, B, C);
}

}  // namespace krex
