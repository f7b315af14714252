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
//             (Section 6.3, Eq. 1).
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

#include <tuple>
#include <utility>

#include "krex_device.hpp"
#include "launch.hpp"

namespace krex {

// hipLaunchKernel with the kernel's own parameter types, returning the
// launch status directly instead of through the sticky last-error state.
template <typename... KArgs, typename... Actual>
static hipError_t launch(void (*kern)(KArgs...), dim3 grid, dim3 block, hipStream_t s, Actual &&...a)
{
    std::tuple<KArgs...> args(std::forward<Actual>(a)...);
    void *argv[sizeof...(KArgs)];
    std::apply([&](auto &...x) {
        int i = 0;
        ((argv[i++] = (void *)&x), ...);
    }, args);
    return hipLaunchKernel((const void *)kern, grid, block, argv, 0, s);
}

static constexpr int kThreads = 256;

template <int DT> struct group_of { static constexpr int G = 4 / dtype_traits<DT>::size; };

// ------------------------------------------------------------------ generation

struct GenParams {
    uint8_t *dst;
    uint64_t n;
    uint64_t offset;
    uint32_t k0, k1;
    float p0, p1;      // uniform: lo and fl(hi - lo); normal: mean and std
    float c;           // uniform with a power-of-two range: range 2^-24
    int pow2;          // uniform range is a power of two (c normal)
    uint64_t b0;       // first Philox block
    uint64_t ngroups;  // groups of G blocks
    uint32_t U;        // groups per thread, block-contiguous
    int vec;           // offset % 4 == 0 and dst 16-byte aligned
};

// POW2: uniform with a power-of-two range (the fused transform; P.c).
template <int DT, int DIST, bool POW2>
__global__ __launch_bounds__(kThreads) void k_gen(GenParams P)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int G = group_of<DT>::G;
    for (uint32_t u = 0; u < P.U; ++u) {
        const uint64_t g = ((uint64_t)blockIdx.x * P.U + u) * kThreads + threadIdx.x;
        if (g >= P.ngroups) break;
        const uint64_t bfirst = P.b0 + g * G;
        union {
            uint4 v;
            uint32_t w[4];
            T s[4 * G];
        } pk;
        if constexpr (DT == U32) {
            const words4 w = philox_block(bfirst, P.k0, P.k1);
#pragma unroll
            for (int l = 0; l < 4; ++l) pk.w[l] = w.v[l];
        } else {
            words4 wb[G];
#pragma unroll
            for (int i = 0; i < G; ++i) wb[i] = philox_block(bfirst + i, P.k0, P.k1);
            float v[4 * G];
#pragma unroll
            for (int i = 0; i < G; ++i) transform4<DIST, POW2>(wb[i], P.p0, POW2 ? P.c : P.p1, v + 4 * i);
            pack_narrow<DT, DIST == BITCAST>(v, pk.w);
        }
        const uint64_t j0 = 4 * bfirst - P.offset;
        if (P.vec && j0 + 4 * G <= P.n) {
            // vec: offset % 4 == 0; the block's first group starts at element
            // jb (uniform across the block) and lane t's 16 bytes at jb + 4 G t
            const uint64_t gb = ((uint64_t)blockIdx.x * P.U + u) * kThreads;
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
// units [b 256 U, (b + 1) 256 U). One unit per thread (a one-shot grid in
// address order) streams HBM fastest on gfx950; U grows only to keep a
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

static uint32_t tune_env(const char *name, uint32_t dflt)
{
    const char *e = getenv(name);
    if (!e) return dflt;
    const unsigned long v = strtoul(e, nullptr, 10);
    return v ? (uint32_t)v : dflt;
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

template <int DT, int DIST>
static hipError_t gen_dt_dist(GenParams P, hipStream_t s)
{
    static const uint32_t u_pref = tune_env("KREX_GEN_U", 1);
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
    P.k0 = (uint32_t)seed;
    P.k1 = (uint32_t)(seed >> 32);
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
// The narrow-dtype generator that spends W bits of the word stream per
// element (W = 16 for bf16 / fp16 and fp8 normal, 8 for fp8 uniform and
// bitcast): field q is bits (q mod K) W .. of word q / K, K = 32 / W, low
// bits first; element j uses field offset + j. One thread unit is one
// 16-byte output vector, E elements = E fields = GB Philox blocks, so every
// narrow dtype needs one block per 16 bytes (two for fp8 normal) instead of
// one word per element. Uniform maps field f through the uniform transform
// of the word f << (32 - W); normal runs Box-Muller on the two 16-bit fields
// of one word widened to the top half (low field -> cosine, high field ->
// sine); bitcast stores the fields, i.e. the words' bytes.

template <int DT, int DIST>
struct packed_of {
    static constexpr int W = (DT == F8 && DIST != NORMAL) ? 8 : 16;
    static constexpr int E = 16 / dtype_traits<DT>::size;
    static constexpr int GB = E * W / 128;
};

struct PackedParams {
    uint8_t *dst;
    uint64_t n;
    uint64_t offset;   // in fields
    uint32_t k0, k1;
    float p0, p1;      // uniform: lo and fl(hi - lo); normal: mean and std
    float rs;          // uniform: fl(hi - lo) 2^-W when that is exact
    int umode;         // uniform: UM_WORD, UM_SCALED or UM_FUSED
    uint64_t u0;       // first unit (units are E fields, E-aligned)
    uint64_t nunits;
    uint32_t U;        // units per thread, block-contiguous
    int vec;           // offset % E == 0 and dst 16-byte aligned
};

// Uniform transform of a W-bit field f: UM_WORD applies the word-stream
// transform to f << (32 - W); UM_SCALED when rs = fl(hi - lo) 2^-W is exact
// (u = f 2^-W exactly, so rs f is the same real number as fl(hi - lo) u and
// rounds the same: one conversion, one multiply, one add); UM_FUSED when rs f
// is exact as well, so lo + rs f has one rounding: one fused multiply-add.
enum : int { UM_WORD = 0, UM_SCALED = 1, UM_FUSED = 2 };

template <int DT, int DIST, int UM>
__global__ __launch_bounds__(kThreads) void k_gen_packed(PackedParams P)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int W = packed_of<DT, DIST>::W;
    constexpr int K = 32 / W;
    constexpr int E = packed_of<DT, DIST>::E;
    constexpr int GB = packed_of<DT, DIST>::GB;
    constexpr uint32_t kMask = (1u << W) - 1u;
    for (uint32_t u = 0; u < P.U; ++u) {
        const uint64_t g = ((uint64_t)blockIdx.x * P.U + u) * kThreads + threadIdx.x;
        if (g >= P.nunits) break;
        const uint64_t unit = P.u0 + g;
        uint32_t wv[4 * GB];
#pragma unroll
        for (int i = 0; i < GB; ++i) {
            const words4 w = philox_block(unit * GB + i, P.k0, P.k1);
#pragma unroll
            for (int l = 0; l < 4; ++l) wv[4 * i + l] = w.v[l];
        }
        union {
            uint4 v;
            uint32_t w[4];
            T s[E];
        } pk;
        if constexpr (DIST == BITCAST) {
            static_assert(GB == 1, "bitcast units are one block");
#pragma unroll
            for (int l = 0; l < 4; ++l) pk.w[l] = wv[l];
        } else if constexpr (DIST == UNIFORM) {
            float v[E];
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const uint32_t f = (wv[e / K] >> ((e % K) * W)) & kMask;
                if constexpr (UM == UM_FUSED) {
                    v[e] = __builtin_fmaf(P.rs, (float)f, P.p0);
                } else if constexpr (UM == UM_SCALED) {
                    const float t = P.rs * (float)f;
                    v[e] = P.p0 + t;
                } else {
                    v[e] = uniform_f32(f << (32 - W), P.p0, P.p1);
                }
            }
            if constexpr (DT == F8) {
                // Two values per conversion (bytes 0-1, then 2-3 of the word).
#pragma unroll
                for (int i = 0; i < E / 4; ++i) {
                    uint32_t wd = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(v[4 * i], v[4 * i + 1], 0, false);
                    wd = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(v[4 * i + 2], v[4 * i + 3], (int)wd, true);
                    pk.w[i] = wd;
                }
            } else {
                pack_narrow<DT, false>(v, pk.w);
            }
        } else {
            static_assert(W == 16 && E == 8 * GB, "normal fields are 16 bits, two per word");
            float v[E];
#pragma unroll
            for (int i = 0; i < 4 * GB; ++i) {
                float z0, z1;
                normal_pair(wv[i] << 16, wv[i] & 0xFFFF0000u, z0, z1);
                const float s0 = P.p1 * z0;
                const float s1 = P.p1 * z1;
                v[2 * i] = P.p0 + s0;
                v[2 * i + 1] = P.p0 + s1;
            }
            pack_narrow<DT, false>(v, pk.w);
        }
        const uint64_t q0 = unit * (uint64_t)E;
        if (P.vec && q0 >= P.offset && q0 - P.offset + E <= P.n) {
            const uint64_t gb = ((uint64_t)blockIdx.x * P.U + u) * kThreads;
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

template <int DT, int DIST>
static hipError_t gen_packed_dt_dist(PackedParams P, hipStream_t s)
{
    constexpr int E = packed_of<DT, DIST>::E;
    constexpr int W = packed_of<DT, DIST>::W;
    P.umode = UM_WORD;
    P.rs = 0.0f;
    if (DIST == UNIFORM) {
        P.rs = ldexpf(P.p1, -W);
        float c;
        if (ldexpf(P.rs, W) == P.p1) P.umode = exact_scale(P.p1, W, &c) ? UM_FUSED : UM_SCALED;
    }
    P.u0 = P.offset / E;
    P.nunits = (P.offset + (P.n - 1)) / E - P.u0 + 1;
    P.vec = (P.offset % E == 0 && ((uintptr_t)P.dst & 15u) == 0) ? 1 : 0;
    uint32_t grid;
    shape(P.nunits, 1, &P.U, &grid);
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
    P.k0 = (uint32_t)seed;
    P.k1 = (uint32_t)(seed >> 32);
    P.p0 = p0;
    P.p1 = (dist == UNIFORM) ? (p1 - p0) : p1;
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
    uint32_t k0, k1;
    uint64_t T;        // threshold in [0, 2^32]
    float delta;
    uint64_t b0;
    uint64_t ngroups;
    uint32_t U;
    int vec;
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

template <int DT, int MODE>
__global__ __launch_bounds__(kThreads) void k_inject(InjectParams P)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int G = group_of<DT>::G;
    for (uint32_t u = 0; u < P.U; ++u) {
        const uint64_t g = ((uint64_t)blockIdx.x * P.U + u) * kThreads + threadIdx.x;
        if (g >= P.ngroups) break;
        const uint64_t bfirst = P.b0 + g * G;
        const uint64_t j0 = 4 * bfirst - P.moff;
        if (P.vec && j0 + 4 * G <= P.n) {
            union {
                uint4 v;
                T s[4 * G];
            } pk;
            pk.v = load16_stream(P.x + j0 * ES);
#pragma unroll
            for (int i = 0; i < G; ++i) {
                const words4 w = philox_block(bfirst + i, P.k0, P.k1);
#pragma unroll
                for (int l = 0; l < 4; ++l)
                    if ((uint64_t)w.v[l] < P.T) pk.s[4 * i + l] = perturb<DT, MODE>(pk.s[4 * i + l], P.delta);
            }
            const uint64_t gb = ((uint64_t)blockIdx.x * P.U + u) * kThreads;
            const uint64_t jb = 4 * (P.b0 + gb * G) - P.moff;
            store16_stream(P.y + jb * ES, 16u * threadIdx.x, pk.v);
        } else {
            for (int i = 0; i < G; ++i) {
                const words4 w = philox_block(bfirst + i, P.k0, P.k1);
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
    static const uint32_t u_pref = tune_env("KREX_INJECT_U", 1);
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
    P.k0 = (uint32_t)mseed;
    P.k1 = (uint32_t)(mseed >> 32);
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
    uint32_t m0, m1;   // mask key
    uint64_t mb0;      // first mask block: mask offset / 4
    uint64_t T;        // threshold in [0, 2^32]
    float delta;
};

template <int DT, int DIST, bool POW2, int MODE>
__global__ __launch_bounds__(kThreads) void k_gen_inject(GenInjectParams Q)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int G = group_of<DT>::G;
    const GenParams &P = Q.g;
    for (uint32_t u = 0; u < P.U; ++u) {
        const uint64_t g = ((uint64_t)blockIdx.x * P.U + u) * kThreads + threadIdx.x;
        if (g >= P.ngroups) break;
        const uint64_t bfirst = P.b0 + g * G;
        const uint64_t mfirst = Q.mb0 + g * G;
        union {
            uint4 v;
            uint32_t w[4];
            T s[4 * G];
        } px, py;
        float v[4 * G];
#pragma unroll
        for (int i = 0; i < G; ++i)
            transform4<DIST, POW2>(philox_block(bfirst + i, P.k0, P.k1), P.p0, POW2 ? P.c : P.p1, v + 4 * i);
        pack_narrow<DT, DIST == BITCAST>(v, px.w);
        py.v = px.v;
#pragma unroll
        for (int i = 0; i < G; ++i) {
            const words4 m = philox_block(mfirst + i, Q.m0, Q.m1);
#pragma unroll
            for (int l = 0; l < 4; ++l)
                if ((uint64_t)m.v[l] < Q.T) py.s[4 * i + l] = perturb<DT, MODE>(py.s[4 * i + l], Q.delta);
        }
        const uint64_t j0 = 4 * bfirst - P.offset;
        if (P.vec && j0 + 4 * G <= P.n) {
            const uint64_t gb = ((uint64_t)blockIdx.x * P.U + u) * kThreads;
            const uint64_t jb = 4 * (P.b0 + gb * G) - P.offset;
            store16_stream(P.dst + jb * ES, 16u * threadIdx.x, px.v);
            store16_stream(Q.y + jb * ES, 16u * threadIdx.x, py.v);
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
    uint32_t grid;
    shape(Q.g.ngroups, 1, &Q.g.U, &grid);
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
    Q.m0 = (uint32_t)mseed;
    Q.m1 = (uint32_t)(mseed >> 32);
    Q.mb0 = moff >> 2;
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
// Two launches and no atomics. k_check: block b owns chunks
// [b 256 U, (b + 1) 256 U) of E elements (one 16-byte vector of the
// narrower operand); thread t takes chunk b 256 U + u 256 + t for u < U, so
// every step of a wave reads contiguous memory. Per element the verdict is
// branch-free; mismatch and NaN counts are wave ballots summed on the scalar
// unit; the per-lane maximum |a - b| is tracked per chunk, and the first
// index of the wave's maximum is recovered at the end by its winning lane
// re-reading that one chunk. Each block writes one
// 32-byte partial with plain stores; k_check_final reduces the partials and
// writes the result record.
//
// max_rel without a division per element: a lane keeps the pair (d*, b*)
// with the largest exact ratio d / |b| among its elements with finite
// positive d, comparing d b* > d* |b| in fp64, where the products of two
// fp32 values are exact. One correctly rounded fp32 division per lane then
// gives fl(max d / |b|), which equals max fl(d / |b|) because rounding is
// monotone. Infinite d (an infinite operand, or overflow) enters as the pair
// (inf, 0), ratio +inf.
//
// (A per-block atomic finish costs ~12 ns per same-address device atomic on
// this GPU, serialised: 2048 blocks x 5 atomics is ~130 us, longer than
// reading 100 MB.)

static constexpr uint64_t kIdxMask = (1ull << 33) - 1;   // n < 2^33
static constexpr int kMaxCheckBlocks = 4096;
static constexpr int kFinalThreads = 256;

struct CheckPartial {
    uint64_t mism;
    uint64_t nan;
    uint64_t key;       // (bits(max d) << 33) | (kIdxMask - index); 0 = no NaN-free element
    uint32_t rel_bits;  // max rel (non-negative fp32 bits)
    uint32_t pad;
};

static_assert(sizeof(CheckPartial) == 32, "partial layout");

size_t check_scratch_bytes() { return (size_t)kMaxCheckBlocks * sizeof(CheckPartial); }

struct LaneAcc {
    uint32_t wmism, wnan;   // wave totals (exact in the wave's first lane)
    float rd, rb;           // element with the largest ratio d / |b| (rb = 0: +inf)
};

__device__ __forceinline__ uint32_t popc(uint64_t m) { return (uint32_t)__builtin_popcountll(m); }

// Every d > 0 has d / |b| >= 2^-26 (fp32 operands that differ are at least
// one spacing of the nearer one apart, or |b| / 2 when far apart; b = 0 gives
// +inf), so 2^-32 is a lower bound of any ratio that can raise a maximum
// above its initial 0.
static constexpr float kRatioFloor = 0x1p-32f;

// Exact ratio update of one element: the pair (d, bn) replaces (rd, rb) when
// d / bn > rd / rb, compared as d rb > rd bn in fp64 (products of two fp32
// values are exact there). An infinite d enters as (inf, 0), ratio +inf, which no
// later pair exceeds; d = 0 and NaN never compare greater.
__device__ __forceinline__ void ratio_update(float A, float B, LaneAcc &acc)
{
    const float d0 = __builtin_fabsf(A - B);
    const bool dinf = d0 == __builtin_inff();
    const float bn = dinf ? 0.0f : __builtin_fabsf(B);
    const bool greater = (double)d0 * (double)acc.rb > (double)acc.rd * (double)bn;
    acc.rd = greater ? d0 : acc.rd;
    acc.rb = greater ? bn : acc.rb;
}

// Counts and verdict of one element, accumulated as wave ballots of plain
// comparisons (each lowers to one compare writing a lane mask). The element
// mismatches when a != b (unordered included) and not d0 <= min(thr,
// FLT_MAX): d0 is +inf exactly when the operands differ and one is infinite,
// or their difference overflows, and is then never close; clamping the
// threshold to the largest float excludes it in the same comparison (a NaN
// threshold, 0 x inf, arises only with |b| = inf, where d0 is inf or NaN and
// the verdict is a mismatch either way). CLAMP = false when neither operand
// type has an infinity and their difference cannot overflow (fp8 e4m3fn
// pairs: |a|, |b| <= 448): d0 is then never +inf and the threshold never
// NaN, so the clamp cannot change a verdict.
template <bool CLAMP = true>
__device__ __forceinline__ uint64_t count_elem(float A, float B, float d0, float ab, float rtol, float atol,
                                               LaneAcc &acc)
{
    const float rt = rtol * ab;
    const float thr = CLAMP ? __builtin_fminf(atol + rt, 0x1.fffffep127f) : atol + rt;
    const uint64_t ne = __ballot(A != B);
    const uint64_t far = __ballot(!(d0 <= thr));
    const uint64_t unord = __ballot(__builtin_isunordered(A, B));
    acc.wmism += popc(ne & far);
    acc.wnan += popc(unord);
    return ne & ~unord;             // lanes whose operands are ordered and differ
}

// One element with its exact ratio update; returns d (0 when equal, NaN when
// unordered) for the |a - b| maximum. Used for the n mod E tail.
__device__ __forceinline__ float check_elem(float A, float B, float rtol, float atol, LaneAcc &acc)
{
    const float d0 = __builtin_fabsf(A - B);
    count_elem(A, B, d0, __builtin_fabsf(B), rtol, atol, acc);
    ratio_update(A, B, acc);
    return (A == B) ? 0.0f : d0;
}

// The same d, for re-reading the best chunk.
__device__ __forceinline__ float elem_d(float A, float B)
{
    return (A == B) ? 0.0f : __builtin_fabsf(A - B);
}

template <int DA, int DB, bool VEC>
struct ChunkIO {
    using TA = typename dtype_traits<DA>::storage;
    using TB = typename dtype_traits<DB>::storage;
    static constexpr int SA = dtype_traits<DA>::size;
    static constexpr int SB = dtype_traits<DB>::size;
    static constexpr int E = 16 / (SA < SB ? SA : SB);
    static constexpr int VA = E * SA / 16;
    static constexpr int VB = E * SB / 16;

    // Raw bytes of one chunk: 16-byte vectors of each operand.
    struct Raw {
        union {
            uint4 v[VA];
            uint32_t w[4 * VA];
            TA s[E];
        } a;
        union {
            uint4 v[VB];
            uint32_t w[4 * VB];
            TB s[E];
        } b;
    };

    __device__ __forceinline__ static void load_raw(const uint8_t *a, const uint8_t *b, uint64_t c, Raw &r)
    {
#pragma unroll
        for (int i = 0; i < VA; ++i) r.a.v[i] = load16_stream(a + (c * VA + i) * 16);
#pragma unroll
        for (int i = 0; i < VB; ++i) r.b.v[i] = load16_stream(b + (c * VB + i) * 16);
    }

    // fp8 elements are converted two at a time straight from their 32-bit
    // words (the packed converter's half-word select: no shifts or masks).
    template <int DT, int NW>
    __device__ __forceinline__ static void widen_words(const uint32_t (&w)[NW],
                                                       const typename dtype_traits<DT>::storage (&s)[E], float (&X)[E])
    {
        if constexpr (DT == F8) {
            typedef float f2 __attribute__((ext_vector_type(2)));
#pragma unroll
            for (int i = 0; i < NW; ++i) {
                const f2 lo = __builtin_amdgcn_cvt_pk_f32_fp8((int)w[i], false);
                const f2 hi = __builtin_amdgcn_cvt_pk_f32_fp8((int)w[i], true);
                X[4 * i + 0] = lo.x;
                X[4 * i + 1] = lo.y;
                X[4 * i + 2] = hi.x;
                X[4 * i + 3] = hi.y;
            }
        } else {
#pragma unroll
            for (int e = 0; e < E; ++e) X[e] = widen<DT>(s[e]);
        }
    }

    __device__ __forceinline__ static void widen_raw(const Raw &r, float (&A)[E], float (&B)[E])
    {
        widen_words<DA, 4 * VA>(r.a.w, r.a.s, A);
        widen_words<DB, 4 * VB>(r.b.w, r.b.s, B);
    }

    __device__ __forceinline__ static void load(const uint8_t *a, const uint8_t *b, uint64_t c, float (&A)[E],
                                                float (&B)[E])
    {
        if constexpr (VEC) {
            Raw r;
            load_raw(a, b, c, r);
            widen_raw(r, A, B);
        } else {
#pragma unroll
            for (int e = 0; e < E; ++e) {
                A[e] = widen<DA>(reinterpret_cast<const TA *>(a)[c * E + e]);
                B[e] = widen<DB>(reinterpret_cast<const TB *>(b)[c * E + e]);
            }
        }
    }
};

// max_rel with a wave-wide filter: R (wave-uniform) is a lower bound of the
// largest exact ratio the wave holds. An element whose ratio is at least R
// has d >= R |b| exactly, hence d >= fl(R |b|) (rounding is monotone and d
// is a float); so an element with d < fl(R |b|) cannot raise the maximum and
// skips the exact fp64 update. Only when some lane of the wave has a
// candidate does the wave run the exact updates for the chunk and raise R to
// the wave maximum of one-ulp-lowered fl(rd / rb). Only ordered, differing
// elements are candidates; a NaN product (inf x 0) counts as one. Called by
// every lane of the wave (the shuffles read
// all lanes) with the wave's candidate mask; lanes without a chunk pass
// valid = false.
template <int E>
struct RatioFilter {
    float R = kRatioFloor;

    __device__ __forceinline__ void chunk(const float (&A)[E], const float (&B)[E], bool valid, uint64_t cand,
                                          LaneAcc &acc)
    {
        if (cand == 0) return;                  // wave-uniform
        if (valid) {
#pragma unroll
            for (int e = 0; e < E; ++e) ratio_update(A[e], B[e], acc);
        }
        const float q = acc.rd / acc.rb;        // 0, a positive float, or +inf
        float lo = (q > 0.0f && q < __builtin_inff()) ? __uint_as_float(__float_as_uint(q) - 1u) : q;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) lo = __builtin_fmaxf(lo, __shfl_xor(lo, off, 64));
        lo = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(lo)));
        R = __builtin_fmaxf(R, lo);
    }
};

template <int DA, int DB, bool VEC, int D>
__global__ __launch_bounds__(kThreads) void k_check(const uint8_t *a, const uint8_t *b, uint64_t n, float rtol,
                                                    float atol, CheckPartial *partials, uint32_t U)
{
    using IO = ChunkIO<DA, DB, VEC>;
    constexpr int E = IO::E;
    const uint32_t t = threadIdx.x;
    const uint64_t nchunks = n / E;
    const uint64_t base = (uint64_t)blockIdx.x * kThreads * U;
    LaneAcc acc{0u, 0u, 0.0f, 1.0f};
    RatioFilter<E> rf;
    float best_d = -1.0f;               // largest non-NaN d seen by this lane
    uint32_t best_c = 0;                // its chunk
    // Counts and |a - b| maximum of one chunk; returns the lanes of the wave
    // whose chunk has a max_rel candidate.
    auto process = [&](const float (&A)[E], const float (&B)[E], uint64_t c) -> uint64_t {
        float cmax = -1.0f;             // NaN d (unordered) is ignored by the maximum
        uint64_t cand = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const float d0 = __builtin_fabsf(A[e] - B[e]);
            const float ab = __builtin_fabsf(B[e]);
            const uint64_t differ = count_elem<!(DA == F8 && DB == F8)>(A[e], B[e], d0, ab, rtol, atol, acc);
            // Equal operands (ratio 0, or 0/0) and unordered ones (NaN d)
            // never raise the maximum: only ordered, differing elements are
            // candidates (otherwise every zero reference would be one).
            cand |= __ballot(!(d0 < rf.R * ab)) & differ;
            cmax = __builtin_fmaxf(cmax, (A[e] == B[e]) ? 0.0f : d0);
        }
        if (cmax > best_d) {
            best_d = cmax;
            best_c = (uint32_t)c;
        }
        return cand;
    };
    if constexpr (VEC) {
        // Software pipeline over a ring of D chunk buffers: the loads of the
        // next D - 1 chunks are in flight while the current one is
        // evaluated. Every load is unconditional (a lane with nothing left
        // re-reads the last chunk, which stays in L2), so the compiler's
        // memory-counter waits stay exact: an evaluation waits for its own
        // buffer only, never for the loads issued after it. A lane's chunks
        // only grow with j, so the first lane of a wave holds a chunk
        // whenever any lane does.
        if (nchunks != 0) {
            const uint64_t last = nchunks - 1;
            auto cj = [&](uint32_t j) { return base + t + (uint64_t)j * kThreads; };
            auto hj = [&](uint32_t j) { return j < U && cj(j) < nchunks; };
            typename IO::Raw r[D];
#pragma unroll
            for (int k = 0; k < D - 1; ++k) IO::load_raw(a, b, hj(k) ? cj(k) : last, r[k]);
            for (uint32_t u = 0; u < U; u += D) {
#pragma unroll
                for (int k = 0; k < D; ++k) {
                    const uint32_t jn = u + k + D - 1;
                    IO::load_raw(a, b, hj(jn) ? cj(jn) : last, r[(k + D - 1) % D]);
                    const uint32_t j = u + k;
                    const bool h = hj(j);
                    float A[E], B[E];   // read only where h holds
                    uint64_t cand = 0;
                    if (h) {
                        IO::widen_raw(r[k], A, B);
                        cand = process(A, B, cj(j));
                    }
                    rf.chunk(A, B, h, cand, acc);
                }
            }
        }
    } else {
        for (uint32_t u = 0; u < U; ++u) {
            const uint64_t c = base + (uint64_t)u * kThreads + t;
            const bool have = c < nchunks;
            float A[E], B[E];           // read only where have holds
            uint64_t cand = 0;
            if (have) {
                IO::load(a, b, c, A, B);
                cand = process(A, B, c);
            }
            rf.chunk(A, B, have, cand, acc);
        }
    }
    // The lane's candidate for the |a - b| maximum: best_d at position pos,
    // the first index of its best chunk (the chunk holds the lane's first
    // element attaining best_d), or a tail index.
    uint64_t pos = (uint64_t)best_c * E;
    bool in_chunk = true;
    // The n mod E tail: the first block's first lanes, one element each.
    const uint64_t tail0 = nchunks * E;
    if (blockIdx.x == 0 && tail0 + t < n) {
        const uint64_t i = tail0 + t;
        const float A = widen<DA>(reinterpret_cast<const typename IO::TA *>(a)[i]);
        const float B = widen<DB>(reinterpret_cast<const typename IO::TB *>(b)[i]);
        const float d = check_elem(A, B, rtol, atol, acc);
        if (d > best_d) {     // tail indices exceed every chunk index
            best_d = d;
            pos = i;
            in_chunk = false;
        }
    }
    // Only the wave's winner, the largest best_d at the lowest position,
    // re-reads its chunk for the exact index (one chunk per wave, not per
    // lane: a chunk's two operands span two 128-byte lines). Chunks are
    // disjoint and ordered by position, so no other lane of the wave holds
    // an element attaining best_d below the winner's chunk, and the exact
    // key stays the wave's largest.
    uint64_t key = best_d >= 0.0f ? (((uint64_t)__float_as_uint(best_d) << 33) | (kIdxMask - pos)) : 0ull;
    uint64_t wkey = key;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint64_t k2 = __shfl_xor((unsigned long long)wkey, off, 64);
        wkey = k2 > wkey ? k2 : wkey;
    }
    if (key != 0 && key == wkey && in_chunk) {
        float A[E], B[E];
        IO::load(a, b, best_c, A, B);
        uint64_t best_i = pos;
        for (int e = E - 1; e >= 0; --e)
            if (elem_d(A[e], B[e]) == best_d) best_i = pos + (uint64_t)e;
        key = ((uint64_t)__float_as_uint(best_d) << 33) | (kIdxMask - best_i);
    }
    float rel = acc.rd / acc.rb;                 // +inf when rb = 0 < rd; 0 for the initial (0, 1)
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint64_t k2 = __shfl_xor((unsigned long long)key, off, 64);
        key = k2 > key ? k2 : key;
        const float r2 = __shfl_xor(rel, off, 64);
        rel = r2 > rel ? r2 : rel;
    }
    const uint32_t wm = __shfl(acc.wmism, 0, 64), wn = __shfl(acc.wnan, 0, 64);
    __shared__ uint64_t s_key[kThreads / 64];
    __shared__ uint32_t s_m[kThreads / 64], s_n[kThreads / 64];
    __shared__ float s_r[kThreads / 64];
    const int w = t / 64;
    if ((t & 63) == 0) {
        s_key[w] = key;
        s_m[w] = wm;
        s_n[w] = wn;
        s_r[w] = rel;
    }
    __syncthreads();
    if (t == 0) {
        CheckPartial p;
        p.mism = 0;
        p.nan = 0;
        p.key = 0;
        float r = 0.0f;
#pragma unroll
        for (int i = 0; i < kThreads / 64; ++i) {
            p.mism += s_m[i];
            p.nan += s_n[i];
            p.key = s_key[i] > p.key ? s_key[i] : p.key;
            r = s_r[i] > r ? s_r[i] : r;
        }
        p.rel_bits = __float_as_uint(r);
        p.pad = 0;
        partials[blockIdx.x] = p;
    }
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

// Blocks of k_check<DA, DB, VEC, D> the current device holds at once, capped
// at the partial buffer's capacity; cached per device.
template <int DA, int DB, bool VEC, int D>
static uint32_t check_resident()
{
    constexpr int kDevCache = 64;
    static uint32_t cache[kDevCache] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevCache) dev = -1;
    if (dev >= 0 && cache[dev]) return cache[dev];
    int per_cu = 0, cus = 0;
    uint32_t r = kMaxCheckBlocks / 2;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_check<DA, DB, VEC, D>, kThreads, 0) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev < 0 ? 0 : dev) == hipSuccess &&
        per_cu > 0 && cus > 0)
        r = (uint32_t)per_cu * (uint32_t)cus;
    if (r > (uint32_t)kMaxCheckBlocks) r = kMaxCheckBlocks;
    if (dev >= 0) cache[dev] = r;
    return r;
}

template <int DA, int DB, int D>
static hipError_t check_ab_d(const void *a, const void *b, uint64_t n, float rtol, float atol, void *scratch,
                             krex_check_result *out, hipStream_t s)
{
    constexpr int SA = dtype_traits<DA>::size, SB = dtype_traits<DB>::size;
    constexpr int E = 16 / (SA < SB ? SA : SB);
    const bool vec = (((uintptr_t)a & 15u) == 0 && ((uintptr_t)b & 15u) == 0);
    const uint64_t nchunks = n / E;
    // One resident round: the grid is at most the number of blocks the
    // device holds at once (occupancy x compute units), so no partial last
    // round of blocks idles most of the chip. Chunks per thread: enough to
    // cover n with that grid, and at least u_floor (the pipeline's depth per
    // lane, and fewer partials for small n).
    static const uint32_t u_floor = tune_env("KREX_CHECK_U", 8);
    const uint64_t resident = vec ? check_resident<DA, DB, true, D>() : check_resident<DA, DB, false, 2>();
    uint64_t U = (nchunks + (uint64_t)kThreads * resident - 1) / ((uint64_t)kThreads * resident);
    if (U < u_floor) U = u_floor;
    if (U == 0) U = 1;
    uint64_t G = (nchunks + (uint64_t)kThreads * U - 1) / ((uint64_t)kThreads * U);
    if (G == 0) G = 1;   // the tail alone
    CheckPartial *parts = (CheckPartial *)scratch;
    hipError_t e;
    if (vec)
        e = launch(k_check<DA, DB, true, D>, dim3((uint32_t)G), dim3(kThreads), s, (const uint8_t *)a, (const uint8_t *)b,
                   n, rtol, atol, parts, (uint32_t)U);
    else
        e = launch(k_check<DA, DB, false, 2>, dim3((uint32_t)G), dim3(kThreads), s, (const uint8_t *)a,
                   (const uint8_t *)b, n, rtol, atol, parts, (uint32_t)U);
    if (e != hipSuccess) return e;
    return launch(k_check_final, dim3(1), dim3(kFinalThreads), s, (const CheckPartial *)parts, (uint32_t)G, n, out);
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
// The stores (store16_stream, raw buffer stores) carry the system-scope
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
    if (i < nvec) store16_stream(buf + (uint64_t)blockIdx.x * kThreads, 16u * threadIdx.x,
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

__global__ __launch_bounds__(kThreads) void k_probe(uint64_t iters, float *sink)
{
    const uint32_t g = blockIdx.x * kThreads + threadIdx.x;
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
    sink[g] = s;
}

hipError_t launch_probe(uint64_t iters, float *sink, hipStream_t s)
{
    return launch(k_probe, dim3(256), dim3(kThreads), s, iters, sink);
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
