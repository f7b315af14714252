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
//             operands, per-thread counters and maxima, wave64 shuffles,
//             LDS across the block's four waves, one atomic per field per
//             block, and the last block to finish decodes the packed argmax.
//   k_flush   16-byte allocating stores of a pattern (Section 2.1 flush
//             between iterations; Section 4.2 step 5).
//   k_probe   fixed-work FMA kernel timed by the fidelity measurement
//             (Section 6.3, Eq. 1).
//   k_sgemm   naive fp32 GEMM standing in for a candidate kernel.
//
// All loops are grid-stride with a grid sized to the device (a few blocks
// per CU), so the launch shape never changes a result: every element's
// value depends only on its index.
#include <hip/hip_runtime.h>

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

static uint32_t grid_for(uint64_t units, int blocks_per_cu)
{
    const uint64_t need = (units + kThreads - 1) / kThreads;
    const uint64_t cap = (uint64_t)device_cus() * (uint64_t)blocks_per_cu;
    uint64_t g = need < cap ? need : cap;
    return (uint32_t)(g == 0 ? 1 : g);
}

// ------------------------------------------------------------------ generation

struct GenParams {
    uint8_t *dst;
    uint64_t n;
    uint64_t offset;
    uint32_t k0, k1;
    float p0, p1;      // uniform: lo and fl(hi - lo); normal: mean and std
    uint64_t b0;       // first Philox block
    uint64_t ngroups;  // groups of G blocks
    int vec;           // offset % 4 == 0 and dst 16-byte aligned
};

template <int DT, int DIST>
__global__ __launch_bounds__(kThreads) void k_gen(GenParams P)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int G = group_of<DT>::G;
    const uint64_t stride = (uint64_t)gridDim.x * kThreads;
    for (uint64_t g = (uint64_t)blockIdx.x * kThreads + threadIdx.x; g < P.ngroups; g += stride) {
        const uint64_t bfirst = P.b0 + g * G;
        union {
            uint4 v;
            T s[4 * G];
        } pk;
#pragma unroll
        for (int i = 0; i < G; ++i) {
            const words4 w = philox_block(bfirst + i, P.k0, P.k1);
            if constexpr (DT == U32) {
#pragma unroll
                for (int l = 0; l < 4; ++l) pk.s[4 * i + l] = w.v[l];
            } else {
                float v[4];
                transform4<DIST>(w, P.p0, P.p1, v);
#pragma unroll
                for (int l = 0; l < 4; ++l) pk.s[4 * i + l] = narrow<DT>(v[l]);
            }
        }
        const uint64_t j0 = 4 * bfirst - P.offset;
        if (P.vec && j0 + 4 * G <= P.n) {
            *reinterpret_cast<uint4 *>(P.dst + j0 * ES) = pk.v;
        } else {
#pragma unroll
            for (int e = 0; e < 4 * G; ++e) {
                const uint64_t w = 4 * bfirst + (uint64_t)e;
                if (w >= P.offset && w - P.offset < P.n) reinterpret_cast<T *>(P.dst)[w - P.offset] = pk.s[e];
            }
        }
    }
}

template <int DT, int DIST>
static hipError_t gen_dt_dist(const GenParams &P, hipStream_t s)
{
    const uint32_t grid = grid_for(P.ngroups, 8);
    return launch(k_gen<DT, DIST>, dim3(grid), dim3(kThreads), s, P);
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

hipError_t launch_gen(void *dst, int dt, uint64_t n, uint64_t seed, uint64_t offset, int dist, float p0,
                      float p1, hipStream_t s)
{
    if (n == 0) return hipSuccess;
    GenParams P;
    P.dst = (uint8_t *)dst;
    P.n = n;
    P.offset = offset;
    P.k0 = (uint32_t)seed;
    P.k1 = (uint32_t)(seed >> 32);
    P.p0 = p0;
    P.p1 = (dist == UNIFORM) ? (p1 - p0) : p1;
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
    switch (dt) {
    case F32: return gen_dt<F32>(P, dist, s);
    case BF16: return gen_dt<BF16>(P, dist, s);
    case F16: return gen_dt<F16>(P, dist, s);
    case F8: return gen_dt<F8>(P, dist, s);
    default: return gen_dt<U32>(P, dist, s);
    }
}

// ------------------------------------------------------------- words transform

struct XformParams {
    uint8_t *dst;
    const uint32_t *words;
    uint64_t n;
    float p0, p1;
    uint64_t ngroups;
    int vec;
};

template <int DT, int DIST>
__global__ __launch_bounds__(kThreads) void k_xform(XformParams P)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int G = group_of<DT>::G;
    const uint64_t stride = (uint64_t)gridDim.x * kThreads;
    for (uint64_t g = (uint64_t)blockIdx.x * kThreads + threadIdx.x; g < P.ngroups; g += stride) {
        const uint64_t j0 = g * 4 * G;
        if (P.vec && j0 + 4 * G <= P.n) {
            union {
                uint4 v;
                T s[4 * G];
            } pk;
#pragma unroll
            for (int i = 0; i < G; ++i) {
                const uint4 raw = reinterpret_cast<const uint4 *>(P.words + j0)[i];
                words4 w;
                w.v[0] = raw.x; w.v[1] = raw.y; w.v[2] = raw.z; w.v[3] = raw.w;
                if constexpr (DT == U32) {
#pragma unroll
                    for (int l = 0; l < 4; ++l) pk.s[4 * i + l] = w.v[l];
                } else {
                    float v[4];
                    transform4<DIST>(w, P.p0, P.p1, v);
#pragma unroll
                    for (int l = 0; l < 4; ++l) pk.s[4 * i + l] = narrow<DT>(v[l]);
                }
            }
            *reinterpret_cast<uint4 *>(P.dst + j0 * ES) = pk.v;
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
                        v = uniform_f32(P.words[j], P.p0, P.p1);
                    } else if constexpr (DIST == NORMAL) {
                        float z0, z1;
                        normal_pair(P.words[j & ~(uint64_t)1], P.words[j | 1u], z0, z1);
                        const float sz = P.p1 * ((j & 1u) ? z1 : z0);
                        v = P.p0 + sz;
                    } else {
                        v = __uint_as_float(P.words[j]);
                    }
                    out = narrow<DT>(v);
                }
                reinterpret_cast<T *>(P.dst)[j] = out;
            }
        }
    }
}

template <int DT>
static hipError_t xform_dt(const XformParams &P, int dist, hipStream_t s)
{
    const uint32_t grid = grid_for(P.ngroups, 8);
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
        if (dp == delta && widen<DT>(narrow<DT>(sp)) == sp) return narrow<DT>(sp);
        const float sm = X - delta;
        const float dm = X - sm;
        if (dm == delta && widen<DT>(narrow<DT>(sm)) == sm) return narrow<DT>(sm);
        return bits;
    }
}

template <int DT, int MODE>
__global__ __launch_bounds__(kThreads) void k_inject(InjectParams P)
{
    using T = typename dtype_traits<DT>::storage;
    constexpr int ES = dtype_traits<DT>::size;
    constexpr int G = group_of<DT>::G;
    const uint64_t stride = (uint64_t)gridDim.x * kThreads;
    for (uint64_t g = (uint64_t)blockIdx.x * kThreads + threadIdx.x; g < P.ngroups; g += stride) {
        const uint64_t bfirst = P.b0 + g * G;
        const uint64_t j0 = 4 * bfirst - P.moff;
        if (P.vec && j0 + 4 * G <= P.n) {
            union {
                uint4 v;
                T s[4 * G];
            } pk;
            pk.v = *reinterpret_cast<const uint4 *>(P.x + j0 * ES);
#pragma unroll
            for (int i = 0; i < G; ++i) {
                const words4 w = philox_block(bfirst + i, P.k0, P.k1);
#pragma unroll
                for (int l = 0; l < 4; ++l)
                    if ((uint64_t)w.v[l] < P.T) pk.s[4 * i + l] = perturb<DT, MODE>(pk.s[4 * i + l], P.delta);
            }
            *reinterpret_cast<uint4 *>(P.y + j0 * ES) = pk.v;
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
static hipError_t inject_dt(const InjectParams &P, int mode, hipStream_t s)
{
    const uint32_t grid = grid_for(P.ngroups, 8);
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

// ---------------------------------------------------------------------- check

static constexpr uint64_t kIdxMask = (1ull << 33) - 1;   // n < 2^33

struct CheckAcc {
    uint32_t mism;
    uint32_t nan;
    uint64_t key;     // (bits(d) << 33) | (kIdxMask - i): max = largest d, lowest i
    float rel;
};

__device__ __forceinline__ void check_one(float A, float B, uint64_t i, float rtol, float atol, CheckAcc &acc)
{
    if (A != A || B != B) {
        acc.mism += 1u;
        acc.nan += 1u;
        return;
    }
    float d, r;
    if (A == B) {
        d = 0.0f;
        r = 0.0f;
    } else if (__builtin_fabsf(A) == __builtin_inff() || __builtin_fabsf(B) == __builtin_inff()) {
        acc.mism += 1u;
        d = __builtin_inff();
        r = __builtin_inff();
    } else {
        const float diff = A - B;
        d = __builtin_fabsf(diff);
        const float ab = __builtin_fabsf(B);
        const float rt = rtol * ab;
        const float thr = atol + rt;
        acc.mism += (d <= thr) ? 0u : 1u;
        r = d / ab;
    }
    const uint64_t k = ((uint64_t)__float_as_uint(d) << 33) | (kIdxMask - i);
    acc.key = k > acc.key ? k : acc.key;
    acc.rel = r > acc.rel ? r : acc.rel;
}

template <int DA, int DB>
__global__ __launch_bounds__(kThreads) void k_check(const uint8_t *a, const uint8_t *b, uint64_t n, float rtol,
                                                    float atol, krex_check_result *out, int vec)
{
    using TA = typename dtype_traits<DA>::storage;
    using TB = typename dtype_traits<DB>::storage;
    constexpr int SA = dtype_traits<DA>::size;
    constexpr int SB = dtype_traits<DB>::size;
    constexpr int E = 16 / (SA < SB ? SA : SB);      // elements per chunk
    constexpr int VA = E * SA / 16;                  // 16-byte vectors of a per chunk
    constexpr int VB = E * SB / 16;
    CheckAcc acc{0u, 0u, 0ull, 0.0f};
    const uint64_t tid = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
    const uint64_t stride = (uint64_t)gridDim.x * kThreads;
    const uint64_t nchunks = vec ? n / E : 0;
    for (uint64_t c = tid; c < nchunks; c += stride) {
        union {
            uint4 v[VA];
            TA s[E];
        } ua;
        union {
            uint4 v[VB];
            TB s[E];
        } ub;
#pragma unroll
        for (int i = 0; i < VA; ++i) ua.v[i] = reinterpret_cast<const uint4 *>(a)[c * VA + i];
#pragma unroll
        for (int i = 0; i < VB; ++i) ub.v[i] = reinterpret_cast<const uint4 *>(b)[c * VB + i];
#pragma unroll
        for (int e = 0; e < E; ++e)
            check_one(widen<DA>(ua.s[e]), widen<DB>(ub.s[e]), c * E + e, rtol, atol, acc);
    }
    for (uint64_t i = nchunks * E + tid; i < n; i += stride)
        check_one(widen<DA>(reinterpret_cast<const TA *>(a)[i]), widen<DB>(reinterpret_cast<const TB *>(b)[i]), i,
                  rtol, atol, acc);

    // wave64 reduction
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        acc.mism += __shfl_xor(acc.mism, off, 64);
        acc.nan += __shfl_xor(acc.nan, off, 64);
        const uint64_t k = __shfl_xor((unsigned long long)acc.key, off, 64);
        acc.key = k > acc.key ? k : acc.key;
        const float r = __shfl_xor(acc.rel, off, 64);
        acc.rel = r > acc.rel ? r : acc.rel;
    }
    __shared__ uint32_t s_mism[kThreads / 64], s_nan[kThreads / 64];
    __shared__ uint64_t s_key[kThreads / 64];
    __shared__ float s_rel[kThreads / 64];
    const int wave = threadIdx.x / 64;
    if ((threadIdx.x & 63) == 0) {
        s_mism[wave] = acc.mism;
        s_nan[wave] = acc.nan;
        s_key[wave] = acc.key;
        s_rel[wave] = acc.rel;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t m = 0, nn = 0, key = 0;
        float rel = 0.0f;
#pragma unroll
        for (int w = 0; w < kThreads / 64; ++w) {
            m += s_mism[w];
            nn += s_nan[w];
            key = s_key[w] > key ? s_key[w] : key;
            rel = s_rel[w] > rel ? s_rel[w] : rel;
        }
        if (m) atomicAdd((unsigned long long *)&out->mismatches, (unsigned long long)m);
        if (nn) atomicAdd((unsigned long long *)&out->nan_count, (unsigned long long)nn);
        if (key) atomicMax((unsigned long long *)&out->reserved[0], (unsigned long long)key);
        if (rel > 0.0f) atomicMax((unsigned int *)&out->max_rel, __float_as_uint(rel));
        __threadfence();
        const unsigned int ticket = atomicAdd((unsigned int *)&out->reserved[1], 1u);
        if (ticket == gridDim.x - 1) {
            __threadfence();
            const uint64_t K = __hip_atomic_load(&out->reserved[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (K == 0) {
                out->argmax_abs = ~0ull;
                out->max_abs = 0.0f;
            } else {
                out->max_abs = __uint_as_float((uint32_t)(K >> 33));
                out->argmax_abs = kIdxMask - (K & kIdxMask);
            }
        }
    }
}

__global__ void k_check_init(krex_check_result *out, uint64_t n)
{
    out->n = n;
    out->mismatches = 0;
    out->nan_count = 0;
    out->argmax_abs = ~0ull;
    out->max_abs = 0.0f;
    out->max_rel = 0.0f;
    out->reserved[0] = 0;
    out->reserved[1] = 0;
    out->reserved[2] = 0;
}

template <int DA, int DB>
static hipError_t check_ab(const void *a, const void *b, uint64_t n, float rtol, float atol, krex_check_result *out,
                           hipStream_t s)
{
    constexpr int SA = dtype_traits<DA>::size, SB = dtype_traits<DB>::size;
    constexpr int E = 16 / (SA < SB ? SA : SB);
    const int vec = (((uintptr_t)a & 15u) == 0 && ((uintptr_t)b & 15u) == 0) ? 1 : 0;
    const uint64_t units = vec ? (n / E > 0 ? n / E : 1) : n;
    const uint32_t grid = grid_for(units, 8);
    return launch(k_check<DA, DB>, dim3(grid), dim3(kThreads), s, (const uint8_t *)a, (const uint8_t *)b, n, rtol,
                  atol, out, vec);
}

template <int DA>
static hipError_t check_a(const void *a, int dtb, const void *b, uint64_t n, float rtol, float atol,
                          krex_check_result *out, hipStream_t s)
{
    switch (dtb) {
    case F32: return check_ab<DA, F32>(a, b, n, rtol, atol, out, s);
    case BF16: return check_ab<DA, BF16>(a, b, n, rtol, atol, out, s);
    case F16: return check_ab<DA, F16>(a, b, n, rtol, atol, out, s);
    default: return check_ab<DA, F8>(a, b, n, rtol, atol, out, s);
    }
}

hipError_t launch_check(const void *a, int dta, const void *b, int dtb, uint64_t n, float rtol, float atol,
                        krex_check_result *out, hipStream_t s)
{
    hipError_t e = launch(k_check_init, dim3(1), dim3(1), s, out, n);
    if (e != hipSuccess || n == 0) return e;
    switch (dta) {
    case F32: return check_a<F32>(a, dtb, b, n, rtol, atol, out, s);
    case BF16: return check_a<BF16>(a, dtb, b, n, rtol, atol, out, s);
    case F16: return check_a<F16>(a, dtb, b, n, rtol, atol, out, s);
    default: return check_a<F8>(a, dtb, b, n, rtol, atol, out, s);
    }
}

// ---------------------------------------------------------------------- flush

__global__ __launch_bounds__(kThreads) void k_flush(uint4 *buf, uint64_t nvec, uint32_t pattern)
{
    const uint4 v = make_uint4(pattern, pattern, pattern, pattern);
    const uint64_t stride = (uint64_t)gridDim.x * kThreads;
    uint64_t i = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
    for (; i + 3 * stride < nvec; i += 4 * stride) {
        buf[i] = v;
        buf[i + stride] = v;
        buf[i + 2 * stride] = v;
        buf[i + 3 * stride] = v;
    }
    for (; i < nvec; i += stride) buf[i] = v;
}

hipError_t launch_flush(void *buf, uint64_t bytes, uint32_t pattern, hipStream_t s)
{
    const uint64_t nvec = bytes / 16;
    if (nvec == 0) return hipSuccess;
    const uint32_t grid = grid_for(nvec, 8);
    return launch(k_flush, dim3(grid), dim3(kThreads), s, (uint4 *)buf, nvec, pattern);
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
