// krex_device.hpp -- device-side building blocks of the gfx950 hot path:
// the Philox4x32-10 block function, the value transforms (uniform, Box-Muller
// normal with own fp32 ln / sin / cos, bitcast) and round-to-nearest-even
// narrowing to bf16 / fp16 / fp8-e4m3fn plus exact upcasts.
//
// Every definition here is the generation / check reading of the paper's
// command phases (KREX, Section 1 and Section 2.1: generate inputs, check
// against a reference, then time). The paper names no RNG or transform; the
// stream is Philox4x32-10 (Salmon et al., SC'11) so that each element's value
// is a pure function of (seed, offset + j), independent of launch shape and
// of colocated work (Section 2.1, "Benchmarking command").
//
// All arithmetic is fp32 with contraction disabled at build time; a fused
// multiply-add appears only where __builtin_fmaf is written. Division and
// square root are the correctly rounded IEEE operations (the normal
// transform reaches them through shorter sequences that equal them on its
// own input domain).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace krex {

enum : int { F32 = 0, BF16 = 1, F16 = 2, F8 = 3, U32 = 4 };
enum : int { UNIFORM = 0, NORMAL = 1, BITCAST = 2 };
enum : int { INJ_ROUND = 0, INJ_EXACT = 1 };

template <int DT> struct dtype_traits;
template <> struct dtype_traits<F32> { using storage = uint32_t; static constexpr int size = 4; };
template <> struct dtype_traits<BF16> { using storage = uint16_t; static constexpr int size = 2; };
template <> struct dtype_traits<F16> { using storage = uint16_t; static constexpr int size = 2; };
template <> struct dtype_traits<F8> { using storage = uint8_t; static constexpr int size = 1; };
template <> struct dtype_traits<U32> { using storage = uint32_t; static constexpr int size = 4; };

struct words4 {
    uint32_t v[4];
};

// The key schedule of one seed: round r uses (k0 + r 0x9E3779B9, k1 + r
// 0xBB67AE85), mod 2^32. Computed once on the host and passed as kernel
// arguments, so no wave spends scalar instructions rebuilding it.
struct RoundKeys {
    uint32_t k[20];
};

__host__ __device__ inline RoundKeys round_keys(uint64_t seed)
{
    RoundKeys r;
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int i = 0; i < 10; ++i) {
        r.k[2 * i] = k0;
        r.k[2 * i + 1] = k1;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return r;
}

// Philox4x32-10 on counter (b mod 2^32, b >> 32, 0, 0) with the key schedule
// rk. Per round the two 32x32->64 products M0*x0 and M1*x2 are formed and the
// state becomes (hi(M1 x2) ^ x1 ^ k0, lo(M1 x2), hi(M0 x0) ^ x3 ^ k1,
// lo(M0 x0)) with that round's key (k0, k1). The schedule is wave-uniform
// and lives in scalar registers. Each three-way xor is one gfx950
// v_bitop3_b32 (truth table 0x96: odd parity of the three inputs).
__device__ __forceinline__ words4 philox_block(uint64_t b, const RoundKeys &rk)
{
    uint32_t x0 = (uint32_t)b, x1 = (uint32_t)(b >> 32), x2 = 0u, x3 = 0u;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)x0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)x2;
        const uint32_t n0 = __builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), x1, rk.k[2 * r], 0x96);
        const uint32_t n1 = (uint32_t)p1;
        const uint32_t n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), x3, rk.k[2 * r + 1], 0x96);
        const uint32_t n3 = (uint32_t)p0;
        x0 = n0; x1 = n1; x2 = n2; x3 = n3;
    }
    words4 o;
    o.v[0] = x0; o.v[1] = x1; o.v[2] = x2; o.v[3] = x3;
    return o;
}

// G consecutive blocks b, b + 1, ... in lockstep, the same values as G
// philox_block calls. On gfx950 a run of v_mad_u64_u32 products issues
// faster than products interleaved one by one with other vector
// instructions (eight products, then eight xors: 8.3-8.4 cycles per pair;
// alternating: 9.5, whether or not the xor reads the product and whatever
// the register banks), and the compiler's schedule places each three-way
// xor next to its product. Here each round forms all 2 G products, then
// (behind a scheduling fence, so the two phases stay apart) all 2 G xors.
// In a plain two-block round chain this took 10% fewer cycles per block
// than the compiler's interleaving; in the kernels it took fp8 normal
// generation 8% and packed fp8 normal 5% faster (generation with
// injection, normal: 4-6%, value and mask blocks each in lockstep), left
// the uniform generators (also with two units' blocks in one lockstep) and
// the packed stream's check (its two-block fp8 normal units included)
// unchanged, and made the check against a regenerated word-stream
// reference 3% slower (the fence also holds back the check's own work),
// which therefore keeps separate philox_block calls.
template <int G>
__device__ __forceinline__ void philox_blocks(uint64_t b, const RoundKeys &rk, words4 (&o)[G])
{
    uint32_t x0[G], x1[G], x2[G], x3[G];
#pragma unroll
    for (int i = 0; i < G; ++i) {
        x0[i] = (uint32_t)(b + (uint64_t)i);
        x1[i] = (uint32_t)((b + (uint64_t)i) >> 32);
        x2[i] = 0u;
        x3[i] = 0u;
    }
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        uint64_t p0[G], p1[G];
#pragma unroll
        for (int i = 0; i < G; ++i) {
            p0[i] = (uint64_t)0xD2511F53u * (uint64_t)x0[i];
            p1[i] = (uint64_t)0xCD9E8D57u * (uint64_t)x2[i];
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < G; ++i) {
            x0[i] = __builtin_amdgcn_bitop3_b32((uint32_t)(p1[i] >> 32), x1[i], rk.k[2 * r], 0x96);
            x1[i] = (uint32_t)p1[i];
            x2[i] = __builtin_amdgcn_bitop3_b32((uint32_t)(p0[i] >> 32), x3[i], rk.k[2 * r + 1], 0x96);
            x3[i] = (uint32_t)p0[i];
        }
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = 0; i < G; ++i) {
        o[i].v[0] = x0[i];
        o[i].v[1] = x1[i];
        o[i].v[2] = x2[i];
        o[i].v[3] = x3[i];
    }
}

// ------------------------------------------------------- streaming memory

// 16-byte load of a streamed operand, non-temporal: it does not allocate in
// the Infinity Cache, which on gfx950 lets two concurrent read streams run at
// ~6.9 TB/s instead of ~6.4 TB/s (the data are read once; a line already
// cached is still returned from the cache).
__device__ __forceinline__ uint4 load16_stream(const void *p)
{
    typedef unsigned int v4u __attribute__((ext_vector_type(4)));
    const v4u v = __builtin_nontemporal_load(reinterpret_cast<const v4u *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// 16-byte raw buffer store with cache-policy bits POL. A raw buffer store,
// so the compiler sees it and keeps the wait states a store needs before its
// data registers are overwritten. `base` must be the same for every lane of
// the wave (a block's first byte); `off` is the lane's byte offset from it,
// below 2^31.
template <int POL>
__device__ __forceinline__ void store16_policy(void *base, uint32_t off, const uint4 &u)
{
    typedef unsigned int v4u __attribute__((ext_vector_type(4)));
    constexpr int kRawDword3 = 0x00020000;     // raw buffer: 32-bit data format, no swizzle
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(base, (short)0, 0x7FFFFFFF, kRawDword3);
    const v4u v = {u.x, u.y, u.z, u.w};
    __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)off, 0, POL);
}

// Store of a generated or injected output: non-temporal at device scope
// (nt sc1). It streams as fast as an allocating store and leaves no dirty
// lines of the output in the Infinity Cache. A kernel that reads an output
// still dirty there pays for it: on gfx950 a 1 GiB check right after the
// generation that wrote its operands with allocating stores took 222 us
// against 172 us once they had left the cache, and 173 us after this store.
__device__ __forceinline__ void store16_stream(void *base, uint32_t off, const uint4 &u)
{
    constexpr int kNtSc1 = 2 | 16;
    store16_policy<kNtSc1>(base, off, u);
}

// Store of the cache flush: system scope (sc0 sc1), written through L2
// without allocating there and allocated in the Infinity Cache like an
// ordinary store (~2% faster than one for streamed writes), so the flush
// evicts that cache's previous contents.
__device__ __forceinline__ void store16_alloc(void *base, uint32_t off, const uint4 &u)
{
    constexpr int kSc0Sc1 = 1 | 16;
    store16_policy<kSc0Sc1>(base, off, u);
}

// ---------------------------------------------------------------- narrowing

// gfx950 conversion instructions (v_cvt_pk_bf16_f32, v_cvt_f16_f32,
// v_cvt_pk_fp8_f32 without clamp, v_cvt_f32_f16, v_cvt_f32_fp8): round to
// nearest even with subnormals kept, fp8 e4m3fn non-saturating. Compared
// with the CPU definitions on gfx950 over all 2^32 fp32 inputs once, and by
// the parity tests over every 251st fp32 pattern, every pattern of the
// exponent windows where the rounding rules change and every 2^16 / 2^8
// narrow input: identical for every input that is not a NaN; a NaN input
// gives a NaN with another payload or sign. `narrow` therefore uses them
// directly only where no NaN can reach it and maps NaN to the canonical
// pattern otherwise. The upcasts' NaN payloads differ too, which no caller
// observes (a NaN is only tested as a NaN or narrowed again).
__device__ __forceinline__ uint16_t to_bf16_hw(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ uint16_t to_f16_hw(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }
__device__ __forceinline__ uint8_t to_f8_hw(float f)
{
    return (uint8_t)(__builtin_amdgcn_cvt_pk_fp8_f32(f, 0.0f, 0, false) & 0xFF);
}

// NAN_IN: whether v may be a NaN.
template <int DT, bool NAN_IN = true>
__device__ __forceinline__ typename dtype_traits<DT>::storage narrow(float v)
{
    if constexpr (DT == F32) {
        return __float_as_uint(v);
    } else if constexpr (DT == BF16) {
        const uint16_t h = to_bf16_hw(v);
        if constexpr (NAN_IN) return (v != v) ? (uint16_t)0x7FC0u : h;
        return h;
    } else if constexpr (DT == F16) {
        const uint16_t h = to_f16_hw(v);
        if constexpr (NAN_IN) return (v != v) ? (uint16_t)0x7E00u : h;
        return h;
    } else {
        const uint8_t h = to_f8_hw(v);
        if constexpr (NAN_IN) return (v != v) ? (uint8_t)0x7Fu : h;
        return h;
    }
}

// N values narrowed into N size / 4 words, element i at bits
// [8 size (i mod K), 8 size (i mod K + 1)) of word i / K (K = 4 / size), i.e.
// the little-endian layout of the narrow array. Two values per packed
// conversion (v_cvt_pk_bf16_f32, v_cvt_pk_f16_f32, v_cvt_pk_fp8_f32; the same
// rounding as the one-value conversions), then the canonical NaN where a NaN
// can occur.
template <int DT, bool NAN_IN, int N>
__device__ __forceinline__ void pack_narrow(const float (&v)[N], uint32_t (&w)[N * dtype_traits<DT>::size / 4])
{
    if constexpr (DT == F32 || DT == U32) {
#pragma unroll
        for (int i = 0; i < N; ++i) w[i] = __float_as_uint(v[i]);
    } else if constexpr (DT == BF16 || DT == F16) {
        static_assert(N % 2 == 0, "pairs");
        typedef float f2 __attribute__((ext_vector_type(2)));
        constexpr uint32_t qnan = (DT == BF16) ? 0x7FC0u : 0x7E00u;
#pragma unroll
        for (int i = 0; i < N / 2; ++i) {
            const f2 x = {v[2 * i], v[2 * i + 1]};
            uint32_t h;
            if constexpr (DT == BF16) {
                typedef __bf16 n2 __attribute__((ext_vector_type(2)));
                h = __builtin_bit_cast(uint32_t, __builtin_convertvector(x, n2));
            } else {
                typedef _Float16 n2 __attribute__((ext_vector_type(2)));
                h = __builtin_bit_cast(uint32_t, __builtin_convertvector(x, n2));
            }
            if constexpr (NAN_IN) {
                if (v[2 * i] != v[2 * i]) h = (h & 0xFFFF0000u) | qnan;
                if (v[2 * i + 1] != v[2 * i + 1]) h = (h & 0x0000FFFFu) | (qnan << 16);
            }
            w[i] = h;
        }
    } else {
        static_assert(N % 4 == 0, "quads");
#pragma unroll
        for (int i = 0; i < N / 4; ++i) {
            uint32_t h = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(v[4 * i], v[4 * i + 1], 0, false);
            h = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(v[4 * i + 2], v[4 * i + 3], (int)h, true);
            if constexpr (NAN_IN) {
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    if (v[4 * i + b] != v[4 * i + b]) h = (h & ~(0xFFu << (8 * b))) | (0x7Fu << (8 * b));
            }
            w[i] = h;
        }
    }
}

template <int DT>
__device__ __forceinline__ float widen(uint32_t bits)
{
    if constexpr (DT == F32) return __uint_as_float(bits);
    else if constexpr (DT == BF16) return __uint_as_float(bits << 16);
    else if constexpr (DT == F16) return (float)__builtin_bit_cast(_Float16, (uint16_t)bits);
    else return __builtin_amdgcn_cvt_f32_fp8((int)bits, 0);
}

// ---------------------------------------------------------------- fp32 math

// The correctly rounded quotient f / den for the operands ln_f32 forms:
// f = m - 1 with m an fp32 value in [sqrt(1/2), sqrt 2], den = fl(2 + f) in
// [1.7, 2.5]. The hardware reciprocal (v_rcp_f32, within one ulp) gives
// q0 = fl(f r); the residual f - den q0 is exact in one fused multiply-add,
// and one correction step q0 + r (f - den q0) rounds to the IEEE quotient.
// That the result equals IEEE division was checked on gfx950 for every one of
// the 8,388,609 fp32 values of m in that interval, and the normal
// transform's parity with the oracle is tested over every u1. Outside this
// domain (denormal, huge or zero den) the sequence is not claimed exact.
__device__ __forceinline__ float div_on_ln_domain(float f, float den)
{
    const float r = __builtin_amdgcn_rcpf(den);
    const float q0 = f * r;
    const float e = __builtin_fmaf(-den, q0, f);
    return __builtin_fmaf(e, r, q0);
}

// The correctly rounded square root of t = +0 or a normal t (no scaling of
// denormal inputs, no infinity or NaN handling): the hardware root s (within
// one ulp) is replaced by its lower or upper neighbour when the exact
// residual t - s' s shows that neighbour is the nearer root. At t = +0 the
// residuals are NaN and +0, so s = +0 stays. Equal to IEEE sqrt on all 2^24
// values -2 ln u1 the normal transform forms (checked on gfx950, and the
// transform's parity with the oracle is tested over every u1).
__device__ __forceinline__ float sqrt_nonneg_normal(float t)
{
    const float s = __builtin_amdgcn_sqrtf(t);
    const float sm = __uint_as_float(__float_as_uint(s) - 1u);
    const float sp = __uint_as_float(__float_as_uint(s) + 1u);
    const float vm = __builtin_fmaf(-sm, s, t);
    const float vp = __builtin_fmaf(-sp, s, t);
    const float r = (vm <= 0.0f) ? sm : s;
    return (vp > 0.0f) ? sp : r;
}

// ln x for a positive normal x: x = 2^e m, m in [sqrt(1/2), sqrt 2);
// f = m - 1 (exact), s = f / (2 + f), ln m = 2 atanh s, written as
// f - (f^2/2 - s (f^2/2 + R)) with R = z (2/3 + z (2/5 + z (2/7 + z (2/9 + z 2/11)))),
// z = s^2; then e ln2 is added as e * head + (e * tail + ln m) with a
// 16-bit head of ln 2.
__device__ __forceinline__ float ln_f32(float x)
{
    // The split without a compare: adding 0x4AFB0C to the bits of x carries
    // into the exponent exactly when the mantissa field exceeds 0x3504F3
    // (that of fp32(sqrt 2)); the low 23 bits plus the bits of
    // fp32(sqrt(1/2)) + 1 ulp, 0x3F3504F4, then give 1.mb or 0.5 x 1.mb.
    const uint32_t iy = __float_as_uint(x) + 0x004AFB0Cu;
    const int32_t e = (int32_t)(iy >> 23) - 127;
    const float m = __uint_as_float((iy & 0x7FFFFFu) + 0x3F3504F4u);
    const float f = m - 1.0f;
    const float den = 2.0f + f;
    const float s = div_on_ln_domain(f, den);
    const float z = s * s;
    float p = 0x1.745d18p-3f;
    p = __builtin_fmaf(p, z, 0x1.c71c72p-3f);
    p = __builtin_fmaf(p, z, 0x1.24924ap-2f);
    p = __builtin_fmaf(p, z, 0x1.99999ap-2f);
    p = __builtin_fmaf(p, z, 0x1.555556p-1f);
    const float R = z * p;
    const float hf = 0.5f * f;
    const float hfsq = hf * f;
    const float a = hfsq + R;
    const float b = s * a;
    const float c = hfsq - b;
    const float lnm = f - c;
    const float dk = (float)e;
    const float tail = __builtin_fmaf(dk, 0x1.7f7d1cp-20f, lnm);
    const float head = dk * 0x1.62e4p-1f;
    return head + tail;
}

// sin and cos of 2 pi k 2^-24, k in [0, 2^24): quadrant q = round(k 2^-22),
// r = (k - q 2^22) 2^-22 in [-1/2, 1/2) (exact integer steps), Taylor
// polynomials of sin(pi r / 2) through r^9 and cos(pi r / 2) through r^10 in
// Horner form on r^2, then the quadrant's swap and signs.
__device__ __forceinline__ void sincos_2pi_q24(uint32_t k, float &sn, float &cs)
{
    const uint32_t q = (k + (1u << 21)) >> 22;
    const int32_t ri = (int32_t)k - (int32_t)(q << 22);
    const float r = (float)ri * 0x1p-22f;
    const float y = r * r;
    float ps = 0x1.507834p-13f;
    ps = __builtin_fmaf(ps, y, -0x1.32d2ccp-8f);
    ps = __builtin_fmaf(ps, y, 0x1.466bc6p-4f);
    ps = __builtin_fmaf(ps, y, -0x1.4abbcep-1f);
    ps = __builtin_fmaf(ps, y, 0x1.921fb6p+0f);
    const float S = r * ps;
    float pc = -0x1.a6d1f2p-16f;
    pc = __builtin_fmaf(pc, y, 0x1.e1f506p-11f);
    pc = __builtin_fmaf(pc, y, -0x1.55d3c8p-6f);
    pc = __builtin_fmaf(pc, y, 0x1.03c1f0p-2f);
    pc = __builtin_fmaf(pc, y, -0x1.3bd3ccp+0f);
    const float C = __builtin_fmaf(pc, y, 1.0f);
    // Quadrant q mod 4: (sin, cos) = (S, C), (C, -S), (-S, -C), (-C, S).
    // Selected without branches (lanes take random quadrants): odd q swaps
    // the pair, bit 1 of q negates the sine, bit 1 of q + 1 the cosine; a
    // negation is the sign-bit flip.
    const bool swap = (q & 1u) != 0u;
    const float a = swap ? C : S;
    const float b = swap ? S : C;
    sn = __uint_as_float(__float_as_uint(a) ^ ((q & 2u) << 30));
    cs = __uint_as_float(__float_as_uint(b) ^ (((q + 1u) & 2u) << 30));
}

// Box-Muller on (w0, w1): u1 = ((w0 >> 8) + 1) 2^-24 in (0, 1],
// rho = sqrt(0 - 2 ln u1) (so rho = +0 at u1 = 1), z0 = rho cos, z1 = rho sin
// of 2 pi (w1 >> 8) 2^-24.
__device__ __forceinline__ void normal_pair(uint32_t w0, uint32_t w1, float &z0, float &z1)
{
    const float u1 = (float)((w0 >> 8) + 1u) * 0x1p-24f;
    const float L = ln_f32(u1);
    const float t2 = 2.0f * L;
    const float t = 0.0f - t2;
    const float rho = sqrt_nonneg_normal(t);
    float sn, cs;
    sincos_2pi_q24(w1 >> 8, sn, cs);
    z0 = rho * cs;
    z1 = rho * sn;
}

__device__ __forceinline__ float uniform_f32(uint32_t w, float lo, float range)
{
    // range = fl(hi - lo), computed once on the host with the same rounding
    const float u = (float)(w >> 8) * 0x1p-24f;
    const float t = range * u;
    return lo + t;
}

// The uniform transform when range = fl(hi - lo) is a power of two with
// c = range 2^-24 normal: range u = c (w >> 8) is then exact (a 24-bit
// integer times a power of two), so lo + fl(range u) has a single rounding
// and one fused multiply-add gives the same value.
__device__ __forceinline__ float uniform_f32_pow2(uint32_t w, float lo, float c)
{
    return __builtin_fmaf(c, (float)(w >> 8), lo);
}

// Four values from four consecutive words (two normal pairs). POW2: the
// uniform range is a power of two and p1 holds c = range 2^-24.
template <int DIST, bool POW2 = false>
__device__ __forceinline__ void transform4(const words4 &w, float p0, float p1, float v[4])
{
    if constexpr (DIST == UNIFORM) {
#pragma unroll
        for (int l = 0; l < 4; ++l) v[l] = POW2 ? uniform_f32_pow2(w.v[l], p0, p1) : uniform_f32(w.v[l], p0, p1);
    } else if constexpr (DIST == NORMAL) {
        float z[4];
        normal_pair(w.v[0], w.v[1], z[0], z[1]);
        normal_pair(w.v[2], w.v[3], z[2], z[3]);
#pragma unroll
        for (int l = 0; l < 4; ++l) {
            const float sz = p1 * z[l];
            v[l] = p0 + sz;
        }
    } else {
#pragma unroll
        for (int l = 0; l < 4; ++l) v[l] = __uint_as_float(w.v[l]);
    }
}

// ------------------------------------------------------------- packed stream
//
// The narrow-dtype stream that spends W bits of the word stream per
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

// Uniform transform of a W-bit field f: UM_WORD applies the word-stream
// transform to f << (32 - W); UM_SCALED when rs = fl(hi - lo) 2^-W is exact
// (u = f 2^-W exactly, so rs f is the same real number as fl(hi - lo) u and
// rounds the same: one conversion, one multiply, one add); UM_FUSED when rs f
// is exact as well, so lo + rs f has one rounding: one fused multiply-add.
enum : int { UM_WORD = 0, UM_SCALED = 1, UM_FUSED = 2 };

// Packed unit `unit` of the stream with key schedule rk: its GB Philox
// blocks (unit GB onward) give E = 16 / size fields, each transformed and
// narrowed to DT, packed little-endian into the 16 bytes w. p0, p1: lo and
// fl(hi - lo) (uniform) or mean and std (normal); rs: fl(hi - lo) 2^-W when
// UM is UM_SCALED or UM_FUSED.
template <int DT, int DIST, int UM>
__device__ __forceinline__ void packed_unit(uint64_t unit, const RoundKeys &rk, float p0, float p1, float rs,
                                            uint32_t (&w)[4])
{
    constexpr int W = packed_of<DT, DIST>::W;
    constexpr int K = 32 / W;
    constexpr int E = packed_of<DT, DIST>::E;
    constexpr int GB = packed_of<DT, DIST>::GB;
    constexpr uint32_t kMask = (1u << W) - 1u;
    uint32_t wv[4 * GB];
    words4 blk[GB];
    if constexpr (GB > 1) philox_blocks<GB>(unit * GB, rk, blk);
    else blk[0] = philox_block(unit, rk);
#pragma unroll
    for (int i = 0; i < GB; ++i) {
#pragma unroll
        for (int l = 0; l < 4; ++l) wv[4 * i + l] = blk[i].v[l];
    }
    if constexpr (DIST == BITCAST) {
        static_assert(GB == 1, "bitcast units are one block");
#pragma unroll
        for (int l = 0; l < 4; ++l) w[l] = wv[l];
    } else if constexpr (DIST == UNIFORM) {
        float v[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const uint32_t f = (wv[e / K] >> ((e % K) * W)) & kMask;
            if constexpr (UM == UM_FUSED) {
                v[e] = __builtin_fmaf(rs, (float)f, p0);
            } else if constexpr (UM == UM_SCALED) {
                const float t = rs * (float)f;
                v[e] = p0 + t;
            } else {
                v[e] = uniform_f32(f << (32 - W), p0, p1);
            }
        }
        if constexpr (DT == F8) {
            // Two values per conversion (bytes 0-1, then 2-3 of the word).
#pragma unroll
            for (int i = 0; i < E / 4; ++i) {
                uint32_t wd = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(v[4 * i], v[4 * i + 1], 0, false);
                wd = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(v[4 * i + 2], v[4 * i + 3], (int)wd, true);
                w[i] = wd;
            }
        } else {
            pack_narrow<DT, false>(v, w);
        }
    } else {
        static_assert(W == 16 && E == 8 * GB, "normal fields are 16 bits, two per word");
        float v[E];
#pragma unroll
        for (int i = 0; i < 4 * GB; ++i) {
            float z0, z1;
            normal_pair(wv[i] << 16, wv[i] & 0xFFFF0000u, z0, z1);
            const float s0 = p1 * z0;
            const float s1 = p1 * z1;
            v[2 * i] = p0 + s0;
            v[2 * i + 1] = p0 + s1;
        }
        pack_narrow<DT, false>(v, w);
    }
}

}  // namespace krex
