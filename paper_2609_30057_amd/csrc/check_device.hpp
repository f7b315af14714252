// check_device.hpp -- the fused allclose check (Section 1; Section 2.1: the
// command checks the candidate's output against a reference) as a device
// body shared by its kernels, which differ in where the reference comes
// from: k_check reads it from memory, k_check_gen and k_check_gen_packed
// regenerate it from the word or the packed Philox stream (the values
// generation would have written), so only the candidate is read.
//
// Two launches and no atomics. k_check: block b owns chunks
// [b 256 U, (b + 1) 256 U) of E elements (one 16-byte vector of the
// narrower operand); thread t takes chunk b 256 U + u 256 + t for u < U, so
// every step of a wave reads contiguous memory. Per element the verdict is
// branch-free: each lane counts its mismatches in a vector register (summed
// over the wave at the end), max_rel candidates are one wave ballot, and
// unordered pairs are counted with ballots only in the rare chunks whose
// maximum of d is NaN. The per-lane maximum |a - b| is tracked per chunk,
// and the first index of the wave's maximum is recovered at the end by its
// winning lane re-reading that one chunk. Each block writes one 32-byte
// partial with plain stores; k_check_final reduces the partials and writes
// the result record.
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
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hip_launch.hpp"
#include "krex.h"
#include "krex_device.hpp"

namespace krex {

static constexpr int kThreads = 256;

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

struct LaneAcc {
    uint32_t mism;          // this lane's mismatches
    uint32_t wnan;          // the wave's unordered pairs (exact in its first lane)
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

// The smallest positive fp32 value (denormals are kept): d > 0 exactly when
// d >= kMinPositive.
static constexpr float kMinPositive = 0x1p-149f;

// Verdict of one element: the lane's mismatch count and the wave's max_rel
// candidate mask (one compare writing a lane mask). d is 0 when a == b (an
// infinity equal to itself included), NaN when the pair is unordered, else
// |a - b|. The
// element mismatches exactly when not d <= min(atol + rtol |b|, FLT_MAX): an
// equal pair has d = 0, below any threshold (atol, rtol >= 0; a NaN
// threshold, 0 x inf with |b| = inf, becomes FLT_MAX); an unordered pair has
// d = NaN, never <= anything; a differing pair is close exactly when d is
// finite and within the threshold (d = +inf, an infinite operand or an
// overflowing difference, exceeds FLT_MAX). It is a max_rel candidate when
// d >= max(fl(R |b|), kMinPositive), i.e. it differs, is ordered and its
// ratio may reach R (the filter's bound; R |b| is NaN only for an unordered
// pair). NOINF: neither operand type has an infinity and their difference
// cannot overflow (fp8 e4m3fn pairs: |a|, |b| <= 448), so |a - b| is already
// 0 for equal operands and the threshold is finite: no select, no clamp; and
// the candidate test is d Rup > |b| with Rup >= (1/R)(1 + 2^-21) (see
// RatioFilter), decided exactly by the sign of fma(d, Rup, -|b|): the lane's
// largest such residual over a chunk goes to tmax (the non-propagating
// maximum, so an unordered pair, NaN there, hides no other element) and the
// caller takes one ballot of tmax > 0 per chunk instead of one per element.
// Mismatches are counted here; unordered pairs are counted by the caller.
template <bool NOINF>
__device__ __forceinline__ float elem_verdict(float A, float B, float rtol, float atol, float R, float Rup,
                                              LaneAcc &acc, uint64_t &cand, float &tmax)
{
    const float d0 = __builtin_fabsf(A - B);
    const float ab = __builtin_fabsf(B);
    const float d = NOINF ? d0 : ((A == B) ? 0.0f : d0);
    const float rt = rtol * ab;
    const float thr = NOINF ? atol + rt : __builtin_fminf(atol + rt, 0x1.fffffep127f);
    acc.mism += (d <= thr) ? 0u : 1u;
    if constexpr (NOINF) tmax = __builtin_fmaxf(tmax, __builtin_fmaf(d, Rup, -ab));
    else cand |= __ballot(d >= __builtin_fmaxf(R * ab, kMinPositive));
    return d;
}

// One element with its exact ratio update and unordered count; returns d.
// Used for the n mod E tail.
template <bool NOINF>
__device__ __forceinline__ float check_elem(float A, float B, float rtol, float atol, LaneAcc &acc)
{
    uint64_t cand = 0;
    float tmax = 0.0f;
    const float d = elem_verdict<NOINF>(A, B, rtol, atol, kRatioFloor, 0.0f, acc, cand, tmax);
    acc.wnan += popc(__ballot(__builtin_isunordered(A, B)));
    ratio_update(A, B, acc);
    return d;
}

// The same d, for re-reading the best chunk.
__device__ __forceinline__ float elem_d(float A, float B)
{
    return (A == B) ? 0.0f : __builtin_fabsf(A - B);
}

// Elements of a chunk: one 16-byte vector of the narrower operand.
template <int DA, int DB>
constexpr int chunk_elems()
{
    return 16 / (dtype_traits<DA>::size < dtype_traits<DB>::size ? dtype_traits<DA>::size : dtype_traits<DB>::size);
}

// The E elements of a chunk widened to fp32 from the little-endian words of
// its 16-byte vectors. fp8 elements are converted two at a time straight
// from their 32-bit words (the packed converter's half-word select: no
// shifts or masks).
template <int DT, int NW, int E>
__device__ __forceinline__ void widen_words(const uint32_t (&w)[NW], const typename dtype_traits<DT>::storage (&s)[E],
                                            float (&X)[E])
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

// The candidate operand's chunk c: E elements in VA 16-byte vectors.
template <int DA, int E>
struct ChunkA {
    using TA = typename dtype_traits<DA>::storage;
    static constexpr int VA = E * dtype_traits<DA>::size / 16;
    union Raw {
        uint4 v[VA];
        uint32_t w[4 * VA];
        TA s[E];
    };

    __device__ __forceinline__ static void load_raw(const uint8_t *a, uint64_t c, Raw &r)
    {
#pragma unroll
        for (int i = 0; i < VA; ++i) r.v[i] = load16_stream(a + (c * VA + i) * 16);
    }
    __device__ __forceinline__ static void values(const Raw &r, float (&A)[E]) { widen_words<DA, 4 * VA, E>(r.w, r.s, A); }
    __device__ __forceinline__ static float elem(const uint8_t *a, uint64_t i)
    {
        return widen<DA>(reinterpret_cast<const TA *>(a)[i]);
    }
};

// Reference operand in memory (dtype DB, 16-byte aligned in the vector path).
// The interface every reference source gives the check body:
//   Raw, load_raw(c, raw)   the chunk's bytes, loaded ahead in the ring;
//   values(raw, c, B)       chunk c widened, from its raw bytes;
//   elems(c, B)             chunk c widened, outside the ring and for
//                           unaligned operands;
//   elem(i)                 element i widened (the n mod E tail).
template <int DB, int E>
struct RefMem {
    using TB = typename dtype_traits<DB>::storage;
    static constexpr int VB = E * dtype_traits<DB>::size / 16;
    union Raw {
        uint4 v[VB];
        uint32_t w[4 * VB];
        TB s[E];
    };
    const uint8_t *b;

    __device__ __forceinline__ void load_raw(uint64_t c, Raw &r) const
    {
#pragma unroll
        for (int i = 0; i < VB; ++i) r.v[i] = load16_stream(b + (c * VB + i) * 16);
    }
    __device__ __forceinline__ void values(const Raw &r, uint64_t, float (&B)[E]) const
    {
        widen_words<DB, 4 * VB, E>(r.w, r.s, B);
    }
    __device__ __forceinline__ void elems(uint64_t c, float (&B)[E]) const
    {
#pragma unroll
        for (int e = 0; e < E; ++e) B[e] = elem(c * E + e);
    }
    __device__ __forceinline__ float elem(uint64_t i) const { return widen<DB>(reinterpret_cast<const TB *>(b)[i]); }
};

// Reference regenerated from its word stream: element i is the value
// generation writes for word offset + i (Philox block (offset + i) / 4, lane
// (offset + i) mod 4, the distribution's transform, round to DB), read back
// as fp32. Nothing is loaded. p1 holds what generation's transform takes:
// the range fl(hi - lo), c = range 2^-24 when POW2, or the std.
template <int DB, int DIST, bool POW2, int E>
struct RefGen {
    using TB = typename dtype_traits<DB>::storage;
    static constexpr int NW = E * dtype_traits<DB>::size / 4;
    struct Raw {};
    uint64_t offset;    // word of element 0
    RoundKeys rk;       // the seed's Philox key schedule
    float p0, p1;
    uint32_t shift;     // offset mod 4

    // Round each value to DB and widen it back, as the stored reference
    // would read (pairs and quads through the packed conversions).
    __device__ __forceinline__ static void finish(const float (&v)[E], float (&B)[E])
    {
        union {
            uint32_t w[NW];
            TB s[E];
        } u;
        pack_narrow<DB, DIST == BITCAST>(v, u.w);
        widen_words<DB, NW, E>(u.w, u.s, B);
    }
    __device__ __forceinline__ void load_raw(uint64_t, Raw &) const {}
    // Chunk c when offset is a multiple of 4: E / 4 whole Philox blocks.
    __device__ __forceinline__ void values(const Raw &, uint64_t c, float (&B)[E]) const
    {
        const uint64_t b0 = (offset >> 2) + c * (E / 4);
        float v[E];
#pragma unroll
        for (int k = 0; k < E / 4; ++k) transform4<DIST, POW2>(philox_block(b0 + k, rk), p0, p1, v + 4 * k);
        finish(v, B);
    }
    // Any offset: the E / 4 + 1 blocks the chunk's words touch, the values
    // taken from position shift on (a wave-uniform choice).
    __device__ __forceinline__ void elems(uint64_t c, float (&B)[E]) const
    {
        const uint64_t b0 = (offset >> 2) + c * (E / 4);
        float v[E + 4];
#pragma unroll
        for (int k = 0; k < E / 4 + 1; ++k) transform4<DIST, POW2>(philox_block(b0 + k, rk), p0, p1, v + 4 * k);
        float x[E];
#pragma unroll
        for (int e = 0; e < E; ++e)
            x[e] = shift == 0 ? v[e] : shift == 1 ? v[e + 1] : shift == 2 ? v[e + 2] : v[e + 3];
        finish(x, B);
    }
    __device__ __forceinline__ float elem(uint64_t i) const
    {
        const uint64_t w = offset + i;
        float v[4];
        transform4<DIST, POW2>(philox_block(w >> 2, rk), p0, p1, v);
        const uint32_t l = (uint32_t)w & 3u;
        const float x = l == 0 ? v[0] : l == 1 ? v[1] : l == 2 ? v[2] : v[3];
        return widen<DB>(narrow<DB, DIST == BITCAST>(x));
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
// Reference regenerated from the packed stream (krex_gen_packed): element i
// is field offset + i, position (offset + i) mod EP of packed unit
// (offset + i) / EP (EP = 16 / size of DB fields per unit), read back as
// fp32. A chunk holds E / EP units' worth of fields; p0, p1 and rs are the
// packed transform's constants and UM its uniform mode.
template <int DB, int DIST, int UM, int E>
struct RefGenPacked {
    using TB = typename dtype_traits<DB>::storage;
    static constexpr int SB = dtype_traits<DB>::size;
    static constexpr int EP = packed_of<DB, DIST>::E;
    static constexpr int NU = E / EP;        // units per chunk
    static constexpr int NW = 4 * NU;        // words per chunk
    static constexpr int PER = 4 / SB;       // fields per word
    static_assert(E % EP == 0, "a chunk holds whole units");
    struct Raw {};
    uint64_t offset;    // field of element 0
    RoundKeys rk;
    float p0, p1, rs;

    __device__ __forceinline__ static void widen_chunk(const uint32_t (&w)[NW], float (&B)[E])
    {
        union {
            uint32_t w[NW];
            TB s[E];
        } u;
#pragma unroll
        for (int j = 0; j < NW; ++j) u.w[j] = w[j];
        widen_words<DB, NW, E>(u.w, u.s, B);
    }
    __device__ __forceinline__ void load_raw(uint64_t, Raw &) const {}
    // Chunk c when offset is a multiple of EP: NU whole units.
    __device__ __forceinline__ void values(const Raw &, uint64_t c, float (&B)[E]) const
    {
        const uint64_t u0 = offset / EP + c * NU;
        uint32_t w[NW];
#pragma unroll
        for (int k = 0; k < NU; ++k) {
            uint32_t w4[4];
            packed_unit<DB, DIST, UM>(u0 + k, rk, p0, p1, rs, w4);
#pragma unroll
            for (int l = 0; l < 4; ++l) w[4 * k + l] = w4[l];
        }
        widen_chunk(w, B);
    }
    // Any offset: the NU + 1 units the chunk's fields touch, shifted by
    // s = offset mod EP fields (s / PER words, then a funnel shift of the
    // rest; s is wave-uniform).
    __device__ __forceinline__ void elems(uint64_t c, float (&B)[E]) const
    {
        const uint64_t u0 = (offset + c * E) / EP;
        const uint32_t s = (uint32_t)(offset % EP);
        uint32_t w[NW + 4];
#pragma unroll
        for (int k = 0; k < NU + 1; ++k) {
            uint32_t w4[4];
            packed_unit<DB, DIST, UM>(u0 + k, rk, p0, p1, rs, w4);
#pragma unroll
            for (int l = 0; l < 4; ++l) w[4 * k + l] = w4[l];
        }
        const uint32_t ws = s / PER, bs = (s % PER) * 8 * SB;
        uint32_t o[NW];
#pragma unroll
        for (int j = 0; j < NW; ++j) {
            const uint32_t lo = ws == 0 ? w[j] : ws == 1 ? w[j + 1] : ws == 2 ? w[j + 2] : w[j + 3];
            const uint32_t hi = ws == 0 ? w[j + 1] : ws == 1 ? w[j + 2] : ws == 2 ? w[j + 3] : w[j + 4];
            o[j] = __builtin_amdgcn_alignbit(hi, lo, bs);   // (hi:lo) >> bs, bs < 32
        }
        widen_chunk(o, B);
    }
    __device__ __forceinline__ float elem(uint64_t i) const
    {
        const uint64_t q = offset + i;
        uint32_t w4[4];
        packed_unit<DB, DIST, UM>(q / EP, rk, p0, p1, rs, w4);
        const uint32_t k = (uint32_t)(q % EP);
        const uint32_t wk = k / PER;
        const uint32_t word = wk == 0 ? w4[0] : wk == 1 ? w4[1] : wk == 2 ? w4[2] : w4[3];
        const uint32_t bits = (word >> (8 * SB * (k % PER))) & ((SB == 2) ? 0xFFFFu : 0xFFu);
        return widen<DB>(bits);
    }
};

template <int E>
struct RatioFilter {
    float R = kRatioFloor;
    // An upper bound of 1/R, at least (1/R)(1 + 2^-21): fl(1/R) (correctly
    // rounded) times 1 + 2^-20. For fp8 pairs an element with ratio
    // d/|b| > R has d Rup > |b| exactly, so fma(d, Rup, -|b|), the rounded
    // exact residual, is positive (no underflow to zero: d and |b| are
    // multiples of 2^-9 and Rup, at least 2^-20 when finite R <= 896 2^9, a
    // multiple of 2^-43, so a nonzero residual is at least 2^-52); an
    // element whose residual is not positive has ratio
    // <= R, below the maximum, and is skipped. R = +inf gives Rup = 0.
    float Rup = 0x1.00001p32f;

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
        Rup = (1.0f / R) * 0x1.00001p0f;
    }
};

// The check of n elements of the candidate a (dtype DA) against the
// reference source ref (dtype DB); block partials into
// partials[blockIdx.x]. VEC: a is 16-byte aligned and ref takes its vector
// path (a ring of D chunk buffers in flight); otherwise element loads.
template <int DA, int DB, bool VEC, int D, class Ref>
__device__ __forceinline__ void check_body(const uint8_t *a, const Ref &ref, uint64_t n, float rtol, float atol,
                                           CheckPartial *partials, uint32_t U)
{
    constexpr int E = chunk_elems<DA, DB>();
    using CA = ChunkA<DA, E>;
    struct Slot {
        typename CA::Raw a;
        typename Ref::Raw b;
    };
    // Chunk c of both operands, outside the ring.
    auto load_chunk = [&](uint64_t c, float (&A)[E], float (&B)[E]) {
        if constexpr (VEC) {
            Slot r;
            CA::load_raw(a, c, r.a);
            ref.load_raw(c, r.b);
            CA::values(r.a, A);
            ref.values(r.b, c, B);
        } else {
#pragma unroll
            for (int e = 0; e < E; ++e) A[e] = CA::elem(a, c * E + e);
            ref.elems(c, B);
        }
    };
    const uint32_t t = threadIdx.x;
    const uint64_t nchunks = n / E;
    const uint64_t base = (uint64_t)blockIdx.x * kThreads * U;
    LaneAcc acc{0u, 0u, 0.0f, 1.0f};
    RatioFilter<E> rf;
    float best_d = -1.0f;               // largest non-NaN d seen by this lane
    uint32_t best_c = 0;                // its chunk
    constexpr bool NOINF = DA == F8 && DB == F8;
    // Counts and |a - b| maximum of one chunk; returns the lanes of the wave
    // whose chunk has a max_rel candidate. The chunk's maximum of d is taken
    // with the NaN-propagating maximum, so it is NaN exactly when some pair
    // is unordered (d is NaN only then); those rare chunks count their
    // unordered pairs and take the maximum again without them.
    auto process = [&](const float (&A)[E], const float (&B)[E], uint64_t c) -> uint64_t {
        float cmax = -1.0f;
        float tmax = 0.0f;
        uint64_t cand = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const float d = elem_verdict<NOINF>(A[e], B[e], rtol, atol, rf.R, rf.Rup, acc, cand, tmax);
            cmax = __builtin_elementwise_maximum(cmax, d);
        }
        if constexpr (NOINF) cand = __ballot(tmax > 0.0f);
        // the counts are complete here: kept from being moved past the rare
        // branch below, where their operands would need extra registers
        __asm__ volatile("" : "+v"(acc.mism));
        if (__ballot(cmax != cmax) != 0) {
#pragma unroll
            for (int e = 0; e < E; ++e) acc.wnan += popc(__ballot(__builtin_isunordered(A[e], B[e])));
            if (cmax != cmax) {
                cmax = -1.0f;           // the maximum without the unordered pairs
#pragma unroll
                for (int e = 0; e < E; ++e) cmax = __builtin_fmaxf(cmax, elem_d(A[e], B[e]));
            }
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
            Slot r[D];
            auto ring_load = [&](uint64_t c, Slot &s) {
                CA::load_raw(a, c, s.a);
                ref.load_raw(c, s.b);
            };
#pragma unroll
            for (int k = 0; k < D - 1; ++k) ring_load(hj(k) ? cj(k) : last, r[k]);
            for (uint32_t u = 0; u < U; u += D) {
#pragma unroll
                for (int k = 0; k < D; ++k) {
                    const uint32_t jn = u + k + D - 1;
                    ring_load(hj(jn) ? cj(jn) : last, r[(k + D - 1) % D]);
                    const uint32_t j = u + k;
                    const bool h = hj(j);
                    float A[E], B[E];   // read only where h holds
                    uint64_t cand = 0;
                    if (h) {
                        CA::values(r[k].a, A);
                        ref.values(r[k].b, cj(j), B);
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
                load_chunk(c, A, B);
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
        const float A = CA::elem(a, i);
        const float B = ref.elem(i);
        const float d = check_elem<NOINF>(A, B, rtol, atol, acc);
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
        load_chunk(best_c, A, B);
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
    uint32_t wm = acc.mism;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) wm += __shfl_xor(wm, off, 64);
    const uint32_t wn = __shfl(acc.wnan, 0, 64);
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

// ------------------------------------------------------------ host helpers

// Blocks of `kern` (kThreads threads) the current device holds at once, at
// most per_cu_cap per compute unit (0: no cap; KREX_CHECK_BLOCKS_PER_CU
// overrides a nonzero cap), capped at the partial buffer's capacity; cached
// per device in `cache`.
inline uint32_t resident_blocks(const void *kern, uint32_t (&cache)[64], uint32_t per_cu_cap = 0)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = -1;
    if (dev >= 0 && cache[dev]) return cache[dev];
    int per_cu = 0, cus = 0;
    uint32_t r = kMaxCheckBlocks / 2;
    static const uint32_t cap_env = tune_env("KREX_CHECK_BLOCKS_PER_CU", 0);
    if (per_cu_cap && cap_env) per_cu_cap = cap_env;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kThreads, 0) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev < 0 ? 0 : dev) == hipSuccess &&
        per_cu > 0 && cus > 0) {
        if (per_cu_cap && (uint32_t)per_cu > per_cu_cap) per_cu = (int)per_cu_cap;
        r = (uint32_t)per_cu * (uint32_t)cus;
    }
    if (r > (uint32_t)kMaxCheckBlocks) r = kMaxCheckBlocks;
    if (dev >= 0) cache[dev] = r;
    return r;
}

// Grid of a check launch over nchunks chunks: one resident round (the grid
// is at most the blocks the device holds at once, so no partial last round
// idles most of the chip). Chunks per thread U: enough to cover n with that
// grid, and at least KREX_CHECK_U (default 8: the pipeline's depth per lane,
// and fewer partials for small n). G >= 1 (the tail alone).
inline void check_grid(uint64_t nchunks, uint64_t resident, uint32_t *U_out, uint32_t *G_out)
{
    static const uint32_t u_floor = tune_env("KREX_CHECK_U", 8);
    uint64_t U = (nchunks + (uint64_t)kThreads * resident - 1) / ((uint64_t)kThreads * resident);
    if (U < u_floor) U = u_floor;
    if (U == 0) U = 1;
    uint64_t G = (nchunks + (uint64_t)kThreads * U - 1) / ((uint64_t)kThreads * U);
    if (G == 0) G = 1;
    *U_out = (uint32_t)U;
    *G_out = (uint32_t)G;
}

// The result record from the partials of `nblocks` check blocks (n = 0:
// none), launched after the check kernel on the same stream.
hipError_t launch_check_final(const CheckPartial *partials, uint32_t nblocks, uint64_t n, krex_check_result *out,
                              hipStream_t s);

}  // namespace krex
