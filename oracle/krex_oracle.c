/*
 * krex_oracle.c -- CPU oracle for the device-side hot path of a kernel
 * benchmarking command: seeded input generation, mismatch injection, the
 * allclose correctness check with its error reductions, the cache-flush
 * fill, the FMA probe and the fp32 reference GEMM of the tiny GEMM command.
 *
 * TEST INFRASTRUCTURE. Only the test suite, the smoke entry point and the
 * benchmark's cpu_baseline leg may load this library. The product path
 * (paper_2609_30057_amd) never calls it, and the two share no source: this
 * file includes nothing from the product and the product includes nothing
 * from here.
 *
 * Form: plain, single-threaded, scalar C99. Build flags: -O2
 * -ffp-contract=off -fno-fast-math, so every float operation below is one
 * IEEE-754 binary32 operation rounded to nearest-even, and an fused
 * multiply-add happens only where fmaf() is written out.
 *
 * What the paper fixes and what is read into it. The paper (KREX,
 * "Concurrent Kernel Benchmarking on Shared GPUs via Region-Granular
 * Exclusivity") describes this work only in prose: a command generates
 * inputs and checks its result against a reference before it times the
 * kernel (Section 1; Section 2.1, "Kernel agent" and "Benchmarking
 * command"); timing is warm-up, repeated timed launches and a median, with
 * a cache flush between iterations (Section 2.1); region entry flushes the
 * cache with a memset over a cache-sized buffer (Section 4.2, step 5); and
 * colocated work must not change the generated tensors or the verdict
 * (Section 2.1, "Benchmarking command"). It names no RNG, no tolerance
 * rule and no reduction. The definitions here are this project's readings:
 *
 *   words    W_s[w] = lane (w mod 4) of Philox4x32-10 (Salmon, Moraes, Dror,
 *            Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3", SC'11)
 *            with key (s mod 2^32, s >> 32) and counter
 *            (b mod 2^32, b >> 32, 0, 0), b = w >> 2. Element j of a tensor
 *            generated at offset o uses word o + j.
 *   uniform  u = (W >> 8) * 2^-24;  v = lo + (hi - lo) * u, two roundings.
 *   normal   Box & Muller (1958) on the word pair (2p, 2p + 1), p = w >> 1,
 *            with this file's own fp32 ln, sin/cos(2 pi k / 2^24) and the
 *            IEEE square root; element w takes the cosine branch if w is
 *            even, the sine branch if odd; v = mu + sigma * z.
 *   bitcast  v = the word's 32 bits read as an fp32 value (any pattern).
 *   convert  fp32 -> bf16 / fp16 / fp8-e4m3fn, round to nearest even,
 *            subnormals kept; fp8 is non-saturating (beyond 448 -> NaN).
 *   check    b is the reference: per element, upcast both to fp32; NaN on
 *            either side is a mismatch counted in nan_count and left out of
 *            the maxima; equal values are close with d = 0, rel = 0; else an
 *            infinity on either side is a mismatch with d = rel = +inf; else
 *            d = |A - B|, close iff d is finite and d <= atol + rtol * |B|
 *            (two roundings), rel = d / |B|. Reported: mismatch count, NaN count, max d with
 *            the lowest index attaining it, max rel.
 *   inject   mask_i = [W_mseed[moff + i] < floor(rate * 2^32)]; ROUND mode
 *            y = cvt(x + delta); EXACT mode perturbs by exactly +delta, else
 *            exactly -delta, else leaves the element untouched.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define KO_F32 0
#define KO_BF16 1
#define KO_F16 2
#define KO_F8E4M3 3
#define KO_U32 4

#define KO_UNIFORM 0
#define KO_NORMAL 1
#define KO_BITCAST 2

#define KO_INJ_ROUND 0
#define KO_INJ_EXACT 1

#define KO_OK 0
#define KO_EINVAL (-1)

static uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

static size_t dtype_size(int dt)
{
    switch (dt) {
    case KO_F32: return 4;
    case KO_BF16: return 2;
    case KO_F16: return 2;
    case KO_F8E4M3: return 1;
    case KO_U32: return 4;
    default: return 0;
    }
}

/* ------------------------------------------------------------------------
 * Philox4x32-10, straight from the SC'11 definition: ten rounds; each round
 * forms the two 64-bit products M0 * x0 and M1 * x2 and permutes
 *   (x0, x1, x2, x3) <- (hi(M1 x2) ^ x1 ^ k0, lo(M1 x2), hi(M0 x0) ^ x3 ^ k1, lo(M0 x0))
 * and the key is bumped by the Weyl constants between rounds.
 * ---------------------------------------------------------------------- */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void ko_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)x0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)x2;
        uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
        uint32_t y1 = (uint32_t)p1;
        uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
        uint32_t y3 = (uint32_t)p0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
        k0 += PHILOX_W0;
        k1 += PHILOX_W1;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* One word of the stream W_seed. */
uint32_t ko_word(uint64_t seed, uint64_t w)
{
    uint64_t b = w >> 2;
    uint32_t ctr[4] = {(uint32_t)b, (uint32_t)(b >> 32), 0u, 0u};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t out[4];
    ko_philox4x32_10(ctr, key, out);
    return out[w & 3u];
}

/* Words W_seed[offset .. offset + n). A one-block cache avoids running the
 * same Philox block four times; the result is the same as ko_word per
 * element. */
void ko_words(uint32_t *dst, uint64_t n, uint64_t seed, uint64_t offset)
{
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint64_t cached = 0;
    int have = 0;
    uint32_t out[4];
    for (uint64_t j = 0; j < n; ++j) {
        uint64_t w = offset + j;
        uint64_t b = w >> 2;
        if (!have || b != cached) {
            uint32_t ctr[4] = {(uint32_t)b, (uint32_t)(b >> 32), 0u, 0u};
            ko_philox4x32_10(ctr, key, out);
            cached = b;
            have = 1;
        }
        dst[j] = out[w & 3u];
    }
}

/* ------------------------------------------------------------------------
 * Conversions. Narrowing is round-to-nearest-even with subnormals kept.
 * A NaN input gives the format's one canonical NaN (bf16 0x7FC0, fp16
 * 0x7E00, fp8 0x7F), whatever its sign and payload: IEEE-754 does not fix
 * the sign or payload a NaN keeps through arithmetic, so only a canonical
 * encoding makes a NaN result reproducible across machines. fp8-e4m3fn has
 * no infinity: infinity and any value whose rounded magnitude would exceed
 * 448 give 0x7F with the input's sign.
 * ---------------------------------------------------------------------- */
uint16_t ko_f32_to_bf16(float f)
{
    uint32_t x = f2u(f);
    if ((x & 0x7FFFFFFFu) > 0x7F800000u)
        return 0x7FC0u;
    /* Nearest-even on the 16 discarded bits: add 0x7FFF plus the bit that
     * will become the last kept bit; a carry out of the mantissa bumps the
     * exponent, which also turns the largest finite values into infinity. */
    uint32_t lsb = (x >> 16) & 1u;
    x += 0x7FFFu + lsb;
    return (uint16_t)(x >> 16);
}

/* Round m / 2^s to nearest even (s >= 1, m < 2^25). */
static uint32_t rne_shift(uint32_t m, int s)
{
    if (s >= 32)
        return 0;
    uint32_t q = m >> s;
    uint32_t rem = m & ((1u << s) - 1u);
    uint32_t half = 1u << (s - 1);
    if (rem > half || (rem == half && (q & 1u)))
        q += 1u;
    return q;
}

uint16_t ko_f32_to_f16(float f)
{
    uint32_t x = f2u(f);
    uint16_t sign = (uint16_t)((x >> 16) & 0x8000u);
    uint32_t ax = x & 0x7FFFFFFFu;
    if (ax > 0x7F800000u)
        return 0x7E00u;
    if (ax >= 0x477FF000u)          /* >= 65520: rounds past 65504 */
        return (uint16_t)(sign | 0x7C00u);
    if (ax >= 0x38800000u) {        /* >= 2^-14: a normal half */
        uint32_t lsb = (ax >> 13) & 1u;
        uint32_t r = ax + 0xFFFu + lsb;
        return (uint16_t)(sign | ((r - (112u << 23)) >> 13));
    }
    /* Below 2^-14: the result counts units of 2^-24. |f| = m * 2^(e - 150)
     * with the implicit bit in m, so |f| / 2^-24 = m / 2^(126 - e). */
    uint32_t e = ax >> 23;
    if (e == 0)                     /* fp32 subnormal: far below 2^-25 */
        return sign;
    uint32_t m = (ax & 0x7FFFFFu) | 0x800000u;
    return (uint16_t)(sign | rne_shift(m, (int)(126u - e)));
}

uint8_t ko_f32_to_f8e4m3(float f)
{
    uint32_t x = f2u(f);
    uint8_t sign = (uint8_t)((x >> 24) & 0x80u);
    uint32_t ax = x & 0x7FFFFFFFu;
    if (ax > 0x7F800000u)           /* NaN: the canonical NaN */
        return 0x7Fu;
    if (ax > 0x43E80000u)           /* inf, or > 464: rounds to 480+ */
        return (uint8_t)(sign | 0x7Fu);
    if (ax >= 0x3C800000u) {        /* >= 2^-6: a normal e4m3 value */
        uint32_t lsb = (ax >> 20) & 1u;
        uint32_t r = ax + 0x7FFFFu + lsb;
        return (uint8_t)(sign | ((r - (120u << 23)) >> 20));
    }
    /* Below 2^-6: units of 2^-9, |f| / 2^-9 = m / 2^(141 - e). */
    uint32_t e = ax >> 23;
    if (e == 0)
        return sign;
    uint32_t m = (ax & 0x7FFFFFu) | 0x800000u;
    return (uint8_t)(sign | rne_shift(m, (int)(141u - e)));
}

float ko_bf16_to_f32(uint16_t h) { return u2f((uint32_t)h << 16); }

float ko_f16_to_f32(uint16_t h)
{
    uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
    uint32_t e = (h >> 10) & 0x1Fu;
    uint32_t m = h & 0x3FFu;
    if (e == 0x1Fu)
        return u2f(sign | 0x7F800000u | (m << 13));
    if (e == 0) {
        float v = (float)m * 0x1p-24f;
        return sign ? -v : v;
    }
    return u2f(sign | ((e + 112u) << 23) | (m << 13));
}

float ko_f8e4m3_to_f32(uint8_t h)
{
    uint32_t sign = (uint32_t)(h & 0x80u) << 24;
    uint32_t e = (h >> 3) & 0xFu;
    uint32_t m = h & 0x7u;
    if (e == 0xFu && m == 0x7u)
        return u2f(sign | 0x7FC00000u);
    if (e == 0) {
        float v = (float)m * 0x1p-9f;
        return sign ? -v : v;
    }
    return u2f(sign | ((e + 120u) << 23) | (m << 20));
}

static float load_f32(const void *p, int dt, uint64_t i)
{
    switch (dt) {
    case KO_F32: return ((const float *)p)[i];
    case KO_BF16: return ko_bf16_to_f32(((const uint16_t *)p)[i]);
    case KO_F16: return ko_f16_to_f32(((const uint16_t *)p)[i]);
    default: return ko_f8e4m3_to_f32(((const uint8_t *)p)[i]);
    }
}

static void store_f32(void *p, int dt, uint64_t i, float v)
{
    switch (dt) {
    case KO_F32: ((float *)p)[i] = v; break;
    case KO_BF16: ((uint16_t *)p)[i] = ko_f32_to_bf16(v); break;
    case KO_F16: ((uint16_t *)p)[i] = ko_f32_to_f16(v); break;
    default: ((uint8_t *)p)[i] = ko_f32_to_f8e4m3(v); break;
    }
}

/* fp32 -> dtype -> fp32 */
static float round_trip(float v, int dt)
{
    switch (dt) {
    case KO_F32: return v;
    case KO_BF16: return ko_bf16_to_f32(ko_f32_to_bf16(v));
    case KO_F16: return ko_f16_to_f32(ko_f32_to_f16(v));
    default: return ko_f8e4m3_to_f32(ko_f32_to_f8e4m3(v));
    }
}

/* Bulk conversions for the pin tests. */
void ko_convert_from_f32(void *dst, int dt, const float *src, uint64_t n)
{
    for (uint64_t i = 0; i < n; ++i)
        store_f32(dst, dt, i, src[i]);
}

void ko_convert_to_f32(float *dst, const void *src, int dt, uint64_t n)
{
    for (uint64_t i = 0; i < n; ++i)
        dst[i] = load_f32(src, dt, i);
}

/* ------------------------------------------------------------------------
 * Value transforms.
 * ---------------------------------------------------------------------- */

/* Uniform [lo, hi): u on the 2^-24 grid, then lo + (hi - lo) * u with two
 * separate roundings. */
float ko_uniform(uint32_t word, float lo, float hi)
{
    float u = (float)(word >> 8) * 0x1p-24f;
    float r = hi - lo;
    float t = r * u;
    return lo + t;
}

/* Natural log of a positive normal x. x = 2^e * m with m in
 * [sqrt(1/2), sqrt(2)); with f = m - 1 and s = f / (2 + f),
 * ln m = 2 atanh(s) = 2s + s R(s^2), R(z) = sum_{k>=1} 2 z^k / (2k + 1),
 * truncated after z^5 (|s| < 0.172, so the first dropped term is below
 * 1e-10 relative). Since 2s = f - s f and s f = f^2/2 - s f^2/2, the sum is
 * evaluated as f - (f^2/2 - s (f^2/2 + R)), which keeps the exact f as the
 * leading term. ln 2 is split into a 16-bit head (so e * head is exact for
 * |e| < 256) and an fp32 tail. */
#define LN_C1 0x1.555556p-1f   /* 2/3  */
#define LN_C2 0x1.99999ap-2f   /* 2/5  */
#define LN_C3 0x1.24924ap-2f   /* 2/7  */
#define LN_C4 0x1.c71c72p-3f   /* 2/9  */
#define LN_C5 0x1.745d18p-3f   /* 2/11 */
#define LN2_HEAD 0x1.62e4p-1f
#define LN2_TAIL 0x1.7f7d1cp-20f

float ko_ln(float x)
{
    uint32_t ix = f2u(x);
    int32_t e = (int32_t)(ix >> 23) - 127;
    uint32_t mb = ix & 0x7FFFFFu;
    float m = u2f(mb | 0x3F800000u);        /* [1, 2) */
    if (mb > 0x3504F3u) {                   /* m > fp32(sqrt 2) */
        m = m * 0.5f;
        e = e + 1;
    }
    float f = m - 1.0f;                     /* exact (Sterbenz) */
    float den = 2.0f + f;
    float s = f / den;
    float z = s * s;
    float p = LN_C5;
    p = fmaf(p, z, LN_C4);
    p = fmaf(p, z, LN_C3);
    p = fmaf(p, z, LN_C2);
    p = fmaf(p, z, LN_C1);
    float R = z * p;
    float hf = 0.5f * f;
    float hfsq = hf * f;
    float a = hfsq + R;
    float b = s * a;
    float c = hfsq - b;
    float lnm = f - c;
    float dk = (float)e;
    float tail = fmaf(dk, LN2_TAIL, lnm);
    float head = dk * LN2_HEAD;
    return head + tail;
}

/* sin and cos of 2 pi k / 2^24 for an integer k in [0, 2^24). The angle is
 * (pi/2)(q + r) with q = round(k / 2^22) and r = (k - q 2^22) / 2^22 in
 * [-1/2, 1/2); both steps are exact integer arithmetic. S(r) = sin(pi r / 2)
 * and C(r) = cos(pi r / 2) are their Taylor polynomials through r^9 and
 * r^10 (for |pi r / 2| <= pi/4 the next terms are below 2^-28 relative),
 * evaluated by Horner's rule in r^2 with fmaf. The quadrant q mod 4 then
 * swaps and negates: (sin, cos) = (S, C), (C, -S), (-S, -C), (-C, S). */
#define SN_1 0x1.921fb6p+0f
#define SN_3 (-0x1.4abbcep-1f)
#define SN_5 0x1.466bc6p-4f
#define SN_7 (-0x1.32d2ccp-8f)
#define SN_9 0x1.507834p-13f
#define CS_2 (-0x1.3bd3ccp+0f)
#define CS_4 0x1.03c1f0p-2f
#define CS_6 (-0x1.55d3c8p-6f)
#define CS_8 0x1.e1f506p-11f
#define CS_10 (-0x1.a6d1f2p-16f)

void ko_sincos_2pi_q24(uint32_t k, float *sn, float *cs)
{
    uint32_t q = (k + (1u << 21)) >> 22;    /* 0..4 */
    int32_t ri = (int32_t)k - (int32_t)(q << 22);
    float r = (float)ri * 0x1p-22f;          /* exact */
    float y = r * r;
    float ps = SN_9;
    ps = fmaf(ps, y, SN_7);
    ps = fmaf(ps, y, SN_5);
    ps = fmaf(ps, y, SN_3);
    ps = fmaf(ps, y, SN_1);
    float S = r * ps;
    float pc = CS_10;
    pc = fmaf(pc, y, CS_8);
    pc = fmaf(pc, y, CS_6);
    pc = fmaf(pc, y, CS_4);
    pc = fmaf(pc, y, CS_2);
    float C = fmaf(pc, y, 1.0f);
    switch (q & 3u) {
    case 0: *sn = S; *cs = C; break;
    case 1: *sn = C; *cs = -S; break;
    case 2: *sn = -S; *cs = -C; break;
    default: *sn = -C; *cs = S; break;
    }
}

/* Box-Muller on one word pair: u1 = ((w0 >> 8) + 1) 2^-24 in (0, 1],
 * rho = sqrt(0 - 2 ln u1) (the subtraction from +0 makes rho = +0, not -0,
 * at u1 = 1), angle 2 pi (w1 >> 8) 2^-24. z0 = rho cos, z1 = rho sin. */
void ko_normal_pair(uint32_t w0, uint32_t w1, float *z0, float *z1)
{
    float u1 = (float)((w0 >> 8) + 1u) * 0x1p-24f;
    float L = ko_ln(u1);
    float t2 = 2.0f * L;
    float t = 0.0f - t2;
    float rho = sqrtf(t);
    float sn, cs;
    ko_sincos_2pi_q24(w1 >> 8, &sn, &cs);
    *z0 = rho * cs;
    *z1 = rho * sn;
}

/* ------------------------------------------------------------------------
 * Generation: element j of dst gets word offset + j, transformed and
 * rounded to dt. KO_U32 stores the raw words.
 * ---------------------------------------------------------------------- */
static int params_ok(int dist, float p0, float p1)
{
    if (dist == KO_UNIFORM)
        return isfinite(p0) && isfinite(p1) && p0 <= p1 && isfinite(p1 - p0);
    if (dist == KO_NORMAL)
        return isfinite(p0) && isfinite(p1) && p1 >= 0.0f;
    return dist == KO_BITCAST;
}

int ko_gen(void *dst, int dt, uint64_t n, uint64_t seed, uint64_t offset,
           int dist, float p0, float p1)
{
    if (dtype_size(dt) == 0)
        return KO_EINVAL;
    if (dt != KO_U32 && !params_ok(dist, p0, p1))
        return KO_EINVAL;
    if (n > 0 && offset > UINT64_MAX - (n - 1))
        return KO_EINVAL;
    for (uint64_t j = 0; j < n; ++j) {
        uint64_t w = offset + j;
        uint32_t W = ko_word(seed, w);
        if (dt == KO_U32) {
            ((uint32_t *)dst)[j] = W;
            continue;
        }
        float v;
        if (dist == KO_UNIFORM) {
            v = ko_uniform(W, p0, p1);
        } else if (dist == KO_BITCAST) {
            v = u2f(W);
        } else {
            uint64_t wp = w & ~(uint64_t)1;  /* first word of the pair */
            uint32_t w0 = ko_word(seed, wp);
            uint32_t w1 = ko_word(seed, wp + 1);
            float z0, z1;
            ko_normal_pair(w0, w1, &z0, &z1);
            float z = (w & 1u) ? z1 : z0;
            float sz = p1 * z;
            v = p0 + sz;
        }
        store_f32(dst, dt, j, v);
    }
    return KO_OK;
}

/* ------------------------------------------------------------------------
 * Packed stream: the narrow-dtype form of the generator, which spends w < 32
 * bits of the word stream per element. The stream is cut into w-bit fields,
 * low bits first: field q is bits [(q mod k) w, (q mod k) w + w) of word
 * W_s[q / k], k = 32 / w. w = 16 for bf16 and fp16 (every distribution)
 * and for fp8 normal; w = 8 for fp8 uniform and bitcast; fp32 and u32 have
 * no packed form. Element j of a tensor generated at field offset o uses
 * field q = o + j:
 *   uniform  the uniform transform above of the word f << (32 - w), i.e.
 *            u = f 2^-w;
 *   normal   the Box-Muller transform above of the word pair
 *            (f_{2p} << 16, f_{2p+1} << 16), p = q >> 1 (both fields lie in
 *            word p), the cosine branch for even q, the sine branch for odd
 *            q; v = mu + sigma z;
 *   bitcast  the element's bits are the field itself.
 * ---------------------------------------------------------------------- */
int ko_packed_width(int dt, int dist)
{
    if (dist != KO_UNIFORM && dist != KO_NORMAL && dist != KO_BITCAST)
        return 0;
    if (dt == KO_BF16 || dt == KO_F16)
        return 16;
    if (dt == KO_F8E4M3)
        return dist == KO_NORMAL ? 16 : 8;
    return 0;
}

/* Field q of the stream of seed. */
static uint32_t packed_field(uint64_t seed, uint64_t q, int w)
{
    uint64_t k = 32u / (unsigned)w;
    uint32_t W = ko_word(seed, q / k);
    uint32_t shift = (uint32_t)(q % k) * (uint32_t)w;
    uint32_t mask = (w == 32) ? 0xFFFFFFFFu : ((1u << w) - 1u);
    return (W >> shift) & mask;
}

int ko_gen_packed(void *dst, int dt, uint64_t n, uint64_t seed, uint64_t offset,
                  int dist, float p0, float p1)
{
    int w = ko_packed_width(dt, dist);
    if (w == 0 || !params_ok(dist, p0, p1))
        return KO_EINVAL;
    if (n > 0 && offset > UINT64_MAX - (n - 1))
        return KO_EINVAL;
    for (uint64_t j = 0; j < n; ++j) {
        uint64_t q = offset + j;
        uint32_t f = packed_field(seed, q, w);
        if (dist == KO_BITCAST) {
            if (w == 16)
                ((uint16_t *)dst)[j] = (uint16_t)f;
            else
                ((uint8_t *)dst)[j] = (uint8_t)f;
            continue;
        }
        float v;
        if (dist == KO_UNIFORM) {
            v = ko_uniform(f << (32 - w), p0, p1);
        } else {
            uint64_t qp = q & ~(uint64_t)1;  /* first field of the pair */
            uint32_t fa = packed_field(seed, qp, w);
            uint32_t fb = packed_field(seed, qp + 1, w);
            float z0, z1;
            ko_normal_pair(fa << 16, fb << 16, &z0, &z1);
            float z = (q & 1u) ? z1 : z0;
            float sz = p1 * z;
            v = p0 + sz;
        }
        store_f32(dst, dt, j, v);
    }
    return KO_OK;
}

/* The same transforms on caller-supplied words: element j uses words[j];
 * the normal pair of element j is (words[j & ~1], words[j | 1]). */
int ko_transform_words(void *dst, int dt, uint64_t n, const uint32_t *words,
                       int dist, float p0, float p1)
{
    if (dtype_size(dt) == 0)
        return KO_EINVAL;
    if (dt != KO_U32 && !params_ok(dist, p0, p1))
        return KO_EINVAL;
    if (dist == KO_NORMAL && dt != KO_U32 && (n & 1u))
        return KO_EINVAL;
    for (uint64_t j = 0; j < n; ++j) {
        uint32_t W = words[j];
        if (dt == KO_U32) {
            ((uint32_t *)dst)[j] = W;
            continue;
        }
        float v;
        if (dist == KO_UNIFORM) {
            v = ko_uniform(W, p0, p1);
        } else if (dist == KO_BITCAST) {
            v = u2f(W);
        } else {
            float z0, z1;
            ko_normal_pair(words[j & ~(uint64_t)1], words[j | 1u], &z0, &z1);
            float z = (j & 1u) ? z1 : z0;
            float sz = p1 * z;
            v = p0 + sz;
        }
        store_f32(dst, dt, j, v);
    }
    return KO_OK;
}

/* ------------------------------------------------------------------------
 * Mismatch injection. y may alias x.
 * ---------------------------------------------------------------------- */
uint64_t ko_inject_threshold(double rate)
{
    double t = floor(rate * 4294967296.0);
    if (t <= 0.0)
        return 0;
    if (t >= 4294967296.0)
        return (uint64_t)1 << 32;
    return (uint64_t)t;
}

/* Returns the number of elements actually perturbed (EXACT mode may leave a
 * masked element untouched), or a negative error code. */
int64_t ko_inject(void *y, const void *x, int dt, uint64_t n, uint64_t mseed,
                  uint64_t moff, double rate, float delta, int mode)
{
    if (dtype_size(dt) == 0 || dt == KO_U32)
        return KO_EINVAL;
    if (!(rate >= 0.0 && rate <= 1.0) || (mode != KO_INJ_ROUND && mode != KO_INJ_EXACT))
        return KO_EINVAL;
    if (n > 0 && moff > UINT64_MAX - (n - 1))
        return KO_EINVAL;
    uint64_t T = ko_inject_threshold(rate);
    size_t es = dtype_size(dt);
    int64_t perturbed = 0;
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t W = ko_word(mseed, moff + i);
        if ((uint64_t)W >= T) {
            if (y != x)
                memcpy((char *)y + i * es, (const char *)x + i * es, es);
            continue;
        }
        float X = load_f32(x, dt, i);
        if (mode == KO_INJ_ROUND) {
            float s = X + delta;
            store_f32(y, dt, i, s);
            perturbed++;
            continue;
        }
        float sp = X + delta;
        float dp = sp - X;
        if (dp == delta && round_trip(sp, dt) == sp) {
            store_f32(y, dt, i, sp);
            perturbed++;
            continue;
        }
        float sm = X - delta;
        float dm = X - sm;
        if (dm == delta && round_trip(sm, dt) == sm) {
            store_f32(y, dt, i, sm);
            perturbed++;
            continue;
        }
        if (y != x)
            memcpy((char *)y + i * es, (const char *)x + i * es, es);
    }
    return perturbed;
}

/* ------------------------------------------------------------------------
 * The allclose check with its reductions.
 * ---------------------------------------------------------------------- */
typedef struct {
    uint64_t n;
    uint64_t mismatches;
    uint64_t nan_count;
    uint64_t argmax_abs;   /* UINT64_MAX when no element is NaN-free */
    float max_abs;
    float max_rel;
} ko_check_result;

int ko_check(const void *a, int dta, const void *b, int dtb, uint64_t n,
             float rtol, float atol, ko_check_result *out)
{
    if (dtype_size(dta) == 0 || dtype_size(dtb) == 0 || dta == KO_U32 || dtb == KO_U32)
        return KO_EINVAL;
    if (!(rtol >= 0.0f) || !(atol >= 0.0f) || isinf(rtol) || isinf(atol))
        return KO_EINVAL;
    ko_check_result r;
    r.n = n;
    r.mismatches = 0;
    r.nan_count = 0;
    r.argmax_abs = UINT64_MAX;
    r.max_abs = 0.0f;
    r.max_rel = 0.0f;
    int have = 0;
    for (uint64_t i = 0; i < n; ++i) {
        float A = load_f32(a, dta, i);
        float B = load_f32(b, dtb, i);
        float d, rel;
        if (isnan(A) || isnan(B)) {
            r.mismatches++;
            r.nan_count++;
            continue;
        }
        if (A == B) {
            d = 0.0f;
            rel = 0.0f;
        } else if (isinf(A) || isinf(B)) {
            r.mismatches++;
            d = INFINITY;
            rel = INFINITY;
        } else {
            float diff = A - B;
            d = fabsf(diff);
            float absb = fabsf(B);
            float rt = rtol * absb;
            float thr = atol + rt;
            if (!(d <= thr) || isinf(d))   /* an overflowed difference is never close */
                r.mismatches++;
            rel = d / absb;
        }
        if (!have || d > r.max_abs) {
            r.max_abs = d;
            r.argmax_abs = i;
            have = 1;
        }
        if (rel > r.max_rel)
            r.max_rel = rel;
    }
    *out = r;
    return KO_OK;
}

/* ------------------------------------------------------------------------
 * Cache-flush fill: every 32-bit word of the buffer gets the pattern.
 * ---------------------------------------------------------------------- */
int ko_flush(void *buf, uint64_t bytes, uint32_t pattern)
{
    if (bytes % 4 != 0)
        return KO_EINVAL;
    uint32_t *p = (uint32_t *)buf;
    for (uint64_t i = 0; i < bytes / 4; ++i)
        p[i] = pattern;
    return KO_OK;
}

/* ------------------------------------------------------------------------
 * FMA probe: thread g of `threads` runs 8 independent chains
 * x <- fma(x, a, b), a = 1 - 2^-10, b = 2^-10, starting from
 * x_c = (g * 8 + c) 2^-19, for iters steps, and writes the chains' sum in
 * chain order.
 * ---------------------------------------------------------------------- */
void ko_probe(uint64_t iters, float *sink, uint32_t threads)
{
    const float a = 1.0f - 0x1p-10f;
    const float bb = 0x1p-10f;
    for (uint32_t g = 0; g < threads; ++g) {
        float x[8];
        for (int c = 0; c < 8; ++c)
            x[c] = (float)(g * 8u + (uint32_t)c) * 0x1p-19f;
        for (uint64_t it = 0; it < iters; ++it)
            for (int c = 0; c < 8; ++c)
                x[c] = fmaf(x[c], a, bb);
        float s = x[0];
        for (int c = 1; c < 8; ++c)
            s = s + x[c];
        sink[g] = s;
    }
}

/* ------------------------------------------------------------------------
 * fp32 reference GEMM of the tiny GEMM command: row-major C = A B,
 * C[i][j] = fma-accumulated sum over k ascending from +0.
 * ---------------------------------------------------------------------- */
void ko_sgemm(uint32_t M, uint32_t N, uint32_t K, const float *A, const float *B, float *C)
{
    for (uint32_t i = 0; i < M; ++i)
        for (uint32_t j = 0; j < N; ++j) {
            float acc = 0.0f;
            for (uint32_t k = 0; k < K; ++k)
                acc = fmaf(A[(uint64_t)i * K + k], B[(uint64_t)k * N + j], acc);
            C[(uint64_t)i * N + j] = acc;
        }
}

/* ------------------------------------------------------------------------
 * Bulk forms of the transforms, for the exhaustive pin sweeps.
 * ---------------------------------------------------------------------- */
void ko_ln_many(const float *x, float *out, uint64_t n)
{
    for (uint64_t i = 0; i < n; ++i)
        out[i] = ko_ln(x[i]);
}

void ko_sincos_many(const uint32_t *k, float *sn, float *cs, uint64_t n)
{
    for (uint64_t i = 0; i < n; ++i)
        ko_sincos_2pi_q24(k[i], &sn[i], &cs[i]);
}

/* z[2i], z[2i + 1] from the word pair (w[2i], w[2i + 1]). */
void ko_normal_pairs(const uint32_t *w, float *z, uint64_t npairs)
{
    for (uint64_t i = 0; i < npairs; ++i)
        ko_normal_pair(w[2 * i], w[2 * i + 1], &z[2 * i], &z[2 * i + 1]);
}

void ko_uniform_many(const uint32_t *w, float *out, uint64_t n, float lo, float hi)
{
    for (uint64_t i = 0; i < n; ++i)
        out[i] = ko_uniform(w[i], lo, hi);
}
