// valu_rates.hip -- issue cost of the gfx950 vector instructions the hot-path
// kernels use, in cycles per wave64 instruction per SIMD.
//
// Each kernel runs one instruction in eight independent register chains per
// lane (no dependency stalls at eight resident waves per SIMD) over a grid of
// 32 waves per SIMD, and is timed with HIP events. Costs are relative to
// v_fma_f32, whose issue cost follows from the published fp32 vector peak:
// 157.3 TFLOP/s = 256 CUs x 2.4 GHz x 256 flop per CU per cycle, i.e. one
// wave64 FMA per SIMD every 2 cycles. Only vector-register instructions appear
// (plus VCC for the compare), and the one store is a guarded vector store.
//
// Three scalar instructions (the wave ballots' mask and count arithmetic and
// the key-schedule adds) run the same way on eight SGPR chains: a CU's four
// SIMDs share one scalar unit, so their cost per wave instruction per SIMD
// is about four cycles. The last entry alternates one v_fma_f32 and one
// s_add_u32 per chain step (eight of each per iteration): its cost per
// v_fma_f32 shows whether the two units issue side by side (the scalar
// chain's cost) or one after the other (their sum).
//
// Two entries measure the Philox multiply in context: a v_mad_u64_u32 whose
// high word the next instruction reads (eight chains of the pair, cost per
// pair), and whole Philox4x32-10 blocks as the generators form them (the
// library's philox_block, two per group as the compiler interleaves them,
// and philox_blocks<2>, the lockstep form; key schedule in kernel
// arguments; cost per wave-block).
//
// Output: one JSON line {"reference": ..., "cycles": {instruction: cost},
// "ms": {instruction: median kernel time}}.
#include <hip/hip_runtime.h>

#include "krex_device.hpp"

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <vector>

#define CHECK(x)                                                                      \
    do {                                                                              \
        hipError_t e_ = (x);                                                          \
        if (e_ != hipSuccess) {                                                       \
            fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
            exit(1);                                                                  \
        }                                                                             \
    } while (0)

static constexpr int kIter = 2048;
static constexpr uint32_t kThreads = 256;

#define ONE(INS, v) asm volatile(INS : "+v"(v))
#define CHAIN8(INS)                                                                            \
    for (int it = 0; it < kIter; ++it) {                                                       \
        ONE(INS, x0); ONE(INS, x1); ONE(INS, x2); ONE(INS, x3);                                \
        ONE(INS, x4); ONE(INS, x5); ONE(INS, x6); ONE(INS, x7);                                \
    }

enum Op {
    FMA_F32, ADD_F32, MUL_F32, ADD_U32, AND_B32, LSHR_B32, BITOP3, FMAAK_F32,
    MAX_F32, MAX3_F32, CNDMASK, PERM, BFE, MUL_HI_U32, MAD_U64_U32,
    CVT_F32_U32, CVT_F32_F16, CVT_F32_FP8, CVT_PK_BF16_F32, CVT_PK_F16_F32,
    CMP_F32, RCP_F32, SQRT_F32, CVT_PK_FP8_F32, S_ADD_U32, S_AND_B64, S_BCNT1_I32_B64, FMA_AND_SADD, MAD_XOR_DEP,
    NUM_OPS
};

// The Philox block entries, timed by k_philox (not k_rate).
enum PhiloxForm { PHILOX_PAIR, PHILOX_LOCKSTEP, NUM_PHILOX };
static const char *kPhiloxNames[NUM_PHILOX] = {"philox4x32_10 block (philox_block, two per group)",
                                               "philox4x32_10 block (philox_blocks<2>)"};
static constexpr int kPhiloxIter = kIter / 16;   // 8 blocks per iteration

static const char *kNames[NUM_OPS] = {
    "v_fma_f32", "v_add_f32", "v_mul_f32", "v_add_u32", "v_and_b32", "v_lshrrev_b32", "v_bitop3_b32", "v_fmaak_f32",
    "v_max_f32", "v_max3_f32", "v_cndmask_b32", "v_perm_b32", "v_bfe_u32", "v_mul_hi_u32", "v_mad_u64_u32",
    "v_cvt_f32_u32", "v_cvt_f32_f16", "v_cvt_f32_fp8", "v_cvt_pk_bf16_f32", "v_cvt_pk_f16_f32",
    "v_cmp_lt_f32", "v_rcp_f32", "v_sqrt_f32", "v_cvt_pk_fp8_f32", "s_add_u32", "s_and_b64", "s_bcnt1_i32_b64",
    "v_fma_f32+s_add_u32", "v_mad_u64_u32+v_xor_b32 (reads its high word)"};

template <int K>
__global__ __launch_bounds__(kThreads) void k_rate(uint32_t *out, uint32_t seed)
{
    const uint32_t t = blockIdx.x * kThreads + threadIdx.x + seed;
    uint32_t x0 = t, x1 = t ^ 1u, x2 = t ^ 2u, x3 = t ^ 3u, x4 = t ^ 4u, x5 = t ^ 5u, x6 = t ^ 6u, x7 = t ^ 7u;
    if constexpr (K == FMA_F32) CHAIN8("v_fma_f32 %0, %0, %0, 1.0")
    if constexpr (K == ADD_F32) CHAIN8("v_add_f32 %0, %0, 1.0")
    if constexpr (K == MUL_F32) CHAIN8("v_mul_f32 %0, %0, 0.5")
    if constexpr (K == ADD_U32) CHAIN8("v_add_u32 %0, %0, 1")
    if constexpr (K == AND_B32) CHAIN8("v_and_b32 %0, 0x7fffff, %0")
    if constexpr (K == LSHR_B32) CHAIN8("v_lshrrev_b32 %0, 8, %0")
    if constexpr (K == BITOP3) CHAIN8("v_bitop3_b32 %0, %0, 1, 2 bitop3:0x96")
    if constexpr (K == FMAAK_F32) CHAIN8("v_fmaak_f32 %0, %0, %0, 0x3e800000")
    if constexpr (K == MAX_F32) CHAIN8("v_max_f32 %0, %0, 1.0")
    if constexpr (K == MAX3_F32) CHAIN8("v_max3_f32 %0, %0, %0, %0")
    if constexpr (K == CNDMASK) CHAIN8("v_cndmask_b32 %0, %0, 1, vcc")
    if constexpr (K == PERM) CHAIN8("v_perm_b32 %0, %0, %0, %0")
    if constexpr (K == BFE) CHAIN8("v_bfe_u32 %0, %0, 8, %0")
    if constexpr (K == MUL_HI_U32) CHAIN8("v_mul_hi_u32 %0, %0, %0")
    if constexpr (K == CVT_F32_U32) CHAIN8("v_cvt_f32_u32 %0, %0")
    if constexpr (K == CVT_F32_F16) CHAIN8("v_cvt_f32_f16 %0, %0")
    if constexpr (K == CVT_F32_FP8) CHAIN8("v_cvt_f32_fp8 %0, %0")
    if constexpr (K == CVT_PK_BF16_F32) CHAIN8("v_cvt_pk_bf16_f32 %0, %0, %0")
    if constexpr (K == CVT_PK_F16_F32) CHAIN8("v_cvt_pk_f16_f32 %0, %0, %0")
    if constexpr (K == RCP_F32) CHAIN8("v_rcp_f32 %0, %0")
    if constexpr (K == SQRT_F32) CHAIN8("v_sqrt_f32 %0, %0")
    if constexpr (K == CVT_PK_FP8_F32) CHAIN8("v_cvt_pk_fp8_f32 %0, %0, %0")
    if constexpr (K == CMP_F32) {
        // Compares write VCC; a chain of them into one VCC has no register
        // dependency, the select afterwards keeps the result live.
        for (int it = 0; it < kIter; ++it) {
            asm volatile("v_cmp_lt_f32 vcc, %0, 1.0" ::"v"(x0) : "vcc");
            asm volatile("v_cmp_lt_f32 vcc, %0, 1.0" ::"v"(x1) : "vcc");
            asm volatile("v_cmp_lt_f32 vcc, %0, 1.0" ::"v"(x2) : "vcc");
            asm volatile("v_cmp_lt_f32 vcc, %0, 1.0" ::"v"(x3) : "vcc");
            asm volatile("v_cmp_lt_f32 vcc, %0, 1.0" ::"v"(x4) : "vcc");
            asm volatile("v_cmp_lt_f32 vcc, %0, 1.0" ::"v"(x5) : "vcc");
            asm volatile("v_cmp_lt_f32 vcc, %0, 1.0" ::"v"(x6) : "vcc");
            asm volatile("v_cmp_lt_f32 vcc, %0, 1.0" ::"v"(x7) : "vcc");
        }
        asm volatile("v_cndmask_b32 %0, %0, 1, vcc" : "+v"(x0)::"vcc");
    }
    if constexpr (K == MAD_U64_U32) {
        uint64_t a0 = t, a1 = t + 1u, a2 = t + 2u, a3 = t + 3u;
        for (int it = 0; it < kIter; ++it) {
#define MAD(a) asm volatile("v_mad_u64_u32 %0, vcc, %1, %1, 0" : "=v"(a) : "v"((uint32_t)(a)) : "vcc")
            MAD(a0); MAD(a1); MAD(a2); MAD(a3); MAD(a0); MAD(a1); MAD(a2); MAD(a3);
#undef MAD
        }
        x0 = (uint32_t)(a0 ^ a1 ^ a2 ^ a3);
    }
    if constexpr (K == MAD_XOR_DEP) {
        uint64_t a[8];
        a[0] = t; a[1] = t + 1u; a[2] = t + 2u; a[3] = t + 3u; a[4] = t + 4u; a[5] = t + 5u; a[6] = t + 6u; a[7] = t + 7u;
        for (int it = 0; it < kIter; ++it) {
#define P(j, y)                                                                                 \
    asm volatile("v_mad_u64_u32 %0, vcc, %1, %1, 0" : "=v"(a[j]) : "v"((uint32_t)a[j]) : "vcc");  \
    asm volatile("v_xor_b32 %0, %0, %1" : "+v"(y) : "v"((uint32_t)(a[j] >> 32)))
            P(0, x0); P(1, x1); P(2, x2); P(3, x3); P(4, x4); P(5, x5); P(6, x6); P(7, x7);
#undef P
        }
        x0 ^= (uint32_t)(a[0] ^ a[1] ^ a[2] ^ a[3] ^ a[4] ^ a[5] ^ a[6] ^ a[7]);
    }
    if constexpr (K == FMA_AND_SADD) {
        uint32_t s0 = blockIdx.x + seed, s1 = s0 ^ 1u, s2 = s0 ^ 2u, s3 = s0 ^ 3u;
        uint32_t s4 = s0 ^ 4u, s5 = s0 ^ 5u, s6 = s0 ^ 6u, s7 = s0 ^ 7u;
#define V(v) asm volatile("v_fma_f32 %0, %0, %0, 1.0" : "+v"(v))
#define S(v) asm volatile("s_add_u32 %0, %0, 1" : "+s"(v)::"scc")
        for (int it = 0; it < kIter; ++it) {
            V(x0); S(s0); V(x1); S(s1); V(x2); S(s2); V(x3); S(s3);
            V(x4); S(s4); V(x5); S(s5); V(x6); S(s6); V(x7); S(s7);
        }
#undef V
#undef S
        x0 ^= s0 ^ s1 ^ s2 ^ s3 ^ s4 ^ s5 ^ s6 ^ s7;
    }
    if constexpr (K == S_ADD_U32 || K == S_AND_B64 || K == S_BCNT1_I32_B64) {
        // wave-uniform chains in scalar registers
        uint32_t s0 = blockIdx.x + seed, s1 = s0 ^ 1u, s2 = s0 ^ 2u, s3 = s0 ^ 3u;
        uint32_t s4 = s0 ^ 4u, s5 = s0 ^ 5u, s6 = s0 ^ 6u, s7 = s0 ^ 7u;
        uint64_t m0 = s0, m1 = s1, m2 = s2, m3 = s3;
        for (int it = 0; it < kIter; ++it) {
            if constexpr (K == S_ADD_U32) {
#define S(v) asm volatile("s_add_u32 %0, %0, 1" : "+s"(v)::"scc")
                S(s0); S(s1); S(s2); S(s3); S(s4); S(s5); S(s6); S(s7);
#undef S
            } else if constexpr (K == S_AND_B64) {
#define S(m) asm volatile("s_and_b64 %0, %0, 0x7fffffff" : "+s"(m)::"scc")
                S(m0); S(m1); S(m2); S(m3); S(m0); S(m1); S(m2); S(m3);
#undef S
            } else {
#define S(d, m) asm volatile("s_bcnt1_i32_b64 %0, %1" : "=s"(d) : "s"(m) : "scc")
                S(s0, m0); S(s1, m1); S(s2, m2); S(s3, m3); S(s4, m0); S(s5, m1); S(s6, m2); S(s7, m3);
#undef S
            }
        }
        x0 ^= s0 ^ s1 ^ s2 ^ s3 ^ s4 ^ s5 ^ s6 ^ s7 ^ (uint32_t)(m0 ^ m1 ^ m2 ^ m3);
    }
    const uint32_t r = x0 ^ x1 ^ x2 ^ x3 ^ x4 ^ x5 ^ x6 ^ x7;
    if (r == 0x9E3779B9u) out[0] = r;
}

// Eight Philox blocks per iteration and thread, in four groups of two; each
// block's output feeds its next counter, so no iteration can be skipped.
template <int F>
__global__ __launch_bounds__(kThreads) void k_philox(krex::RoundKeys rk, uint32_t *out, uint32_t seed)
{
    const uint32_t t = blockIdx.x * kThreads + threadIdx.x + seed;
    uint64_t c[4] = {(uint64_t)t << 3, ((uint64_t)t << 3) + 2, ((uint64_t)t << 3) + 4, ((uint64_t)t << 3) + 6};
    uint32_t acc = 0;
    for (int it = 0; it < kPhiloxIter; ++it) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            krex::words4 w[2];
            if constexpr (F == PHILOX_PAIR) {
                w[0] = krex::philox_block(c[g], rk);
                w[1] = krex::philox_block(c[g] + 1, rk);
            } else {
                krex::philox_blocks<2>(c[g], rk, w);
            }
            c[g] = ((uint64_t)(w[0].v[1] ^ w[1].v[3]) << 32 | (w[0].v[0] ^ w[1].v[2])) & ~1ull;
            acc ^= w[0].v[2] ^ w[1].v[1];
        }
    }
    acc ^= (uint32_t)(c[0] ^ c[1] ^ c[2] ^ c[3]);
    if (acc == 0x9E3779B9u) out[0] = acc;
}

template <int F>
static float time_philox(uint32_t grid, uint32_t *out, hipEvent_t a, hipEvent_t b)
{
    const krex::RoundKeys rk = krex::round_keys(0x0123456789ABCDEFull);
    std::vector<float> ts;
    for (int r = 0; r < 7; ++r) {
        CHECK(hipEventRecord(a, 0));
        k_philox<F><<<grid, kThreads>>>(rk, out, (uint32_t)r);
        CHECK(hipGetLastError());
        CHECK(hipEventRecord(b, 0));
        CHECK(hipEventSynchronize(b));
        float ms = 0.0f;
        CHECK(hipEventElapsedTime(&ms, a, b));
        ts.push_back(ms);
    }
    std::sort(ts.begin(), ts.end());
    return ts[ts.size() / 2];
}

template <int K>
static float time_op(uint32_t grid, uint32_t *out, hipEvent_t a, hipEvent_t b)
{
    std::vector<float> ts;
    for (int r = 0; r < 7; ++r) {
        CHECK(hipEventRecord(a, 0));
        k_rate<K><<<grid, kThreads>>>(out, (uint32_t)r);
        CHECK(hipGetLastError());
        CHECK(hipEventRecord(b, 0));
        CHECK(hipEventSynchronize(b));
        float ms = 0.0f;
        CHECK(hipEventElapsedTime(&ms, a, b));
        ts.push_back(ms);
    }
    std::sort(ts.begin(), ts.end());
    return ts[ts.size() / 2];
}

template <int... Ks>
static void time_all(std::integer_sequence<int, Ks...>, uint32_t grid, uint32_t *out, hipEvent_t a, hipEvent_t b,
                     float *ms)
{
    ((ms[Ks] = time_op<Ks>(grid, out, a, b)), ...);
}

int main()
{
    int cus = 0;
    CHECK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0));
    uint32_t *out = nullptr;
    CHECK(hipMalloc(&out, sizeof(uint32_t)));
    hipEvent_t a, b;
    CHECK(hipEventCreate(&a));
    CHECK(hipEventCreate(&b));
    const uint32_t grid = (uint32_t)cus * 32u;   // 32 waves per SIMD over the run
    float ms[NUM_OPS];
    time_all(std::make_integer_sequence<int, NUM_OPS>{}, grid, out, a, b, ms);
    const double waves = (double)grid * kThreads / 64.0;
    const double insts_per_simd = waves * kIter * 8.0 / (cus * 4.0);
    const double clock_ghz = insts_per_simd * 2.0 / (ms[FMA_F32] * 1e6);   // FMA at 2 cycles
    printf("{\"reference\": \"v_fma_f32 = 2 cycles per wave64 (fp32 vector peak)\", \"cus\": %d, "
           "\"implied_clock_ghz\": %.3f, \"cycles\": {", cus, clock_ghz);
    for (int k = 0; k < NUM_OPS; ++k)
        printf("%s\"%s\": %.2f", k ? ", " : "", kNames[k], 2.0 * ms[k] / ms[FMA_F32]);
    // a k_philox wave forms 8 kPhiloxIter blocks against 8 kIter instructions
    // of a k_rate wave
    float pms[NUM_PHILOX];
    pms[PHILOX_PAIR] = time_philox<PHILOX_PAIR>(grid, out, a, b);
    pms[PHILOX_LOCKSTEP] = time_philox<PHILOX_LOCKSTEP>(grid, out, a, b);
    for (int f = 0; f < NUM_PHILOX; ++f)
        printf(", \"%s\": %.1f", kPhiloxNames[f], 2.0 * pms[f] / ms[FMA_F32] * kIter / kPhiloxIter);
    printf("}, \"ms\": {");
    for (int k = 0; k < NUM_OPS; ++k) printf("%s\"%s\": %.4f", k ? ", " : "", kNames[k], ms[k]);
    for (int f = 0; f < NUM_PHILOX; ++f) printf(", \"%s\": %.4f", kPhiloxNames[f], pms[f]);
    printf("}}\n");
    CHECK(hipFree(out));
    return 0;
}
