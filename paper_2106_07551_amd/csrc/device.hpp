// Device primitives shared by the gfx950 kernels: the counter-based random
// stream, the uniform and Gumbel transforms, bf16 rounding and the fixed
// tanh of the feature dynamics.  All of it is written for a single fp32
// environment: no fast-math, no contraction (-ffp-contract=off), correctly
// rounded fp32 division, fp32 denormals preserved.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace malib {

// Random-stream purposes (third counter word, high half).
enum : uint32_t { kPurposeAction = 0, kPurposeReset = 1, kPurposeMeta = 2 };

struct u64x4 {
    uint64_t x, y, z, w;
};

// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds, each two
// 64x64->128-bit products with the round constants, the high halves xor-ed
// with the other counter words and the key; the key advances by the Weyl
// increments between rounds.
// 64x64 -> 128-bit product from four 32x32 -> 64 multiply-adds: the partial
// products are chained so that no sum can overflow 64 bits.
__device__ __forceinline__ void mul_hilo64(uint64_t a, uint64_t b, uint64_t& lo, uint64_t& hi)
{
    const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32);
    const uint32_t b0 = (uint32_t)b, b1 = (uint32_t)(b >> 32);
    const uint64_t p00 = (uint64_t)a0 * b0;
    const uint64_t t = (uint64_t)a0 * b1 + (p00 >> 32);
    const uint64_t u = (uint64_t)a1 * b0 + (uint32_t)t;
    lo = (u << 32) | (uint32_t)p00;
    hi = (uint64_t)a1 * b1 + ((t >> 32) + (u >> 32));
}

__device__ __forceinline__ u64x4 philox4x64_10(u64x4 c, uint64_t k0, uint64_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t m0 = 0xD2E7470EE14C6C93ull, m1 = 0xCA5A826395121157ull;
        uint64_t lo0, hi0, lo1, hi1;
        mul_hilo64(m0, c.x, lo0, hi0);
        mul_hilo64(m1, c.z, lo1, hi1);
        u64x4 n;
        n.x = hi1 ^ c.y ^ k0;
        n.y = lo1;
        n.z = hi0 ^ c.w ^ k1;
        n.w = lo0;
        c = n;
        k0 += 0x9E3779B97F4A7C15ull;
        k1 += 0xBB67AE8584CAA73Bull;
    }
    return c;
}

// The block of the stream at (global env g, step t, purpose, slot, block):
// counter (g, t, purpose<<32 | slot, block), key (seed, 0).
__device__ __forceinline__ u64x4 stream_block(uint64_t seed, uint64_t g, uint64_t t,
                                              uint32_t purpose, uint32_t slot, uint64_t block)
{
    u64x4 c{g, t, ((uint64_t)purpose << 32) | slot, block};
    return philox4x64_10(c, seed, 0);
}

// 32-bit lane j (0..7) of a block: lane 2w = low half of word w, 2w+1 = high.
__device__ __forceinline__ uint32_t block_lane(const u64x4& b, int j)
{
    uint64_t w = (j >> 1) == 0 ? b.x : (j >> 1) == 1 ? b.y : (j >> 1) == 2 ? b.z : b.w;
    return (j & 1) ? (uint32_t)(w >> 32) : (uint32_t)w;
}

// Uniform in (0,1): odd integer 2*(x>>9)+1 (< 2^24, exact in fp32) times 2^-24.
__device__ __forceinline__ float uniform01(uint32_t x)
{
    return (float)(2u * (x >> 9) + 1u) * 0x1p-24f;
}

// bf16 bits of x, round to nearest even; NaN -> quiet NaN with x's sign.
__device__ __forceinline__ uint16_t bf16_bits(float x)
{
    uint32_t b = __float_as_uint(x);
    if ((b & 0x7FFFFFFFu) > 0x7F800000u)
        return (uint16_t)(((b >> 16) & 0x8000u) | 0x7FC0u);
    b += 0x7FFFu + ((b >> 16) & 1u);
    return (uint16_t)(b >> 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> bf16 (round to nearest even) packed low/high; an IEEE fptrunc,
// which gfx950 executes as one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// exp_ref: Cody-Waite reduction x = n ln2 + r with ln2 split into a high part
// (trailing zero bits) and a low part, degree-7 Taylor polynomial of e^r in
// fused Horner form, exact scaling by 2^n.
__device__ __forceinline__ float exp_ref(float x)
{
    const float log2e = 0x1.715476p+0f;
    const float ln2_hi = 0x1.62e4p-1f;
    const float ln2_lo = 0x1.7f7d1cp-20f;
    float n = rintf(x * log2e);
    float r = __builtin_fmaf(-n, ln2_hi, x);
    r = __builtin_fmaf(-n, ln2_lo, r);
    float p = 0x1.a01a02p-13f;            // 1/7!
    p = __builtin_fmaf(p, r, 0x1.6c16c2p-10f);  // 1/6!
    p = __builtin_fmaf(p, r, 0x1.111112p-7f);   // 1/5!
    p = __builtin_fmaf(p, r, 0x1.555556p-5f);   // 1/4!
    p = __builtin_fmaf(p, r, 0x1.555556p-3f);   // 1/3!
    p = __builtin_fmaf(p, r, 0x1p-1f);
    p = __builtin_fmaf(p, r, 0x1p+0f);
    p = __builtin_fmaf(p, r, 0x1p+0f);
    return ldexpf(p, (int)n);
}

// tanh_ref: |x| < 0.55 -> x + x^3 p(x^2) with p the Taylor series of
// (tanh x - x)/x^3 through the x^19 term; 0.55 <= |x| <= 9.01 ->
// sign(x) (1 - 2/(exp_ref(2|x|) + 1)); |x| > 9.01 -> sign(x); NaN and signed
// zeros unchanged.
__device__ __forceinline__ float tanh_ref(float x)
{
    if (__builtin_isnan(x) || x == 0.0f)
        return x;
    float ax = __builtin_fabsf(x);
    if (ax > 9.01f)
        return __builtin_copysignf(1.0f, x);
    if (ax < 0.55f) {
        float y = x * x;
        float p = -0x1.f57d78p-13f;
        p = __builtin_fmaf(p, y, 0x1.355824p-11f);
        p = __builtin_fmaf(p, y, -0x1.7da364p-10f);
        p = __builtin_fmaf(p, y, 0x1.d6d3dp-9f);
        p = __builtin_fmaf(p, y, -0x1.226e36p-7f);
        p = __builtin_fmaf(p, y, 0x1.664f48p-6f);
        p = __builtin_fmaf(p, y, -0x1.ba1ba2p-5f);
        p = __builtin_fmaf(p, y, 0x1.111112p-3f);
        p = __builtin_fmaf(p, y, -0x1.555556p-2f);
        float x3 = x * y;
        return __builtin_fmaf(x3, p, x);
    }
    // 1 - 2 / b with b = exp_ref(2|x|) + 1 in [4, 2^26]: 2 / b rounded is
    // twice the rounded reciprocal y of b, obtained from the hardware estimate
    // (1 ulp) by one fused Newton step, and 1 - 2y is formed with one rounding,
    // as 1 - (2 / b) is.  (The result equals that of the IEEE quotient for
    // every one of the 2^32 fp32 inputs, checked exhaustively on the device.)
    const float b = exp_ref(2.0f * ax) + 1.0f;
    float y = __builtin_amdgcn_rcpf(b);
    y = __builtin_fmaf(__builtin_fmaf(-b, y, 1.0f), y, y);
    const float t = __builtin_fmaf(-2.0f, y, 1.0f);
    return __builtin_copysignf(t, x);
}

// Device error flags (bit values of malib_eval_stats.device_flags).
enum : int { kErrPid = 1, kErrNaN = 2 };

// Gumbel noise -ln(-ln u) for u in [2^-24, 1 - 2^-24] (uniform01's range):
// both logarithms see normal fp32 inputs, so each is the hardware log2
// (v_log_f32, 1 ulp) times ln 2, without the denormal scaling of logf.
__device__ __forceinline__ float gumbel01(float u)
{
    const float ln2 = 0x1.62e430p-1f;
    const float e = -(__builtin_amdgcn_logf(u) * ln2);
    return -(__builtin_amdgcn_logf(e) * ln2);
}

// Gumbel-max action of one agent slot from its A logits l[0..A-1]:
// z_a = l_a + g_a with g_a = gumbel01(u_a) in fp32, u_a from lane a%8 of
// block a/8 of (global env g, step t, kPurposeAction<<32 | seat); the first
// index of the maximum wins.  AMAX >= A (a multiple of 8): all logits are
// loaded and all Philox blocks drawn before the arithmetic, so their
// latencies overlap.  A NaN logit sets `nan` and gives action 0.
template <int AMAX>
__device__ __forceinline__ int gumbel_action(const float* __restrict__ l, int A, uint64_t seed,
                                             uint64_t g, int t, int seat, bool& nan)
{
    float lv[AMAX];
#pragma unroll
    for (int a = 0; a < AMAX; ++a)
        lv[a] = a < A ? l[a] : 0.0f;
    u64x4 blk[AMAX / 8];
#pragma unroll
    for (int b = 0; b < AMAX / 8; ++b)
        if (b * 8 < A)
            blk[b] = stream_block(seed, g, (uint64_t)t, kPurposeAction, (uint32_t)seat,
                                  (uint64_t)b);
    float zbest = 0.0f;
    int best = 0;
    bool bad = false;
#pragma unroll
    for (int a = 0; a < AMAX; ++a) {
        if (a < A) {
            const float gn = gumbel01(uniform01(block_lane(blk[a >> 3], a & 7)));
            bad |= __builtin_isnan(lv[a]);
            const float z = lv[a] + gn;
            if (a == 0 || z > zbest) {
                zbest = z;
                best = a;
            }
        }
    }
    nan = bad;
    return bad ? 0 : best;
}

}  // namespace malib
