// gem_device.hpp -- device-side numerics of the GEM commit pipeline (gfx950).
//
// Counter-based noise and the elementwise GEM step, evaluated in IEEE binary32
// with round-to-nearest-even in a fixed operation order: explicit fma where
// written, correctly rounded division and square root (hipcc's IEEE lowering
// on gfx950, or its core steps where the operand range leaves the rest
// nothing to do), denormals kept, no contraction (built with
// -ffp-contract=off).
// Any IEEE implementation of the same steps -- in particular the host-side
// test oracle, written separately -- produces the same bits.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gemk {

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror & Shaw, SC'11).  Each round multiplies
// words 0 and 2 by the two Philox multipliers and mixes the high halves with
// the odd words and the key; the key advances by the two Weyl increments
// after every round.
// ---------------------------------------------------------------------------
struct Words4 {
    uint32_t x0, x1, x2, x3;
};

// a ^ b ^ c.  On the device one V_BITOP3_B32 (gfx950's three-input bitwise
// operation; truth table 0x96 is the odd-parity function), which the compiler
// does not form from two XORs by itself.
__host__ __device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c)
{
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
#else
    return a ^ b ^ c;
#endif
}

__host__ __device__ __forceinline__ Words4 philox10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                          uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t pa = static_cast<uint64_t>(0xD2511F53u) * c0;
        const uint64_t pb = static_cast<uint64_t>(0xCD9E8D57u) * c2;
        const uint32_t y0 = xor3(static_cast<uint32_t>(pb >> 32), c1, k0);
        const uint32_t y2 = xor3(static_cast<uint32_t>(pa >> 32), c3, k1);
        c1 = static_cast<uint32_t>(pb);
        c3 = static_cast<uint32_t>(pa);
        c0 = y0;
        c2 = y2;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return Words4{c0, c1, c2, c3};
}

// ---------------------------------------------------------------------------
// Correctly rounded division and square root for operand ranges where the
// general IEEE sequences' range handling has nothing to do.  hipcc lowers a / b
// to scale operands near the ends of the exponent range, refine a hardware
// reciprocal by Newton steps with fma residual corrections, and fix up special
// values; sqrt(x) to scale tiny x, take the hardware root and step to the
// neighbour whose fma residual has the right sign, then handle 0 and inf.  On
// operands with no scaling and no special value the core steps alone give the
// same, correctly rounded, result -- which the self-test library checks
// exhaustively over the domains used below and on a wide random sample for
// the guarded quotient.
// ---------------------------------------------------------------------------

// a / b, correctly rounded, for normal b and a quotient well inside the
// normal range (no scaling of either operand).
__device__ __forceinline__ float div_rn_core(float a, float b)
{
    float r = __builtin_amdgcn_rcpf(b);
    const float e = __builtin_fmaf(-b, r, 1.0f);
    r = __builtin_fmaf(e, r, r);                    // refined reciprocal
    float q = a * r;
    const float e2 = __builtin_fmaf(-b, q, a);
    q = __builtin_fmaf(e2, r, q);
    const float e3 = __builtin_fmaf(-b, q, a);
    return __builtin_fmaf(e3, r, q);
}

// sqrt(x), correctly rounded, for x = +0 or normal x (no scaling).
__device__ __forceinline__ float sqrt_rn_core(float x)
{
    const float y = __builtin_amdgcn_sqrtf(x);
    const float dn = __uint_as_float(__float_as_uint(y) - 1u);
    const float up = __uint_as_float(__float_as_uint(y) + 1u);
    const float r_dn = __builtin_fmaf(-dn, y, x);
    const float r_up = __builtin_fmaf(-up, y, x);
    float r = (r_dn <= 0.0f) ? dn : y;
    r = (r_up > 0.0f) ? up : r;
    return r;
}

// num / den, correctly rounded for every input: the core steps when both
// magnitudes lie in [2^-60, 2^60] (quotient in [2^-120, 2^120]), the general
// division otherwise (zero, tiny, huge, infinite or NaN operands).
__device__ __forceinline__ float div_rn(float num, float den)
{
    const float an = __builtin_fabsf(num), ad = __builtin_fabsf(den);
    const bool core = an >= 0x1p-60f && an <= 0x1p60f && ad >= 0x1p-60f && ad <= 0x1p60f;
    float q;
    if (core) q = div_rn_core(num, den);
    else q = num / den;
    return q;
}

// (f - 1) / (f + 1), correctly rounded, for the binary32 f in (sqrt(1/2),
// sqrt(2)] the logarithm below reduces to: the hardware reciprocal r of
// f + 1 and one residual correction of the quotient (f - 1) r.  f - 1 is exact,
// f + 1 lies in (1.7, 2.5), and on these 2^23 operand pairs the two steps
// give the correctly rounded quotient every time (the self-test library
// checks all of them on the device against the IEEE division); the general
// core above takes four more steps.
__device__ __forceinline__ float ln_quotient(float a, float b)
{
    const float r = __builtin_amdgcn_rcpf(b);
    const float q = a * r;
    const float e = __builtin_fmaf(-b, q, a);
    return __builtin_fmaf(e, r, q);
}

// ---------------------------------------------------------------------------
// Natural logarithm of u = k * 2^-24 for an integer k in [1, 2^24] (the Box-
// Muller radius argument).  u = 2^e f with f in (sqrt(1/2), sqrt(2)];
// ln f = 2 atanh((f-1)/(f+1)) by its series to the s^9 term (Abramowitz &
// Stegun 4.1.27); ln u = e ln2 + ln f with ln 2 split into a 15-bit head and
// a binary32 tail so that e * head is exact.
// ---------------------------------------------------------------------------

// ln of the positive normal binary32 value with bit pattern `bits`, scaled by
// 2^(127 - bias): bias 127 gives ln of the value itself.
__device__ __forceinline__ float ln_from_bits(uint32_t bits, int bias)
{
    int e = static_cast<int>(bits >> 23) - bias;  // positive: the sign bit is clear
    const uint32_t mant = bits & 0x007FFFFFu;
    const bool upper = mant > 0x003504F3u;        // 1.mant above sqrt(2) in binary32
    const uint32_t fbits = mant | (upper ? 0x3F000000u : 0x3F800000u);
    e += upper ? 1 : 0;
    const float f = __uint_as_float(fbits);
    const float s = ln_quotient(f - 1.0f, f + 1.0f);
    const float z = s * s;
    float p = 1.0f / 9.0f;
    p = __builtin_fmaf(p, z, 1.0f / 7.0f);
    p = __builtin_fmaf(p, z, 1.0f / 5.0f);
    p = __builtin_fmaf(p, z, 1.0f / 3.0f);
    p = p * z;
    const float two_s = s + s;
    const float ln_f = __builtin_fmaf(two_s, p, two_s);
    const float ef = static_cast<float>(e);
    const float ln2_tail = 0x1.7f7d1cp-20f;   // RN(ln 2 - ln2_head)
    const float ln2_head = 0x1.62e4p-1f;
    float r = __builtin_fmaf(ef, ln2_tail, ln_f);
    r = __builtin_fmaf(ef, ln2_head, r);
    return r;
}

// ln u for u = k 2^-24 in (0, 1].
__device__ __forceinline__ float ln_of_unit(float u) { return ln_from_bits(__float_as_uint(u), 127); }

// The same from k: the binary32 k (exact) has the significand of u and an
// exponent 24 larger, so the scaling by 2^-24 folds into the exponent's bias
// instead of a multiplication.
__device__ __forceinline__ float ln_of_k24(uint32_t k)
{
    return ln_from_bits(__float_as_uint(static_cast<float>(k)), 127 + 24);
}

// sin and cos of 2 pi k / 2^24, k in [0, 2^24).  The angle is reduced to the
// nearest quarter turn on the integer, exactly; the rest, |x| <= pi/4, goes
// through the Taylor series of sin (to x^9) and cos (to x^10).
__device__ __forceinline__ void sincos_of_turn(uint32_t k, float& sn, float& cs)
{
    const uint32_t quarter = (k + 0x00200000u) >> 22;
    const int rem = static_cast<int>(k) - static_cast<int>(quarter << 22);
    const float step = 6.28318530717958647692f * 0x1p-24f;   // RN(2 pi) 2^-24
    const float x = static_cast<float>(rem) * step;
    const float x2 = x * x;

    float ps = 1.0f / 362880.0f;
    ps = __builtin_fmaf(ps, x2, -1.0f / 5040.0f);
    ps = __builtin_fmaf(ps, x2, 1.0f / 120.0f);
    ps = __builtin_fmaf(ps, x2, -1.0f / 6.0f);
    ps = ps * x2;
    const float sx = __builtin_fmaf(x, ps, x);

    float pc = -1.0f / 3628800.0f;
    pc = __builtin_fmaf(pc, x2, 1.0f / 40320.0f);
    pc = __builtin_fmaf(pc, x2, -1.0f / 720.0f);
    pc = __builtin_fmaf(pc, x2, 1.0f / 24.0f);
    pc = __builtin_fmaf(pc, x2, -0.5f);
    const float cx = __builtin_fmaf(pc, x2, 1.0f);

    // Quadrant q = quarter mod 4 (bits 22 and 23 of k + 2^21): sin takes sx, cx,
    // -sx, -cx and cos cx, -sx, -cx, sx.  On the bits: an odd quadrant swaps
    // the two (a bit-select under a mask of bit 22), quadrants 2 and 3 negate
    // sin (bit 23 into the sign) and quadrants 1 and 2 negate cos (bit 22 xor
    // bit 23) -- negation flips the sign bit, as -x does.
    const uint32_t kq = k + 0x00200000u;
    const uint32_t odd = static_cast<uint32_t>(static_cast<int32_t>(kq << 9) >> 31);
    const uint32_t sxb = __float_as_uint(sx), cxb = __float_as_uint(cx);
    const uint32_t a = (odd & cxb) | (~odd & sxb);     // |sin| candidate
    const uint32_t b = (odd & sxb) | (~odd & cxb);     // |cos| candidate
    const uint32_t neg_s = (kq << 8) & 0x80000000u;
    const uint32_t neg_c = ((kq << 8) ^ (kq << 9)) & 0x80000000u;
    sn = __uint_as_float(a ^ neg_s);
    cs = __uint_as_float(b ^ neg_c);
}

// Box-Muller (1958): from two words, u1 = ((xa >> 8) + 1) 2^-24 in (0, 1] and
// the angle index xb >> 8, the pair r cos(phi), r sin(phi), r = sqrt(-2 ln u1).
__device__ __forceinline__ void box_muller(uint32_t xa, uint32_t xb, float& zc, float& zs)
{
    // -2 ln u1 is +0 (u1 = 1) or at least 1.1e-7: no scaling.
    const float r = sqrt_rn_core(-2.0f * ln_of_k24((xa >> 8) + 1u));
    float sn, cs;
    sincos_of_turn(xb >> 8, sn, cs);
    zc = r * cs;
    zs = r * sn;
}

// Four standard normals for elements 4q..4q+3 at clock t.
__device__ __forceinline__ float4 normals4(uint64_t q, uint32_t t, uint32_t k0, uint32_t k1)
{
    const Words4 w = philox10(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32), t, 0u,
                              k0, k1);
    float4 z;
    box_muller(w.x0, w.x1, z.x, z.y);
    box_muller(w.x2, w.x3, z.z, z.w);
    return z;
}

// binary32 -> bfloat16 -> binary32, nearest-even; NaN stays a (quiet) NaN.
__device__ __forceinline__ float round_to_bf16(float x)
{
    uint32_t b = __float_as_uint(x);
    if ((b & 0x7FFFFFFFu) > 0x7F800000u) {
        b = (b | 0x00400000u) & 0xFFFF0000u;
    } else {
        b = (b + 0x7FFFu + ((b >> 16) & 1u)) & 0xFFFF0000u;
    }
    return __uint_as_float(b);
}

}  // namespace gemk
