// Per-parameter arithmetic shared by the dense and sparse FASGD kernels, and
// the counter-based generator used by the B-FASGD selection.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fasgd {

enum : int { MATH_IEEE = 0, MATH_FAST = 1 };
// Which v the update keeps (bit 1 of a kernel variant; bit 0 is the math mode):
//   V_EQUATIONS  v averages 1/sqrt(n - b^2 + eps), Sec. 2.2's equation for v;
//   V_PROSE      v averages sqrt(n - b^2 + eps), the moving average of the
//                standard deviation that Sec. 2.2's text describes.
// Both divide the rate by v.
enum : int { V_EQUATIONS = 0, V_PROSE = 2 };
constexpr int kernel_variant(int math_mode, int v_reading) { return math_mode | (v_reading ? V_PROSE : 0); }

// Scalars of one weight update that are the same for every parameter.
struct Hyper {
    float gamma;   // decay of n and b
    float omg;     // 1 - gamma
    float beta;    // decay of v
    float omb;     // 1 - beta
    float eps;     // inside the square root
    float alpha;   // master rate
    int32_t rn_short;   // IEEE mode: eps >= 2^-96 and 2^-20 <= |alpha| < 2^20 (set by the host), so the
                        // short correctly rounded sequences below hold; otherwise the general ones run
};

// Correctly rounded square root, reciprocal and division in fewer
// instructions than the general sequences, for the operand ranges the IEEE
// update meets once the host has checked eps and alpha.  Each starts from
// the hardware estimate (within 1 ulp) and corrects it with exact residuals
// computed by fused multiply-adds.  fasgd_check_ieee_sequences compares them
// with the general sequences bit for bit, exhaustively over their ranges.
//
// sqrt(x), x >= 2^-96, +inf or NaN: of the estimate s and its neighbours
// s-, s+ (one ulp away), the residuals x - s- s and x - s+ s tell on which
// side of each midpoint the root lies (a root of a float is never exactly a
// midpoint); at x >= 2^-96 the residuals are normal numbers, so their signs
// are exact.
__device__ __forceinline__ float sqrt_rn_short(float x)
{
    float s = __builtin_amdgcn_sqrtf(x);
    const float sm = __int_as_float(__float_as_int(s) - 1);
    const float sp = __int_as_float(__float_as_int(s) + 1);
    const float rm = fmaf(-sm, s, x);
    const float rp = fmaf(-sp, s, x);
    s = rm <= 0.0f ? sm : s;
    s = rp > 0.0f ? sp : s;
    return s;
}

// 1/r for r = sqrt_rn_short(x), x >= 2^-96 (r in [2^-48, 2^64], +inf or
// NaN): one Newton step y + y (1 - r y) with the residual exact in the fma;
// the fix-up gives 1/inf = 0.
__device__ __forceinline__ float rcp_of_root_rn_short(float r)
{
    const float y0 = __builtin_amdgcn_rcpf(r);
    const float e = fmaf(-r, y0, 1.0f);
    return __builtin_amdgcn_div_fixupf(fmaf(e, y0, y0), r, 1.0f);
}

// a / d for 2^-20 <= |a| < 2^20: the reciprocal as above, the quotient
// q0 = a y, then q0 + y (a - d q0) with the remainder exact in the fma
// (Markstein's correction).  Lanes whose |d| lies outside [2^-100, 2^100]
// (zero, subnormal, huge, infinite or NaN divisors) take the general division.
__device__ __forceinline__ float div_rn_short(float a, float d)
{
    const float y0 = __builtin_amdgcn_rcpf(d);
    const float e = fmaf(-d, y0, 1.0f);
    const float y = fmaf(e, y0, y0);
    const float q0 = a * y;
    const float r = fmaf(-d, q0, a);
    float q = fmaf(r, y, q0);
    const bool in_range = __builtin_fabsf(d) >= 0x1p-100f && __builtin_fabsf(d) <= 0x1p100f;
    if (__builtin_expect(__ballot(!in_range) != 0, 0)) q = in_range ? q : a / d;
    return q;
}

// One parameter, one gradient: the FASGD update of Sec. 2.2.
//   n <- gamma n + (1-gamma) g^2 ; b <- gamma b + (1-gamma) g
//   v <- beta v + (1-beta) / sqrt(max(n - b^2, 0) + eps)     (V_EQUATIONS)
//   v <- beta v + (1-beta) * sqrt(max(n - b^2, 0) + eps)     (V_PROSE)
//   theta <- theta - alpha / (v tau) g
// VARIANT = math mode | v reading.  `coef` carries the staleness: tau (as
// float) in IEEE mode, and the precomputed alpha / tau in FAST mode (so
// that the only per-parameter division becomes one hardware reciprocal).
template <int VARIANT>
__device__ __forceinline__ void fasgd_step(float& th, float& n, float& b, float& v, float g,
                                           float coef, const Hyper& h)
{
    constexpr bool fast = (VARIANT & MATH_FAST) != 0;
    constexpr bool prose = (VARIANT & V_PROSE) != 0;
    const float a = h.omg * g;                 // (1 - gamma) g
    n = fmaf(h.gamma, n, a * g);
    b = fmaf(h.gamma, b, a);
    float var = fmaf(-b, b, n);                // n - b^2, one rounding
    var = fmaxf(var, 0.0f);
    const float x = var + h.eps;
    if constexpr (fast) {
        const float s = prose ? __builtin_amdgcn_sqrtf(x) : __builtin_amdgcn_rsqf(x);
        v = fmaf(h.beta, v, h.omb * s);
        th = fmaf(-(coef * __builtin_amdgcn_rcpf(v)), g, th);
    } else if (h.rn_short) {
        // the same correctly rounded operations as below, in the short sequences
        const float r = sqrt_rn_short(x);
        const float s = prose ? r : rcp_of_root_rn_short(r);
        v = fmaf(h.beta, v, h.omb * s);
        th = fmaf(-div_rn_short(h.alpha, v * coef), g, th);
    } else {
        const float s = prose ? sqrtf(x) : 1.0f / sqrtf(x);
        v = fmaf(h.beta, v, h.omb * s);
        th = fmaf(-(h.alpha / (v * coef)), g, th);
    }
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11).  Per round, words 0 and
// 2 are multiplied by the round multipliers; the high halves, xored with
// words 1 and 3 and the round key, become the new words 0 and 2, the low
// halves the new words 3 and 1.  The key steps by the Weyl increments
// between rounds.  The key is uniform across a wave and stays in SGPRs.
// Each three-way xor is one v_bitop3_b32 (truth table 0x96) on gfx950.
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c)
{
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

__device__ __forceinline__ uint4 philox4x32_10(uint4 x, uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int i = 0; i < 10; ++i) {
        const uint64_t m0 = static_cast<uint64_t>(x.x) * 0xD2511F53ull;
        const uint64_t m2 = static_cast<uint64_t>(x.z) * 0xCD9E8D57ull;
        x = make_uint4(xor3(static_cast<uint32_t>(m2 >> 32), x.y, k0), static_cast<uint32_t>(m2),
                       xor3(static_cast<uint32_t>(m0 >> 32), x.w, k1), static_cast<uint32_t>(m0));
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return x;
}

// B-FASGD transmit test of Sec. 2.3, r < 1/(1 + c/(v + eps_c)), in the
// division-free form r (t + c) < t with t = v + eps_c: both sums are fp32
// and the fused multiply-add rounds once, so the sign of r*u - t is exact.
// r is the top 24 bits of a Philox word scaled into [0, 1).
__device__ __forceinline__ uint32_t transmit_bit(uint32_t word, float v, float c, float eps_c)
{
#pragma clang fp contract(off)
    const float r = static_cast<float>(word >> 8) * 0x1p-24f;
    const float t = v + eps_c;
    const float u = t + c;
    return fmaf(r, u, -t) < 0.0f ? 1u : 0u;
}

}  // namespace fasgd
