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
};

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
