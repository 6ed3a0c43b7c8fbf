// Device self-check of the IEEE update's short correctly rounded sequences
// (sqrt_rn_short, rcp_of_root_rn_short, div_rn_short) against the general
// sequences the compiler emits for sqrtf and '/', bit for bit:
//   - the square root and the reciprocal of the root over every float
//     x >= 2^-96 (+inf and the positive NaNs included);
//   - the division alpha / d over every one of the 2^32 bit patterns of d;
//   - whole updates (fasgd_step, IEEE mode, both readings of v) on
//     pseudo-random states, with rn_short set and cleared.
// NaN results compare equal to NaN results whatever their payloads.
#include "kernels.hpp"

namespace fasgd {
namespace {

constexpr int kCheckBlock = 256;
constexpr unsigned kCheckGrid = 65536;   // grid-stride over 2^24 threads

__device__ __forceinline__ bool same_bits(float a, float b)
{
    return __float_as_uint(a) == __float_as_uint(b) || (a != a && b != b);
}

__device__ __forceinline__ uint64_t thread_index()
{
    return static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
}

__device__ __forceinline__ uint64_t thread_count() { return static_cast<uint64_t>(gridDim.x) * blockDim.x; }

__global__ __launch_bounds__(kCheckBlock) void clear_counts(unsigned long long* counts)
{
    if (threadIdx.x < kIeeeChecks) counts[threadIdx.x] = 0ull;
}

// counts[0]: sqrt, counts[1]: 1 / sqrt (two roundings), x in [2^-96, NaN]
__global__ __launch_bounds__(kCheckBlock) void check_roots(unsigned long long* counts)
{
    constexpr uint64_t lo = 0x0F800000u;   // 2^-96
    constexpr uint64_t hi = 0x7FFFFFFFu;   // the last positive NaN
    unsigned long long bad_root = 0, bad_rcp = 0;
    for (uint64_t i = lo + thread_index(); i <= hi; i += thread_count()) {
        const float x = __uint_as_float(static_cast<uint32_t>(i));
        const float r = sqrt_rn_short(x);
        const float want = sqrtf(x);
        bad_root += !same_bits(r, want);
        bad_rcp += !same_bits(rcp_of_root_rn_short(r), 1.0f / want);
    }
    if (bad_root) atomicAdd(counts + 0, bad_root);
    if (bad_rcp) atomicAdd(counts + 1, bad_rcp);
}

// counts[2]: alpha / d over every bit pattern of d
__global__ __launch_bounds__(kCheckBlock) void check_division(float alpha, unsigned long long* counts)
{
    unsigned long long bad = 0;
    for (uint64_t i = thread_index(); i <= 0xFFFFFFFFull; i += thread_count()) {
        const float d = __uint_as_float(static_cast<uint32_t>(i));
        bad += !same_bits(div_rn_short(alpha, d), alpha / d);
    }
    if (bad) atomicAdd(counts + 2, bad);
}

__device__ __forceinline__ uint32_t mix32(uint64_t x)
{
    x ^= x >> 33;
    x *= 0xff51afd7ed558ccdull;
    x ^= x >> 33;
    x *= 0xc4ceb9fe1a85ec53ull;
    x ^= x >> 33;
    return static_cast<uint32_t>(x);
}

// A state value: one in four any bit pattern (zeros, subnormals, infinities
// and NaNs among them), the others of the magnitudes the method produces.
__device__ __forceinline__ float draw(uint64_t key, float scale)
{
    const uint32_t w = mix32(key);
    if ((w & 3u) == 0u) return __uint_as_float(mix32(key ^ 0x5bd1e995ull));
    const float u = static_cast<float>(w >> 8) * 0x1p-24f;       // [0, 1)
    const float e = static_cast<float>((w >> 2) & 31u) - 16.0f;  // 2^-16 .. 2^15 spread
    return scale * ldexpf(u, static_cast<int>(e));
}

// counts[3]: whole IEEE updates, short against general sequences
template <int VARIANT>
__global__ __launch_bounds__(kCheckBlock) void check_updates(Hyper h, uint64_t seed, int64_t n_updates,
                                                             unsigned long long* counts)
{
    static_assert((VARIANT & MATH_FAST) == 0, "IEEE mode");
    Hyper hs = h, hg = h;
    hs.rn_short = 1;
    hg.rn_short = 0;
    unsigned long long bad = 0;
    for (uint64_t i = thread_index(); i < static_cast<uint64_t>(n_updates); i += thread_count()) {
        const uint64_t k = (seed ^ (static_cast<uint64_t>(VARIANT) << 60)) + 8 * i;
        float th = draw(k, 1.0f), n = fabsf(draw(k + 1, 1e-3f)), b = draw(k + 2, 1e-2f), v = draw(k + 3, 10.0f);
        const float g = draw(k + 4, 1e-2f);
        const float coef = 1.0f + static_cast<float>(mix32(k + 5) & 1023u);   // tau
        float th2 = th, n2 = n, b2 = b, v2 = v;
        fasgd_step<VARIANT>(th, n, b, v, g, coef, hs);
        fasgd_step<VARIANT>(th2, n2, b2, v2, g, coef, hg);
        bad += !(same_bits(th, th2) && same_bits(n, n2) && same_bits(b, b2) && same_bits(v, v2));
    }
    if (bad) atomicAdd(counts + 3, bad);
}

}  // namespace

hipError_t launch_check_ieee(const Hyper& h, uint64_t seed, int64_t n_updates, unsigned long long* counts,
                             hipStream_t s)
{
    clear_counts<<<1, kCheckBlock, 0, s>>>(counts);
    check_roots<<<kCheckGrid, kCheckBlock, 0, s>>>(counts);
    check_division<<<kCheckGrid, kCheckBlock, 0, s>>>(h.alpha, counts);
    if (n_updates > 0) {
        check_updates<kernel_variant(MATH_IEEE, 0)><<<kCheckGrid, kCheckBlock, 0, s>>>(h, seed, n_updates, counts);
        check_updates<kernel_variant(MATH_IEEE, 1)><<<kCheckGrid, kCheckBlock, 0, s>>>(h, seed, n_updates, counts);
    }
    return hipGetLastError();
}

}  // namespace fasgd
