// The bandwidth anchor: a plain streaming copy of a float array, one 16-byte
// vector per thread over an exact-cover grid, non-temporal loads and stores
// (the access pattern of the library's passes).  Its rate on a box is what
// that box's HBM achieves for one read and one write stream, the yardstick
// the passes' rates are set against.
#include "anchor.hpp"

namespace fasgd {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kAnchorBlock = 256;

// n4 vectors, then the n % 4 trailing floats (by the thread past the last vector)
__global__ __launch_bounds__(kAnchorBlock) void copy_anchor(const float* __restrict__ src, float* __restrict__ dst,
                                                            int64_t n4, int tail)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kAnchorBlock + threadIdx.x;
    if (i < n4) {
        const f4 x = __builtin_nontemporal_load(reinterpret_cast<const f4*>(src) + i);
        __builtin_nontemporal_store(x, reinterpret_cast<f4*>(dst) + i);
    } else if (i == n4) {
        for (int k = 0; k < tail; ++k) dst[4 * n4 + k] = src[4 * n4 + k];
    }
}

}  // namespace

hipError_t launch_copy_anchor(const float* src, float* dst, int64_t n, hipStream_t s)
{
    const int64_t n4 = n / 4;
    const int tail = static_cast<int>(n % 4);
    const int64_t blocks = (n4 + 1 + kAnchorBlock - 1) / kAnchorBlock;   // n4 + 1 threads
    copy_anchor<<<static_cast<unsigned>(blocks), kAnchorBlock, 0, s>>>(src, dst, n4, tail);
    return hipGetLastError();
}

}  // namespace fasgd
