// B-FASGD as the paper states it: one transmit decision per push from v
// averaged over all parameters (Sec. 2.3), or one per tensor segment from
// that segment's mean (the per-tensor direction of Sec. 5), and the server
// apply of a push decided that way.
//
// Segments are handled in groups of up to kSegGroup whose offsets and block
// counts travel in the kernel arguments, so the host never copies to the
// device.  Every segment is cut into blocks of kSegSpan parameters:
//   seg_partial  one fp64 partial sum of v per block, in a fixed order;
//   seg_decide   one block of 1024 threads per segment folds its partials in
//                a fixed order, divides by the length and decides in fp64;
//   seg_apply    the FASGD update on the blocks of transmitted segments.
// Sums are deterministic run to run (fixed assignment and reduction order).
#include "kernels.hpp"

namespace fasgd {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kThreads = 256;
constexpr int kPerThread = 16;                         // 4 vectors of 4
constexpr int64_t kSegSpan = int64_t(kThreads) * kPerThread;

// block b of the group -> (segment i of the group, first parameter, end)
__device__ __forceinline__ void block_range(const SegGroup& g, int64_t b, int& i, int64_t& lo, int64_t& hi)
{
    i = 0;
    while (i + 1 < g.n && b >= g.block_prefix[i + 1]) ++i;
    lo = g.start[i] + (b - g.block_prefix[i]) * kSegSpan;
    hi = lo + kSegSpan < g.start[i + 1] ? lo + kSegSpan : g.start[i + 1];
}

constexpr int kDecideThreads = 1024;   // one block folds a segment's partials
constexpr int kDecideAcc = 4;          // independent accumulators per thread
static_assert(kDecideAcc == 4, "the fold below combines four sums");

template <int THREADS>
__device__ __forceinline__ double block_sum(double x)
{
    __shared__ double wave_sum[THREADS / kWave];
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) x += __shfl_xor(x, d, kWave);
    if ((threadIdx.x & (kWave - 1)) == 0) wave_sum[threadIdx.x / kWave] = x;
    __syncthreads();
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < THREADS / kWave; ++w) s += wave_sum[w];
    return s;
}

__global__ __launch_bounds__(kThreads) void seg_partial(const SegGroup g, const float* __restrict__ v,
                                                        double* __restrict__ partial)
{
    int i;
    int64_t lo, hi;
    block_range(g, blockIdx.x, i, lo, hi);
    double acc = 0.0;
    if ((lo & 3) == 0 && (reinterpret_cast<uintptr_t>(v) & 15) == 0 && hi - lo == kSegSpan) {
#pragma unroll
        for (int k = 0; k < kPerThread / 4; ++k) {
            const f4 x = __builtin_nontemporal_load(reinterpret_cast<const f4*>(v + lo) + k * kThreads + threadIdx.x);
            acc += static_cast<double>(x[0]) + static_cast<double>(x[1]) + static_cast<double>(x[2]) +
                   static_cast<double>(x[3]);
        }
    } else {
        for (int64_t j = lo + threadIdx.x; j < hi; j += kThreads) acc += static_cast<double>(v[j]);
    }
    const double s = block_sum<kThreads>(acc);
    if (threadIdx.x == 0) partial[g.partial_base + blockIdx.x] = s;
}

__global__ __launch_bounds__(kDecideThreads) void seg_decide(const SegGroup g, const double* __restrict__ partial,
                                                       float c, float eps_c, uint32_t key0, uint32_t key1,
                                                       uint32_t ctr_T, uint32_t ctr_client,
                                                       uint8_t* __restrict__ transmit)
{
    const int i = blockIdx.x;
    // thread t folds partials t, t + 1024, ... into kDecideAcc running sums
    // (loads of one round issued together), then the sums in a fixed order
    double acc[kDecideAcc] = {0.0, 0.0, 0.0, 0.0};
    const int64_t end = g.block_prefix[i + 1];
    for (int64_t b = g.block_prefix[i] + threadIdx.x; b < end; b += kDecideAcc * kDecideThreads) {
#pragma unroll
        for (int q = 0; q < kDecideAcc; ++q) {
            const int64_t bq = b + q * kDecideThreads;
            if (bq < end) acc[q] += partial[g.partial_base + bq];
        }
    }
    const double sum = block_sum<kDecideThreads>((acc[0] + acc[1]) + (acc[2] + acc[3]));
    if (threadIdx.x == 0) {
        const int64_t s = g.first_seg + i;
        const double mean = sum / static_cast<double>(g.start[i + 1] - g.start[i]);
        const uint4 w = philox4x32_10(
            make_uint4(static_cast<uint32_t>(s), 0x80000000u | static_cast<uint32_t>(static_cast<uint64_t>(s) >> 32),
                       ctr_T, ctr_client),
            key0, key1);
        const double r = static_cast<double>(w.x >> 8) * 0x1p-24;
        const double t = mean + static_cast<double>(eps_c);
        const double u = t + static_cast<double>(c);
        transmit[s] = fma(r, u, -t) < 0.0 ? 1 : 0;
    }
}

template <int MODE>
__global__ __launch_bounds__(kThreads) void seg_apply(const SegGroup g, const SegApplyArgs a)
{
    int i;
    int64_t lo, hi;
    block_range(g, blockIdx.x, i, lo, hi);
    if (!a.transmit[g.first_seg + i]) return;
    const Hyper h = a.h;
    const bool vec = (lo & 3) == 0 && hi - lo == kSegSpan && a.aligned;
    if (vec) {
#pragma unroll
        for (int k = 0; k < kPerThread / 4; ++k) {
            const int64_t o = lo + (static_cast<int64_t>(k) * kThreads + threadIdx.x) * 4;
            f4 th = *reinterpret_cast<const f4*>(a.theta + o), n = *reinterpret_cast<const f4*>(a.n + o);
            f4 b = *reinterpret_cast<const f4*>(a.b + o), v = *reinterpret_cast<const f4*>(a.v + o);
            const f4 gr = __builtin_nontemporal_load(reinterpret_cast<const f4*>(a.grad + o));
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) {
                float t = th[cc], nn = n[cc], bb = b[cc], vv = v[cc];
                fasgd_step<MODE>(t, nn, bb, vv, gr[cc], a.coef, h);
                th[cc] = t; n[cc] = nn; b[cc] = bb; v[cc] = vv;
            }
            *reinterpret_cast<f4*>(a.theta + o) = th;
            *reinterpret_cast<f4*>(a.n + o) = n;
            *reinterpret_cast<f4*>(a.b + o) = b;
            *reinterpret_cast<f4*>(a.v + o) = v;
            const int32_t T = a.last_T_value;
            *reinterpret_cast<int4*>(a.last_T + o) = make_int4(T, T, T, T);
        }
    } else {
        for (int64_t j = lo + threadIdx.x; j < hi; j += kThreads) {
            float th = a.theta[j], n = a.n[j], b = a.b[j], v = a.v[j];
            fasgd_step<MODE>(th, n, b, v, a.grad[j], a.coef, h);
            a.theta[j] = th; a.n[j] = n; a.b[j] = b; a.v[j] = v;
            a.last_T[j] = a.last_T_value;
        }
    }
}

}  // namespace

int64_t seg_blocks(int64_t length) { return (length + kSegSpan - 1) / kSegSpan; }

size_t segments_workspace_bytes(int64_t P, int32_t S)
{
    const int64_t blocks = (P + kSegSpan - 1) / kSegSpan + S;
    return ((size_t(blocks) * sizeof(double)) + 255) & ~size_t(255);
}

hipError_t launch_seg_decide(const SegGroup& g, const float* v, double* partial, float c, float eps_c,
                             uint64_t seed, uint32_t ctr_T, uint32_t ctr_client, uint8_t* transmit,
                             hipStream_t s)
{
    const unsigned blocks = static_cast<unsigned>(g.block_prefix[g.n]);
    seg_partial<<<blocks, kThreads, 0, s>>>(g, v, partial);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    seg_decide<<<static_cast<unsigned>(g.n), kDecideThreads, 0, s>>>(g, partial, c, eps_c, static_cast<uint32_t>(seed),
                                                              static_cast<uint32_t>(seed >> 32), ctr_T, ctr_client,
                                                              transmit);
    return hipGetLastError();
}

hipError_t launch_seg_apply(const SegGroup& g, const SegApplyArgs& a, int variant, hipStream_t s)
{
    const unsigned blocks = static_cast<unsigned>(g.block_prefix[g.n]);
    switch (variant) {
    case kernel_variant(MATH_FAST, 0): seg_apply<kernel_variant(MATH_FAST, 0)><<<blocks, kThreads, 0, s>>>(g, a); break;
    case kernel_variant(MATH_IEEE, 0): seg_apply<kernel_variant(MATH_IEEE, 0)><<<blocks, kThreads, 0, s>>>(g, a); break;
    case kernel_variant(MATH_FAST, 1): seg_apply<kernel_variant(MATH_FAST, 1)><<<blocks, kThreads, 0, s>>>(g, a); break;
    case kernel_variant(MATH_IEEE, 1): seg_apply<kernel_variant(MATH_IEEE, 1)><<<blocks, kThreads, 0, s>>>(g, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace fasgd
