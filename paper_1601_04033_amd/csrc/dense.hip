// Dense server updates: state initialisation, the K-fused FASGD apply and
// the K-fused SASGD apply.
//
// Every update is elementwise and HBM-bound, so the kernels are plain
// streaming passes: each thread owns 4 consecutive parameters (one 16-byte
// vector per state array), loads their state once, applies the K queued
// gradients in arrival order with the state in registers, and stores the
// state once.  Gradients are read once and never reused, so they are loaded
// non-temporally.  Grid-stride loops keep the launch at a fixed size.
#include <stdlib.h>

#include "kernels.hpp"

namespace fasgd {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef int i4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;
constexpr int kBatch = 8;          // gradients loaded together before use

__device__ __forceinline__ f4 ld4(const float* p) { return *reinterpret_cast<const f4*>(p); }
__device__ __forceinline__ f4 ld4_stream(const float* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const f4*>(p));
}
__device__ __forceinline__ void st4(float* p, f4 x) { *reinterpret_cast<f4*>(p) = x; }

template <int MODE>
__device__ __forceinline__ void fasgd_step4(f4& th, f4& n, f4& b, f4& v, const f4 g, float coef,
                                            const Hyper& h)
{
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        float t = th[c], nn = n[c], bb = b[c], vv = v[c];
        fasgd_step<MODE>(t, nn, bb, vv, g[c], coef, h);
        th[c] = t; n[c] = nn; b[c] = bb; v[c] = vv;
    }
}

int grid_for(int64_t work_items)
{
    // Enough resident waves to cover HBM latency on 256 CUs; more blocks
    // only add scheduling overhead to a grid-stride loop.
    static const int64_t cap = [] {
        const char* e = getenv("FASGD_DENSE_MAX_BLOCKS");
        int64_t v = e ? atoll(e) : 0;
        return v > 0 ? v : int64_t(256) * 16;
    }();
    int64_t g = (work_items + kBlock - 1) / kBlock;
    if (g > cap) g = cap;
    return static_cast<int>(g < 1 ? 1 : g);
}

__global__ __launch_bounds__(kBlock) void init_kernel(float* __restrict__ n, float* __restrict__ b,
                                                      float* __restrict__ v, int32_t* __restrict__ last_T,
                                                      int64_t P, float n0, float b0, float v0)
{
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; j < P; j += stride) {
        if (n) n[j] = n0;
        if (b) b[j] = b0;
        if (v) v[j] = v0;
        if (last_T) last_T[j] = -1;
    }
}

// K-fused FASGD over 16-byte aligned arrays.
template <int MODE>
__global__ __launch_bounds__(kBlock) void fasgd_dense_vec(const DenseArgs a)
{
    const Hyper h = a.h;
    const int K = a.K;
    const int64_t nvec = a.P >> 2;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    const i4 stamp = {a.last_T_value, a.last_T_value, a.last_T_value, a.last_T_value};
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < nvec; i += stride) {
        const int64_t o = i * 4;
        f4 th = ld4(a.theta + o), n = ld4(a.n + o), b = ld4(a.b + o), v = ld4(a.v + o);
        int k = 0;
        for (; k + kBatch <= K; k += kBatch) {
            f4 g[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) g[u] = ld4_stream(a.grad[k + u] + o);
#pragma unroll
            for (int u = 0; u < kBatch; ++u) fasgd_step4<MODE>(th, n, b, v, g[u], a.coef[k + u], h);
        }
        for (; k < K; ++k) fasgd_step4<MODE>(th, n, b, v, ld4_stream(a.grad[k] + o), a.coef[k], h);
        st4(a.theta + o, th);
        st4(a.n + o, n);
        st4(a.b + o, b);
        st4(a.v + o, v);
        *reinterpret_cast<i4*>(a.last_T + o) = stamp;
    }
    // the last P mod 4 parameters
    if (blockIdx.x == 0 && threadIdx.x < static_cast<unsigned>(a.P & 3)) {
        const int64_t j = nvec * 4 + threadIdx.x;
        float th = a.theta[j], n = a.n[j], b = a.b[j], v = a.v[j];
        for (int k = 0; k < K; ++k) fasgd_step<MODE>(th, n, b, v, a.grad[k][j], a.coef[k], h);
        a.theta[j] = th; a.n[j] = n; a.b[j] = b; a.v[j] = v;
        a.last_T[j] = a.last_T_value;
    }
}

// Same update, one parameter per thread, for arrays that are only 4-byte aligned.
template <int MODE>
__global__ __launch_bounds__(kBlock) void fasgd_dense_scalar(const DenseArgs a)
{
    const Hyper h = a.h;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; j < a.P; j += stride) {
        float th = a.theta[j], n = a.n[j], b = a.b[j], v = a.v[j];
        for (int k = 0; k < a.K; ++k) fasgd_step<MODE>(th, n, b, v, a.grad[k][j], a.coef[k], h);
        a.theta[j] = th; a.n[j] = n; a.b[j] = b; a.v[j] = v;
        a.last_T[j] = a.last_T_value;
    }
}

// K-fused SASGD: theta <- theta - (alpha / tau_k) g_k; coef[k] = alpha / tau_k.
__global__ __launch_bounds__(kBlock) void sasgd_dense_vec(const DenseArgs a)
{
    const int K = a.K;
    const int64_t nvec = a.P >> 2;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    const i4 stamp = {a.last_T_value, a.last_T_value, a.last_T_value, a.last_T_value};
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < nvec; i += stride) {
        const int64_t o = i * 4;
        f4 th = ld4(a.theta + o);
        int k = 0;
        for (; k + kBatch <= K; k += kBatch) {
            f4 g[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) g[u] = ld4_stream(a.grad[k + u] + o);
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const float r = -a.coef[k + u];
#pragma unroll
                for (int c = 0; c < 4; ++c) th[c] = fmaf(r, g[u][c], th[c]);
            }
        }
        for (; k < K; ++k) {
            const f4 g = ld4_stream(a.grad[k] + o);
            const float r = -a.coef[k];
#pragma unroll
            for (int c = 0; c < 4; ++c) th[c] = fmaf(r, g[c], th[c]);
        }
        st4(a.theta + o, th);
        if (a.last_T) *reinterpret_cast<i4*>(a.last_T + o) = stamp;
    }
    if (blockIdx.x == 0 && threadIdx.x < static_cast<unsigned>(a.P & 3)) {
        const int64_t j = nvec * 4 + threadIdx.x;
        float th = a.theta[j];
        for (int k = 0; k < K; ++k) th = fmaf(-a.coef[k], a.grad[k][j], th);
        a.theta[j] = th;
        if (a.last_T) a.last_T[j] = a.last_T_value;
    }
}

__global__ __launch_bounds__(kBlock) void sasgd_dense_scalar(const DenseArgs a)
{
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; j < a.P; j += stride) {
        float th = a.theta[j];
        for (int k = 0; k < a.K; ++k) th = fmaf(-a.coef[k], a.grad[k][j], th);
        a.theta[j] = th;
        if (a.last_T) a.last_T[j] = a.last_T_value;
    }
}

}  // namespace

hipError_t launch_init(float* n, float* b, float* v, int32_t* last_T, int64_t P,
                       float n0, float b0, float v0, hipStream_t s)
{
    init_kernel<<<grid_for(P), kBlock, 0, s>>>(n, b, v, last_T, P, n0, b0, v0);
    return hipGetLastError();
}

hipError_t launch_fasgd_dense(const DenseArgs& a, int mode, bool aligned, hipStream_t s)
{
    if (aligned) {
        const int grid = grid_for(a.P >> 2 > 0 ? a.P >> 2 : 1);
        if (mode == MATH_FAST)
            fasgd_dense_vec<MATH_FAST><<<grid, kBlock, 0, s>>>(a);
        else
            fasgd_dense_vec<MATH_IEEE><<<grid, kBlock, 0, s>>>(a);
    } else {
        const int grid = grid_for(a.P);
        if (mode == MATH_FAST)
            fasgd_dense_scalar<MATH_FAST><<<grid, kBlock, 0, s>>>(a);
        else
            fasgd_dense_scalar<MATH_IEEE><<<grid, kBlock, 0, s>>>(a);
    }
    return hipGetLastError();
}

hipError_t launch_sasgd_dense(const DenseArgs& a, bool aligned, hipStream_t s)
{
    if (aligned)
        sasgd_dense_vec<<<grid_for(a.P >> 2 > 0 ? a.P >> 2 : 1), kBlock, 0, s>>>(a);
    else
        sasgd_dense_scalar<<<grid_for(a.P), kBlock, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace fasgd
