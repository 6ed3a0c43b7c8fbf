// Dense server updates: state initialisation, the K-fused FASGD apply (also
// with a compacted B-FASGD push applied ahead of the K gradients in the same
// pass, and then optionally with the next push's transmit decisions taken
// from the v the pass leaves), the K-fused SASGD apply and the
// synchronous-SGD step.
//
// Every update is elementwise and HBM-bound, so the kernels are plain
// streaming passes: each thread owns 4 consecutive parameters (one 16-byte
// vector per state array; one parameter for a single-gradient pass), loads
// their state once, applies the K queued gradients in arrival order with the
// state in registers, and stores the state once.  Measured on MI355X:
//   - the grid covers the arrays exactly (one 16-byte chunk per thread) in
//     blocks of 128 threads; grid-stride loops over a few thousand blocks
//     lose 10-25 % of HBM bandwidth on streaming passes, and 128-thread
//     blocks beat 256 by up to 8 % on short (25M-parameter) passes;
//   - every load and store is non-temporal: nothing is re-read within a
//     pass, and streaming hints help the mixed read/write traffic most at
//     small K;
//   - the pass writes no per-parameter timestamps (the state records the
//     dense timestamp once), so the minimum traffic is 32/K + 4 bytes per
//     parameter-update for FASGD and 8/K + 4 for SASGD.
#include "kernels.hpp"

namespace fasgd {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 128;        // measured best for the streaming passes (2 waves)
constexpr int kBatch = 8;          // gradients loaded together before use

__device__ __forceinline__ f4 ld4(const float* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const f4*>(p));
}
__device__ __forceinline__ void st4(float* p, f4 x)
{
    __builtin_nontemporal_store(x, reinterpret_cast<f4*>(p));
}

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

unsigned grid_for(int64_t items)
{
    const int64_t g = (items + kBlock - 1) / kBlock;
    return static_cast<unsigned>(g < 1 ? 1 : g);
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
        last_T[j] = -1;
    }
}

// K-fused FASGD over 16-byte aligned arrays; thread i owns parameters
// 4i .. 4i+3, and the thread after the last full chunk owns the P mod 4 tail.
template <int MODE>
__global__ __launch_bounds__(kBlock) void fasgd_dense_vec(const DenseArgs a)
{
    const Hyper h = a.h;
    const int K = a.K;
    const int64_t nvec = a.P >> 2;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i < nvec) {
        const int64_t o = i * 4;
        f4 th = ld4(a.theta + o), n = ld4(a.n + o), b = ld4(a.b + o), v = ld4(a.v + o);
        int k = 0;
        for (; k + kBatch <= K; k += kBatch) {
            f4 g[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) g[u] = ld4(a.grad[k + u] + o);
#pragma unroll
            for (int u = 0; u < kBatch; ++u) fasgd_step4<MODE>(th, n, b, v, g[u], a.coef[k + u], h);
        }
        for (; k < K; ++k) fasgd_step4<MODE>(th, n, b, v, ld4(a.grad[k] + o), a.coef[k], h);
        st4(a.theta + o, th);
        st4(a.n + o, n);
        st4(a.b + o, b);
        st4(a.v + o, v);
    } else if (i == nvec) {
        for (int64_t j = nvec * 4; j < a.P; ++j) {
            float th = a.theta[j], n = a.n[j], b = a.b[j], v = a.v[j];
            for (int k = 0; k < K; ++k) fasgd_step<MODE>(th, n, b, v, a.grad[k][j], a.coef[k], h);
            a.theta[j] = th; a.n[j] = n; a.b[j] = b; a.v[j] = v;
        }
    }
}

// A compacted push applied in the same pass, before the K gradients (the
// arrival order when the push came in ahead of them).  Every wave of the
// vector kernel owns one kPushSeg-parameter segment (64 chunks of 4), so it
// finds the push's entries for its parameters at [seg_start[s],
// seg_start[s + 1]) of the list, clipped to min(count, capacity), and stages
// them in its LDS slice: one value and one flag byte per parameter.
// last_T is not written: the K gradients that follow update every parameter
// later than the push, and that last update is recorded once as dense_T
// (scattered 4-byte timestamp writes cost this pass about 8 % at 1e9
// parameters and a 10 % push; without them the pass takes as long as the
// dense pass alone).
constexpr int kWave = 64;
constexpr int kWavesPerBlock = kBlock / kWave;
static_assert(kWave * 4 == kPushSeg, "one vector-kernel wave covers one list-index segment");

__device__ __forceinline__ void wave_lds_order()
{
    // the wave's LDS operations execute in order; keep the compiler from
    // moving the reads of other lanes' entries above the writes
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Entries of segment seg, clipped to the list's usable length.
__device__ __forceinline__ void push_range(const PushArgs& p, int64_t seg, int64_t& lo, int64_t& hi)
{
    int64_t m = *p.d_count;
    m = m < p.capacity ? m : p.capacity;
    m = m > 0 ? m : 0;
    lo = hi = m;
    if (seg < p.n_segs) {
        const int64_t a0 = p.seg_start[seg], a1 = p.seg_start[seg + 1];
        lo = a0 < m ? a0 : m;
        hi = a1 < m ? a1 : m;
    }
}

// Stage the entries of [lo, hi) whose index lies in [first, first + span)
// (and below P): value at s_val[j - first], flag byte s_flag[j - first] = 1.
// The flags must have been cleared.
__device__ __forceinline__ void stage_push(const PushArgs& p, int64_t lo, int64_t hi, int64_t first, int span,
                                           int64_t P, float* s_val, uint8_t* s_flag, int lane)
{
    for (int64_t e = lo + lane; e < hi; e += kWave) {
        const int64_t x = static_cast<int64_t>(p.idx[e]) - first;
        if (x >= 0 && x < span && first + x < P) {
            s_val[x] = p.val[e];
            s_flag[x] = 1;
        }
    }
}

// MARK: the pass also takes the transmit decisions of the next push (Sec.
// 2.3) from the v it leaves, i.e. the selection's mark step on the v that a
// selection after the pass would read: one Philox call per chunk of 4, and
// the segment's 4 ballot words (word c: bit c of each of the 64 chunks) in
// the selection workspace, laid out as the mark launch lays them out.
template <int MODE, bool MARK>
__global__ __launch_bounds__(kBlock) void fasgd_dense_push_vec(const DenseArgs a, const PushArgs p, const SelectArgs m)
{
    __shared__ float s_val[kWavesPerBlock][kPushSeg];
    __shared__ uint32_t s_flag[kWavesPerBlock][kWave];    // byte c of word l: parameter 4 l + c listed
    const Hyper h = a.h;
    const int K = a.K;
    const int64_t nvec = a.P >> 2;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t seg = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + w;
    const int64_t first = seg * kPushSeg;
    const int64_t o = i * 4;
    // Loads in the order their data is needed, so that waiting for the list
    // entries does not wait for the state and gradient loads behind them:
    // the first 64 entries of the segment, then the state, then the first
    // batch of gradients.
    int64_t lo, hi;
    push_range(p, seg, lo, hi);
    int32_t e_idx = -1;
    float e_val = 0.0f;
    if (lo + lane < hi) { e_idx = p.idx[lo + lane]; e_val = p.val[lo + lane]; }
    const bool own = i < nvec;
    f4 th, n, b, v;
    if (own) { th = ld4(a.theta + o); n = ld4(a.n + o); b = ld4(a.b + o); v = ld4(a.v + o); }
    const int k0 = K < kBatch ? K : kBatch;
    f4 g0[kBatch];
    if (own) {
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
            if (u < k0) g0[u] = ld4(a.grad[u] + o);
    }
    // stage the push's entries for this segment
    s_flag[w][lane] = 0u;
    wave_lds_order();
    {
        const int64_t x = static_cast<int64_t>(e_idx) - first;
        if (e_idx >= 0 && x >= 0 && x < kPushSeg && first + x < a.P) {
            s_val[w][x] = e_val;
            reinterpret_cast<uint8_t*>(s_flag[w])[x] = 1;
        }
    }
    if (hi - lo > kWave)   // more than 64 entries in 256 parameters (transmit fraction above 1/4)
        stage_push(p, lo + kWave, hi, first, kPushSeg, a.P, s_val[w], reinterpret_cast<uint8_t*>(s_flag[w]), lane);
    wave_lds_order();
    const uint32_t flags = s_flag[w][lane];
    const f4 pv = *reinterpret_cast<const f4*>(&s_val[w][4 * lane]);
    if (own) {
        if (flags) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if ((flags >> (8 * c)) & 0xffu) {
                    float t = th[c], nn = n[c], bb = b[c], vv = v[c];
                    fasgd_step<MODE>(t, nn, bb, vv, pv[c], p.coef, h);
                    th[c] = t; n[c] = nn; b[c] = bb; v[c] = vv;
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
            if (u < k0) fasgd_step4<MODE>(th, n, b, v, g0[u], a.coef[u], h);
        int k = k0;
        for (; k + kBatch <= K; k += kBatch) {
            f4 g[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) g[u] = ld4(a.grad[k + u] + o);
#pragma unroll
            for (int u = 0; u < kBatch; ++u) fasgd_step4<MODE>(th, n, b, v, g[u], a.coef[k + u], h);
        }
        for (; k < K; ++k) fasgd_step4<MODE>(th, n, b, v, ld4(a.grad[k] + o), a.coef[k], h);
        st4(a.theta + o, th);
        st4(a.n + o, n);
        st4(a.b + o, b);
        st4(a.v + o, v);
    } else if (i == nvec) {
        for (int64_t j = nvec * 4; j < a.P; ++j) {
            const int c = static_cast<int>(j - nvec * 4);
            float tt = a.theta[j], nn = a.n[j], bb = a.b[j], vv = a.v[j];
            if ((flags >> (8 * c)) & 0xffu) fasgd_step<MODE>(tt, nn, bb, vv, pv[c], p.coef, h);
            for (int k = 0; k < K; ++k) fasgd_step<MODE>(tt, nn, bb, vv, a.grad[k][j], a.coef[k], h);
            a.theta[j] = tt; a.n[j] = nn; a.b[j] = bb; a.v[j] = vv;
            if (MARK) v[c] = vv;
        }
    }
    if (MARK) {
        if (blockIdx.x == 0 && threadIdx.x == 0) *m.groups_done = 0u;   // for the scan launch
        const int n_own = own ? 4 : (i == nvec ? static_cast<int>(a.P - 4 * nvec) : 0);
        uint32_t nib = 0;
        if (n_own > 0) {
            const uint64_t qg = m.chunk_base + static_cast<uint64_t>(i);   // global chunk index
            const uint4 wd = philox4x32_10(
                make_uint4(static_cast<uint32_t>(qg), static_cast<uint32_t>(qg >> 32), m.ctr_T, m.ctr_client),
                m.key0, m.key1);
            const uint32_t wds[4] = {wd.x, wd.y, wd.z, wd.w};
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (c < n_own) nib |= transmit_bit(wds[c], v[c], m.c, m.eps_c) << c;
        }
        uint64_t words[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) words[c] = __builtin_amdgcn_ballot_w64(((nib >> c) & 1u) != 0);
        const int64_t tile_segs = m.n_tiles * 4;   // segments the ballot array holds
        const uint64_t mine = lane == 0 ? words[0] : lane == 1 ? words[1] : lane == 2 ? words[2] : words[3];
        if (seg < tile_segs && lane < 4) m.ballots[seg * 4 + lane] = mine;
        // segments of the last tile beyond the grid hold no chunk: no bits
        const int64_t last_seg = static_cast<int64_t>(gridDim.x) * kWavesPerBlock - 1;
        if (seg == last_seg && lane < 4)
            for (int64_t s2 = seg + 1; s2 < tile_segs; ++s2) m.ballots[s2 * 4 + lane] = 0;
    }
}

// A push whose dropped values re-apply the client's most recent gradient
// (Sec. 2.3) in one pass: every wave merges its segment's list entries into
// the client's cache segment (staged as in the pass above), writes the
// segment back whole when it has entries, and applies the merged values as
// one gradient.  Bit for bit the list copy into the cache followed by a
// one-gradient pass over it, without the partial-sector writes of the copy.
template <int MODE>
__global__ __launch_bounds__(kBlock) void fasgd_cached_push_vec(const DenseArgs a, const PushArgs p,
                                                                float* __restrict__ cache)
{
    __shared__ float s_val[kWavesPerBlock][kPushSeg];
    __shared__ uint32_t s_flag[kWavesPerBlock][kWave];    // byte c of word l: parameter 4 l + c listed
    const Hyper h = a.h;
    const int64_t nvec = a.P >> 2;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t seg = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + w;
    const int64_t first = seg * kPushSeg;
    const int64_t o = i * 4;
    int64_t lo, hi;
    push_range(p, seg, lo, hi);
    int32_t e_idx = -1;
    float e_val = 0.0f;
    if (lo + lane < hi) { e_idx = p.idx[lo + lane]; e_val = p.val[lo + lane]; }
    const bool own = i < nvec;
    f4 th, n, b, v, cv;
    if (own) {
        th = ld4(a.theta + o); n = ld4(a.n + o); b = ld4(a.b + o); v = ld4(a.v + o);
        cv = ld4(cache + o);
    }
    s_flag[w][lane] = 0u;
    wave_lds_order();
    {
        const int64_t x = static_cast<int64_t>(e_idx) - first;
        if (e_idx >= 0 && x >= 0 && x < kPushSeg && first + x < a.P) {
            s_val[w][x] = e_val;
            reinterpret_cast<uint8_t*>(s_flag[w])[x] = 1;
        }
    }
    if (hi - lo > kWave)
        stage_push(p, lo + kWave, hi, first, kPushSeg, a.P, s_val[w], reinterpret_cast<uint8_t*>(s_flag[w]), lane);
    wave_lds_order();
    const uint32_t flags = s_flag[w][lane];
    const f4 pv = *reinterpret_cast<const f4*>(&s_val[w][4 * lane]);
    if (own) {
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if ((flags >> (8 * c)) & 0xffu) cv[c] = pv[c];
        if (hi > lo) st4(cache + o, cv);       // the segment has entries (wave-uniform)
        fasgd_step4<MODE>(th, n, b, v, cv, a.coef[0], h);
        st4(a.theta + o, th);
        st4(a.n + o, n);
        st4(a.b + o, b);
        st4(a.v + o, v);
    } else if (i == nvec) {
        for (int64_t j = nvec * 4; j < a.P; ++j) {
            const int c = static_cast<int>(j - nvec * 4);
            float gj = cache[j];
            if ((flags >> (8 * c)) & 0xffu) {
                gj = pv[c];
                cache[j] = gj;
            }
            float tt = a.theta[j], nn = a.n[j], bb = a.b[j], vv = a.v[j];
            fasgd_step<MODE>(tt, nn, bb, vv, gj, a.coef[0], h);
            a.theta[j] = tt; a.n[j] = nn; a.b[j] = bb; a.v[j] = vv;
        }
    }
}

// The listed values written into a dense array segment by segment (the
// fetch refresh of a client's copy of theta): a wave reads its segment
// whole, puts the segment's entries in and writes it back whole; segments
// without entries are not touched.  Full-line writes instead of one partial
// 32-byte sector per entry.
__global__ __launch_bounds__(kBlock) void merge_list_vec(float* __restrict__ dst, int64_t P, const PushArgs p)
{
    __shared__ float s_val[kWavesPerBlock][kPushSeg];
    __shared__ uint32_t s_flag[kWavesPerBlock][kWave];
    const int64_t nvec = P >> 2;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t seg = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + w;
    const int64_t first = seg * kPushSeg;
    int64_t lo, hi;
    push_range(p, seg, lo, hi);
    if (hi == lo) return;                      // wave-uniform: nothing listed here
    const bool own = i < nvec;
    f4 d;
    if (own) d = ld4(dst + i * 4);
    s_flag[w][lane] = 0u;
    wave_lds_order();
    stage_push(p, lo, hi, first, kPushSeg, P, s_val[w], reinterpret_cast<uint8_t*>(s_flag[w]), lane);
    wave_lds_order();
    const uint32_t flags = s_flag[w][lane];
    const f4 pv = *reinterpret_cast<const f4*>(&s_val[w][4 * lane]);
    if (own) {
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if ((flags >> (8 * c)) & 0xffu) d[c] = pv[c];
        st4(dst + i * 4, d);
    } else if (i == nvec) {
        for (int64_t j = nvec * 4; j < P; ++j) {
            const int c = static_cast<int>(j - nvec * 4);
            if ((flags >> (8 * c)) & 0xffu) dst[j] = pv[c];
        }
    }
}

// The same, one parameter per thread (arrays only 4-byte aligned): a wave
// covers 64 parameters, a quarter of a list-index segment.
template <int MODE>
__global__ __launch_bounds__(kBlock) void fasgd_dense_push_scalar(const DenseArgs a, const PushArgs p)
{
    __shared__ float s_val[kWavesPerBlock][kWave];
    __shared__ uint8_t s_flag[kWavesPerBlock][kWave];
    const Hyper h = a.h;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t first = static_cast<int64_t>(blockIdx.x) * kBlock + w * kWave;   // the wave's first parameter
    const int64_t j = first + lane;
    int64_t lo, hi;
    push_range(p, first / kPushSeg, lo, hi);
    s_flag[w][lane] = 0;
    wave_lds_order();
    stage_push(p, lo, hi, first, kWave, a.P, s_val[w], s_flag[w], lane);
    wave_lds_order();
    if (j >= a.P) return;
    float th = a.theta[j], n = a.n[j], b = a.b[j], v = a.v[j];
    if (s_flag[w][lane]) fasgd_step<MODE>(th, n, b, v, s_val[w][lane], p.coef, h);
    for (int k = 0; k < a.K; ++k) fasgd_step<MODE>(th, n, b, v, a.grad[k][j], a.coef[k], h);
    a.theta[j] = th; a.n[j] = n; a.b[j] = b; a.v[j] = v;
}

// Same update, one parameter per thread: for arrays that are only 4-byte
// aligned, and for passes with one gradient (K = 1), where it measured
// 3-8 % faster than 4 parameters per thread at 1e9 parameters and 2.5 %
// at 25M (at K = 32 the two are within 1 %).
template <int MODE>
__global__ __launch_bounds__(kBlock) void fasgd_dense_scalar(const DenseArgs a)
{
    const Hyper h = a.h;
    const int K = a.K;
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (j >= a.P) return;
    float th = __builtin_nontemporal_load(a.theta + j), n = __builtin_nontemporal_load(a.n + j);
    float b = __builtin_nontemporal_load(a.b + j), v = __builtin_nontemporal_load(a.v + j);
    int k = 0;
    for (; k + kBatch <= K; k += kBatch) {
        float g[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) g[u] = __builtin_nontemporal_load(a.grad[k + u] + j);
#pragma unroll
        for (int u = 0; u < kBatch; ++u) fasgd_step<MODE>(th, n, b, v, g[u], a.coef[k + u], h);
    }
    for (; k < K; ++k) fasgd_step<MODE>(th, n, b, v, __builtin_nontemporal_load(a.grad[k] + j), a.coef[k], h);
    __builtin_nontemporal_store(th, a.theta + j);
    __builtin_nontemporal_store(n, a.n + j);
    __builtin_nontemporal_store(b, a.b + j);
    __builtin_nontemporal_store(v, a.v + j);
}

// K-fused SASGD: theta <- theta - (alpha / tau_k) g_k; coef[k] = alpha / tau_k.
__global__ __launch_bounds__(kBlock) void sasgd_dense_vec(const DenseArgs a)
{
    const int K = a.K;
    const int64_t nvec = a.P >> 2;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i < nvec) {
        const int64_t o = i * 4;
        f4 th = ld4(a.theta + o);
        int k = 0;
        for (; k + kBatch <= K; k += kBatch) {
            f4 g[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) g[u] = ld4(a.grad[k + u] + o);
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const float r = -a.coef[k + u];
#pragma unroll
                for (int c = 0; c < 4; ++c) th[c] = fmaf(r, g[u][c], th[c]);
            }
        }
        for (; k < K; ++k) {
            const f4 g = ld4(a.grad[k] + o);
            const float r = -a.coef[k];
#pragma unroll
            for (int c = 0; c < 4; ++c) th[c] = fmaf(r, g[c], th[c]);
        }
        st4(a.theta + o, th);
    } else if (i == nvec) {
        for (int64_t j = nvec * 4; j < a.P; ++j) {
            float th = a.theta[j];
            for (int k = 0; k < K; ++k) th = fmaf(-a.coef[k], a.grad[k][j], th);
            a.theta[j] = th;
        }
    }
}

__global__ __launch_bounds__(kBlock) void sasgd_dense_scalar(const DenseArgs a)
{
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (j >= a.P) return;
    float th = a.theta[j];
    for (int k = 0; k < a.K; ++k) th = fmaf(-a.coef[k], a.grad[k][j], th);
    a.theta[j] = th;
}

// Synchronous SGD (the apply-update listing of Sec. 3): every gradient is
// divided by lambda, then theta <- theta - lr * that, in client order.
__global__ __launch_bounds__(kBlock) void sync_sgd_vec(const DenseArgs a)
{
    const int K = a.K;
    const float lam = a.lambda;
    const int64_t nvec = a.P >> 2;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i < nvec) {
        const int64_t o = i * 4;
        f4 th = ld4(a.theta + o);
        int k = 0;
        for (; k + kBatch <= K; k += kBatch) {
            f4 g[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) g[u] = ld4(a.grad[k + u] + o);
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const float r = -a.coef[k + u];
#pragma unroll
                for (int c = 0; c < 4; ++c) th[c] = fmaf(r, g[u][c] / lam, th[c]);
            }
        }
        for (; k < K; ++k) {
            const f4 g = ld4(a.grad[k] + o);
            const float r = -a.coef[k];
#pragma unroll
            for (int c = 0; c < 4; ++c) th[c] = fmaf(r, g[c] / lam, th[c]);
        }
        st4(a.theta + o, th);
    } else if (i == nvec) {
        for (int64_t j = nvec * 4; j < a.P; ++j) {
            float th = a.theta[j];
            for (int k = 0; k < K; ++k) th = fmaf(-a.coef[k], a.grad[k][j] / lam, th);
            a.theta[j] = th;
        }
    }
}

__global__ __launch_bounds__(kBlock) void sync_sgd_scalar(const DenseArgs a)
{
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (j >= a.P) return;
    float th = a.theta[j];
    for (int k = 0; k < a.K; ++k) th = fmaf(-a.coef[k], a.grad[k][j] / a.lambda, th);
    a.theta[j] = th;
}

}  // namespace

hipError_t launch_init(float* n, float* b, float* v, int32_t* last_T, int64_t P,
                       float n0, float b0, float v0, hipStream_t s)
{
    init_kernel<<<grid_for(P < kMaxScalarItems ? P : kMaxScalarItems), kBlock, 0, s>>>(n, b, v, last_T, P, n0, b0, v0);
    return hipGetLastError();
}

template <int VARIANT>
void launch_dense_variant(const DenseArgs& a, bool aligned, unsigned grid, hipStream_t s)
{
    if (aligned)
        fasgd_dense_vec<VARIANT><<<grid, kBlock, 0, s>>>(a);
    else
        fasgd_dense_scalar<VARIANT><<<grid, kBlock, 0, s>>>(a);
}

template <int VARIANT>
void launch_push_variant(const DenseArgs& a, const PushArgs& p, const SelectArgs* m, bool aligned, unsigned grid,
                         hipStream_t s)
{
    if (m)
        fasgd_dense_push_vec<VARIANT, true><<<grid, kBlock, 0, s>>>(a, p, *m);
    else if (aligned)
        fasgd_dense_push_vec<VARIANT, false><<<grid, kBlock, 0, s>>>(a, p, SelectArgs{});
    else
        fasgd_dense_push_scalar<VARIANT><<<grid, kBlock, 0, s>>>(a, p);
}

hipError_t launch_fasgd_dense_push(const DenseArgs& a, const PushArgs& p, const SelectArgs* mark, int variant,
                                   bool aligned, hipStream_t s)
{
    if (mark && !aligned) return hipErrorInvalidValue;   // the decisions ride on the vector kernel only
    const unsigned grid = aligned ? grid_for((a.P >> 2) + 1) : grid_for(a.P);
    switch (variant) {
    case kernel_variant(MATH_FAST, 0): launch_push_variant<kernel_variant(MATH_FAST, 0)>(a, p, mark, aligned, grid, s); break;
    case kernel_variant(MATH_IEEE, 0): launch_push_variant<kernel_variant(MATH_IEEE, 0)>(a, p, mark, aligned, grid, s); break;
    case kernel_variant(MATH_FAST, 1): launch_push_variant<kernel_variant(MATH_FAST, 1)>(a, p, mark, aligned, grid, s); break;
    case kernel_variant(MATH_IEEE, 1): launch_push_variant<kernel_variant(MATH_IEEE, 1)>(a, p, mark, aligned, grid, s); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_fasgd_dense(const DenseArgs& a, int variant, bool aligned, hipStream_t s)
{
    // vector path (nvec chunks plus one thread for the tail) for K > 1 over
    // 16-byte aligned arrays, and for any K beyond the one-per-thread limit;
    // one parameter per thread otherwise
    const bool vec = aligned && (a.K > 1 || a.P > kMaxScalarItems);
    if (!vec && a.P > kMaxScalarItems) return hipErrorInvalidValue;   // the API rejects this first
    const unsigned grid = vec ? grid_for((a.P >> 2) + 1) : grid_for(a.P);
    switch (variant) {
    case kernel_variant(MATH_FAST, 0): launch_dense_variant<kernel_variant(MATH_FAST, 0)>(a, vec, grid, s); break;
    case kernel_variant(MATH_IEEE, 0): launch_dense_variant<kernel_variant(MATH_IEEE, 0)>(a, vec, grid, s); break;
    case kernel_variant(MATH_FAST, 1): launch_dense_variant<kernel_variant(MATH_FAST, 1)>(a, vec, grid, s); break;
    case kernel_variant(MATH_IEEE, 1): launch_dense_variant<kernel_variant(MATH_IEEE, 1)>(a, vec, grid, s); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_fasgd_cached_push(const DenseArgs& a, const PushArgs& p, float* cache, int variant, hipStream_t s)
{
    const unsigned grid = grid_for((a.P >> 2) + 1);
    switch (variant) {
    case kernel_variant(MATH_FAST, 0): fasgd_cached_push_vec<kernel_variant(MATH_FAST, 0)><<<grid, kBlock, 0, s>>>(a, p, cache); break;
    case kernel_variant(MATH_IEEE, 0): fasgd_cached_push_vec<kernel_variant(MATH_IEEE, 0)><<<grid, kBlock, 0, s>>>(a, p, cache); break;
    case kernel_variant(MATH_FAST, 1): fasgd_cached_push_vec<kernel_variant(MATH_FAST, 1)><<<grid, kBlock, 0, s>>>(a, p, cache); break;
    case kernel_variant(MATH_IEEE, 1): fasgd_cached_push_vec<kernel_variant(MATH_IEEE, 1)><<<grid, kBlock, 0, s>>>(a, p, cache); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_merge_list(float* dst, int64_t P, const PushArgs& p, hipStream_t s)
{
    merge_list_vec<<<grid_for((P >> 2) + 1), kBlock, 0, s>>>(dst, P, p);
    return hipGetLastError();
}

hipError_t launch_sasgd_dense(const DenseArgs& a, bool aligned, hipStream_t s)
{
    if (aligned)
        sasgd_dense_vec<<<grid_for((a.P >> 2) + 1), kBlock, 0, s>>>(a);
    else
        sasgd_dense_scalar<<<grid_for(a.P), kBlock, 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_sync_sgd(const DenseArgs& a, bool aligned, hipStream_t s)
{
    if (aligned)
        sync_sgd_vec<<<grid_for((a.P >> 2) + 1), kBlock, 0, s>>>(a);
    else
        sync_sgd_scalar<<<grid_for(a.P), kBlock, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace fasgd
