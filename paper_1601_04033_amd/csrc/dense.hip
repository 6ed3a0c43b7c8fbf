// Dense server updates: state initialisation, the K-fused FASGD apply (also
// with a compacted B-FASGD push applied ahead of the K gradients in the same
// pass, and then optionally with the next push's transmit decisions taken
// from the v the pass leaves), the K-fused SASGD apply and the
// synchronous-SGD step.
//
// Every update is elementwise and HBM-bound, so the kernels are plain
// streaming passes: each thread loads its parameters' state once, applies
// the K queued gradients in arrival order with the state in registers, and
// stores the state once.  Below kMaxScalarItems parameters every pass runs
// one parameter per thread (any 4-byte alignment); beyond it, where one
// thread per parameter no longer fits a launch, 16-byte aligned arrays run 4
// parameters per thread.  Measured on MI355X:
//   - one parameter per thread with a few gradient loads in flight (few
//     VGPRs, the full 8 waves per SIMD) beats 4 per thread (16-byte loads,
//     4-6 waves per SIMD) by 5-10 % on the K-fused passes, see kLaneBlock;
//   - the grid covers the arrays exactly; grid-stride loops over a few
//     thousand blocks lose 10-25 % of HBM bandwidth on streaming passes;
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

constexpr int kBlock = 128;        // the 4-per-thread passes (2 waves)
constexpr int kBatch = 8;          // their gradients loaded together before use

// One parameter per thread: the form of every pass below kMaxScalarItems.
// Measured on MI355X at K = 32 against 4 parameters per thread (78-104
// VGPRs, 4-6 waves per SIMD), same box: the FASGD pass 648 against 714 us at
// 25M parameters (77 % against 70 % of 8 TB/s) and 26.9 against 28.9 ms at
// 1e9; at K = 8, 80 % against 73 %.  The FASGD pass loads its gradients
// kLaneBatch at a time (25 VGPRs, 8 waves per SIMD, the most a SIMD holds;
// batches of 2, 4, 6 measured 2-7 % slower) in blocks of kLaneBlock threads
// (128 and 512: 2-5 % slower).  The pass with a push, SASGD and synchronous
// SGD take 4 at a time (measured best for each; SASGD 0.52 against 0.56 ms
// at 25M).
constexpr int kLaneBlock = 256;
constexpr int kLaneBatch = 3;
constexpr int kPushBatch = 4;      // the pass with a push: 647 against 694 us at 25M with 3, 28.1 against 29.3 ms at 1e9
constexpr int kSgdBatch = 4;       // SASGD and synchronous SGD

unsigned lane_grid(int64_t P) { return static_cast<unsigned>((P + kLaneBlock - 1) / kLaneBlock); }

__device__ __forceinline__ f4 ld4(const float* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const f4*>(p));
}
__device__ __forceinline__ void st4(float* p, f4 x)
{
    __builtin_nontemporal_store(x, reinterpret_cast<f4*>(p));
}
__device__ __forceinline__ float ldnt(const float* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void stnt(float* p, float x) { __builtin_nontemporal_store(x, p); }

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

// The pass with a push, 4 parameters per thread, for 16-byte aligned
// arrays beyond kMaxScalarItems parameters (below it fasgd_dense_push_lane).
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

// Block barrier that orders the block's LDS accesses only: outstanding
// global loads are not waited for.
__device__ __forceinline__ void block_barrier_lds()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Stage, in the block's LDS, the entries of list-index segment blockIdx.x
// (thread t: entry lo + t, at most kPushSeg of them) at their parameters:
// value s_val[x] and flag byte s_flag[x] for parameter first + x.  e_idx and
// e_val are the thread's entry, loaded by the caller (entry lo + t when
// lo + t < hi).  Ends with the block's LDS ordered.
__device__ __forceinline__ void stage_segment(int32_t e_idx, float e_val, bool entry, int64_t first, int64_t P,
                                              float* s_val, uint8_t* s_flag)
{
    s_flag[threadIdx.x] = 0;
    block_barrier_lds();
    if (entry) {
        const int64_t x = static_cast<int64_t>(e_idx) - first;
        if (x >= 0 && x < kPushSeg && first + x < P) {
            s_val[x] = e_val;
            s_flag[x] = 1;
        }
    }
    block_barrier_lds();
}

// The pass with a compacted push applied ahead of the K gradients, one
// parameter per thread (any 4-byte alignment).  Block s owns list-index
// segment s (kPushSeg parameters).  Thread t loads entry lo + t of the
// segment's list range [lo, hi) (a segment holds at most kPushSeg entries:
// the indices are distinct) and stages it in the block's LDS, a value and a
// flag byte at its parameter.  Every global load is issued by every thread
// (addresses kept inside the arrays), so waits are for the loads they need.
// MARK: the pass also takes the next push's transmit decisions from the v it
// leaves: each thread draws the Philox call of its parameter's chunk of 4
// and keeps the word of its parameter; the wave's ballot (64 parameters, 16
// chunks) gives bits 16 w .. 16 w + 15 of each of the segment's 4 ballot
// words (word c: bit c of each of the segment's 64 chunks), which lanes
// 0..3 store as 16-bit pieces, in the layout the selection's mark launch
// writes.
template <int MODE, bool MARK>
__global__ __launch_bounds__(kLaneBlock) void fasgd_dense_push_lane(const DenseArgs a, const PushArgs p,
                                                                    const SelectArgs m)
{
    static_assert(kLaneBlock == kPushSeg, "a block covers one list-index segment");
    __shared__ float s_val[kPushSeg];
    __shared__ uint8_t s_flag[kPushSeg];
    const Hyper h = a.h;
    const int K = a.K;
    const int t = threadIdx.x;
    const int64_t seg = blockIdx.x;
    const int64_t first = seg * kPushSeg;
    const int64_t j = first + t;
    const bool own = j < a.P;
    const int64_t jl = own ? j : a.P - 1;      // loads stay inside [0, P)
    int64_t lo, hi;
    push_range(p, seg, lo, hi);
    const bool entry = lo + t < hi;
    const int64_t e = entry ? lo + t : 0;      // entry 0 is readable (the launcher sees to it)
    const int32_t e_idx = p.idx[e];
    const float e_val = p.val[e];
    float th = ldnt(a.theta + jl), n = ldnt(a.n + jl), b = ldnt(a.b + jl), v = ldnt(a.v + jl);
    const int k0 = K < kPushBatch ? K : kPushBatch;
    float g0[kPushBatch];
#pragma unroll
    for (int u = 0; u < kPushBatch; ++u) g0[u] = ldnt(a.grad[u < k0 ? u : 0] + jl);
    stage_segment(e_idx, e_val, entry, first, a.P, s_val, s_flag);
    if (s_flag[t]) fasgd_step<MODE>(th, n, b, v, s_val[t], p.coef, h);
#pragma unroll
    for (int u = 0; u < kPushBatch; ++u)
        if (u < k0) fasgd_step<MODE>(th, n, b, v, g0[u], a.coef[u], h);
    int k = k0;
    for (; k + kPushBatch <= K; k += kPushBatch) {
        float g[kPushBatch];
#pragma unroll
        for (int u = 0; u < kPushBatch; ++u) g[u] = ldnt(a.grad[k + u] + jl);
#pragma unroll
        for (int u = 0; u < kPushBatch; ++u) fasgd_step<MODE>(th, n, b, v, g[u], a.coef[k + u], h);
    }
    for (; k < K; ++k) fasgd_step<MODE>(th, n, b, v, ldnt(a.grad[k] + jl), a.coef[k], h);
    if (own) {
        stnt(a.theta + j, th);
        stnt(a.n + j, n);
        stnt(a.b + j, b);
        stnt(a.v + j, v);
    }
    if (MARK) {
        if (blockIdx.x == 0 && t == 0) *m.groups_done = 0u;   // for the scan launch
        const int lane = t & (kWave - 1);
        const int w = __builtin_amdgcn_readfirstlane(t / kWave);
        uint32_t bit = 0;
        if (own) {
            const uint64_t qg = m.chunk_base + static_cast<uint64_t>(j >> 2);   // global chunk index
            const uint4 wd = philox4x32_10(
                make_uint4(static_cast<uint32_t>(qg), static_cast<uint32_t>(qg >> 32), m.ctr_T, m.ctr_client),
                m.key0, m.key1);
            const int c = static_cast<int>(j & 3);
            const uint32_t word = c == 0 ? wd.x : c == 1 ? wd.y : c == 2 ? wd.z : wd.w;
            bit = transmit_bit(word, v, m.c, m.eps_c);
        }
        // bit l: parameter first + 64 w + l, bit (l mod 4) of the segment's chunk 16 w + l / 4
        const uint64_t wave_bits = __builtin_amdgcn_ballot_w64(bit != 0);
        uint32_t piece = 0;   // lane c < 4: bits 16 w .. 16 w + 15 of the segment's word c
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const uint64_t wc = __builtin_amdgcn_ballot_w64(lane < 16 && ((wave_bits >> (4 * lane + c)) & 1u) != 0);
            if (lane == c) piece = static_cast<uint32_t>(wc) & 0xFFFFu;
        }
        const int64_t tile_segs = m.n_tiles * 4;   // segments the ballot array holds
        if (seg < tile_segs && lane < 4)
            reinterpret_cast<uint16_t*>(m.ballots + seg * 4 + lane)[w] = static_cast<uint16_t>(piece);
        // segments of the last tile beyond the grid hold no parameter: no bits
        if (seg == static_cast<int64_t>(gridDim.x) - 1 && w == 0 && lane < 4)
            for (int64_t s2 = seg + 1; s2 < tile_segs; ++s2) m.ballots[s2 * 4 + lane] = 0;
    }
}

// A cached push in one pass, one parameter per thread (block s: list-index
// segment s): the segment's entries merged into the client's cache, the
// cache segment written back whole when the push lists any of it, and the
// merged values applied as one gradient.  As fasgd_cached_push_vec, bit for
// bit; measured 6.35 against 7.03 ms at 1e9 parameters (10 % listed), equal
// at 25M.
template <int MODE>
__global__ __launch_bounds__(kLaneBlock) void fasgd_cached_push_lane(const DenseArgs a, const PushArgs p,
                                                                     float* __restrict__ cache)
{
    __shared__ float s_val[kPushSeg];
    __shared__ uint8_t s_flag[kPushSeg];
    const int t = threadIdx.x;
    const int64_t seg = blockIdx.x;
    const int64_t first = seg * kPushSeg;
    const int64_t j = first + t;
    const bool own = j < a.P;
    const int64_t jl = own ? j : a.P - 1;
    int64_t lo, hi;
    push_range(p, seg, lo, hi);
    const bool entry = lo + t < hi;
    const int64_t e = entry ? lo + t : 0;      // entry 0 is readable (the launcher sees to it)
    const int32_t e_idx = p.idx[e];
    const float e_val = p.val[e];
    float th = ldnt(a.theta + jl), n = ldnt(a.n + jl), b = ldnt(a.b + jl), v = ldnt(a.v + jl);
    float g = ldnt(cache + jl);
    stage_segment(e_idx, e_val, entry, first, a.P, s_val, s_flag);
    if (!own) return;
    if (s_flag[t]) g = s_val[t];
    if (hi > lo) stnt(cache + j, g);           // block-uniform: the push lists part of this segment
    fasgd_step<MODE>(th, n, b, v, g, a.coef[0], a.h);
    stnt(a.theta + j, th);
    stnt(a.n + j, n);
    stnt(a.b + j, b);
    stnt(a.v + j, v);
}

// K-fused FASGD, one parameter per thread (any 4-byte alignment): the pass
// for every P below kMaxScalarItems.
template <int MODE>
__global__ __launch_bounds__(kLaneBlock) void fasgd_dense_lane(const DenseArgs a)
{
    const Hyper h = a.h;
    const int K = a.K;
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kLaneBlock + threadIdx.x;
    if (j >= a.P) return;
    float th = ldnt(a.theta + j), n = ldnt(a.n + j), b = ldnt(a.b + j), v = ldnt(a.v + j);
    int k = 0;
    for (; k + kLaneBatch <= K; k += kLaneBatch) {
        float g[kLaneBatch];
#pragma unroll
        for (int u = 0; u < kLaneBatch; ++u) g[u] = ldnt(a.grad[k + u] + j);
#pragma unroll
        for (int u = 0; u < kLaneBatch; ++u) fasgd_step<MODE>(th, n, b, v, g[u], a.coef[k + u], h);
    }
    for (; k < K; ++k) fasgd_step<MODE>(th, n, b, v, ldnt(a.grad[k] + j), a.coef[k], h);
    stnt(a.theta + j, th);
    stnt(a.n + j, n);
    stnt(a.b + j, b);
    stnt(a.v + j, v);
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

// SYNC: synchronous SGD (the apply-update listing of Sec. 3), every gradient
// divided by lambda before the step; otherwise K-fused SASGD.  One parameter
// per thread, below kMaxScalarItems.
template <bool SYNC>
__global__ __launch_bounds__(kLaneBlock) void sgd_dense_lane(const DenseArgs a)
{
    const int K = a.K;
    const float lam = a.lambda;
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kLaneBlock + threadIdx.x;
    if (j >= a.P) return;
    float th = ldnt(a.theta + j);
    int k = 0;
    for (; k + kSgdBatch <= K; k += kSgdBatch) {
        float g[kSgdBatch];
#pragma unroll
        for (int u = 0; u < kSgdBatch; ++u) g[u] = ldnt(a.grad[k + u] + j);
#pragma unroll
        for (int u = 0; u < kSgdBatch; ++u) th = fmaf(-a.coef[k + u], SYNC ? g[u] / lam : g[u], th);
    }
    for (; k < K; ++k) {
        const float g = ldnt(a.grad[k] + j);
        th = fmaf(-a.coef[k], SYNC ? g / lam : g, th);
    }
    stnt(a.theta + j, th);
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


}  // namespace

hipError_t launch_init(float* n, float* b, float* v, int32_t* last_T, int64_t P,
                       float n0, float b0, float v0, hipStream_t s)
{
    init_kernel<<<grid_for(P < kMaxScalarItems ? P : kMaxScalarItems), kBlock, 0, s>>>(n, b, v, last_T, P, n0, b0, v0);
    return hipGetLastError();
}

// Every thread of a segment pass reads list entry 0 or later: a list
// without capacity (its pointers may be NULL) reads the list index instead,
// which has at least two entries; no entry is then used.
PushArgs readable_list(const PushArgs& p)
{
    PushArgs q = p;
    if (q.capacity == 0 || !q.idx || !q.val) {
        q.idx = reinterpret_cast<const int32_t*>(q.seg_start);
        q.val = reinterpret_cast<const float*>(q.seg_start);
    }
    return q;
}

// one parameter per thread below kMaxScalarItems; beyond it (16-byte
// aligned arrays only: the API rejects others first) 4 per thread
template <int VARIANT>
void launch_dense_variant(const DenseArgs& a, hipStream_t s)
{
    if (a.P <= kMaxScalarItems)
        fasgd_dense_lane<VARIANT><<<lane_grid(a.P), kLaneBlock, 0, s>>>(a);
    else
        fasgd_dense_vec<VARIANT><<<grid_for((a.P >> 2) + 1), kBlock, 0, s>>>(a);
}

template <int VARIANT>
void launch_push_variant(const DenseArgs& a, const PushArgs& p, const SelectArgs* m, hipStream_t s)
{
    if (a.P <= kMaxScalarItems) {
        const PushArgs q = readable_list(p);
        if (m)
            fasgd_dense_push_lane<VARIANT, true><<<lane_grid(a.P), kLaneBlock, 0, s>>>(a, q, *m);
        else
            fasgd_dense_push_lane<VARIANT, false><<<lane_grid(a.P), kLaneBlock, 0, s>>>(a, q, SelectArgs{});
    } else if (m) {
        fasgd_dense_push_vec<VARIANT, true><<<grid_for((a.P >> 2) + 1), kBlock, 0, s>>>(a, p, *m);
    } else {
        fasgd_dense_push_vec<VARIANT, false><<<grid_for((a.P >> 2) + 1), kBlock, 0, s>>>(a, p, SelectArgs{});
    }
}

hipError_t launch_fasgd_dense_push(const DenseArgs& a, const PushArgs& p, const SelectArgs* mark, int variant,
                                   bool aligned, hipStream_t s)
{
    if (a.P > kMaxScalarItems && !aligned) return hipErrorInvalidValue;   // the API rejects this first
    switch (variant) {
    case kernel_variant(MATH_FAST, 0): launch_push_variant<kernel_variant(MATH_FAST, 0)>(a, p, mark, s); break;
    case kernel_variant(MATH_IEEE, 0): launch_push_variant<kernel_variant(MATH_IEEE, 0)>(a, p, mark, s); break;
    case kernel_variant(MATH_FAST, 1): launch_push_variant<kernel_variant(MATH_FAST, 1)>(a, p, mark, s); break;
    case kernel_variant(MATH_IEEE, 1): launch_push_variant<kernel_variant(MATH_IEEE, 1)>(a, p, mark, s); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_fasgd_dense(const DenseArgs& a, int variant, bool aligned, hipStream_t s)
{
    if (a.P > kMaxScalarItems && !aligned) return hipErrorInvalidValue;   // the API rejects this first
    switch (variant) {
    case kernel_variant(MATH_FAST, 0): launch_dense_variant<kernel_variant(MATH_FAST, 0)>(a, s); break;
    case kernel_variant(MATH_IEEE, 0): launch_dense_variant<kernel_variant(MATH_IEEE, 0)>(a, s); break;
    case kernel_variant(MATH_FAST, 1): launch_dense_variant<kernel_variant(MATH_FAST, 1)>(a, s); break;
    case kernel_variant(MATH_IEEE, 1): launch_dense_variant<kernel_variant(MATH_IEEE, 1)>(a, s); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int VARIANT>
void launch_cached_variant(const DenseArgs& a, const PushArgs& p, float* cache, hipStream_t s)
{
    if (a.P <= kMaxScalarItems)
        fasgd_cached_push_lane<VARIANT><<<lane_grid(a.P), kLaneBlock, 0, s>>>(a, readable_list(p), cache);
    else
        fasgd_cached_push_vec<VARIANT><<<grid_for((a.P >> 2) + 1), kBlock, 0, s>>>(a, p, cache);
}

hipError_t launch_fasgd_cached_push(const DenseArgs& a, const PushArgs& p, float* cache, int variant, hipStream_t s)
{
    switch (variant) {
    case kernel_variant(MATH_FAST, 0): launch_cached_variant<kernel_variant(MATH_FAST, 0)>(a, p, cache, s); break;
    case kernel_variant(MATH_IEEE, 0): launch_cached_variant<kernel_variant(MATH_IEEE, 0)>(a, p, cache, s); break;
    case kernel_variant(MATH_FAST, 1): launch_cached_variant<kernel_variant(MATH_FAST, 1)>(a, p, cache, s); break;
    case kernel_variant(MATH_IEEE, 1): launch_cached_variant<kernel_variant(MATH_IEEE, 1)>(a, p, cache, s); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_merge_list(float* dst, int64_t P, const PushArgs& p, hipStream_t s)
{
    // 4 parameters per thread at every size: one parameter per thread was
    // twice as slow (3.04 against 1.55 ms at 1e9, 10 %), each of its blocks
    // doing one load and one store per thread
    merge_list_vec<<<grid_for((P >> 2) + 1), kBlock, 0, s>>>(dst, P, p);
    return hipGetLastError();
}

hipError_t launch_sasgd_dense(const DenseArgs& a, bool aligned, hipStream_t s)
{
    if (a.P <= kMaxScalarItems)
        sgd_dense_lane<false><<<lane_grid(a.P), kLaneBlock, 0, s>>>(a);
    else if (aligned)
        sasgd_dense_vec<<<grid_for((a.P >> 2) + 1), kBlock, 0, s>>>(a);
    else
        return hipErrorInvalidValue;   // the API rejects this first
    return hipGetLastError();
}

hipError_t launch_sync_sgd(const DenseArgs& a, bool aligned, hipStream_t s)
{
    if (a.P <= kMaxScalarItems)
        sgd_dense_lane<true><<<lane_grid(a.P), kLaneBlock, 0, s>>>(a);
    else if (aligned)
        sync_sgd_vec<<<grid_for((a.P >> 2) + 1), kBlock, 0, s>>>(a);
    else
        return hipErrorInvalidValue;   // the API rejects this first
    return hipGetLastError();
}

}  // namespace fasgd
