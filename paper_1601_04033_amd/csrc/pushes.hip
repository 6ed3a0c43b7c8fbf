// Several compacted B-FASGD pushes applied in one pass (Sec. 2.3): pushes
// that reached the server together, from different clients, are applied in
// arrival order b = 0 .. B-1 at timestamps T0 + b, with every parameter's
// state loaded once, carried through the B pushes in registers and stored
// once.  The result is the one B sparse applies in a row give, bit for bit,
// including last_T (T0 + the last push that lists the parameter).
//
// Each list is one that the selection wrote with its list index, so the
// entries of push b for the 256-parameter segment s are at [seg_start_b[s],
// seg_start_b[s + 1]) of its list, clipped to min(count_b, capacity).  One
// wave owns one segment (64 lanes x 4 parameters): lane b of the wave first
// finds push b's range; the wave loads its segment's state into LDS and the
// first 64 entries of kGroup pushes at once, and applies the pushes one at
// a time, each lane updating the LDS state of the parameter its entry
// names.  A push thus costs one update per listed parameter (a lane-owns-
// parameters layout would evaluate the update for all four parameters of
// every lane in every push, and be bound by the vector ALU).
//
// Traffic: the state is read and written once (16 + 16 bytes per parameter,
// plus 4 bytes of last_T per parameter that some push lists) and every list
// entry is read once (8 bytes), instead of one gather/scatter of the listed
// state per push.
#include "kernels.hpp"

namespace fasgd {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef int i4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 128;
constexpr int kWave = 64;
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kGroup = 8;   // pushes whose entries are loaded together
constexpr int kEntries = 1; // entries per lane of each push loaded ahead (64 each)
static_assert(kWave * 4 == kPushSeg, "one wave covers one list-index segment");
static_assert(kMaxBatch <= kWave, "lane b holds the range of push b");

__device__ __forceinline__ f4 ld4(const float* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const f4*>(p));
}
__device__ __forceinline__ void st4(float* p, f4 x)
{
    __builtin_nontemporal_store(x, reinterpret_cast<f4*>(p));
}

__device__ __forceinline__ void wave_lds_order()
{
    // the wave's LDS operations execute in order; keep the compiler from
    // moving one lane's LDS accesses across those of the others
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Lane b < B: the entries [lo, hi) of push b that fall in segment seg.
__device__ __forceinline__ void lane_range(const PushBatchArgs& a, int64_t seg, int lane, uint32_t& lo,
                                           uint32_t& hi)
{
    lo = hi = 0;
    if (lane < a.B) {
        int64_t m = a.d_count[lane];
        m = m < a.list_stride ? m : a.list_stride;
        m = m > 0 ? m : 0;
        int64_t l = m, h = m;
        if (seg < a.n_segs) {
            const uint32_t* ss = a.seg_start + static_cast<int64_t>(lane) * (a.n_segs + 1);
            const int64_t s0 = ss[seg], s1 = ss[seg + 1];
            l = s0 < m ? s0 : m;
            h = s1 < m ? s1 : m;
        }
        lo = static_cast<uint32_t>(l);
        hi = static_cast<uint32_t>(h > l ? h : l);
    }
}

// Stage entry e of push b (whose index lies in [first, first + span) and
// below P) at s_val[j - first], with flag byte 1.
__device__ __forceinline__ void stage_entry(int32_t j, float x, int64_t first, int span, int64_t P, float* s_val,
                                            uint8_t* s_flag)
{
    const int64_t r = static_cast<int64_t>(j) - first;
    if (j >= 0 && r >= 0 && r < span && first + r < P) {
        s_val[r] = x;
        s_flag[r] = 1;
    }
}

// The wave's 256 parameters: theta, n, b, v and the last push that listed
// each one, in LDS for the whole pass.
struct SegState {
    float x[4][kPushSeg];
    int last[kPushSeg];
};

// Apply list entry (j, g) of push pb to the LDS copy of the state, when j
// lies in this wave's segment and below P.
template <int MODE>
__device__ __forceinline__ void apply_entry(SegState& s, int32_t j, float g, int pb, float coef, int64_t first,
                                            int64_t P, const Hyper& h)
{
    const int64_t r = static_cast<int64_t>(j) - first;
    if (j >= 0 && r >= 0 && r < kPushSeg && first + r < P) {
        float t = s.x[0][r], nn = s.x[1][r], bb = s.x[2][r], vv = s.x[3][r];
        fasgd_step<MODE>(t, nn, bb, vv, g, coef, h);
        s.x[0][r] = t; s.x[1][r] = nn; s.x[2][r] = bb; s.x[3][r] = vv;
        s.last[r] = pb;
    }
}

// Thread i of the vector kernel loads and stores parameters 4i .. 4i+3 (the
// thread after the last full chunk the P mod 4 tail); in between, the state
// of the wave's segment lives in LDS and each push's entries are applied
// there, one entry per lane, so a push costs one update per listed
// parameter rather than one per parameter.
template <int MODE>
__global__ __launch_bounds__(kBlock) void apply_pushes_vec(const PushBatchArgs a)
{
    __shared__ SegState s_seg[kWavesPerBlock];
    const Hyper h = a.h;
    const int B = a.B;
    const int64_t nvec = a.P >> 2;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t seg = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + w;
    const int64_t first = seg * kPushSeg;
    const int64_t o = i * 4;
    SegState& S = s_seg[w];
    uint32_t lo, hi;
    lane_range(a, seg, lane, lo, hi);
    if (__builtin_amdgcn_ballot_w64(hi > lo) == 0) return;   // no push lists a parameter of this segment
    const int valid = i < nvec ? 4 : (i == nvec ? static_cast<int>(a.P - 4 * nvec) : 0);
    f4 th = {0, 0, 0, 0}, n = th, b = th, v = th;
    if (valid == 4) {
        th = ld4(a.theta + o); n = ld4(a.n + o); b = ld4(a.b + o); v = ld4(a.v + o);
    } else {
        for (int c = 0; c < valid; ++c) { th[c] = a.theta[o + c]; n[c] = a.n[o + c]; b[c] = a.b[o + c]; v[c] = a.v[o + c]; }
    }
    for (int g0 = 0; g0 < B; g0 += kGroup) {
        int32_t e_idx[kGroup][kEntries];
        float e_val[kGroup][kEntries];
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            const int pb = g0 + u;
            const uint32_t l = pb < B ? __builtin_amdgcn_readlane(lo, pb) : 0u;
            const uint32_t e = pb < B ? __builtin_amdgcn_readlane(hi, pb) : 0u;
#pragma unroll
            for (int q = 0; q < kEntries; ++q) {
                e_idx[u][q] = -1;
                e_val[u][q] = 0.0f;
                if (l + q * kWave + lane < e) {
                    const int64_t at = static_cast<int64_t>(pb) * a.list_stride + l + q * kWave + lane;
                    e_idx[u][q] = a.idx[at];
                    e_val[u][q] = a.val[at];
                }
            }
        }
        if (g0 == 0) {   // the state, once its loads (issued before the entries') are in
            *reinterpret_cast<f4*>(&S.x[0][4 * lane]) = th;
            *reinterpret_cast<f4*>(&S.x[1][4 * lane]) = n;
            *reinterpret_cast<f4*>(&S.x[2][4 * lane]) = b;
            *reinterpret_cast<f4*>(&S.x[3][4 * lane]) = v;
            *reinterpret_cast<i4*>(&S.last[4 * lane]) = i4{-1, -1, -1, -1};
        }
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            const int pb = g0 + u;
            if (pb >= B) break;
            const uint32_t l = __builtin_amdgcn_readlane(lo, pb), e = __builtin_amdgcn_readlane(hi, pb);
            if (l == e) continue;   // push pb lists nothing here
            const float coef = a.coef[pb];
            // the entries of one push are distinct parameters; the previous
            // push's updates are in LDS before this push reads them
            wave_lds_order();
#pragma unroll
            for (int q = 0; q < kEntries; ++q)
                apply_entry<MODE>(S, e_idx[u][q], e_val[u][q], pb, coef, first, a.P, h);
            if (e - l > static_cast<uint32_t>(kEntries * kWave)) {   // more entries than were loaded ahead
                const int64_t base = static_cast<int64_t>(pb) * a.list_stride;
                for (uint32_t x = l + kEntries * kWave + lane; x < e; x += kWave)
                    apply_entry<MODE>(S, a.idx[base + x], a.val[base + x], pb, coef, first, a.P, h);
            }
        }
    }
    wave_lds_order();
    th = *reinterpret_cast<const f4*>(&S.x[0][4 * lane]);
    n = *reinterpret_cast<const f4*>(&S.x[1][4 * lane]);
    b = *reinterpret_cast<const f4*>(&S.x[2][4 * lane]);
    v = *reinterpret_cast<const f4*>(&S.x[3][4 * lane]);
    const i4 last = *reinterpret_cast<const i4*>(&S.last[4 * lane]);
    if (valid == 4) {
        st4(a.theta + o, th); st4(a.n + o, n); st4(a.b + o, b); st4(a.v + o, v);
        if ((last[0] | last[1] | last[2] | last[3]) >= 0) {   // all four listed
            const i4 t = {a.T0 + last[0], a.T0 + last[1], a.T0 + last[2], a.T0 + last[3]};
            __builtin_nontemporal_store(t, reinterpret_cast<i4*>(a.last_T + o));
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (last[c] >= 0) a.last_T[o + c] = a.T0 + last[c];
        }
    } else {
        for (int c = 0; c < valid; ++c) {
            a.theta[o + c] = th[c]; a.n[o + c] = n[c]; a.b[o + c] = b[c]; a.v[o + c] = v[c];
            if (last[c] >= 0) a.last_T[o + c] = a.T0 + last[c];
        }
    }
}

// The same, one parameter per thread (arrays only 4-byte aligned): a wave
// covers 64 parameters, a quarter of a list-index segment.
template <int MODE>
__global__ __launch_bounds__(kBlock) void apply_pushes_scalar(const PushBatchArgs a)
{
    __shared__ float s_val[kWavesPerBlock][kWave];
    __shared__ uint8_t s_flag[kWavesPerBlock][kWave];
    const Hyper h = a.h;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t first = static_cast<int64_t>(blockIdx.x) * kBlock + w * kWave;   // the wave's first parameter
    const int64_t j = first + lane;
    uint32_t lo, hi;
    lane_range(a, first / kPushSeg, lane, lo, hi);
    if (__builtin_amdgcn_ballot_w64(hi > lo) == 0) return;
    const bool own = j < a.P;
    float th = 0.0f, n = 0.0f, b = 0.0f, v = 0.0f;
    if (own) { th = a.theta[j]; n = a.n[j]; b = a.b[j]; v = a.v[j]; }
    int last = -1;
    for (int pb = 0; pb < a.B; ++pb) {
        const uint32_t l = __builtin_amdgcn_readlane(lo, pb), e = __builtin_amdgcn_readlane(hi, pb);
        if (l == e) continue;
        wave_lds_order();
        s_flag[w][lane] = 0;
        wave_lds_order();
        const int64_t base = static_cast<int64_t>(pb) * a.list_stride;
        for (uint32_t x = l + lane; x < e; x += kWave)
            stage_entry(a.idx[base + x], a.val[base + x], first, kWave, a.P, s_val[w], s_flag[w]);
        wave_lds_order();
        if (own && s_flag[w][lane]) {
            fasgd_step<MODE>(th, n, b, v, s_val[w][lane], a.coef[pb], h);
            last = pb;
        }
    }
    if (!own) return;
    a.theta[j] = th; a.n[j] = n; a.b[j] = b; a.v[j] = v;
    if (last >= 0) a.last_T[j] = a.T0 + last;
}

// One push (B = 1), one parameter per thread: block s owns list-index
// segment s.  A segment no entry names is skipped.  One with at least
// kWholeEntries entries is read and written whole, every thread loading and
// storing its parameter (last_T too, rewritten with its old value where
// the push lists nothing), so its lines are written in full; one with fewer
// touches only its listed parameters.  The push's entries are staged in the
// block's LDS (value and flag byte per parameter) as in the dense pass with
// a push.  Listed parameters get last_T = T0.
// Measured on MI355X against bfasgd_apply_sparse (one gather and scatter
// per entry): 1e9 parameters, 10 % listed, 7.16 against 9.37 ms; 25 %, 7.26
// against 9.95 ms; 25M, 10 %, 178 against 231 us; but 1.8 %, 4.9 against
// 3.6 ms (almost every segment holds an entry, so every block runs for one
// or two updates).  Thresholds of 16, 32 and 64 entries were 1-8 % slower at
// 10 %; writing only the listed last_T of a whole segment (partial lines)
// 4-13 % slower.
constexpr int kSegBlock = kPushSeg;
constexpr int kWholeEntries = 8;
constexpr bool kWholeLastT = true;

__device__ __forceinline__ void block_barrier_lds()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <int MODE, bool WHOLE>
__device__ __forceinline__ void push_segment(const PushBatchArgs& a, int64_t lo, int64_t hi, float* s_val,
                                             uint8_t* s_flag)
{
    const Hyper h = a.h;
    const int t = threadIdx.x;
    const int64_t first = static_cast<int64_t>(blockIdx.x) * kPushSeg;
    const int64_t j = first + t;
    const bool own = j < a.P;
    const int64_t jl = own ? j : a.P - 1;       // loads stay inside [0, P)
    const bool entry = lo + t < hi;
    const int64_t e = entry ? lo + t : lo;      // lo < hi: entry lo exists
    const int32_t e_idx = a.idx[e];
    const float e_val = a.val[e];
    float th = 0.0f, n = 0.0f, b = 0.0f, v = 0.0f;
    int32_t lt = 0;
    if (WHOLE) {
        th = a.theta[jl]; n = a.n[jl]; b = a.b[jl]; v = a.v[jl];
        if (kWholeLastT) lt = a.last_T[jl];
    }
    s_flag[t] = 0;
    block_barrier_lds();
    if (entry) {
        const int64_t x = static_cast<int64_t>(e_idx) - first;
        if (e_idx >= 0 && x >= 0 && x < kPushSeg && first + x < a.P) {
            s_val[x] = e_val;
            s_flag[x] = 1;
        }
    }
    block_barrier_lds();
    const bool listed = s_flag[t] != 0;
    if (!own) return;
    if (WHOLE) {
        if (listed) fasgd_step<MODE>(th, n, b, v, s_val[t], a.coef[0], h);
        a.theta[j] = th; a.n[j] = n; a.b[j] = b; a.v[j] = v;
        if (kWholeLastT)
            a.last_T[j] = listed ? a.T0 : lt;
        else if (listed)
            a.last_T[j] = a.T0;
    } else if (listed) {
        th = a.theta[j]; n = a.n[j]; b = a.b[j]; v = a.v[j];
        fasgd_step<MODE>(th, n, b, v, s_val[t], a.coef[0], h);
        a.theta[j] = th; a.n[j] = n; a.b[j] = b; a.v[j] = v;
        a.last_T[j] = a.T0;
    }
}

template <int MODE>
__global__ __launch_bounds__(kSegBlock) void apply_push_segments(const PushBatchArgs a)
{
    __shared__ float s_val[kPushSeg];
    __shared__ uint8_t s_flag[kPushSeg];
    const int64_t seg = blockIdx.x;
    int64_t m = a.d_count[0];
    m = m < a.list_stride ? m : a.list_stride;
    m = m > 0 ? m : 0;
    const int64_t s0 = a.seg_start[seg], s1 = a.seg_start[seg + 1];
    const int64_t lo = s0 < m ? s0 : m, hi = s1 < m ? s1 : m;
    if (hi <= lo) return;                       // no entry names this segment
    if (hi - lo >= kWholeEntries)
        push_segment<MODE, true>(a, lo, hi, s_val, s_flag);
    else
        push_segment<MODE, false>(a, lo, hi, s_val, s_flag);
}

unsigned grid_for(int64_t items)
{
    const int64_t g = (items + kBlock - 1) / kBlock;
    return static_cast<unsigned>(g < 1 ? 1 : g);
}

template <int VARIANT>
void launch_variant(const PushBatchArgs& a, bool aligned, hipStream_t s)
{
    if (a.B == 1)
        apply_push_segments<VARIANT><<<static_cast<unsigned>(a.n_segs), kSegBlock, 0, s>>>(a);
    else if (aligned)
        apply_pushes_vec<VARIANT><<<grid_for((a.P >> 2) + 1), kBlock, 0, s>>>(a);
    else
        apply_pushes_scalar<VARIANT><<<grid_for(a.P), kBlock, 0, s>>>(a);
}

}  // namespace

hipError_t launch_apply_pushes(const PushBatchArgs& a, int variant, bool aligned, hipStream_t s)
{
    if (a.B < 1 || a.B > kMaxBatch) return hipErrorInvalidValue;
    switch (variant) {
    case kernel_variant(MATH_FAST, 0): launch_variant<kernel_variant(MATH_FAST, 0)>(a, aligned, s); break;
    case kernel_variant(MATH_IEEE, 0): launch_variant<kernel_variant(MATH_IEEE, 0)>(a, aligned, s); break;
    case kernel_variant(MATH_FAST, 1): launch_variant<kernel_variant(MATH_FAST, 1)>(a, aligned, s); break;
    case kernel_variant(MATH_IEEE, 1): launch_variant<kernel_variant(MATH_IEEE, 1)>(a, aligned, s); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace fasgd
