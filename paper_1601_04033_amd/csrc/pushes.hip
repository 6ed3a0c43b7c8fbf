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
// wave owns one segment (64 lanes x 4 parameters); lane b of the wave first
// finds push b's range, then the wave loads the first 64 entries of
// kGroup pushes at once and applies them one push at a time through an LDS
// slice holding one value and one flag byte per parameter.
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

// Thread i of the vector kernel owns parameters 4i .. 4i+3; the thread after
// the last full chunk owns the P mod 4 tail.
template <int MODE>
__global__ __launch_bounds__(kBlock) void apply_pushes_vec(const PushBatchArgs a)
{
    __shared__ float s_val[kWavesPerBlock][kPushSeg];
    __shared__ uint32_t s_flag[kWavesPerBlock][kWave];   // byte c of word l: parameter 4 l + c listed
    const Hyper h = a.h;
    const int B = a.B;
    const int64_t nvec = a.P >> 2;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t seg = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + w;
    const int64_t first = seg * kPushSeg;
    const int64_t o = i * 4;
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
    int last[4] = {-1, -1, -1, -1};
    uint8_t* flag_bytes = reinterpret_cast<uint8_t*>(s_flag[w]);
    for (int g0 = 0; g0 < B; g0 += kGroup) {
        int32_t e_idx[kGroup];
        float e_val[kGroup];
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            e_idx[u] = -1;
            e_val[u] = 0.0f;
            const int pb = g0 + u;
            if (pb < B) {
                const uint32_t l = __builtin_amdgcn_readlane(lo, pb), e = __builtin_amdgcn_readlane(hi, pb);
                if (l + lane < e) {
                    const int64_t at = static_cast<int64_t>(pb) * a.list_stride + l + lane;
                    e_idx[u] = a.idx[at];
                    e_val[u] = a.val[at];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            const int pb = g0 + u;
            if (pb >= B) break;
            const uint32_t l = __builtin_amdgcn_readlane(lo, pb), e = __builtin_amdgcn_readlane(hi, pb);
            if (l == e) continue;   // push pb lists nothing here
            wave_lds_order();
            s_flag[w][lane] = 0u;
            wave_lds_order();
            stage_entry(e_idx[u], e_val[u], first, kPushSeg, a.P, s_val[w], flag_bytes);
            if (e - l > static_cast<uint32_t>(kWave)) {   // more than 64 entries in 256 parameters
                const int64_t base = static_cast<int64_t>(pb) * a.list_stride;
                for (uint32_t x = l + kWave + lane; x < e; x += kWave)
                    stage_entry(a.idx[base + x], a.val[base + x], first, kPushSeg, a.P, s_val[w], flag_bytes);
            }
            wave_lds_order();
            const uint32_t flags = s_flag[w][lane];
            if (flags) {
                const f4 pv = *reinterpret_cast<const f4*>(&s_val[w][4 * lane]);
                const float coef = a.coef[pb];
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    if ((flags >> (8 * c)) & 0xffu) {
                        float t = th[c], nn = n[c], bb = b[c], vv = v[c];
                        fasgd_step<MODE>(t, nn, bb, vv, pv[c], coef, h);
                        th[c] = t; n[c] = nn; b[c] = bb; v[c] = vv;
                        last[c] = pb;
                    }
                }
            }
        }
    }
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

unsigned grid_for(int64_t items)
{
    const int64_t g = (items + kBlock - 1) / kBlock;
    return static_cast<unsigned>(g < 1 ? 1 : g);
}

template <int VARIANT>
void launch_variant(const PushBatchArgs& a, bool aligned, hipStream_t s)
{
    if (aligned)
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
