// B-FASGD push selection with deterministic ordered compaction, and the
// sparse server apply of the compacted list.
//
// Selection runs in four launches, none of which waits on another block:
//   mark     one Philox4x32-10 call per 4 parameters (the counter is the
//            chunk index j/4, so one call feeds one 16-byte vector of v),
//            four wave ballots per 64 chunks stored to the workspace (1 bit
//            per parameter), and a per-tile count;
//   scan     one block per 1024 tiles scans their counts (offsets within
//            the group) and records the group total;
//   top      one block scans the group totals and writes the device count;
//   scatter  every wave rebuilds its output position from the ballots of
//            its tile (scalar loads and popcounts) plus the group and tile
//            offsets, stages its (index, value) pairs in LDS and writes its
//            contiguous piece of the output in ascending index order.
// The result depends only on (seed, T, client, v, grad), never on timing.
#include "kernels.hpp"

namespace fasgd {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kBlock = 256;                   // 4 waves
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kItems = 4;                     // 64-chunk segments per wave per tile
constexpr int kSegsPerTile = kWavesPerBlock * kItems;          // 16
constexpr int64_t kChunksPerTile = int64_t(kSegsPerTile) * kWave;  // 1024 chunks = 4096 parameters
constexpr int kScanBlock = 1024;              // tiles per scan group
constexpr int kMaxGroups = 4096;              // 2^31 parameters need 512

__host__ __device__ inline int64_t n_chunks(int64_t P) { return (P + 3) / 4; }
int64_t n_tiles(int64_t P) { return (n_chunks(P) + kChunksPerTile - 1) / kChunksPerTile; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

__device__ __forceinline__ uint64_t lanes_below(int lane)
{
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// v for the 4 parameters of chunk q; parameters at or past P read as NaN,
// which never transmits.
template <bool ALIGNED>
__device__ __forceinline__ f4 load_chunk(const float* p, int64_t q, int64_t P)
{
    const int64_t j = q * 4;
    if (ALIGNED && j + 3 < P) return *reinterpret_cast<const f4*>(p + j);
    f4 x;
#pragma unroll
    for (int c = 0; c < 4; ++c) x[c] = (j + c < P) ? p[j + c] : __builtin_nanf("");
    return x;
}

template <bool ALIGNED>
__global__ __launch_bounds__(kBlock) void select_mark(const SelectArgs a)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t tile = blockIdx.x;
    const int64_t nch = n_chunks(a.P);
    uint32_t count = 0;
#pragma unroll
    for (int it = 0; it < kItems; ++it) {
        const int64_t seg = tile * kSegsPerTile + it * kWavesPerBlock + wave;
        const int64_t q = seg * kWave + lane;
        uint32_t nib = 0;
        if (q < nch) {
            const f4 v = load_chunk<ALIGNED>(a.v, q, a.P);
            const uint4 w = philox4x32_10(
                make_uint4(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32), a.ctr_T, a.ctr_client),
                a.key0, a.key1);
            nib = transmit_bit(w.x, v[0], a.c, a.eps_c) | (transmit_bit(w.y, v[1], a.c, a.eps_c) << 1) |
                  (transmit_bit(w.z, v[2], a.c, a.eps_c) << 2) | (transmit_bit(w.w, v[3], a.c, a.eps_c) << 3);
        }
        const uint64_t b0 = __builtin_amdgcn_ballot_w64((nib & 1u) != 0);
        const uint64_t b1 = __builtin_amdgcn_ballot_w64((nib & 2u) != 0);
        const uint64_t b2 = __builtin_amdgcn_ballot_w64((nib & 4u) != 0);
        const uint64_t b3 = __builtin_amdgcn_ballot_w64((nib & 8u) != 0);
        if (lane < 4) {
            const uint64_t mine = lane == 0 ? b0 : lane == 1 ? b1 : lane == 2 ? b2 : b3;
            a.ballots[seg * 4 + lane] = mine;
        }
        count += __popcll(b0) + __popcll(b1) + __popcll(b2) + __popcll(b3);
    }
    __shared__ uint32_t wave_count[kWavesPerBlock];
    if (lane == 0) wave_count[wave] = count;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t s = 0;
#pragma unroll
        for (int w = 0; w < kWavesPerBlock; ++w) s += wave_count[w];
        a.tile_count[tile] = s;
    }
}

// Block-wide exclusive scan of one value per thread (kScanBlock threads).
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* total)
{
    __shared__ uint32_t wave_total[kScanBlock / kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    uint32_t inc = x;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const uint32_t y = __shfl_up(inc, d, kWave);
        if (lane >= d) inc += y;
    }
    if (lane == kWave - 1) wave_total[wave] = inc;
    __syncthreads();
    if (wave == 0) {
        uint32_t t = lane < kScanBlock / kWave ? wave_total[lane] : 0;
#pragma unroll
        for (int d = 1; d < kScanBlock / kWave; d <<= 1) {
            const uint32_t y = __shfl_up(t, d, kWave);
            if (lane >= d) t += y;
        }
        if (lane < kScanBlock / kWave) wave_total[lane] = t;
    }
    __syncthreads();
    *total = wave_total[kScanBlock / kWave - 1];
    return inc - x + (wave > 0 ? wave_total[wave - 1] : 0u);
}

// Group g of 1024 tiles: offsets of its tiles within the group, and its total.
__global__ __launch_bounds__(kScanBlock) void select_scan(const SelectArgs a)
{
    const int64_t t = static_cast<int64_t>(blockIdx.x) * kScanBlock + threadIdx.x;
    const uint32_t c = t < a.n_tiles ? a.tile_count[t] : 0u;
    uint32_t total;
    const uint32_t off = block_exclusive_scan(c, &total);
    if (t < a.n_tiles) a.tile_offset[t] = off;
    if (threadIdx.x == 0) a.group_total[blockIdx.x] = total;
}

// Offsets of the groups (at most kMaxGroups) and the number transmitted.
__global__ __launch_bounds__(kScanBlock) void select_top(const SelectArgs a)
{
    const int64_t ng = (a.n_tiles + kScanBlock - 1) / kScanBlock;
    uint32_t carry = 0;
    for (int64_t base = 0; base < ng; base += kScanBlock) {
        const int64_t g = base + threadIdx.x;
        const uint32_t c = g < ng ? a.group_total[g] : 0u;
        uint32_t total;
        const uint32_t off = block_exclusive_scan(c, &total);
        if (g < ng) a.group_offset[g] = carry + off;
        carry += total;
        __syncthreads();
    }
    if (threadIdx.x == 0) *a.d_count = static_cast<int64_t>(carry);
}

__device__ __forceinline__ uint32_t seg_count(const uint64_t* b)
{
    return static_cast<uint32_t>(__popcll(b[0]) + __popcll(b[1]) + __popcll(b[2]) + __popcll(b[3]));
}

template <bool ALIGNED>
__global__ __launch_bounds__(kBlock) void select_scatter(const SelectArgs a)
{
    __shared__ int32_t s_idx[kWavesPerBlock][4 * kWave];
    __shared__ float s_val[kWavesPerBlock][4 * kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t tile = blockIdx.x;
    const uint64_t below = lanes_below(lane);
    const uint64_t* tb = a.ballots + tile * kSegsPerTile * 4;

    // output position of segment (0, wave): group and tile offsets plus
    // everything the earlier segments of this tile transmitted
    int64_t seg_base = static_cast<int64_t>(a.group_offset[tile / kScanBlock]) + a.tile_offset[tile];
    for (int s = 0; s < wave; ++s) seg_base += seg_count(tb + 4 * s);

#pragma unroll
    for (int it = 0; it < kItems; ++it) {
        const int s = it * kWavesPerBlock + wave;
        const uint64_t b0 = tb[4 * s], b1 = tb[4 * s + 1], b2 = tb[4 * s + 2], b3 = tb[4 * s + 3];
        const uint32_t n_seg = static_cast<uint32_t>(__popcll(b0) + __popcll(b1) + __popcll(b2) + __popcll(b3));
        const uint32_t nib = static_cast<uint32_t>((b0 >> lane) & 1) | static_cast<uint32_t>(((b1 >> lane) & 1) << 1) |
                             static_cast<uint32_t>(((b2 >> lane) & 1) << 2) |
                             static_cast<uint32_t>(((b3 >> lane) & 1) << 3);
        if (nib) {
            uint32_t p = static_cast<uint32_t>(__popcll(b0 & below) + __popcll(b1 & below) + __popcll(b2 & below) +
                                               __popcll(b3 & below));
            const int64_t q = (tile * kSegsPerTile + s) * kWave + lane;
            const f4 g = load_chunk<ALIGNED>(a.grad, q, a.P);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if ((nib >> c) & 1u) {
                    s_idx[wave][p] = static_cast<int32_t>(q * 4 + c);
                    s_val[wave][p] = g[c];
                    ++p;
                }
            }
        }
        __syncthreads();
        // the segment's n_seg entries are contiguous in the output
        for (uint32_t e = lane; e < n_seg; e += kWave) {
            const int64_t pos = seg_base + e;
            if (pos < a.capacity) {
                a.out_idx[pos] = s_idx[wave][e];
                a.out_val[pos] = s_val[wave][e];
            }
        }
        __syncthreads();
        // advance past this segment and the other waves' segments of this item
        for (int t = s; t < s + kWavesPerBlock && t < kSegsPerTile; ++t) seg_base += seg_count(tb + 4 * t);
    }
}

constexpr int kSparseE = 2;                   // list entries per lane
constexpr int64_t kListMaxBlocks = 65536;     // grid cap of the list kernels (grid-stride)

// A wave owns 64 E consecutive list entries and lane l takes entries
// l, l + 64, ...: every gather instruction covers 64 consecutive entries
// (ascending indices, so few cache lines), and each thread issues all 4 E of
// its gathers before the first update.
template <int MODE>
__global__ __launch_bounds__(kBlock) void sparse_apply(const SparseArgs a)
{
    int64_t m = *a.d_count;
    if (m > a.capacity) m = a.capacity;
    const Hyper h = a.h;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wave_id = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) / kWave;
    const int64_t n_waves = static_cast<int64_t>(gridDim.x) * (kBlock / kWave);
    for (int64_t base = wave_id * kWave * kSparseE; base < m; base += n_waves * kWave * kSparseE) {
        int64_t j[kSparseE];
        float g[kSparseE], th[kSparseE], n[kSparseE], b[kSparseE], v[kSparseE];
#pragma unroll
        for (int e = 0; e < kSparseE; ++e) {
            const int64_t i = base + e * kWave + lane;
            j[e] = -1;
            if (i < m) {
                const int64_t x = a.idx[i];
                if (x >= 0 && x < a.P) { j[e] = x; g[e] = a.val[i]; }
            }
        }
#pragma unroll
        for (int e = 0; e < kSparseE; ++e) {
            if (j[e] >= 0) { th[e] = a.theta[j[e]]; n[e] = a.n[j[e]]; b[e] = a.b[j[e]]; v[e] = a.v[j[e]]; }
        }
#pragma unroll
        for (int e = 0; e < kSparseE; ++e) {
            if (j[e] >= 0) {
                fasgd_step<MODE>(th[e], n[e], b[e], v[e], g[e], a.coef, h);
                a.theta[j[e]] = th[e]; a.n[j[e]] = n[e]; a.b[j[e]] = b[e]; a.v[j[e]] = v[e];
                a.last_T[j[e]] = a.last_T_value;
            }
        }
    }
}

__global__ __launch_bounds__(kBlock) void scatter_list(float* __restrict__ dst, int64_t P,
                                                       const int32_t* __restrict__ idx,
                                                       const float* __restrict__ val,
                                                       const int64_t* __restrict__ d_count, int64_t capacity)
{
    int64_t m = *d_count;
    if (m > capacity) m = capacity;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < m; i += stride) {
        const int64_t j = idx[i];
        if (j >= 0 && j < P) dst[j] = val[i];
    }
}

}  // namespace

size_t select_workspace_bytes(int64_t P)
{
    const int64_t nt = n_tiles(P);
    return align256(size_t(nt) * kSegsPerTile * 4 * sizeof(uint64_t)) + 2 * align256(size_t(nt) * sizeof(uint32_t)) +
           2 * align256(size_t(kMaxGroups) * sizeof(uint32_t));
}

void select_workspace_layout(void* ws, int64_t P, SelectArgs& a)
{
    const int64_t nt = n_tiles(P);
    char* p = static_cast<char*>(ws);
    a.ballots = reinterpret_cast<uint64_t*>(p);
    p += align256(size_t(nt) * kSegsPerTile * 4 * sizeof(uint64_t));
    a.tile_count = reinterpret_cast<uint32_t*>(p);
    p += align256(size_t(nt) * sizeof(uint32_t));
    a.tile_offset = reinterpret_cast<uint32_t*>(p);
    p += align256(size_t(nt) * sizeof(uint32_t));
    a.group_total = reinterpret_cast<uint32_t*>(p);
    p += align256(size_t(kMaxGroups) * sizeof(uint32_t));
    a.group_offset = reinterpret_cast<uint32_t*>(p);
    a.n_tiles = nt;
}

hipError_t launch_select(const SelectArgs& a, bool aligned, hipStream_t s)
{
    const unsigned grid = static_cast<unsigned>(a.n_tiles);
    const unsigned groups = static_cast<unsigned>((a.n_tiles + kScanBlock - 1) / kScanBlock);
    if (groups > static_cast<unsigned>(kMaxGroups)) return hipErrorInvalidValue;
    if (aligned)
        select_mark<true><<<grid, kBlock, 0, s>>>(a);
    else
        select_mark<false><<<grid, kBlock, 0, s>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    select_scan<<<groups, kScanBlock, 0, s>>>(a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    select_top<<<1, kScanBlock, 0, s>>>(a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (aligned)
        select_scatter<true><<<grid, kBlock, 0, s>>>(a);
    else
        select_scatter<false><<<grid, kBlock, 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_sparse(const SparseArgs& a, int mode, hipStream_t s)
{
    // enough lanes for `capacity` entries (the count is only known on the
    // device); lanes past the count exit
    int64_t g = (a.capacity + int64_t(kBlock) * kSparseE - 1) / (int64_t(kBlock) * kSparseE);
    if (g > kListMaxBlocks) g = kListMaxBlocks;
    if (g < 1) g = 1;
    if (mode == MATH_FAST)
        sparse_apply<MATH_FAST><<<static_cast<unsigned>(g), kBlock, 0, s>>>(a);
    else
        sparse_apply<MATH_IEEE><<<static_cast<unsigned>(g), kBlock, 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_scatter(float* dst, int64_t P, const int32_t* idx, const float* val,
                          const int64_t* d_count, int64_t capacity, hipStream_t s)
{
    int64_t g = (capacity + kBlock - 1) / kBlock;
    if (g > kListMaxBlocks) g = kListMaxBlocks;
    if (g < 1) g = 1;
    scatter_list<<<static_cast<unsigned>(g), kBlock, 0, s>>>(dst, P, idx, val, d_count, capacity);
    return hipGetLastError();
}

}  // namespace fasgd
