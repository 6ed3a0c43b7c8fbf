// B-FASGD push selection with deterministic ordered compaction, and the
// sparse server apply of the compacted list.
//
// Selection runs in three launches, none of which waits on another block:
//   mark     one Philox4x32-10 call per 4 parameters (the counter is the
//            chunk index j/4, so one call feeds one 16-byte vector of v),
//            four wave ballots per 64 chunks stored to the workspace (1 bit
//            per parameter), and a per-tile count;
//   scan     one block turns the tile counts into exclusive tile offsets
//            and writes the total to the device count;
//   scatter  every wave rebuilds its output position from the ballots of
//            its tile (scalar loads and popcounts) plus the tile offset,
//            and writes (index, value) pairs in ascending index order.
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
constexpr int kScanBlock = 1024;

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

// Exclusive scan of the tile counts by one block: each thread owns a
// contiguous run of tiles.
__global__ __launch_bounds__(kScanBlock) void select_scan(const SelectArgs a)
{
    const int64_t nt = a.n_tiles;
    const int64_t per = (nt + kScanBlock - 1) / kScanBlock;
    const int64_t t0 = threadIdx.x * per;
    const int64_t t1 = t0 + per < nt ? t0 + per : nt;
    uint32_t sum = 0;
    for (int64_t t = t0; t < t1; ++t) sum += a.tile_count[t];

    // inclusive scan of the per-thread sums across the block
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    uint32_t x = sum;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const uint32_t y = __shfl_up(x, d, kWave);
        if (lane >= d) x += y;
    }
    __shared__ uint32_t wave_total[kScanBlock / kWave];
    if (lane == kWave - 1) wave_total[wave] = x;
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
    uint32_t run = x - sum + (wave > 0 ? wave_total[wave - 1] : 0u);   // exclusive
    for (int64_t t = t0; t < t1; ++t) {
        a.tile_offset[t] = run;
        run += a.tile_count[t];
    }
    if (threadIdx.x == kScanBlock - 1) *a.d_count = static_cast<int64_t>(run);
}

template <bool ALIGNED>
__global__ __launch_bounds__(kBlock) void select_scatter(const SelectArgs a)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t tile = blockIdx.x;
    const uint64_t below = lanes_below(lane);
    const uint64_t* tb = a.ballots + tile * kSegsPerTile * 4;

    // position of segment (0, wave) within the output: tile offset plus
    // everything the earlier segments of this tile transmitted
    uint32_t pos0 = a.tile_offset[tile];
    for (int s = 0; s < wave; ++s)
        pos0 += __popcll(tb[4 * s]) + __popcll(tb[4 * s + 1]) + __popcll(tb[4 * s + 2]) + __popcll(tb[4 * s + 3]);

#pragma unroll
    for (int it = 0; it < kItems; ++it) {
        const int s = it * kWavesPerBlock + wave;
        const uint64_t b0 = tb[4 * s], b1 = tb[4 * s + 1], b2 = tb[4 * s + 2], b3 = tb[4 * s + 3];
        const uint32_t nib = static_cast<uint32_t>((b0 >> lane) & 1) | static_cast<uint32_t>(((b1 >> lane) & 1) << 1) |
                             static_cast<uint32_t>(((b2 >> lane) & 1) << 2) |
                             static_cast<uint32_t>(((b3 >> lane) & 1) << 3);
        if (nib) {
            int64_t pos = static_cast<int64_t>(pos0) + __popcll(b0 & below) + __popcll(b1 & below) +
                          __popcll(b2 & below) + __popcll(b3 & below);
            const int64_t q = (tile * kSegsPerTile + s) * kWave + lane;
            const f4 g = load_chunk<ALIGNED>(a.grad, q, a.P);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if ((nib >> c) & 1u) {
                    if (pos < a.capacity) {
                        a.out_idx[pos] = static_cast<int32_t>(q * 4 + c);
                        a.out_val[pos] = g[c];
                    }
                    ++pos;
                }
            }
        }
        // the remaining segments of this item, then the earlier ones of the next
        for (int t = s; t < s + kWavesPerBlock && t < kSegsPerTile; ++t)
            pos0 += __popcll(tb[4 * t]) + __popcll(tb[4 * t + 1]) + __popcll(tb[4 * t + 2]) + __popcll(tb[4 * t + 3]);
    }
}

template <int MODE>
__global__ __launch_bounds__(kBlock) void sparse_apply(const SparseArgs a)
{
    int64_t m = *a.d_count;
    if (m > a.capacity) m = a.capacity;
    const Hyper h = a.h;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < m; i += stride) {
        const int64_t j = a.idx[i];
        if (j < 0 || j >= a.P) continue;
        float th = a.theta[j], n = a.n[j], b = a.b[j], v = a.v[j];
        fasgd_step<MODE>(th, n, b, v, a.val[i], a.coef, h);
        a.theta[j] = th; a.n[j] = n; a.b[j] = b; a.v[j] = v;
        a.last_T[j] = a.last_T_value;
    }
}

}  // namespace

size_t select_workspace_bytes(int64_t P)
{
    const int64_t nt = n_tiles(P);
    return align256(size_t(nt) * kSegsPerTile * 4 * sizeof(uint64_t)) + 2 * align256(size_t(nt) * sizeof(uint32_t));
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
    a.n_tiles = nt;
}

hipError_t launch_select(const SelectArgs& a, bool aligned, hipStream_t s)
{
    const unsigned grid = static_cast<unsigned>(a.n_tiles);
    if (aligned)
        select_mark<true><<<grid, kBlock, 0, s>>>(a);
    else
        select_mark<false><<<grid, kBlock, 0, s>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    select_scan<<<1, kScanBlock, 0, s>>>(a);
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
    int64_t g = (a.capacity + kBlock - 1) / kBlock;
    if (g > 256 * 16) g = 256 * 16;
    if (g < 1) g = 1;
    if (mode == MATH_FAST)
        sparse_apply<MATH_FAST><<<static_cast<unsigned>(g), kBlock, 0, s>>>(a);
    else
        sparse_apply<MATH_IEEE><<<static_cast<unsigned>(g), kBlock, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace fasgd
