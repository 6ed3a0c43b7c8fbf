// B-FASGD push selection with deterministic ordered compaction, and the
// sparse server apply of the compacted list.
//
// Work is cut into wave tiles of kTileSegs segments of 64 chunks (one chunk is
// 4 consecutive parameters, one 16-byte vector).  Every wave owns one tile and
// never waits on another wave, so no launch has a block barrier in its
// streaming part.  Selection runs in three or four launches (calls of up to
// about 50M parameters: two, described at select_mark_totals):
//   mark     the wave loads its tile of v, draws one Philox4x32-10 call per
//            chunk (the counter is the global chunk index, so one call feeds
//            one vector of v), forms four ballots per segment (1 bit per
//            parameter), stores the tile's ballot words in one store and its
//            transmit count;
//   scan     one block per 1024 tiles scans their counts (offsets within the
//            group) and records the group total; the group totals are
//            scanned and the device count written by the last scan block to
//            finish or, for many groups, by one more single-block launch;
//   scatter  the wave loads its tile of gradients, reads its ballot words
//            (scalar loads), places every transmitted (index, value) pair in
//            an LDS stage at the popcount of the bits before it (ascending
//            index order), and writes the staged run at group offset + tile
//            offset in contiguous stores.
// When the mark step ran inside the preceding dense pass (which leaves the
// ballot words but no tile counts), the scan counts each tile's ballot bits
// (in the two-launch range, a count launch does, for the direct scatter).
// Several pushes selected together run as one set of launches with the push
// as the grid's y index, each with its own gradient, counter words, output
// slice and workspace slice.
// The result depends only on (seed, T, client, v, grad), never on timing.
#include <string.h>

#include "kernels.hpp"

// v_writelane_b32: write a wave-uniform value into one lane of a VGPR.  The
// LLVM intrinsic is reached through its symbol name (this compiler has no
// clang builtin for it), so the backend still schedules it and handles its
// hazards as for any other instruction.
__device__ int amdgcn_writelane(int value, int lane, int old) __asm("llvm.amdgcn.writelane.i32");

namespace fasgd {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kSelBlock = 256;                // 4 independent waves
constexpr int kWavesPerBlock = kSelBlock / kWave;
constexpr int kTileSegs = 4;                  // 64-chunk segments per wave tile
constexpr int kTileWords = 4 * kTileSegs;     // ballot words per tile
constexpr int64_t kChunksPerTile = int64_t(kTileSegs) * kWave;  // 256 chunks = 1024 parameters
constexpr int kScanBlock = 1024;              // tiles per scan group
constexpr int kMaxGroups = 4096;              // 2^31 parameters need 2048
constexpr int kFusedTopGroups = 64;           // up to 64 groups: group scan fused into the scan launch

__host__ __device__ inline int64_t n_chunks(int64_t P) { return (P + 3) / 4; }
int64_t n_tiles(int64_t P) { return (n_chunks(P) + kChunksPerTile - 1) / kChunksPerTile; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

__device__ __forceinline__ uint64_t lanes_below(int lane)
{
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// The 4 values of chunk q, one load each; parameters at or past P read as
// NaN, which never transmits (mark) and is never written (scatter).
__device__ __forceinline__ f4 load_chunk(const float* p, int64_t q, int64_t P)
{
    const int64_t j = q * 4;
    f4 x;
#pragma unroll
    for (int c = 0; c < 4; ++c) x[c] = (j + c < P) ? p[j + c] : __builtin_nanf("");
    return x;
}

// wave tile of this wave (wave-uniform)
__device__ __forceinline__ int64_t wave_tile()
{
    return static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
}

// The arguments of push blockIdx.y of a batch: its gradient, counter words,
// list, count, list index and workspace slice.
__device__ __forceinline__ SelectArgs push_args(const SelectArgs& a0, const SelectBatch& bt)
{
    const int b = blockIdx.y;
    if (b == 0) return a0;
    SelectArgs a = a0;
    a.grad = bt.grad[b];
    a.ctr_T = bt.ctr_T[b];
    a.ctr_client = bt.ctr_client[b];
    if (a0.out_idx) a.out_idx = a0.out_idx + b * bt.list_stride;
    if (a0.out_val) a.out_val = a0.out_val + b * bt.list_stride;
    a.d_count = a0.d_count + b;
    if (a0.seg_start) a.seg_start = a0.seg_start + b * bt.index_stride;
    const size_t off = b * bt.ws_stride;
    a.ballots = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(a0.ballots) + off);
    a.tile_count = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(a0.tile_count) + off);
    a.tile_offset = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(a0.tile_offset) + off);
    a.group_total = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(a0.group_total) + off);
    a.group_offset = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(a0.group_offset) + off);
    a.groups_done = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(a0.groups_done) + off);
    return a;
}

// Mark one tile and return its transmit count (wave-uniform).  FULL: the
// tile lies inside [0, P) and v is 16-byte aligned, so no lane needs a bounds
// check (every tile but the last).  STORE_COUNT: also store the count for the
// scan launch.
template <bool FULL, bool STORE_COUNT>
__device__ __forceinline__ uint32_t mark_tile(const SelectArgs& a, int64_t tile, int lane)
{
    const int64_t nch = n_chunks(a.P);
    const int64_t q0 = tile * kChunksPerTile + lane;
    // every load of the tile before any arithmetic
    f4 v[kTileSegs];
#pragma unroll
    for (int s = 0; s < kTileSegs; ++s) {
        const int64_t q = q0 + s * kWave;
        if (FULL)
            v[s] = *reinterpret_cast<const f4*>(a.v + q * 4);
        else if (q < nch)
            v[s] = load_chunk(a.v, q, a.P);
    }
    // lane k < kTileWords holds ballot word k of the tile (low, high halves)
    int word_lo = 0, word_hi = 0;
    uint32_t count = 0;
#pragma unroll
    for (int s = 0; s < kTileSegs; ++s) {
        const int64_t q = q0 + s * kWave;
        uint32_t nib = 0;
        if (FULL || q < nch) {
            const uint64_t qg = a.chunk_base + static_cast<uint64_t>(q);   // global chunk index
            const uint4 w = philox4x32_10(
                make_uint4(static_cast<uint32_t>(qg), static_cast<uint32_t>(qg >> 32), a.ctr_T, a.ctr_client),
                a.key0, a.key1);
            nib = transmit_bit(w.x, v[s][0], a.c, a.eps_c) | (transmit_bit(w.y, v[s][1], a.c, a.eps_c) << 1) |
                  (transmit_bit(w.z, v[s][2], a.c, a.eps_c) << 2) |
                  (transmit_bit(w.w, v[s][3], a.c, a.eps_c) << 3);
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint64_t bk = __builtin_amdgcn_ballot_w64(((nib >> k) & 1u) != 0);
            count += static_cast<uint32_t>(__popcll(bk));
            word_lo = amdgcn_writelane(static_cast<int>(bk), 4 * s + k, word_lo);
            word_hi = amdgcn_writelane(static_cast<int>(bk >> 32), 4 * s + k, word_hi);
        }
    }
    if (lane < kTileWords)
        a.ballots[tile * kTileWords + lane] =
            (static_cast<uint64_t>(static_cast<uint32_t>(word_hi)) << 32) | static_cast<uint32_t>(word_lo);
    if (STORE_COUNT && lane == 0) a.tile_count[tile] = count;
    return count;
}

__global__ __launch_bounds__(kSelBlock) void select_mark(const SelectArgs a0, const SelectBatch bt, bool aligned)
{
    const SelectArgs a = push_args(a0, bt);
    if (blockIdx.x == 0 && threadIdx.x == 0) *a.groups_done = 0u;   // for the scan launch
    const int64_t tile = wave_tile();
    if (tile >= a.n_tiles) return;
    const int lane = threadIdx.x & (kWave - 1);
    if (aligned && (tile + 1) * kChunksPerTile * 4 <= a.P)
        mark_tile<true, true>(a, tile, lane);
    else
        mark_tile<false, true>(a, tile, lane);
}

// Inclusive prefix sum over the wave's 64 lanes in register-to-register
// DPP adds: row shifts by 1, 2, 4 and 8 give each 16-lane row its own
// prefix sums (lanes shifted in from outside the row read 0), then the last
// lane of row 0 is broadcast into row 1 and of row 2 into row 3, and the
// last lane of row 1 (the sum of lanes 0-31) into rows 2 and 3.
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x)
{
    constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
    constexpr int kRowBcast15 = 0x142, kRowBcast31 = 0x143;
    x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), kRowShr1, 0xf, 0xf, false));
    x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), kRowShr2, 0xf, 0xf, false));
    x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), kRowShr4, 0xf, 0xf, false));
    x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), kRowShr8, 0xf, 0xf, false));
    x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), kRowBcast15, 0xa, 0xf, false));
    x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), kRowBcast31, 0xc, 0xf, false));
    return x;
}

// Block-wide exclusive scan of one value per thread (kScanBlock threads).
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* total)
{
    __shared__ uint32_t wave_total[kScanBlock / kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const uint32_t inc = wave_inclusive_scan(x);
    if (lane == kWave - 1) wave_total[wave] = inc;
    __syncthreads();
    if (wave == 0) {
        const uint32_t t = wave_inclusive_scan(lane < kScanBlock / kWave ? wave_total[lane] : 0u);
        if (lane < kScanBlock / kWave) wave_total[lane] = t;
    }
    __syncthreads();
    *total = wave_total[kScanBlock / kWave - 1];
    return inc - x + (wave > 0 ? wave_total[wave - 1] : 0u);
}

// Offsets of the groups (at most kMaxGroups) from their totals, and the
// number transmitted; run by one block.
__device__ __forceinline__ void scan_groups(const SelectArgs& a, int64_t ng, bool atomic_loads)
{
    uint32_t carry = 0;
    for (int64_t base = 0; base < ng; base += kScanBlock) {
        const int64_t g = base + threadIdx.x;
        uint32_t c = 0;
        if (g < ng)
            c = atomic_loads ? __hip_atomic_load(a.group_total + g, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT)
                             : a.group_total[g];
        uint32_t total;
        const uint32_t off = block_exclusive_scan(c, &total);
        if (g < ng) a.group_offset[g] = carry + off;
        carry += total;
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        *a.d_count = static_cast<int64_t>(carry);
        if (a.seg_start) a.seg_start[a.n_segs] = carry;
    }
}

// Group g of 1024 tiles: offsets of its tiles within the group and the group
// total.  FUSED_TOP: the last group block to arrive (arrival counter, zeroed
// by the mark launch before this one) then scans the group totals itself.
// Each arrival is a device-scope release, which costs more than a launch once
// there are many groups; then select_top does that scan as its own launch.
// FROM_BALLOTS: the tile counts were not written (the mark step ran inside
// another pass); count the tiles' ballot bits instead.  The wave's 64 tiles
// are 8 KB of ballot words, read in 8 rounds of one 16-byte piece per lane
// (8 lanes per tile, contiguous), summed over each group of 8 lanes and
// passed through LDS to the lane of the tile.
__device__ __forceinline__ uint32_t wave_tile_bits(const SelectArgs& a, int64_t wave_first_tile, int lane)
{
    __shared__ uint32_t s_cnt[kScanBlock / kWave][kWave];
    const int w = threadIdx.x / kWave;
    constexpr int kPieces = kTileWords / 2;                 // 16-byte pieces per tile
    constexpr int kTilesPerRound = kWave / kPieces;
    const ulonglong2* base = reinterpret_cast<const ulonglong2*>(a.ballots + wave_first_tile * kTileWords);
#pragma unroll
    for (int r = 0; r < kPieces; ++r) {
        const int t = r * kTilesPerRound + lane / kPieces;  // tile of this lane's piece, within the wave's 64
        uint32_t n = 0;
        if (wave_first_tile + t < a.n_tiles) {
            const ulonglong2 piece = base[r * kWave + lane];
            n = __popcll(piece.x) + __popcll(piece.y);
        }
#pragma unroll
        for (int d = 1; d < kPieces; d <<= 1) n += __shfl_xor(n, d, kWave);
        if (lane % kPieces == 0) s_cnt[w][t] = n;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    return s_cnt[w][lane];
}

template <bool FUSED_TOP, bool FROM_BALLOTS>
__global__ __launch_bounds__(kScanBlock) void select_scan(const SelectArgs a0, const SelectBatch bt)
{
    const SelectArgs a = push_args(a0, bt);
    const int64_t t = static_cast<int64_t>(blockIdx.x) * kScanBlock + threadIdx.x;
    uint32_t c = 0;
    if (FROM_BALLOTS) {
        const int64_t wave_first = t - (threadIdx.x & (kWave - 1));
        c = wave_tile_bits(a, wave_first, threadIdx.x & (kWave - 1));
        if (t >= a.n_tiles) c = 0;
    } else if (t < a.n_tiles) {
        c = a.tile_count[t];
    }
    uint32_t total;
    const uint32_t off = block_exclusive_scan(c, &total);
    if (t < a.n_tiles) a.tile_offset[t] = off;
    if (!FUSED_TOP) {
        if (threadIdx.x == 0) a.group_total[blockIdx.x] = total;
        return;
    }
    __shared__ bool last;
    if (threadIdx.x == 0) {
        __hip_atomic_store(a.group_total + blockIdx.x, total, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        // release: the total is visible before the arrival is counted
        const uint32_t before = __hip_atomic_fetch_add(a.groups_done, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        last = before == gridDim.x - 1;
    }
    __syncthreads();
    if (last) scan_groups(a, gridDim.x, true);
}

__global__ __launch_bounds__(kScanBlock) void select_top(const SelectArgs a0, const SelectBatch bt)
{
    const SelectArgs a = push_args(a0, bt);
    scan_groups(a, (a.n_tiles + kScanBlock - 1) / kScanBlock, false);
}

// Scatter one tile; FULL as for mark_tile.  The tile's entries are staged
// in output order in the wave's LDS slice and leave in contiguous full-wave
// stores (a lane storing its own entries directly issues four sparse masked
// stores per segment).  The slice holds kStageEntries; a segment that would
// overflow it flushes it first, so the slice stays small enough for full
// occupancy while a tile at any transmit fraction up to about 1/4 leaves in
// one flush.
constexpr int kStageEntries = 4 * kWave;     // one segment's worth

__device__ __forceinline__ void wave_lds_order()
{
    // the wave's LDS operations execute in order; keep the compiler from
    // moving the reads of other lanes' entries above the writes
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// entries [0, n) of the stage to output positions [base, base + n)
__device__ __forceinline__ void drain(const SelectArgs& a, const int32_t* s_idx, const float* s_val, uint32_t n,
                                      int64_t base, int lane)
{
    for (uint32_t e = lane; e < n; e += kWave) {
        const int64_t pos = base + e;
        if (pos < a.capacity) {
            a.out_idx[pos] = s_idx[e];
            a.out_val[pos] = s_val[e];
        }
    }
}

// Every gradient load of the tile, issued before anything waits on them (at
// any transmit fraction worth compacting every line holds a transmitted
// value, so loading the whole tile costs no traffic).
template <bool FULL>
__device__ __forceinline__ void load_tile_grad(const SelectArgs& a, int64_t tile, int lane, f4 (&g)[kTileSegs])
{
    const int64_t nch = n_chunks(a.P);
    const int64_t q0 = tile * kChunksPerTile + lane;
#pragma unroll
    for (int s = 0; s < kTileSegs; ++s) {
        const int64_t q = q0 + s * kWave;
        if (FULL)
            g[s] = *reinterpret_cast<const f4*>(a.grad + q * 4);
        else if (q < nch)
            g[s] = load_chunk(a.grad, q, a.P);
    }
}

// The tile's ballot words (wave-uniform, scalar loads).  Loaded together
// with the gradients, ahead of any use: loading them segment by segment
// left up to three dependent scalar round trips in each wave's lifetime.
__device__ __forceinline__ void load_tile_ballots(const SelectArgs& a, int64_t tile, uint64_t (&bw)[kTileWords])
{
    const uint64_t* tb = a.ballots + tile * kTileWords;
#pragma unroll
    for (int k = 0; k < kTileWords; ++k) bw[k] = tb[k];
}

// The tile's entries, with gradients g and ballot words bw (loaded into
// registers already, or the tile's words in the workspace), to list
// positions from `base` on.  Chunks past P carry no ballot bits, so their
// (unloaded) gradients are never read.
__device__ __forceinline__ void scatter_loaded(const SelectArgs& a, int64_t tile, int lane, const f4 (&g)[kTileSegs],
                                               const uint64_t* bw, int64_t base, int32_t* s_idx, float* s_val)
{
    const int64_t q0 = tile * kChunksPerTile + lane;
    const uint64_t below = lanes_below(lane);
    uint32_t staged = 0;
    uint32_t seg_pos = 0;   // lane s < kTileSegs: list position of segment s's first entry
#pragma unroll
    for (int s = 0; s < kTileSegs; ++s) {
        const uint64_t b0 = bw[4 * s], b1 = bw[4 * s + 1], b2 = bw[4 * s + 2], b3 = bw[4 * s + 3];
        const uint32_t nib = static_cast<uint32_t>((b0 >> lane) & 1) | static_cast<uint32_t>(((b1 >> lane) & 1) << 1) |
                             static_cast<uint32_t>(((b2 >> lane) & 1) << 2) |
                             static_cast<uint32_t>(((b3 >> lane) & 1) << 3);
        const uint32_t n_seg = __popcll(b0) + __popcll(b1) + __popcll(b2) + __popcll(b3);
        if (lane == s) seg_pos = static_cast<uint32_t>(base + staged);
        if (staged + n_seg > static_cast<uint32_t>(kStageEntries)) {
            wave_lds_order();
            drain(a, s_idx, s_val, staged, base, lane);
            wave_lds_order();
            base += staged;
            staged = 0;
        }
        // entries of the lanes below come first; within a lane, ascending c
        uint32_t p = staged + __popcll(b0 & below) + __popcll(b1 & below) + __popcll(b2 & below) +
                     __popcll(b3 & below);
        const int64_t q = q0 + s * kWave;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            if ((nib >> c) & 1u) {
                s_idx[p] = static_cast<int32_t>(q * 4 + c);
                s_val[p] = g[s][c];
                ++p;
            }
        }
        staged += n_seg;
    }
    wave_lds_order();
    drain(a, s_idx, s_val, staged, base, lane);
    if (a.seg_start) {
        static_assert(kTileSegs * kWave * 4 == kTileSegs * kPushSeg, "a tile segment is a list-index segment");
        const int64_t sg = tile * kTileSegs + lane;
        if (lane < kTileSegs && sg < a.n_segs) a.seg_start[sg] = seg_pos;
    }
}

// EARLY: every ballot word and the list position are loaded and waited for
// while the gradient loads are in flight.  In calls of at most
// kFusedTopGroups groups (up to 67M parameters: the scan after a pass that
// took the decisions, and standalone calls past the two-launch form) every
// wave's latency is exposed, and this took the 25M selection, then in three
// launches, from 44.0-46.6 to 41.5-45.1 us (same box, lists identical).  Otherwise the compiler issues each part
// where it is first used (three dependent scalar round trips per tile),
// which was 3 % faster at 1e9 (1.63-1.65 against 1.70 ms), where many more
// waves are in flight to cover them.
template <bool FULL, bool EARLY>
__device__ __forceinline__ void scatter_tile(const SelectArgs& a, int64_t tile, int lane, int32_t* s_idx,
                                             float* s_val)
{
    f4 g[kTileSegs];
    load_tile_grad<FULL>(a, tile, lane, g);
    const uint32_t group_off = a.group_offset[tile / kScanBlock];
    const uint32_t tile_off = a.tile_offset[tile];
    const int64_t base = static_cast<int64_t>(group_off) + tile_off;
    if (EARLY) {
        uint64_t bw[kTileWords];
        load_tile_ballots(a, tile, bw);
        // uses that keep the compiler from sinking these loads to the first
        // use of each
#pragma unroll
        for (int k = 0; k < kTileWords; ++k) asm volatile("" ::"s"(bw[k]));
        asm volatile("" ::"s"(base));
        scatter_loaded(a, tile, lane, g, bw, base, s_idx, s_val);
    } else {
        scatter_loaded(a, tile, lane, g, a.ballots + tile * kTileWords, base, s_idx, s_val);
    }
}

// 64 VGPRs keep 8 waves per SIMD (the EARLY form needs 71 uncapped).
template <bool EARLY>
__global__ __launch_bounds__(kSelBlock) __attribute__((amdgpu_waves_per_eu(8, 8))) void select_scatter(
    const SelectArgs a0, const SelectBatch bt, bool aligned)
{
    const SelectArgs a = push_args(a0, bt);
    __shared__ int32_t s_idx[kWavesPerBlock][kStageEntries];
    __shared__ float s_val[kWavesPerBlock][kStageEntries];
    const int64_t tile = wave_tile();
    if (tile >= a.n_tiles) return;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x / kWave;
    if (aligned && (tile + 1) * kChunksPerTile * 4 <= a.P)
        scatter_tile<true, EARLY>(a, tile, lane, s_idx[w], s_val[w]);
    else
        scatter_tile<false, EARLY>(a, tile, lane, s_idx[w], s_val[w]);
}

// Two-launch selection, for calls of at most kDirectMaxTiles tiles per push:
// no scan launch, and no wave waits for another.
//   select_mark_totals  blocks of TPB waves, one tile each, store the
//     tiles' ballot words as select_mark does and their counts in LDS; the
//     last wave to arrive (an LDS arrival counter) stores each tile's offset
//     within the block and the block total as 16 bits (at most 16 x 1024).
//   select_scatter_direct  every wave finds its own list position: the
//     totals of all blocks before its tile's block plus the tile's offset
//     within its block.  KT 16-byte loads per lane cover the totals of
//     512 KT blocks; they are issued before the gradient loads, so the wait
//     for them leaves the gradients in flight, and the wave sums them in
//     registers and across its lanes.
// The result is that of the three launches, bit for bit.  Against them on
// the same box (10 % transmitted, back to back): 8.4M 17.2 against 19.6 us,
// 12M 23.0 against 25.9, 25M 39.2 against 41.0, 33M 51.2 against 52.2 and
// 50M 86.0 against 91.3 us; at 1.8M the kernels take 8.2 us against 10.0 us
// for the two-launch form with 16-wave blocks and a block barrier in the
// scatter that this form replaced.  Blocks of 8 tiles are the faster shape
// where both fit (probes at 25M: 38.6 against 39.2 us with blocks of 16 and
// half the loads).  A mark block of 8 waves takes 1.1-1.4 us longer than one
// of 4 at 25M (it needs 8 free wave slots on a CU to start), but blocks of 4
// would need twice the loads and more registers than the scatter has.
constexpr int kDirectLoads = 6;                                  // 16-byte loads of block totals per lane, at most
constexpr int64_t kDirectMaxBlocks = int64_t(kDirectLoads) * kWave * 8;   // 3072 block totals (6 KB)
constexpr int64_t kDirectMaxTiles = 16 * kDirectMaxBlocks;       // 49,152 tiles: 50.3M parameters
static_assert(kDirectMaxBlocks * sizeof(uint16_t) <= kMaxGroups * sizeof(uint32_t),
              "16-bit block totals fit the group totals");

template <int TPB>
__global__ __launch_bounds__(TPB * kWave) void select_mark_totals(const SelectArgs a0, const SelectBatch bt,
                                                                  bool aligned)
{
    static_assert(TPB * kChunksPerTile * 4 < 65536 && TPB <= kWave, "a block total fits 16 bits");
    const SelectArgs a = push_args(a0, bt);
    __shared__ uint32_t s_cnt[TPB];
    __shared__ uint32_t s_arrived;
    if (threadIdx.x == 0) s_arrived = 0;
    __syncthreads();
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t t0 = static_cast<int64_t>(blockIdx.x) * TPB;
    const int64_t tile = t0 + w;
    const int lane = threadIdx.x & (kWave - 1);
    uint32_t count = 0;
    if (tile < a.n_tiles) {
        if (aligned && (tile + 1) * kChunksPerTile * 4 <= a.P)
            count = mark_tile<true, false>(a, tile, lane);
        else
            count = mark_tile<false, false>(a, tile, lane);
    }
    int last = 0;
    if (lane == 0) {
        s_cnt[w] = count;
        // release / acquire: the last wave to arrive sees every count
        last = __hip_atomic_fetch_add(&s_arrived, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP) == TPB - 1;
    }
    if (__builtin_amdgcn_readfirstlane(last)) {
        const uint32_t c = lane < TPB ? s_cnt[lane] : 0u;
        const uint32_t inc = wave_inclusive_scan(c);
        if (lane < TPB && t0 + lane < a.n_tiles) a.tile_offset[t0 + lane] = inc - c;
        if (lane == TPB - 1) reinterpret_cast<uint16_t*>(a.group_total)[blockIdx.x] = static_cast<uint16_t>(inc);
    }
}

__device__ __forceinline__ uint32_t sum_halves(uint32_t x) { return (x & 0xffffu) + (x >> 16); }

// Mask of the 16-bit halves j < r of 32-bit word i (halves 2i, 2i + 1).
__device__ __forceinline__ uint32_t halves_below(int i, int r)
{
    return (2 * i + 1 < r) ? 0xffffffffu : (2 * i < r ? 0xffffu : 0u);
}

// The list position of the first entry of a tile whose block has
// `blocks_before` blocks before it: the sum of their 16-bit totals plus the
// tile's offset within its block.  Lane l holds the groups l + 64 k of 8
// totals (tv[k]); the group that holds the last totals that count is summed
// in part.
template <int KT>
__device__ __forceinline__ int64_t direct_position(const uint4 (&tv)[KT], int blocks_before, uint32_t tile_off,
                                                   int lane)
{
    const int whole = blocks_before >> 3;   // groups of 8 totals that count in full
    const int r = blocks_before & 7;        // totals of the next group that count
    const uint32_t m0 = halves_below(0, r), m1 = halves_below(1, r), m2 = halves_below(2, r),
                   m3 = halves_below(3, r);
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < KT; ++k) {
        const int grp = lane + kWave * k;
        const bool all = grp < whole;
        const uint32_t x = sum_halves(tv[k].x & (all ? ~0u : m0)) + sum_halves(tv[k].y & (all ? ~0u : m1)) +
                           sum_halves(tv[k].z & (all ? ~0u : m2)) + sum_halves(tv[k].w & (all ? ~0u : m3));
        s += grp <= whole ? x : 0u;
    }
    const uint32_t inc = wave_inclusive_scan(s);
    return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(inc), kWave - 1)) + tile_off;
}

// The call's count (and the list index's last entry) from the last tile.
template <typename Words>
__device__ __forceinline__ void direct_finish(const SelectArgs& a, int64_t tile, int lane, const Words& bw,
                                              int64_t base)
{
    if (tile == a.n_tiles - 1 && lane == 0) {
        uint32_t mine = 0;
#pragma unroll
        for (int k = 0; k < kTileWords; ++k) mine += __popcll(bw[k]);
        *a.d_count = base + mine;
        if (a.seg_start) a.seg_start[a.n_segs] = static_cast<uint32_t>(base + mine);
    }
}

// FULL as for mark_tile.  The partial tile (or every tile of misaligned
// arrays) finds its position before it loads its gradients, and reads its
// ballot words from the workspace where it uses them, which needs fewer
// registers.
template <bool FULL, int TPB, int KT>
__device__ __forceinline__ void scatter_direct_tile(const SelectArgs& a, int64_t tile, int lane, int32_t* s_idx,
                                                    float* s_val)
{
    const int nb = static_cast<int>(tile / TPB);   // blocks before this tile's block
    const uint4* tot = reinterpret_cast<const uint4*>(a.group_total);
    uint4 tv[KT];
#pragma unroll
    for (int k = 0; k < KT; ++k)   // only the groups some lane needs (wave-uniform)
        tv[k] = kWave * k <= (nb >> 3) ? tot[lane + kWave * k] : make_uint4(0u, 0u, 0u, 0u);
    f4 g[kTileSegs];
    if (FULL) {
        // the loads above are issued before the gradients', so waiting for
        // them leaves the gradients in flight
        __builtin_amdgcn_sched_barrier(0);
        load_tile_grad<true>(a, tile, lane, g);
        const uint32_t tile_off = a.tile_offset[tile];
        uint64_t bw[kTileWords];
        load_tile_ballots(a, tile, bw);
        // uses that keep the compiler from sinking these (scalar) loads to
        // the first use of each
#pragma unroll
        for (int k = 0; k < kTileWords; ++k) asm volatile("" ::"s"(bw[k]));
        asm volatile("" ::"s"(tile_off));
        const int64_t base = direct_position<KT>(tv, nb, tile_off, lane);
        scatter_loaded(a, tile, lane, g, bw, base, s_idx, s_val);
        direct_finish(a, tile, lane, bw, base);
    } else {
        const int64_t base = direct_position<KT>(tv, nb, a.tile_offset[tile], lane);
        load_tile_grad<false>(a, tile, lane, g);
        const uint64_t* bw = a.ballots + tile * kTileWords;
        scatter_loaded(a, tile, lane, g, bw, base, s_idx, s_val);
        direct_finish(a, tile, lane, bw, base);
    }
}

template <int TPB, int KT>
__global__ __launch_bounds__(kSelBlock) __attribute__((amdgpu_waves_per_eu(8, 8))) void select_scatter_direct(
    const SelectArgs a0, const SelectBatch bt, bool aligned)
{
    const SelectArgs a = push_args(a0, bt);
    __shared__ int32_t s_idx[kWavesPerBlock][kStageEntries];
    __shared__ float s_val[kWavesPerBlock][kStageEntries];
    const int64_t tile = wave_tile();
    if (tile >= a.n_tiles) return;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x / kWave;
    if (aligned && (tile + 1) * kChunksPerTile * 4 <= a.P)
        scatter_direct_tile<true, TPB, KT>(a, tile, lane, s_idx[w], s_val[w]);
    else
        scatter_direct_tile<false, TPB, KT>(a, tile, lane, s_idx[w], s_val[w]);
}

// After a pass that took the decisions (it leaves ballot words, no counts):
// each tile's offset within its block of TPB tiles and the blocks' 16-bit
// totals, for select_scatter_direct.  A wave counts 64 consecutive tiles,
// one per lane (as the scan from ballots does); a block of tiles is TPB
// consecutive lanes, so a scan within segments of TPB lanes gives both.
template <int TPB>
__global__ __launch_bounds__(kSelBlock) void select_count_totals(const SelectArgs a)
{
    static_assert(kWave % TPB == 0, "a block of tiles lies within one wave");
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t t = static_cast<int64_t>(blockIdx.x) * kSelBlock + threadIdx.x;
    uint32_t c = wave_tile_bits(a, t - lane, lane);
    if (t >= a.n_tiles) c = 0;
    uint32_t inc = c;
#pragma unroll
    for (int d = 1; d < TPB; d <<= 1) {
        const uint32_t up = __shfl_up(inc, d, kWave);
        if (lane % TPB >= d) inc += up;
    }
    if (t < a.n_tiles) a.tile_offset[t] = inc - c;
    if (lane % TPB == TPB - 1 && t - (TPB - 1) < a.n_tiles)
        reinterpret_cast<uint16_t*>(a.group_total)[t / TPB] = static_cast<uint16_t>(inc);
}

// The two-launch selection; from_ballots (one push): the decisions were
// taken by the preceding pass, so the first launch only counts.
template <int TPB>
hipError_t launch_direct(const SelectArgs& a, const SelectBatch& bt, int B, bool aligned, bool from_ballots,
                         hipStream_t s)
{
    const int64_t blocks = (a.n_tiles + TPB - 1) / TPB;
    const int kt = static_cast<int>((blocks + kWave * 8 - 1) / (kWave * 8));
    if (from_ballots) {
        select_count_totals<TPB><<<static_cast<unsigned>((a.n_tiles + kSelBlock - 1) / kSelBlock), kSelBlock, 0,
                                   s>>>(a);
    } else {
        const dim3 mgrid(static_cast<unsigned>(blocks), static_cast<unsigned>(B));
        select_mark_totals<TPB><<<mgrid, TPB * kWave, 0, s>>>(a, bt, aligned);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 grid(static_cast<unsigned>((a.n_tiles + kWavesPerBlock - 1) / kWavesPerBlock), static_cast<unsigned>(B));
    switch (kt) {
    case 1: select_scatter_direct<TPB, 1><<<grid, kSelBlock, 0, s>>>(a, bt, aligned); break;
    case 2: select_scatter_direct<TPB, 2><<<grid, kSelBlock, 0, s>>>(a, bt, aligned); break;
    case 3: select_scatter_direct<TPB, 3><<<grid, kSelBlock, 0, s>>>(a, bt, aligned); break;
    case 4: select_scatter_direct<TPB, 4><<<grid, kSelBlock, 0, s>>>(a, bt, aligned); break;
    case 5: select_scatter_direct<TPB, 5><<<grid, kSelBlock, 0, s>>>(a, bt, aligned); break;
    case 6: select_scatter_direct<TPB, 6><<<grid, kSelBlock, 0, s>>>(a, bt, aligned); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

constexpr int kListBlock = 256;               // list kernels: 4 waves
constexpr int kSparseE = 2;                   // list entries per lane
constexpr int64_t kListMaxBlocks = 65536;     // grid cap of the list kernels (grid-stride)

// A wave owns 64 E consecutive list entries and lane l takes entries
// l, l + 64, ...: every gather instruction covers 64 consecutive entries
// (ascending indices, so few cache lines), and each thread issues all
// kSparseE of its gathers before the first update.
template <int MODE>
__global__ __launch_bounds__(kListBlock) void sparse_apply(const SparseArgs a)
{
    int64_t m = *a.d_count;
    if (m > a.capacity) m = a.capacity;
    const Hyper h = a.h;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wave_id = (static_cast<int64_t>(blockIdx.x) * kListBlock + threadIdx.x) / kWave;
    const int64_t n_waves = static_cast<int64_t>(gridDim.x) * (kListBlock / kWave);
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

__global__ __launch_bounds__(kListBlock) void scatter_list(float* __restrict__ dst, int64_t P,
                                                       const int32_t* __restrict__ idx,
                                                       const float* __restrict__ val,
                                                       const int64_t* __restrict__ d_count, int64_t capacity)
{
    int64_t m = *d_count;
    if (m > capacity) m = capacity;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kListBlock;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kListBlock + threadIdx.x; i < m; i += stride) {
        const int64_t j = idx[i];
        if (j >= 0 && j < P) dst[j] = val[i];
    }
}

}  // namespace

static_assert(kSelTileParams == kChunksPerTile * 4 && kSelTileWords == kTileWords && kSelMaxGroups == kMaxGroups,
              "the workspace size in kernels.hpp follows this file's layout");

size_t select_workspace_bytes(int64_t P) { return select_workspace_bytes_for(P); }

void select_workspace_layout(void* ws, int64_t P, SelectArgs& a)
{
    const int64_t nt = n_tiles(P);
    char* p = static_cast<char*>(ws);
    a.ballots = reinterpret_cast<uint64_t*>(p);
    p += align256(size_t(nt) * kTileWords * sizeof(uint64_t));
    a.tile_count = reinterpret_cast<uint32_t*>(p);
    p += align256(size_t(nt) * sizeof(uint32_t));
    a.tile_offset = reinterpret_cast<uint32_t*>(p);
    p += align256(size_t(nt) * sizeof(uint32_t));
    a.group_total = reinterpret_cast<uint32_t*>(p);
    p += align256(size_t(kMaxGroups) * sizeof(uint32_t));
    a.group_offset = reinterpret_cast<uint32_t*>(p);
    p += align256(size_t(kMaxGroups) * sizeof(uint32_t));
    a.groups_done = reinterpret_cast<uint32_t*>(p);
    a.n_tiles = nt;
}

hipError_t launch_select(const SelectArgs& a, const SelectBatch& bt, int B, bool aligned, hipStream_t s)
{
    const unsigned gx = static_cast<unsigned>((a.n_tiles + kWavesPerBlock - 1) / kWavesPerBlock);
    const unsigned groups = static_cast<unsigned>((a.n_tiles + kScanBlock - 1) / kScanBlock);
    if (groups > static_cast<unsigned>(kMaxGroups) || B < 1 || B > kMaxBatch) return hipErrorInvalidValue;
    if (a.n_tiles <= 8 * kDirectMaxBlocks) return launch_direct<8>(a, bt, B, aligned, false, s);
    if (a.n_tiles <= kDirectMaxTiles) return launch_direct<16>(a, bt, B, aligned, false, s);
    hipError_t e;
    const dim3 grid(gx, static_cast<unsigned>(B));
    select_mark<<<grid, kSelBlock, 0, s>>>(a, bt, aligned);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (groups <= static_cast<unsigned>(kFusedTopGroups)) {
        select_scan<true, false><<<dim3(groups, B), kScanBlock, 0, s>>>(a, bt);
    } else {
        select_scan<false, false><<<dim3(groups, B), kScanBlock, 0, s>>>(a, bt);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        select_top<<<dim3(1, B), kScanBlock, 0, s>>>(a, bt);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (groups <= static_cast<unsigned>(kFusedTopGroups))
        select_scatter<true><<<grid, kSelBlock, 0, s>>>(a, bt, aligned);
    else
        select_scatter<false><<<grid, kSelBlock, 0, s>>>(a, bt, aligned);
    return hipGetLastError();
}

hipError_t launch_select_after_mark(const SelectArgs& a, bool aligned, hipStream_t s)
{
    const unsigned gx = static_cast<unsigned>((a.n_tiles + kWavesPerBlock - 1) / kWavesPerBlock);
    const unsigned groups = static_cast<unsigned>((a.n_tiles + kScanBlock - 1) / kScanBlock);
    if (groups > static_cast<unsigned>(kMaxGroups)) return hipErrorInvalidValue;
    SelectBatch bt;
    memset(&bt, 0, sizeof bt);
    if (a.n_tiles <= 8 * kDirectMaxBlocks) return launch_direct<8>(a, bt, 1, aligned, true, s);
    if (a.n_tiles <= kDirectMaxTiles) return launch_direct<16>(a, bt, 1, aligned, true, s);
    hipError_t e;
    if (groups <= static_cast<unsigned>(kFusedTopGroups)) {
        select_scan<true, true><<<groups, kScanBlock, 0, s>>>(a, bt);
    } else {
        select_scan<false, true><<<groups, kScanBlock, 0, s>>>(a, bt);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        select_top<<<1, kScanBlock, 0, s>>>(a, bt);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (groups <= static_cast<unsigned>(kFusedTopGroups))
        select_scatter<true><<<gx, kSelBlock, 0, s>>>(a, bt, aligned);
    else
        select_scatter<false><<<gx, kSelBlock, 0, s>>>(a, bt, aligned);
    return hipGetLastError();
}

hipError_t launch_sparse(const SparseArgs& a, int variant, hipStream_t s)
{
    // enough lanes for `capacity` entries (the count is only known on the
    // device); lanes past the count exit
    int64_t g = (a.capacity + int64_t(kListBlock) * kSparseE - 1) / (int64_t(kListBlock) * kSparseE);
    if (g > kListMaxBlocks) g = kListMaxBlocks;
    if (g < 1) g = 1;
    const unsigned grid = static_cast<unsigned>(g);
    switch (variant) {
    case kernel_variant(MATH_FAST, 0): sparse_apply<kernel_variant(MATH_FAST, 0)><<<grid, kListBlock, 0, s>>>(a); break;
    case kernel_variant(MATH_IEEE, 0): sparse_apply<kernel_variant(MATH_IEEE, 0)><<<grid, kListBlock, 0, s>>>(a); break;
    case kernel_variant(MATH_FAST, 1): sparse_apply<kernel_variant(MATH_FAST, 1)><<<grid, kListBlock, 0, s>>>(a); break;
    case kernel_variant(MATH_IEEE, 1): sparse_apply<kernel_variant(MATH_IEEE, 1)><<<grid, kListBlock, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_scatter(float* dst, int64_t P, const int32_t* idx, const float* val,
                          const int64_t* d_count, int64_t capacity, hipStream_t s)
{
    int64_t g = (capacity + kListBlock - 1) / kListBlock;
    if (g > kListMaxBlocks) g = kListMaxBlocks;
    if (g < 1) g = 1;
    scatter_list<<<static_cast<unsigned>(g), kListBlock, 0, s>>>(dst, P, idx, val, d_count, capacity);
    return hipGetLastError();
}

}  // namespace fasgd
