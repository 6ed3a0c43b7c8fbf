// Launchers of the device kernels, called by the C ABI after it has
// validated every argument.  Each returns the HIP launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "device_math.hpp"

namespace fasgd {

constexpr int kMaxK = 64;

// One fused pass of K gradients over the whole state.
struct DenseArgs {
    float* theta;
    float* n;
    float* b;
    float* v;
    const float* grad[kMaxK];
    float coef[kMaxK];      // FASGD IEEE: tau_k; FASGD FAST and SASGD: alpha / tau_k
    int64_t P;
    int32_t K;
    float lambda;           // synchronous SGD: gradients are divided by lambda
    Hyper h;
};

// Self-check of the IEEE update's short correctly rounded sequences against
// the general ones: kIeeeChecks mismatch counters (cleared first).
constexpr int kIeeeChecks = 4;
hipError_t launch_check_ieee(const Hyper& h, uint64_t seed, int64_t n_updates, unsigned long long* counts,
                             hipStream_t s);

hipError_t launch_init(float* n, float* b, float* v, int32_t* last_T, int64_t P,
                       float n0, float b0, float v0, hipStream_t s);
// variant: kernel_variant(math mode, v reading)
hipError_t launch_fasgd_dense(const DenseArgs& a, int variant, bool aligned, hipStream_t s);
hipError_t launch_sasgd_dense(const DenseArgs& a, bool aligned, hipStream_t s);
// theta <- theta - coef[k] * (g_k / lambda), k in order (coef[k] = lr)
hipError_t launch_sync_sgd(const DenseArgs& a, bool aligned, hipStream_t s);

// Kernels with one parameter per thread (the paths for arrays that are only
// 4-byte aligned) cover at most this many: a launch has fewer than 2^32
// work-items.
constexpr int64_t kMaxScalarItems = (int64_t(1) << 32) - 256;

// B-FASGD selection: Philox decisions -> per-wave ballots and per-tile
// counts, an exclusive scan of the tile counts, then ordered writes.
struct SelectArgs {
    const float* v;
    const float* grad;
    int32_t* out_idx;
    float* out_val;
    int64_t* d_count;
    uint64_t* ballots;      // 4 per 64 chunks of 4 parameters
    uint32_t* tile_count;
    uint32_t* tile_offset;   // within its group of 1024 tiles
    uint32_t* group_total;
    uint32_t* group_offset;
    uint32_t* groups_done;  // arrival counter of the scan blocks
    int64_t P;
    int64_t capacity;
    int64_t n_tiles;
    float c;
    float eps_c;
    uint32_t key0, key1;    // seed low / high words
    uint32_t ctr_T;         // counter word 2
    uint32_t ctr_client;    // counter word 3
    uint64_t chunk_base;    // global chunk index of chunk 0 (index_base / 4)
    uint32_t* seg_start;    // optional: list position of each kPushSeg-parameter segment, [n_segs + 1]
    int64_t n_segs;
};

// Several pushes selected in one set of launches (the grid's y index is the
// push): SelectArgs describes push 0 and SelectBatch how the others differ.
constexpr int kMaxBatch = 64;
struct SelectBatch {
    const float* grad[kMaxBatch];
    uint32_t ctr_T[kMaxBatch];
    uint32_t ctr_client[kMaxBatch];
    int64_t list_stride;    // entries between consecutive pushes' lists (their capacity)
    int64_t index_stride;   // entries between consecutive pushes' list indexes
    size_t ws_stride;       // workspace bytes per push
};

// Workspace of one selection: 16 ballot words (8 bytes each) per wave tile
// of kSelTileParams parameters, a count and an offset per tile, the totals
// and offsets of at most kSelMaxGroups groups of tiles, and an arrival
// counter, each part 256-byte aligned.
constexpr int64_t kSelTileParams = 1024;
constexpr int kSelTileWords = 16;
constexpr int kSelMaxGroups = 4096;
constexpr size_t sel_align256(size_t x) { return (x + 255) & ~size_t(255); }
constexpr size_t select_workspace_bytes_for(int64_t P)
{
    const size_t nt = static_cast<size_t>((P + kSelTileParams - 1) / kSelTileParams);
    return sel_align256(nt * kSelTileWords * sizeof(uint64_t)) + 2 * sel_align256(nt * sizeof(uint32_t)) +
           2 * sel_align256(size_t(kSelMaxGroups) * sizeof(uint32_t)) + sel_align256(sizeof(uint32_t));
}
size_t select_workspace_bytes(int64_t P);
// Carve the workspace into ballots / tile counts / tile offsets.
void select_workspace_layout(void* ws, int64_t P, SelectArgs& a);
hipError_t launch_select(const SelectArgs& a, const SelectBatch& bt, int B, bool aligned, hipStream_t s);
// The selection after its mark step was taken elsewhere (ballot words in the
// workspace, tile counts not written): scan with the counts taken from the
// ballots, then scatter.  One push.
hipError_t launch_select_after_mark(const SelectArgs& a, bool aligned, hipStream_t s);

struct SparseArgs {
    float* theta;
    float* n;
    float* b;
    float* v;
    int32_t* last_T;
    const int32_t* idx;
    const float* val;
    const int64_t* d_count;
    int64_t capacity;
    int64_t P;
    float coef;             // as DenseArgs::coef for this one push
    int32_t last_T_value;   // T
    Hyper h;
};

hipError_t launch_sparse(const SparseArgs& a, int variant, hipStream_t s);

// Index of a compacted list: seg_start[s] is the position of the first entry
// with index >= kPushSeg * s, seg_start[n_segs] the number of entries.
constexpr int kPushSeg = 256;
inline int64_t push_segments(int64_t P) { return (P + kPushSeg - 1) / kPushSeg; }

// A compacted push applied inside a dense pass, before its K gradients.
struct PushArgs {
    const int32_t* idx;
    const float* val;
    const int64_t* d_count;
    const uint32_t* seg_start;
    int64_t capacity;
    int64_t n_segs;
    float coef;             // as DenseArgs::coef for the push
};

// mark: optional; the selection arguments of the next push, whose transmit
// decisions the pass then takes from the v it leaves.  aligned: every array
// 16-byte aligned (needed only beyond kMaxScalarItems parameters).
hipError_t launch_fasgd_dense_push(const DenseArgs& a, const PushArgs& p, const SelectArgs* mark, int variant,
                                   bool aligned, hipStream_t s);
// A cached push (dropped values re-apply the client's cache) in one pass over
// 16-byte aligned arrays: the list (with its index) merged into the cache,
// then the cache applied as one gradient (a.K = 1, a.coef[0]).
hipError_t launch_fasgd_cached_push(const DenseArgs& a, const PushArgs& p, float* cache, int variant, hipStream_t s);
// dst[idx[i]] = val[i] for the list (with its index) over a 16-byte aligned
// dst, written segment by segment in whole lines.
hipError_t launch_merge_list(float* dst, int64_t P, const PushArgs& p, hipStream_t s);

// B compacted pushes applied in order in one pass (push b at timestamp
// T0 + b); listed parameters get last_T = T0 + the last push that lists them.
struct PushBatchArgs {
    float* theta;
    float* n;
    float* b;
    float* v;
    int32_t* last_T;
    const int32_t* idx;        // [B][list_stride]
    const float* val;          // [B][list_stride]
    const int64_t* d_count;    // [B]
    const uint32_t* seg_start; // [B][n_segs + 1]
    int64_t list_stride;       // the lists' capacity
    int64_t n_segs;
    int64_t P;
    int32_t B;
    int32_t T0;
    float coef[kMaxBatch];
    Hyper h;
};

hipError_t launch_apply_pushes(const PushBatchArgs& a, int variant, bool aligned, hipStream_t s);

// Paper-literal decisions per segment (groups of up to kSegGroup segments).
constexpr int kSegGroup = 32;

struct SegGroup {
    int64_t start[kSegGroup + 1];          // offsets of the group's segments, start[n] = end of the last
    int64_t block_prefix[kSegGroup + 1];   // blocks before segment i within the group
    int32_t n;                             // segments in the group
    int32_t pad;
    int64_t first_seg;                     // global index of the group's first segment
    int64_t partial_base;                  // partial sums of the group start here
};

struct SegApplyArgs {
    float* theta;
    float* n;
    float* b;
    float* v;
    int32_t* last_T;
    const float* grad;
    const uint8_t* transmit;
    float coef;             // as DenseArgs::coef for this push
    int32_t last_T_value;   // T
    int32_t aligned;        // every array 16-byte aligned
    Hyper h;
};

int64_t seg_blocks(int64_t length);
size_t segments_workspace_bytes(int64_t P, int32_t S);
hipError_t launch_seg_decide(const SegGroup& g, const float* v, double* partial, float c, float eps_c,
                             uint64_t seed, uint32_t ctr_T, uint32_t ctr_client, uint8_t* transmit,
                             hipStream_t s);
hipError_t launch_seg_apply(const SegGroup& g, const SegApplyArgs& a, int variant, hipStream_t s);

// dst[idx[i]] = val[i] for i < min(*d_count, capacity); indices outside
// [0, P) are skipped.
hipError_t launch_scatter(float* dst, int64_t P, const int32_t* idx, const float* val,
                          const int64_t* d_count, int64_t capacity, hipStream_t s);

}  // namespace fasgd
