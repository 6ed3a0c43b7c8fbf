// C ABI of libfasgd.so (declared in include/fasgd.h): host-side argument
// checks, step-staleness bookkeeping (Sec. 2.1) and kernel dispatch.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "../../include/fasgd.h"
#include "anchor.hpp"
#include "kernels.hpp"

static_assert(FASGD_MAX_K == fasgd::kMaxK, "K limit mismatch");
static_assert(FASGD_MAX_BATCH == fasgd::kMaxBatch, "batch limit mismatch");

namespace {

thread_local char g_err[512];

// fasgd_record_next_pass: events recorded around the next FASGD pass kernel
// this thread launches (one-shot)
thread_local hipEvent_t g_pass_start = nullptr;
thread_local hipEvent_t g_pass_stop = nullptr;

hipError_t pass_begin(hipStream_t stream)
{
    return g_pass_start ? hipEventRecord(g_pass_start, stream) : hipSuccess;
}

hipError_t pass_end(hipStream_t stream)
{
    if (!g_pass_stop) return hipSuccess;
    const hipError_t e = hipEventRecord(g_pass_stop, stream);
    g_pass_start = g_pass_stop = nullptr;
    return e;
}

fasgd_status fail(fasgd_status s, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return s;
}

fasgd_status ok()
{
    g_err[0] = '\0';
    return FASGD_OK;
}

fasgd_status hip_fail(hipError_t e, const char* what)
{
    return fail(FASGD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

fasgd_status check_state(const fasgd_state* st, bool need_stats)
{
    if (!st) return fail(FASGD_ERR_NULL, "state is NULL");
    if (st->P < 1) return fail(FASGD_ERR_ARG, "P = %lld must be >= 1", (long long)st->P);
    if (st->lambda < 1) return fail(FASGD_ERR_ARG, "lambda = %d must be >= 1", st->lambda);
    if (st->T < 0 || st->T > INT32_MAX) return fail(FASGD_ERR_ARG, "T = %lld out of range", (long long)st->T);
    if (st->dense_T < -1 || st->dense_T >= st->T)
        return fail(FASGD_ERR_ARG, "dense_T = %lld is not in [-1, T)", (long long)st->dense_T);
    if (!st->theta || !st->last_T) return fail(FASGD_ERR_NULL, "theta or last_T is NULL");
    if (need_stats && (!st->n || !st->b || !st->v)) return fail(FASGD_ERR_NULL, "n, b or v is NULL");
    if (!aligned(st->theta, 4) || !aligned(st->last_T, 4) || (st->n && !aligned(st->n, 4)) ||
        (st->b && !aligned(st->b, 4)) || (st->v && !aligned(st->v, 4)))
        return fail(FASGD_ERR_ALIGN, "state arrays must be 4-byte aligned");
    if (need_stats && st->math_mode != FASGD_MATH_IEEE && st->math_mode != FASGD_MATH_FAST)
        return fail(FASGD_ERR_ARG, "math_mode = %d is not a fasgd_math value", st->math_mode);
    if (need_stats && st->v_reading != FASGD_V_EQUATIONS && st->v_reading != FASGD_V_PROSE)
        return fail(FASGD_ERR_ARG, "v_reading = %d is not a fasgd_v_reading value", st->v_reading);
    return FASGD_OK;
}

// Arrays that are not all 16-byte aligned take the one-parameter-per-thread
// kernels, whose launches cover fewer than 2^32 parameters.
fasgd_status scalar_size_ok(int64_t P, bool vec)
{
    if (!vec && P > fasgd::kMaxScalarItems)
        return fail(FASGD_ERR_ALIGN, "P = %lld needs 16-byte aligned arrays (at most %lld otherwise)", (long long)P,
                    (long long)fasgd::kMaxScalarItems);
    return FASGD_OK;
}

// kernel template variant of a validated state
int variant_of(const fasgd_state* st)
{
    return fasgd::kernel_variant(st->math_mode, st->v_reading == FASGD_V_PROSE);
}

// The IEEE update's short correctly rounded sequences hold for these eps and
// alpha (x = max(n - b^2, 0) + eps >= 2^-96 under the square root; the
// quotient alpha / (v tau) stays normal wherever the division takes them).
bool ieee_short_ok(float eps, float alpha)
{
    return isfinite(eps) && eps >= 0x1p-96f && fabsf(alpha) >= 0x1p-20f && fabsf(alpha) < 0x1p20f;
}

fasgd::Hyper hyper_of(const fasgd_state* st)
{
    fasgd::Hyper h;
    h.gamma = st->gamma;
    h.omg = 1.0f - st->gamma;
    h.beta = st->beta;
    h.omb = 1.0f - st->beta;
    h.eps = st->eps;
    h.alpha = st->alpha;
    h.rn_short = ieee_short_ok(st->eps, st->alpha) ? 1 : 0;
    return h;
}

// tau = (T + k) - grad_ts[k] >= 0; the divisor is max(tau, 1).
fasgd_status staleness(const fasgd_state* st, const int32_t* clients, const int64_t* grad_ts, int32_t K,
                       float* tau_div)
{
    for (int32_t k = 0; k < K; ++k) {
        const int64_t Tk = st->T + k;
        if (clients[k] < 0 || clients[k] >= st->lambda)
            return fail(FASGD_ERR_CLIENT, "clients[%d] = %d is outside [0, %d)", k, clients[k], st->lambda);
        if (grad_ts[k] < 0 || grad_ts[k] > Tk)
            return fail(FASGD_ERR_STALENESS, "grad_ts[%d] = %lld is not in [0, T + k = %lld]", k,
                        (long long)grad_ts[k], (long long)Tk);
        const int64_t tau = Tk - grad_ts[k];
        tau_div[k] = static_cast<float>(tau > 0 ? tau : 1);
    }
    return FASGD_OK;
}

fasgd_status dense_common(fasgd_state* st, const float* const* grads, const int32_t* clients,
                          const int64_t* grad_ts, int32_t K, bool fasgd_mode, fasgd::DenseArgs& a, bool& vec)
{
    fasgd_status s = check_state(st, fasgd_mode);
    if (s != FASGD_OK) return s;
    if (!grads || !clients || !grad_ts) return fail(FASGD_ERR_NULL, "grads, clients or grad_ts is NULL");
    if (K < 1 || K > FASGD_MAX_K) return fail(FASGD_ERR_ARG, "K = %d is not in [1, %d]", K, FASGD_MAX_K);
    if (st->T + K - 1 > INT32_MAX) return fail(FASGD_ERR_ARG, "T + K - 1 exceeds the int32 timestamp range");
    float tau_div[FASGD_MAX_K];
    s = staleness(st, clients, grad_ts, K, tau_div);
    if (s != FASGD_OK) return s;
    vec = aligned(st->theta, 16) &&
          (!fasgd_mode || (aligned(st->n, 16) && aligned(st->b, 16) && aligned(st->v, 16)));
    memset(&a, 0, sizeof a);
    for (int32_t k = 0; k < K; ++k) {
        if (!grads[k]) return fail(FASGD_ERR_NULL, "grads[%d] is NULL", k);
        if (!aligned(grads[k], 4)) return fail(FASGD_ERR_ALIGN, "grads[%d] is not 4-byte aligned", k);
        vec = vec && aligned(grads[k], 16);
        a.grad[k] = grads[k];
        const bool rate = !fasgd_mode || st->math_mode == FASGD_MATH_FAST;
        a.coef[k] = rate ? st->alpha / tau_div[k] : tau_div[k];
    }
    s = scalar_size_ok(st->P, vec);
    if (s != FASGD_OK) return s;
    a.theta = st->theta;
    a.n = st->n;
    a.b = st->b;
    a.v = st->v;
    a.P = st->P;
    a.K = K;
    a.h = hyper_of(st);
    return FASGD_OK;
}

bool finite_nonneg(float x) { return isfinite(x) && x >= 0.0f; }

fasgd_status check_segments(const int64_t* seg, int32_t S, int64_t P)
{
    if (!seg) return fail(FASGD_ERR_NULL, "seg is NULL");
    if (S < 1) return fail(FASGD_ERR_ARG, "S = %d must be >= 1", S);
    if (seg[0] != 0 || seg[S] != P) return fail(FASGD_ERR_ARG, "segments must start at 0 and end at P");
    for (int32_t s = 0; s < S; ++s)
        if (seg[s + 1] <= seg[s]) return fail(FASGD_ERR_ARG, "segment %d is empty or out of order", s);
    return FASGD_OK;
}

// Group g0 .. g0 + n - 1 of the segments; partial_base is updated past it.
fasgd::SegGroup segment_group(const int64_t* seg, int32_t S, int32_t g0, int64_t& partial_base)
{
    fasgd::SegGroup g;
    memset(&g, 0, sizeof g);
    g.n = S - g0 < fasgd::kSegGroup ? S - g0 : fasgd::kSegGroup;
    g.first_seg = g0;
    g.partial_base = partial_base;
    int64_t blocks = 0;
    for (int32_t i = 0; i <= g.n; ++i) {
        g.start[i] = seg[g0 + i];
        g.block_prefix[i] = blocks;
        if (i < g.n) blocks += fasgd::seg_blocks(seg[g0 + i + 1] - seg[g0 + i]);
    }
    partial_base += blocks;
    return g;
}

}  // namespace

extern "C" {

fasgd_status fasgd_init_state(fasgd_state* st, int64_t P, int32_t lambda, int32_t mu, float alpha,
                              float gamma, float beta, float eps, int32_t math_mode, float n0, float b0,
                              float v0, float* theta, float* n, float* b, float* v, int32_t* last_T,
                              hipStream_t stream)
{
    if (!st) return fail(FASGD_ERR_NULL, "state is NULL");
    if (P < 1) return fail(FASGD_ERR_ARG, "P = %lld must be >= 1", (long long)P);
    if (lambda < 1 || mu < 1) return fail(FASGD_ERR_ARG, "lambda and mu must be >= 1");
    if (!(isfinite(alpha) && alpha > 0.0f)) return fail(FASGD_ERR_ARG, "alpha must be finite and > 0");
    if (!(gamma >= 0.0f && gamma <= 1.0f) || !(beta >= 0.0f && beta <= 1.0f))
        return fail(FASGD_ERR_ARG, "gamma and beta must be in [0, 1]");
    if (!(isfinite(eps) && eps > 0.0f)) return fail(FASGD_ERR_ARG, "eps must be finite and > 0");
    if (math_mode != FASGD_MATH_IEEE && math_mode != FASGD_MATH_FAST)
        return fail(FASGD_ERR_ARG, "math_mode = %d is not a fasgd_math value", math_mode);
    if (!isfinite(n0) || !isfinite(b0) || !isfinite(v0)) return fail(FASGD_ERR_ARG, "n0, b0, v0 must be finite");
    if (!theta || !last_T) return fail(FASGD_ERR_NULL, "theta or last_T is NULL");
    if ((n || b || v) && !(n && b && v)) return fail(FASGD_ERR_NULL, "n, b and v must be all set or all NULL");
    if (!aligned(theta, 4) || !aligned(last_T, 4) || (n && (!aligned(n, 4) || !aligned(b, 4) || !aligned(v, 4))))
        return fail(FASGD_ERR_ALIGN, "state arrays must be 4-byte aligned");
    const hipError_t e = fasgd::launch_init(n, b, v, last_T, P, n0, b0, v0, stream);
    if (e != hipSuccess) return hip_fail(e, "fasgd_init_state");
    fasgd_state s;
    memset(&s, 0, sizeof s);
    s.P = P;
    s.lambda = lambda;
    s.mu = mu;
    s.alpha = alpha;
    s.gamma = gamma;
    s.beta = beta;
    s.eps = eps;
    s.math_mode = math_mode;
    s.v_reading = FASGD_V_EQUATIONS;
    s.T = 0;
    s.dense_T = -1;
    s.theta = theta;
    s.n = n;
    s.b = b;
    s.v = v;
    s.last_T = last_T;
    *st = s;
    return ok();
}

fasgd_status fasgd_apply_updates(fasgd_state* st, const float* const* grads, const int32_t* clients,
                                 const int64_t* grad_ts, int32_t K, hipStream_t stream)
{
    fasgd::DenseArgs a;
    bool vec = false;
    fasgd_status s = dense_common(st, grads, clients, grad_ts, K, true, a, vec);
    if (s != FASGD_OK) return s;
    hipError_t e = pass_begin(stream);
    if (e == hipSuccess) e = fasgd::launch_fasgd_dense(a, variant_of(st), vec, stream);
    if (e == hipSuccess) e = pass_end(stream);
    if (e != hipSuccess) return hip_fail(e, "fasgd_apply_updates");
    st->dense_T = st->T + K - 1;
    st->T += K;
    return ok();
}

fasgd_status sasgd_apply_updates(fasgd_state* st, const float* const* grads, const int32_t* clients,
                                 const int64_t* grad_ts, int32_t K, hipStream_t stream)
{
    fasgd::DenseArgs a;
    bool vec = false;
    fasgd_status s = dense_common(st, grads, clients, grad_ts, K, false, a, vec);
    if (s != FASGD_OK) return s;
    const hipError_t e = fasgd::launch_sasgd_dense(a, vec, stream);
    if (e != hipSuccess) return hip_fail(e, "sasgd_apply_updates");
    st->dense_T = st->T + K - 1;
    st->T += K;
    return ok();
}

size_t bfasgd_workspace_bytes(int64_t P)
{
    if (P < 1) return 0;
    return fasgd::select_workspace_bytes(P);
}

int64_t bfasgd_list_index_length(int64_t P)
{
    if (P < 1) return 0;
    return fasgd::push_segments(P) + 1;
}

namespace {

// Checks and kernel arguments of B selections; push b's per-push arguments
// are grads[b], T[b], clients[b].  vec: v and every gradient 16-byte aligned.
fasgd_status select_setup(const fasgd_state* st, int32_t B, const float* const* grads, float c, float eps_c,
                          uint64_t seed, const int64_t* T, const int32_t* clients, int32_t* out_idx,
                          float* out_val, int64_t capacity, int64_t* d_count, uint32_t* out_seg_start,
                          void* workspace, size_t workspace_bytes, fasgd::SelectArgs& a, fasgd::SelectBatch& bt,
                          bool& vec)
{
    if (!st) return fail(FASGD_ERR_NULL, "state is NULL");
    if (st->P < 1 || st->P > INT32_MAX) return fail(FASGD_ERR_ARG, "P must be in [1, INT32_MAX] for int32 indices");
    if (st->lambda < 1) return fail(FASGD_ERR_ARG, "lambda = %d must be >= 1", st->lambda);
    if (B < 1 || B > FASGD_MAX_BATCH) return fail(FASGD_ERR_ARG, "B = %d is not in [1, %d]", B, FASGD_MAX_BATCH);
    if (!st->v || !grads || !T || !clients || !d_count || !workspace)
        return fail(FASGD_ERR_NULL, "v, grad, T, clients, d_count or workspace is NULL");
    if (capacity < 0) return fail(FASGD_ERR_ARG, "capacity must be >= 0");
    if (capacity > 0 && (!out_idx || !out_val)) return fail(FASGD_ERR_NULL, "out_idx or out_val is NULL");
    if (!finite_nonneg(c) || !finite_nonneg(eps_c)) return fail(FASGD_ERR_ARG, "c and eps_c must be finite and >= 0");
    for (int32_t p = 0; p < B; ++p) {
        if (!grads[p]) return fail(FASGD_ERR_NULL, "grad of push %d is NULL", p);
        if (T[p] < 0 || T[p] > int64_t(UINT32_MAX))
            return fail(FASGD_ERR_ARG, "T = %lld (push %d) is not in [0, 2^32)", (long long)T[p], p);
        if (clients[p] < 0 || clients[p] >= st->lambda)
            return fail(FASGD_ERR_CLIENT, "client = %d (push %d) is outside [0, %d)", clients[p], p, st->lambda);
        if (!aligned(grads[p], 4)) return fail(FASGD_ERR_ALIGN, "misaligned grad (push %d)", p);
    }
    if (!aligned(st->v, 4) || (out_idx && !aligned(out_idx, 4)) || (out_val && !aligned(out_val, 4)) ||
        !aligned(d_count, 8) || (out_seg_start && !aligned(out_seg_start, 4)))
        return fail(FASGD_ERR_ALIGN, "misaligned v, grad, output list, d_count or out_seg_start");
    if (!aligned(workspace, 256)) return fail(FASGD_ERR_ALIGN, "workspace must be 256-byte aligned");
    if (st->index_base < 0 || (st->index_base & 3) != 0 || st->index_base > (int64_t(1) << 62) - st->P)
        return fail(FASGD_ERR_ARG, "index_base = %lld must be a multiple of 4 in [0, 2^62 - P]",
                    (long long)st->index_base);
    const size_t per_push = fasgd::select_workspace_bytes(st->P);
    if (workspace_bytes / size_t(B) < per_push)
        return fail(FASGD_ERR_CAPACITY, "workspace of %zu bytes is smaller than the %zu needed", workspace_bytes,
                    per_push * size_t(B));
    memset(&a, 0, sizeof a);
    memset(&bt, 0, sizeof bt);
    vec = aligned(st->v, 16);
    for (int32_t p = 0; p < B; ++p) {
        bt.grad[p] = grads[p];
        bt.ctr_T[p] = static_cast<uint32_t>(T[p]);
        bt.ctr_client[p] = static_cast<uint32_t>(clients[p]);
        vec = vec && aligned(grads[p], 16);
    }
    a.v = st->v;
    a.grad = grads[0];
    a.out_idx = out_idx;
    a.out_val = out_val;
    a.d_count = d_count;
    a.P = st->P;
    a.capacity = capacity;
    a.c = c;
    a.eps_c = eps_c;
    a.key0 = static_cast<uint32_t>(seed);
    a.key1 = static_cast<uint32_t>(seed >> 32);
    a.ctr_T = bt.ctr_T[0];
    a.ctr_client = bt.ctr_client[0];
    a.chunk_base = static_cast<uint64_t>(st->index_base) >> 2;
    a.seg_start = out_seg_start;
    a.n_segs = fasgd::push_segments(st->P);
    fasgd::select_workspace_layout(workspace, st->P, a);
    bt.list_stride = capacity;
    bt.index_stride = a.n_segs + 1;
    bt.ws_stride = per_push;
    return FASGD_OK;
}

fasgd_status select_common(const fasgd_state* st, int32_t B, const float* const* grads, float c, float eps_c,
                           uint64_t seed, const int64_t* T, const int32_t* clients, int32_t* out_idx,
                           float* out_val, int64_t capacity, int64_t* d_count, uint32_t* out_seg_start,
                           void* workspace, size_t workspace_bytes, hipStream_t stream, const char* what)
{
    fasgd::SelectArgs a;
    fasgd::SelectBatch bt;
    bool vec = false;
    const fasgd_status s = select_setup(st, B, grads, c, eps_c, seed, T, clients, out_idx, out_val, capacity,
                                        d_count, out_seg_start, workspace, workspace_bytes, a, bt, vec);
    if (s != FASGD_OK) return s;
    const hipError_t e = fasgd::launch_select(a, bt, B, vec, stream);
    if (e != hipSuccess) return hip_fail(e, what);
    return ok();
}

}  // namespace

fasgd_status bfasgd_select_compact(const fasgd_state* st, const float* grad, float c, float eps_c, uint64_t seed,
                                   int64_t T, int32_t client, int32_t* out_idx, float* out_val, int64_t capacity,
                                   int64_t* d_count, uint32_t* out_seg_start, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream)
{
    return select_common(st, 1, &grad, c, eps_c, seed, &T, &client, out_idx, out_val, capacity, d_count,
                         out_seg_start, workspace, workspace_bytes, stream, "bfasgd_select_compact");
}

fasgd_status bfasgd_select_compact_batch(const fasgd_state* st, int32_t B, const float* const* grads, float c,
                                         float eps_c, uint64_t seed, const int64_t* T, const int32_t* clients,
                                         int32_t* out_idx, float* out_val, int64_t capacity, int64_t* d_count,
                                         uint32_t* out_seg_start, void* workspace, size_t workspace_bytes,
                                         hipStream_t stream)
{
    return select_common(st, B, grads, c, eps_c, seed, T, clients, out_idx, out_val, capacity, d_count,
                         out_seg_start, workspace, workspace_bytes, stream, "bfasgd_select_compact_batch");
}

}  // extern "C"

namespace {

// Scratch of bfasgd_select_compact_noalloc: the selection workspace of the
// largest call it accepts, one copy per device, held until the process ends.
// In host code this name is a stand-in for the device array, not its
// address: the calls pass the device address that hipGetSymbolAddress
// returns for the current device.
static_assert(fasgd::select_workspace_bytes_for(FASGD_NOALLOC_MAX_P) == FASGD_NOALLOC_SCRATCH_BYTES,
              "the header states the scratch size");
static __device__ __align__(256) unsigned char scratch[FASGD_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 256;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch` on each device, once looked up

fasgd_status device_scratch(void** out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "bfasgd_select_compact_noalloc: hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(FASGD_ERR_ARG, "bfasgd_select_compact_noalloc: device %d is beyond the %d this library tracks", dev,
                    kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol,
                            "bfasgd_select_compact_noalloc: hipGetSymbolAddress(scratch)");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return FASGD_OK;
}

}  // namespace

extern "C" {

fasgd_status bfasgd_select_compact_noalloc(const fasgd_state* st, const float* grad, float c, float eps_c,
                                           uint64_t seed, int64_t T, int32_t client, int32_t* out_idx,
                                           float* out_val, int64_t capacity, int64_t* d_count,
                                           uint32_t* out_seg_start, hipStream_t stream)
{
    if (!st) return fail(FASGD_ERR_NULL, "state is NULL");
    if (st->P > FASGD_NOALLOC_MAX_P)
        return fail(FASGD_ERR_CAPACITY,
                    "bfasgd_select_compact_noalloc: P = %lld exceeds the %lld parameters its built-in scratch "
                    "holds; use bfasgd_select_compact with a workspace",
                    (long long)st->P, (long long)FASGD_NOALLOC_MAX_P);
    void* ws = nullptr;
    const fasgd_status s = device_scratch(&ws);
    if (s != FASGD_OK) return s;
    return select_common(st, 1, &grad, c, eps_c, seed, &T, &client, out_idx, out_val, capacity, d_count,
                         out_seg_start, ws, FASGD_NOALLOC_SCRATCH_BYTES, stream, "bfasgd_select_compact_noalloc");
}

fasgd_status bfasgd_apply_sparse(fasgd_state* st, const int32_t* idx, const float* val, const int64_t* d_count,
                                 int64_t capacity, int32_t client, int64_t grad_ts, hipStream_t stream)
{
    fasgd_status s = check_state(st, true);
    if (s != FASGD_OK) return s;
    if (!d_count) return fail(FASGD_ERR_NULL, "d_count is NULL");
    if (capacity < 0) return fail(FASGD_ERR_ARG, "capacity must be >= 0");
    if (capacity > 0 && (!idx || !val)) return fail(FASGD_ERR_NULL, "idx or val is NULL");
    if ((idx && !aligned(idx, 4)) || (val && !aligned(val, 4)) || !aligned(d_count, 8))
        return fail(FASGD_ERR_ALIGN, "misaligned idx, val or d_count");
    float tau_div;
    s = staleness(st, &client, &grad_ts, 1, &tau_div);
    if (s != FASGD_OK) return s;
    fasgd::SparseArgs a;
    memset(&a, 0, sizeof a);
    a.theta = st->theta;
    a.n = st->n;
    a.b = st->b;
    a.v = st->v;
    a.last_T = st->last_T;
    a.idx = idx;
    a.val = val;
    a.d_count = d_count;
    a.capacity = capacity;
    a.P = st->P;
    a.coef = st->math_mode == FASGD_MATH_FAST ? st->alpha / tau_div : tau_div;
    a.last_T_value = static_cast<int32_t>(st->T);
    a.h = hyper_of(st);
    if (capacity > 0) {
        const hipError_t e = fasgd::launch_sparse(a, variant_of(st), stream);
        if (e != hipSuccess) return hip_fail(e, "bfasgd_apply_sparse");
    }
    st->T += 1;
    return ok();
}

namespace {

// Checks and kernel arguments of a push followed by K gradients in one pass.
fasgd_status with_push_setup(fasgd_state* st, const int32_t* push_idx, const float* push_val,
                             const int64_t* push_count, const uint32_t* push_seg_start, int64_t capacity,
                             int32_t push_client, int64_t push_grad_ts, const float* const* grads,
                             const int32_t* clients, const int64_t* grad_ts, int32_t K, fasgd::DenseArgs& a,
                             fasgd::PushArgs& p, bool& vec)
{
    fasgd_status s = check_state(st, true);
    if (s != FASGD_OK) return s;
    if (!push_count || !push_seg_start) return fail(FASGD_ERR_NULL, "push_count or push_seg_start is NULL");
    if (capacity < 0) return fail(FASGD_ERR_ARG, "capacity must be >= 0");
    if (capacity > 0 && (!push_idx || !push_val)) return fail(FASGD_ERR_NULL, "push_idx or push_val is NULL");
    if ((push_idx && !aligned(push_idx, 4)) || (push_val && !aligned(push_val, 4)) || !aligned(push_count, 8) ||
        !aligned(push_seg_start, 4))
        return fail(FASGD_ERR_ALIGN, "misaligned push_idx, push_val, push_count or push_seg_start");
    float push_tau;
    s = staleness(st, &push_client, &push_grad_ts, 1, &push_tau);
    if (s != FASGD_OK) return s;
    // the K gradients follow the push: they are applied at T + 1 ... T + K
    fasgd_state after = *st;
    after.T = st->T + 1;
    s = dense_common(&after, grads, clients, grad_ts, K, true, a, vec);
    if (s != FASGD_OK) return s;
    memset(&p, 0, sizeof p);
    p.idx = push_idx;
    p.val = push_val;
    p.d_count = push_count;
    p.seg_start = push_seg_start;
    p.capacity = capacity;
    p.n_segs = fasgd::push_segments(st->P);
    p.coef = st->math_mode == FASGD_MATH_FAST ? st->alpha / push_tau : push_tau;
    return FASGD_OK;
}

}  // namespace

fasgd_status fasgd_apply_with_push(fasgd_state* st, const int32_t* push_idx, const float* push_val,
                                   const int64_t* push_count, const uint32_t* push_seg_start, int64_t capacity,
                                   int32_t push_client, int64_t push_grad_ts, const float* const* grads,
                                   const int32_t* clients, const int64_t* grad_ts, int32_t K, hipStream_t stream)
{
    fasgd::DenseArgs a;
    fasgd::PushArgs p;
    bool vec = false;
    const fasgd_status s = with_push_setup(st, push_idx, push_val, push_count, push_seg_start, capacity,
                                           push_client, push_grad_ts, grads, clients, grad_ts, K, a, p, vec);
    if (s != FASGD_OK) return s;
    hipError_t e = pass_begin(stream);
    if (e == hipSuccess) e = fasgd::launch_fasgd_dense_push(a, p, nullptr, variant_of(st), vec, stream);
    if (e == hipSuccess) e = pass_end(stream);
    if (e != hipSuccess) return hip_fail(e, "fasgd_apply_with_push");
    st->dense_T = st->T + K;
    st->T += K + 1;
    return ok();
}

fasgd_status fasgd_apply_with_push_and_select(fasgd_state* st, const int32_t* push_idx, const float* push_val,
                                              const int64_t* push_count, const uint32_t* push_seg_start,
                                              int64_t push_capacity, int32_t push_client, int64_t push_grad_ts,
                                              const float* const* grads, const int32_t* clients,
                                              const int64_t* grad_ts, int32_t K, const float* next_grad,
                                              int32_t next_client, float c, float eps_c, uint64_t seed,
                                              int32_t* out_idx, float* out_val, int64_t out_capacity,
                                              int64_t* out_count, uint32_t* out_seg_start, void* workspace,
                                              size_t workspace_bytes, hipStream_t stream)
{
    fasgd::DenseArgs a;
    fasgd::PushArgs p;
    bool vec = false;
    fasgd_status s = with_push_setup(st, push_idx, push_val, push_count, push_seg_start, push_capacity,
                                     push_client, push_grad_ts, grads, clients, grad_ts, K, a, p, vec);
    if (s != FASGD_OK) return s;
    // the next push is applied at the timestamp after the pass, and decided
    // from the v the pass leaves
    fasgd_state after = *st;
    after.T = st->T + K + 1;
    const int64_t T_next = after.T;
    fasgd::SelectArgs m;
    fasgd::SelectBatch bt;
    bool sel_vec = false;
    s = select_setup(&after, 1, &next_grad, c, eps_c, seed, &T_next, &next_client, out_idx, out_val, out_capacity,
                     out_count, out_seg_start, workspace, workspace_bytes, m, bt, sel_vec);
    if (s != FASGD_OK) return s;
    // the pass takes the decisions; the selection's own launches scan them
    // and scatter
    hipError_t e = pass_begin(stream);
    if (e == hipSuccess) e = fasgd::launch_fasgd_dense_push(a, p, &m, variant_of(st), vec, stream);
    if (e == hipSuccess) e = pass_end(stream);
    if (e == hipSuccess) e = fasgd::launch_select_after_mark(m, aligned(next_grad, 16), stream);
    if (e != hipSuccess) return hip_fail(e, "fasgd_apply_with_push_and_select");
    st->dense_T = st->T + K;
    st->T += K + 1;
    return ok();
}

fasgd_status fasgd_apply_pushes(fasgd_state* st, int32_t B, const int32_t* idx, const float* val,
                                const int64_t* d_count, const uint32_t* seg_start, int64_t capacity,
                                const int32_t* clients, const int64_t* grad_ts, hipStream_t stream)
{
    fasgd_status s = check_state(st, true);
    if (s != FASGD_OK) return s;
    if (B < 1 || B > FASGD_MAX_BATCH) return fail(FASGD_ERR_ARG, "B = %d is not in [1, %d]", B, FASGD_MAX_BATCH);
    if (st->P > INT32_MAX) return fail(FASGD_ERR_ARG, "P must be <= INT32_MAX for int32 indices");
    if (st->T + B - 1 > INT32_MAX) return fail(FASGD_ERR_ARG, "T + B - 1 exceeds the int32 timestamp range");
    if (!d_count || !seg_start || !clients || !grad_ts)
        return fail(FASGD_ERR_NULL, "d_count, seg_start, clients or grad_ts is NULL");
    if (capacity < 0) return fail(FASGD_ERR_ARG, "capacity must be >= 0");
    if (capacity > 0 && (!idx || !val)) return fail(FASGD_ERR_NULL, "idx or val is NULL");
    if ((idx && !aligned(idx, 4)) || (val && !aligned(val, 4)) || !aligned(d_count, 8) || !aligned(seg_start, 4))
        return fail(FASGD_ERR_ALIGN, "misaligned idx, val, d_count or seg_start");
    float tau_div[FASGD_MAX_BATCH];
    s = staleness(st, clients, grad_ts, B, tau_div);
    if (s != FASGD_OK) return s;
    if (capacity > 0) {
        fasgd::PushBatchArgs a;
        memset(&a, 0, sizeof a);
        a.theta = st->theta;
        a.n = st->n;
        a.b = st->b;
        a.v = st->v;
        a.last_T = st->last_T;
        a.idx = idx;
        a.val = val;
        a.d_count = d_count;
        a.seg_start = seg_start;
        a.list_stride = capacity;
        a.n_segs = fasgd::push_segments(st->P);
        a.P = st->P;
        a.B = B;
        a.T0 = static_cast<int32_t>(st->T);
        for (int32_t p = 0; p < B; ++p)
            a.coef[p] = st->math_mode == FASGD_MATH_FAST ? st->alpha / tau_div[p] : tau_div[p];
        a.h = hyper_of(st);
        const bool vec = aligned(st->theta, 16) && aligned(st->n, 16) && aligned(st->b, 16) &&
                         aligned(st->v, 16) && aligned(st->last_T, 16);
        const hipError_t e = fasgd::launch_apply_pushes(a, variant_of(st), vec, stream);
        if (e != hipSuccess) return hip_fail(e, "fasgd_apply_pushes");
    }
    st->T += B;
    return ok();
}

fasgd_status sgd_sync_apply(fasgd_state* st, const float* const* grads, float lr, hipStream_t stream)
{
    fasgd_status s = check_state(st, false);
    if (s != FASGD_OK) return s;
    if (!grads) return fail(FASGD_ERR_NULL, "grads is NULL");
    if (!(isfinite(lr) && lr > 0.0f)) return fail(FASGD_ERR_ARG, "lr must be finite and > 0");
    if (st->T + 1 > INT32_MAX) return fail(FASGD_ERR_ARG, "T exceeds the int32 timestamp range");
    bool vec = aligned(st->theta, 16);
    for (int32_t k = 0; k < st->lambda; ++k) {
        if (!grads[k]) return fail(FASGD_ERR_NULL, "grads[%d] is NULL", k);
        if (!aligned(grads[k], 4)) return fail(FASGD_ERR_ALIGN, "grads[%d] is not 4-byte aligned", k);
        vec = vec && aligned(grads[k], 16);
    }
    s = scalar_size_ok(st->P, vec);
    if (s != FASGD_OK) return s;
    // lambda gradients in passes of at most FASGD_MAX_K; theta is stored in
    // fp32 between passes exactly as it is held in registers within one
    for (int32_t k0 = 0; k0 < st->lambda; k0 += FASGD_MAX_K) {
        fasgd::DenseArgs a;
        memset(&a, 0, sizeof a);
        const int32_t K = st->lambda - k0 < FASGD_MAX_K ? st->lambda - k0 : FASGD_MAX_K;
        for (int32_t k = 0; k < K; ++k) {
            a.grad[k] = grads[k0 + k];
            a.coef[k] = lr;
        }
        a.theta = st->theta;
        a.P = st->P;
        a.K = K;
        a.lambda = static_cast<float>(st->lambda);
        const hipError_t e = fasgd::launch_sync_sgd(a, vec, stream);
        if (e != hipSuccess) return hip_fail(e, "sgd_sync_apply");
    }
    st->dense_T = st->T;
    st->T += 1;
    return ok();
}

fasgd_status bfasgd_apply_cached(fasgd_state* st, const int32_t* idx, const float* val, const int64_t* d_count,
                                 const uint32_t* seg_start, int64_t capacity, float* cache, int32_t client,
                                 int64_t grad_ts, hipStream_t stream)
{
    fasgd_status s = check_state(st, true);
    if (s != FASGD_OK) return s;
    if (!d_count || !cache) return fail(FASGD_ERR_NULL, "d_count or cache is NULL");
    if (capacity < 0) return fail(FASGD_ERR_ARG, "capacity must be >= 0");
    if (capacity > 0 && (!idx || !val)) return fail(FASGD_ERR_NULL, "idx or val is NULL");
    if ((idx && !aligned(idx, 4)) || (val && !aligned(val, 4)) || !aligned(d_count, 8) || !aligned(cache, 4) ||
        (seg_start && !aligned(seg_start, 4)))
        return fail(FASGD_ERR_ALIGN, "misaligned idx, val, d_count, seg_start or cache");
    float tau_div;
    s = staleness(st, &client, &grad_ts, 1, &tau_div);
    if (s != FASGD_OK) return s;
    const bool vec = aligned(st->theta, 16) && aligned(st->n, 16) && aligned(st->b, 16) && aligned(st->v, 16) &&
                     aligned(cache, 16);
    s = scalar_size_ok(st->P, vec);
    if (s != FASGD_OK) return s;
    const float coef = st->math_mode == FASGD_MATH_FAST ? st->alpha / tau_div : tau_div;
    if (seg_start && (vec || st->P <= fasgd::kMaxScalarItems)) {
        // one pass: the list merged into the cache segment by segment, then applied
        fasgd::DenseArgs a;
        memset(&a, 0, sizeof a);
        a.theta = st->theta;
        a.n = st->n;
        a.b = st->b;
        a.v = st->v;
        a.grad[0] = cache;
        a.coef[0] = coef;
        a.P = st->P;
        a.K = 1;
        a.h = hyper_of(st);
        fasgd::PushArgs p;
        memset(&p, 0, sizeof p);
        p.idx = idx;
        p.val = val;
        p.d_count = d_count;
        p.seg_start = seg_start;
        p.capacity = capacity;
        p.n_segs = fasgd::push_segments(st->P);
        const hipError_t e = fasgd::launch_fasgd_cached_push(a, p, cache, variant_of(st), stream);
        if (e != hipSuccess) return hip_fail(e, "bfasgd_apply_cached");
        st->dense_T = st->T;
        st->T += 1;
        return ok();
    }
    if (capacity > 0) {
        const hipError_t e = fasgd::launch_scatter(cache, st->P, idx, val, d_count, capacity, stream);
        if (e != hipSuccess) return hip_fail(e, "bfasgd_apply_cached (cache update)");
    }
    fasgd::DenseArgs a;
    memset(&a, 0, sizeof a);
    a.theta = st->theta;
    a.n = st->n;
    a.b = st->b;
    a.v = st->v;
    a.grad[0] = cache;
    a.coef[0] = coef;
    a.P = st->P;
    a.K = 1;
    a.h = hyper_of(st);
    const hipError_t e = fasgd::launch_fasgd_dense(a, variant_of(st), vec, stream);
    if (e != hipSuccess) return hip_fail(e, "bfasgd_apply_cached");
    st->dense_T = st->T;
    st->T += 1;
    return ok();
}

fasgd_status bfasgd_apply_fetch(float* theta_client, int64_t P, const int32_t* idx, const float* val,
                                const int64_t* d_count, const uint32_t* seg_start, int64_t capacity,
                                hipStream_t stream)
{
    if (!theta_client || !d_count) return fail(FASGD_ERR_NULL, "theta_client or d_count is NULL");
    if (P < 1) return fail(FASGD_ERR_ARG, "P = %lld must be >= 1", (long long)P);
    if (capacity < 0) return fail(FASGD_ERR_ARG, "capacity must be >= 0");
    if (capacity > 0 && (!idx || !val)) return fail(FASGD_ERR_NULL, "idx or val is NULL");
    if (!aligned(theta_client, 4) || (idx && !aligned(idx, 4)) || (val && !aligned(val, 4)) ||
        !aligned(d_count, 8) || (seg_start && !aligned(seg_start, 4)))
        return fail(FASGD_ERR_ALIGN, "misaligned theta_client, idx, val, d_count or seg_start");
    if (capacity > 0 && seg_start && aligned(theta_client, 16)) {
        fasgd::PushArgs p;
        memset(&p, 0, sizeof p);
        p.idx = idx;
        p.val = val;
        p.d_count = d_count;
        p.seg_start = seg_start;
        p.capacity = capacity;
        p.n_segs = fasgd::push_segments(P);
        const hipError_t e = fasgd::launch_merge_list(theta_client, P, p, stream);
        if (e != hipSuccess) return hip_fail(e, "bfasgd_apply_fetch");
        return ok();
    }
    if (capacity > 0) {
        const hipError_t e = fasgd::launch_scatter(theta_client, P, idx, val, d_count, capacity, stream);
        if (e != hipSuccess) return hip_fail(e, "bfasgd_apply_fetch");
    }
    return ok();
}

size_t bfasgd_segments_workspace_bytes(int64_t P, int32_t S)
{
    if (P < 1 || S < 1) return 0;
    return fasgd::segments_workspace_bytes(P, S);
}

fasgd_status bfasgd_decide_segments(const fasgd_state* st, const int64_t* seg, int32_t S, float c, float eps_c,
                                    uint64_t seed, int64_t T, int32_t client, uint8_t* d_transmit,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream)
{
    if (!st) return fail(FASGD_ERR_NULL, "state is NULL");
    if (st->P < 1) return fail(FASGD_ERR_ARG, "P must be >= 1");
    if (st->lambda < 1) return fail(FASGD_ERR_ARG, "lambda = %d must be >= 1", st->lambda);
    if (!st->v || !d_transmit || !workspace) return fail(FASGD_ERR_NULL, "v, d_transmit or workspace is NULL");
    fasgd_status s = check_segments(seg, S, st->P);
    if (s != FASGD_OK) return s;
    if (!finite_nonneg(c) || !finite_nonneg(eps_c)) return fail(FASGD_ERR_ARG, "c and eps_c must be finite and >= 0");
    if (T < 0 || T > int64_t(UINT32_MAX)) return fail(FASGD_ERR_ARG, "T = %lld is not in [0, 2^32)", (long long)T);
    if (client < 0 || client >= st->lambda)
        return fail(FASGD_ERR_CLIENT, "client = %d is outside [0, %d)", client, st->lambda);
    if (!aligned(st->v, 4)) return fail(FASGD_ERR_ALIGN, "v is not 4-byte aligned");
    if (!aligned(workspace, 256)) return fail(FASGD_ERR_ALIGN, "workspace must be 256-byte aligned");
    if (st->index_base < 0 || (st->index_base & 3) != 0 || st->index_base > (int64_t(1) << 62) - st->P)
        return fail(FASGD_ERR_ARG, "index_base = %lld must be a multiple of 4 in [0, 2^62 - P]",
                    (long long)st->index_base);
    if (workspace_bytes < fasgd::segments_workspace_bytes(st->P, S))
        return fail(FASGD_ERR_CAPACITY, "workspace of %zu bytes is smaller than the %zu needed", workspace_bytes,
                    fasgd::segments_workspace_bytes(st->P, S));
    int64_t base = 0;
    for (int32_t g0 = 0; g0 < S; g0 += fasgd::kSegGroup) {
        const fasgd::SegGroup g = segment_group(seg, S, g0, base);
        const hipError_t e = fasgd::launch_seg_decide(g, st->v, static_cast<double*>(workspace), c, eps_c, seed,
                                                      static_cast<uint32_t>(T), static_cast<uint32_t>(client),
                                                      d_transmit, stream);
        if (e != hipSuccess) return hip_fail(e, "bfasgd_decide_segments");
    }
    return ok();
}

fasgd_status bfasgd_apply_segments(fasgd_state* st, const float* grad, const int64_t* seg, int32_t S,
                                   const uint8_t* d_transmit, int32_t client, int64_t grad_ts, hipStream_t stream)
{
    fasgd_status s = check_state(st, true);
    if (s != FASGD_OK) return s;
    if (!grad || !d_transmit) return fail(FASGD_ERR_NULL, "grad or d_transmit is NULL");
    if (!aligned(grad, 4)) return fail(FASGD_ERR_ALIGN, "grad is not 4-byte aligned");
    s = check_segments(seg, S, st->P);
    if (s != FASGD_OK) return s;
    float tau_div;
    s = staleness(st, &client, &grad_ts, 1, &tau_div);
    if (s != FASGD_OK) return s;
    fasgd::SegApplyArgs a;
    memset(&a, 0, sizeof a);
    a.theta = st->theta;
    a.n = st->n;
    a.b = st->b;
    a.v = st->v;
    a.last_T = st->last_T;
    a.grad = grad;
    a.transmit = d_transmit;
    a.coef = st->math_mode == FASGD_MATH_FAST ? st->alpha / tau_div : tau_div;
    a.last_T_value = static_cast<int32_t>(st->T);
    a.aligned = aligned(st->theta, 16) && aligned(st->n, 16) && aligned(st->b, 16) && aligned(st->v, 16) &&
                aligned(st->last_T, 16) && aligned(grad, 16);
    a.h = hyper_of(st);
    int64_t base = 0;
    for (int32_t g0 = 0; g0 < S; g0 += fasgd::kSegGroup) {
        const fasgd::SegGroup g = segment_group(seg, S, g0, base);
        const hipError_t e = fasgd::launch_seg_apply(g, a, variant_of(st), stream);
        if (e != hipSuccess) return hip_fail(e, "bfasgd_apply_segments");
    }
    st->T += 1;
    return ok();
}

const char* fasgd_status_string(fasgd_status s)
{
    switch (s) {
    case FASGD_OK: return "ok";
    case FASGD_ERR_NULL: return "null pointer";
    case FASGD_ERR_ARG: return "argument out of range";
    case FASGD_ERR_STALENESS: return "negative staleness (gradient timestamp after the update)";
    case FASGD_ERR_CLIENT: return "client id outside [0, lambda)";
    case FASGD_ERR_ALIGN: return "misaligned pointer";
    case FASGD_ERR_CAPACITY: return "workspace too small";
    case FASGD_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

const char* fasgd_last_error(void) { return g_err; }

fasgd_status fasgd_copy_anchor(const float* src, float* dst, int64_t n, hipStream_t stream)
{
    if (!src || !dst) return fail(FASGD_ERR_NULL, "src or dst is NULL");
    if (n < 1) return fail(FASGD_ERR_ARG, "n = %lld must be >= 1", (long long)n);
    if ((n + 3) / 4 + 1 > int64_t(0xffffffff) * 256)
        return fail(FASGD_ERR_ARG, "n = %lld is beyond one launch", (long long)n);
    if (!aligned(src, 16) || !aligned(dst, 16)) return fail(FASGD_ERR_ALIGN, "src and dst must be 16-byte aligned");
    const uintptr_t s = reinterpret_cast<uintptr_t>(src), d = reinterpret_cast<uintptr_t>(dst);
    const uintptr_t len = static_cast<uintptr_t>(n) * sizeof(float);
    if (s < d + len && d < s + len) return fail(FASGD_ERR_ARG, "src and dst overlap");
    const hipError_t e = fasgd::launch_copy_anchor(src, dst, n, stream);
    if (e != hipSuccess) return hip_fail(e, "fasgd_copy_anchor");
    return ok();
}

fasgd_status fasgd_check_ieee_sequences(float gamma, float beta, float eps, float alpha, uint64_t seed,
                                        int64_t n_updates, unsigned long long* d_mismatches, hipStream_t stream)
{
    if (!d_mismatches) return fail(FASGD_ERR_NULL, "d_mismatches is NULL");
    if (!aligned(d_mismatches, 8)) return fail(FASGD_ERR_ALIGN, "d_mismatches must be 8-byte aligned");
    if (!(gamma >= 0.0f && gamma <= 1.0f) || !(beta >= 0.0f && beta <= 1.0f))
        return fail(FASGD_ERR_ARG, "gamma and beta must be in [0, 1]");
    if (!ieee_short_ok(eps, alpha))
        return fail(FASGD_ERR_ARG,
                    "eps = %g and alpha = %g: the short sequences need eps >= 2^-96 (finite) and "
                    "2^-20 <= |alpha| < 2^20",
                    static_cast<double>(eps), static_cast<double>(alpha));
    if (n_updates < 0) return fail(FASGD_ERR_ARG, "n_updates = %lld must be >= 0", (long long)n_updates);
    fasgd::Hyper h;
    h.gamma = gamma;
    h.omg = 1.0f - gamma;
    h.beta = beta;
    h.omb = 1.0f - beta;
    h.eps = eps;
    h.alpha = alpha;
    h.rn_short = 1;
    const hipError_t e = fasgd::launch_check_ieee(h, seed, n_updates, d_mismatches, stream);
    if (e != hipSuccess) return hip_fail(e, "fasgd_check_ieee_sequences");
    return ok();
}

fasgd_status fasgd_record_next_pass(hipEvent_t start, hipEvent_t stop)
{
    if ((start == nullptr) != (stop == nullptr)) return fail(FASGD_ERR_NULL, "start and stop: both or neither");
    g_pass_start = start;
    g_pass_stop = stop;
    return ok();
}

}  // extern "C"
