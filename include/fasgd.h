/*
 * fasgd.h -- C ABI of libfasgd.so, the parameter-server hot path of
 * "Faster Asynchronous SGD" (A. Odena, arXiv:1601.04033) on one AMD
 * Instinct MI355X (gfx950).
 *
 * Notation (Sec. 2.1): lambda clients, mu minibatch size, alpha master
 * learning rate, T server timestamp (starts at 0, +1 per weight update),
 * tau = T - j the step-staleness of a gradient computed on parameters with
 * timestamp j.
 *
 * Conventions shared by every entry point
 *   - Device memory is owned by the caller (allocated e.g. with torch); the
 *     library allocates nothing and keeps no pointer beyond a call (the two
 *     event handles of fasgd_record_next_pass aside, held until used).
 *   - Every call is asynchronous on `stream` (0 = the null stream) and never
 *     synchronises the host.  Results are visible after the stream is
 *     synchronised.
 *   - All arguments are checked on the host before anything is enqueued.
 *     On any error nothing is enqueued and the state (including T) is
 *     unchanged; fasgd_last_error() then describes the problem.
 *   - Device arrays are plain, densely packed 1-D arrays of P elements in
 *     parameter order (structure of arrays).  4-byte alignment is required.
 *     The kernels take one parameter per thread up to P = 2^32 - 256;
 *     beyond that every array must be 16-byte aligned (as torch
 *     allocations are: the kernels then take 4 parameters per thread),
 *     otherwise the call returns FASGD_ERR_ALIGN.
 *   - Calls that share a state must be issued on one stream (or otherwise
 *     ordered by the caller); concurrent calls on one state race.
 */
#ifndef FASGD_H
#define FASGD_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FASGD_MAX_K 64          /* most gradients one fused apply accepts */
#define FASGD_MAX_BATCH 64      /* most pushes one batched selection or apply accepts */

typedef enum fasgd_status {
    FASGD_OK = 0,
    FASGD_ERR_NULL = 1,         /* a required pointer is NULL */
    FASGD_ERR_ARG = 2,          /* a size, count, timestamp or hyper-parameter is out of range */
    FASGD_ERR_STALENESS = 3,    /* a gradient timestamp is later than the update it is applied at */
    FASGD_ERR_CLIENT = 4,       /* a client id is outside [0, lambda) */
    FASGD_ERR_ALIGN = 5,        /* a device pointer is not 4-byte aligned */
    FASGD_ERR_CAPACITY = 6,     /* the B-FASGD workspace is smaller than bfasgd_workspace_bytes(P) */
    FASGD_ERR_HIP = 7           /* the HIP runtime refused a launch */
} fasgd_status;

typedef enum fasgd_math {
    FASGD_MATH_IEEE = 0,        /* correctly rounded fp32 sqrt and divisions */
    FASGD_MATH_FAST = 1         /* hardware (reciprocal) square root and reciprocal (about 1 ulp each) */
} fasgd_math;

/*
 * Which moving average v keeps (Sec. 2.2).  The equation for v averages
 * 1/sqrt(n - b^2 + eps); the text around it describes a moving average of
 * the standard deviation.  The rate is alpha / (v tau) in both.
 */
typedef enum fasgd_v_reading {
    FASGD_V_EQUATIONS = 0,      /* v <- beta v + (1 - beta) / sqrt(n - b^2 + eps)   (default) */
    FASGD_V_PROSE = 1           /* v <- beta v + (1 - beta) * sqrt(n - b^2 + eps) */
} fasgd_v_reading;

/*
 * Server state (Sec. 2.2).  A host-side POD owned by the caller; the device
 * arrays it points to are owned by the caller too.
 *   theta   parameters theta, fp32 [P]
 *   n       moving average of the squared gradient, fp32 [P]
 *   b       moving average of the gradient, fp32 [P]
 *   v       moving average of 1/sqrt(n - b^2 + eps) (or, with
 *           v_reading = FASGD_V_PROSE, of sqrt(n - b^2 + eps)), fp32 [P]
 *   last_T  timestamp of the last sparse (B-FASGD) update of each
 *           parameter, int32 [P], -1 before the first
 * Per-parameter staleness bookkeeping: a dense apply updates every
 * parameter, so it records its timestamp once in dense_T instead of
 * writing P copies of it; the last update that touched parameter j is
 * max(last_T[j], dense_T) (-1: never updated).  A value of last_T[j] at or
 * below dense_T carries no information.
 * index_base: a state may hold the slice [index_base, index_base + P) of a
 * larger parameter vector (one shard of a server split by index range).  The
 * updates are elementwise and ignore it; B-FASGD decisions draw their random
 * word from the global index index_base + j, so they do not depend on how the
 * vector is split.  fasgd_init_state sets 0.
 * Hyper-parameters: alpha (Sec. 2.1), gamma, beta, eps (Sec. 2.2).
 * lambda bounds the client ids; mu is recorded only (a gradient arrives as
 * the minibatch mean, Sec. 2.2).  T and dense_T are advanced by the apply
 * calls.
 */
typedef struct fasgd_state {
    int64_t P;
    int32_t lambda;
    int32_t mu;
    float alpha;
    float gamma;
    float beta;
    float eps;
    int32_t math_mode;          /* fasgd_math */
    int32_t v_reading;          /* fasgd_v_reading; fasgd_init_state sets FASGD_V_EQUATIONS */
    int64_t T;
    int64_t dense_T;            /* timestamp of the last dense update, -1 before the first */
    float* theta;
    float* n;
    float* b;
    float* v;
    int32_t* last_T;
    int64_t index_base;         /* global index of parameter 0 (a multiple of 4); 0 unless this
                                   state is one slice of a larger vector */
} fasgd_state;

/*
 * Initialise a server (the FRED Server initialisation function, Sec. 3):
 * fills n, b and v with n0, b0, v0 and last_T with -1 on `stream`, sets
 * T = 0 (Sec. 2.1) and dense_T = -1, and records the hyper-parameters in
 * *st.  theta must already hold the initial parameters; it is not written.
 * Requires P >= 1, lambda >= 1, mu >= 1, alpha > 0, gamma and beta in
 * [0, 1], eps > 0 (finite), math_mode a fasgd_math value.  v_reading is set
 * to FASGD_V_EQUATIONS; a caller may set it to FASGD_V_PROSE before the
 * first update (the apply calls reject other values with FASGD_ERR_ARG).
 * n, b, v may be NULL for a state used only with sasgd_apply_updates.
 */
fasgd_status fasgd_init_state(fasgd_state* st, int64_t P, int32_t lambda, int32_t mu,
                              float alpha, float gamma, float beta, float eps, int32_t math_mode,
                              float n0, float b0, float v0,
                              float* theta, float* n, float* b, float* v, int32_t* last_T,
                              hipStream_t stream);

/*
 * FASGD apply-update for K client gradients in arrival order (Sec. 2.2):
 * the k-th gradient is applied at server timestamp T + k with staleness
 * tau_k = T + k - grad_ts[k], and for every parameter
 *   n <- gamma n + (1 - gamma) g^2,   b <- gamma b + (1 - gamma) g,
 *   v <- beta v + (1 - beta) / sqrt(max(n - b^2, 0) + eps),
 *   theta <- theta - alpha / (v max(tau_k, 1)) g,
 * one gradient after the other (the server lock serialises arrivals,
 * Sec. 2.1), with each parameter's state held in registers across the K
 * gradients.  dense_T becomes T + K - 1 and T advances by K; last_T is not
 * touched.
 *   grads    host array of K device pointers, each fp32 [P]
 *   clients  host int32 [K], each in [0, lambda)
 *   grad_ts  host int64 [K], 0 <= grad_ts[k] <= T + k
 *   K        1 .. FASGD_MAX_K
 * Errors: FASGD_ERR_STALENESS if some grad_ts[k] > T + k; FASGD_ERR_ARG if
 * K is out of range or T + K - 1 exceeds INT32_MAX (timestamps are kept
 * within the int32 range of last_T).
 */
fasgd_status fasgd_apply_updates(fasgd_state* st, const float* const* grads, const int32_t* clients,
                                 const int64_t* grad_ts, int32_t K, hipStream_t stream);

/*
 * SASGD apply-update (staleness-aware ASGD, Sec. 1 and 2.1): the rate of
 * the k-th gradient is alpha / max(tau_k, 1), theta <- theta - that * g.
 * Reads and writes theta only (n, b, v may be NULL) and sets dense_T as
 * fasgd_apply_updates does.  Same arguments, order and errors.
 */
fasgd_status sasgd_apply_updates(fasgd_state* st, const float* const* grads, const int32_t* clients,
                                 const int64_t* grad_ts, int32_t K, hipStream_t stream);

/* Bytes of device workspace bfasgd_select_compact needs for P parameters. */
size_t bfasgd_workspace_bytes(int64_t P);

/*
 * B-FASGD push selection and compaction (Sec. 2.3, decided per parameter,
 * the per-parameter direction of Sec. 5).  Parameter j of this push is
 * transmitted iff r_j < 1 / (1 + c / (v_j + eps_c)), decided in fp32 as
 *   t = v_j + eps_c,  u = t + c,  transmit <=> r_j * u - t < 0 (one rounding),
 * where r_j is the top 24 bits of word (J mod 4) of Philox4x32-10 at counter
 * (J/4 low 32 bits, J/4 high 32 bits, T, client) with key (seed low, seed
 * high), scaled by 2^-24 into [0, 1), and J = st->index_base + j is the
 * global index (index_base must be a multiple of 4, >= 0, with
 * index_base + P <= 2^62; otherwise FASGD_ERR_ARG).  v is read from the
 * state as it is before this push is applied.
 * The transmitted entries are written in ascending index order:
 * out_idx[i] = j (int32, the state's own index), out_val[i] = grad[j] (bit copy), for the first
 * min(m, capacity) of them; *d_count (device int64) receives m, the number
 * transmitted, even when m > capacity.  capacity >= P never truncates.
 *   grad       device fp32 [P], this client's gradient
 *   out_seg_start  optional (NULL: not written) device uint32
 *              [bfasgd_list_index_length(P)], the list's index: entry s is the
 *              list position of the first transmitted index >= 256 s (counted
 *              before the capacity cut), the last entry is m.  It lets a
 *              consumer find the entries of any 256-parameter segment at once
 *              (fasgd_apply_with_push).
 *   c, eps_c   finite, >= 0
 *   T          server timestamp this push is applied at, 0 <= T < 2^32
 *   client     in [0, lambda)
 *   workspace  device scratch of at least bfasgd_workspace_bytes(P) bytes,
 *              256-byte aligned; its contents need no initialisation
 * Requires P <= INT32_MAX (int32 indices).  The selection is deterministic:
 * it does not depend on launch shape, timing or earlier calls.
 */
fasgd_status bfasgd_select_compact(const fasgd_state* st, const float* grad, float c, float eps_c,
                                   uint64_t seed, int64_t T, int32_t client,
                                   int32_t* out_idx, float* out_val, int64_t capacity,
                                   int64_t* d_count, uint32_t* out_seg_start,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * bfasgd_select_compact without a workspace argument, for callers that
 * cannot allocate device memory: code under HIP graph capture, serving
 * loops that must not call hipMalloc, harnesses that forbid it.  The
 * selection's scratch (ballot words, tile counts and offsets, group totals)
 * lives in a fixed device array built into the library, one per GPU, of
 * FASGD_NOALLOC_SCRATCH_BYTES bytes, which stays allocated until the process
 * ends.  Its device address is looked up once per device on the first call
 * made with that device current.  The call allocates nothing (no hipMalloc,
 * no library allocation) and needs no initialisation of the array: the
 * kernels clear what must start at zero.
 * Arguments, results and errors as bfasgd_select_compact (same lists,
 * counts and list index, bit for bit), plus FASGD_ERR_CAPACITY when P
 * exceeds FASGD_NOALLOC_MAX_P (nothing is enqueued).
 * Every call on a GPU uses that GPU's one array: calls that overlap on one
 * GPU (on different streams, or from different threads, without ordering)
 * race and may produce wrong lists.  Issue them on one stream, or order them.
 */
#define FASGD_NOALLOC_MAX_P 67108864LL            /* 2^26 parameters */
#define FASGD_NOALLOC_SCRATCH_BYTES 8945920ULL    /* bfasgd_workspace_bytes(FASGD_NOALLOC_MAX_P) */
fasgd_status bfasgd_select_compact_noalloc(const fasgd_state* st, const float* grad, float c, float eps_c,
                                           uint64_t seed, int64_t T, int32_t client,
                                           int32_t* out_idx, float* out_val, int64_t capacity,
                                           int64_t* d_count, uint32_t* out_seg_start, hipStream_t stream);

/* Entries of the list index bfasgd_select_compact writes for P parameters:
 * ceil(P / 256) + 1 (0 for P < 1). */
int64_t bfasgd_list_index_length(int64_t P);

/*
 * B pushes selected in one set of launches (Sec. 2.3): push b is exactly
 * bfasgd_select_compact(st, grads[b], c, eps_c, seed, T[b], clients[b],
 * out_idx + b capacity, out_val + b capacity, capacity, d_count + b,
 * out_seg_start + b L, workspace slice b), with L =
 * bfasgd_list_index_length(P): every push is decided from v as the state
 * holds it at this call (the v its client last fetched, before any of the B
 * pushes is applied).  For pushes that arrive at the server together, where
 * one selection per push would be bound by launch latency.
 *   B              1 .. FASGD_MAX_BATCH
 *   grads          host array of B device pointers, each fp32 [P]
 *   T, clients     host arrays [B]; each as for bfasgd_select_compact
 *   out_idx, out_val  device [B][capacity]
 *   d_count        device int64 [B]
 *   out_seg_start  NULL, or device uint32 [B][L]
 *   workspace      at least B * bfasgd_workspace_bytes(P) bytes, 256-byte aligned
 * Errors: those of bfasgd_select_compact for any push, FASGD_ERR_ARG for B
 * out of range; a rejected call enqueues nothing.
 */
fasgd_status bfasgd_select_compact_batch(const fasgd_state* st, int32_t B, const float* const* grads, float c,
                                         float eps_c, uint64_t seed, const int64_t* T, const int32_t* clients,
                                         int32_t* out_idx, float* out_val, int64_t capacity,
                                         int64_t* d_count, uint32_t* out_seg_start,
                                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Server side of a B-FASGD push: the FASGD update of fasgd_apply_updates,
 * applied at timestamp T with staleness T - grad_ts, to the listed
 * parameters only, with g = val[i] for parameter idx[i], for
 * i < min(*d_count, capacity) (*d_count is read on the device, so this can
 * follow bfasgd_select_compact on the same stream without a host
 * round-trip).  Unlisted parameters keep theta, n, b, v and last_T; listed
 * ones get last_T = T.  T advances by one even when the list is empty.
 * Indices must be distinct; an index outside [0, P) is skipped.  Each
 * entry is one gather and one scatter of the listed parameter's state.  A
 * list that comes with its index (bfasgd_select_compact's out_seg_start)
 * can instead be applied segment by segment by fasgd_apply_pushes with
 * B = 1, with the same result: faster above a few percent transmitted
 * (1e9 parameters, 10 %: 7.2 against 9.4 ms), slower below (1.8 %: 4.9
 * against 3.6 ms).
 *   idx, val  device int32 / fp32 [capacity]
 *   d_count   device int64 [1]
 * Errors: as fasgd_apply_updates with K = 1.
 */
fasgd_status bfasgd_apply_sparse(fasgd_state* st, const int32_t* idx, const float* val,
                                 const int64_t* d_count, int64_t capacity, int32_t client,
                                 int64_t grad_ts, hipStream_t stream);

/*
 * One pass that applies a compacted B-FASGD push and then K client gradients
 * (Sec. 2.2, 2.3): the push at timestamp T (staleness T - push_grad_ts) to
 * its listed parameters, exactly as bfasgd_apply_sparse, then the K
 * gradients at T + 1 ... T + K, exactly as fasgd_apply_updates; each
 * parameter's state stays in registers across all K + 1 updates.  theta,
 * n, b and v are bit-identical to those two calls in that order (the order
 * in which the server lock serialises a push that arrived ahead of K dense
 * gradients), but the state is read and written once.  T advances by
 * K + 1 and dense_T becomes T + K.  last_T is not written: every
 * parameter's last update is the dense one at T + K, so the last update
 * max(last_T[j], dense_T) of every parameter is the same as after the two
 * calls, without the push's scattered timestamp writes.
 *   push_idx, push_val, push_count, capacity  the push list, as for
 *                      bfasgd_apply_sparse (indices ascending and distinct,
 *                      as bfasgd_select_compact writes them)
 *   push_seg_start     its index, as bfasgd_select_compact's out_seg_start
 *   push_client, push_grad_ts  as for bfasgd_apply_sparse
 *   grads, clients, grad_ts, K as for fasgd_apply_updates (K >= 1)
 * Errors: those of the two calls it stands for (FASGD_ERR_NULL also for a
 * NULL push_count or push_seg_start).
 */
fasgd_status fasgd_apply_with_push(fasgd_state* st, const int32_t* push_idx, const float* push_val,
                                   const int64_t* push_count, const uint32_t* push_seg_start,
                                   int64_t capacity, int32_t push_client, int64_t push_grad_ts,
                                   const float* const* grads, const int32_t* clients,
                                   const int64_t* grad_ts, int32_t K, hipStream_t stream);

/*
 * The server step of a pipeline: fasgd_apply_with_push (a queued push, then
 * K gradients, in one pass), then the selection of the next push exactly as
 * bfasgd_select_compact(st, next_grad, c, eps_c, seed, T', next_client,
 * out_idx, out_val, out_capacity, out_count, out_seg_start, workspace,
 * workspace_bytes) with T' = the timestamp after the pass (the one the next
 * pass applies that push at) and v as the pass leaves it.  Every output
 * (theta, n, b, v, T, dense_T, the list, its count and its index) is
 * bit-identical to those two calls; when the state and the K gradients are
 * 16-byte aligned the pass itself takes the next push's transmit decisions
 * from the v it holds in registers, so the selection does not read v again.
 * The output list may be the buffers of the push being applied (the pass
 * reads them before the selection writes).
 *   push_*, grads, clients, grad_ts, K  as for fasgd_apply_with_push
 *   next_grad, next_client, c, eps_c, seed, out_*, workspace  as for
 *                  bfasgd_select_compact
 * Errors: those of the two calls it stands for; a rejected call enqueues
 * nothing and leaves T alone.
 */
fasgd_status fasgd_apply_with_push_and_select(fasgd_state* st, const int32_t* push_idx, const float* push_val,
                                              const int64_t* push_count, const uint32_t* push_seg_start,
                                              int64_t push_capacity, int32_t push_client, int64_t push_grad_ts,
                                              const float* const* grads, const int32_t* clients,
                                              const int64_t* grad_ts, int32_t K, const float* next_grad,
                                              int32_t next_client, float c, float eps_c, uint64_t seed,
                                              int32_t* out_idx, float* out_val, int64_t out_capacity,
                                              int64_t* out_count, uint32_t* out_seg_start, void* workspace,
                                              size_t workspace_bytes, hipStream_t stream);

/*
 * B compacted pushes applied in one pass (Sec. 2.3): the same state, T and
 * last_T, bit for bit, as B calls of bfasgd_apply_sparse in order b = 0 ..
 * B-1, push b at timestamp T + b with staleness T + b - grad_ts[b], but
 * each parameter's state is read and written once.  A parameter listed by
 * some push gets last_T = T + the last such b; T advances by B; dense_T is
 * unchanged.  With B = 1 this is bfasgd_apply_sparse applied segment by
 * segment through the list's index: a segment the push lists nothing of is
 * skipped, one with 8 or more entries is read and rewritten whole, one
 * with fewer touches its listed parameters only.
 *   idx, val       device int32 / fp32 [B][capacity]; list b as
 *                  bfasgd_select_compact writes it (ascending, distinct)
 *   d_count        device int64 [B]
 *   seg_start      device uint32 [B][bfasgd_list_index_length(P)], each
 *                  list's index as bfasgd_select_compact writes it
 *   clients, grad_ts  host arrays [B], as for bfasgd_apply_sparse
 * Errors: those of the B calls it stands for; FASGD_ERR_ARG for B outside
 * 1 .. FASGD_MAX_BATCH or T + B - 1 beyond INT32_MAX; FASGD_ERR_NULL for a
 * NULL d_count or seg_start.
 */
fasgd_status fasgd_apply_pushes(fasgd_state* st, int32_t B, const int32_t* idx, const float* val,
                                const int64_t* d_count, const uint32_t* seg_start, int64_t capacity,
                                const int32_t* clients, const int64_t* grad_ts, hipStream_t stream);

/*
 * Synchronous SGD server (Sec. 3, the apply-update listing): with the
 * gradients of all lambda clients collected, apply each one, in client
 * order 0 .. lambda-1, as theta <- theta - lr * (g / lambda) (the division
 * and the step are separate fp32 operations); then dense_T = T and T
 * advances by one, since the weights changed once.  Reads and writes theta
 * only (n, b, v may be NULL).
 *   grads  host array of lambda device pointers, each fp32 [P]
 *   lr     finite, > 0
 */
fasgd_status sgd_sync_apply(fasgd_state* st, const float* const* grads, float lr, hipStream_t stream);

/*
 * B-FASGD push with its dropped values re-applied: the server re-applies
 * the client's most recent gradient (Sec. 2.3), kept per parameter.
 * cache is this client's gradient cache, fp32 [P] (device, owned by the
 * caller, zero before the client's first push).  The first
 * min(*d_count, capacity) listed pairs are written into it
 * (cache[idx[i]] = val[i]); then the whole cache is applied as one FASGD
 * gradient at timestamp T with staleness T - grad_ts.  dense_T = T, T += 1.
 * Indices outside [0, P) are skipped.
 *   seg_start  optional (NULL: not used) device uint32, the list's index as
 *              bfasgd_select_compact writes it.  With it (and, beyond
 *              2^32 - 256 parameters, the state and the cache 16-byte
 *              aligned), the list is merged into the cache inside the one
 *              pass that applies it (the same state and cache bit for bit,
 *              without a separate scattered copy).
 * Errors: as bfasgd_apply_sparse, and FASGD_ERR_NULL for a NULL cache.
 */
fasgd_status bfasgd_apply_cached(fasgd_state* st, const int32_t* idx, const float* val,
                                 const int64_t* d_count, const uint32_t* seg_start, int64_t capacity,
                                 float* cache, int32_t client, int64_t grad_ts, hipStream_t stream);

/*
 * Fetch side of B-FASGD (Sec. 2.3): a client refreshes its copy of theta
 * only where the transmit rule, with the fetch threshold, says so.  Select
 * with bfasgd_select_compact, passing the server's theta as the values (and
 * a seed that keeps fetch draws apart from push draws); this call then
 * copies the listed values into the client's copy:
 * theta_client[idx[i]] = val[i] for i < min(*d_count, capacity).  Indices
 * outside [0, P) are skipped.  No state is changed.
 *   theta_client  device fp32 [P]
 *   seg_start     optional (NULL: not used) device uint32, the list's index
 *                 as bfasgd_select_compact writes it.  With it (and
 *                 theta_client 16-byte aligned) every 256-parameter segment
 *                 holding an entry is read and rewritten whole instead of
 *                 one partial sector per entry: faster when most segments
 *                 hold an entry (above a few percent transmitted) and the
 *                 copy does not fit the 256 MB Infinity Cache (1e9
 *                 parameters at 10 %: 1.5 against 2.0 ms), slower otherwise
 *                 (1e9 at 1 %: 0.73 against 0.43 ms).  The result is the same.
 */
fasgd_status bfasgd_apply_fetch(float* theta_client, int64_t P, const int32_t* idx, const float* val,
                                const int64_t* d_count, const uint32_t* seg_start, int64_t capacity,
                                hipStream_t stream);

/*
 * B-FASGD decision as the paper states it (Sec. 2.3): one decision per push
 * (or fetch) opportunity, from v averaged over all parameters; or, per
 * tensor (Sec. 5), one decision per segment s = [seg[s], seg[s+1]) from that
 * segment's mean of v.  In fp64: mean_s = (sum of v over s) / its length,
 * t = mean_s + eps_c, u = t + c, transmit <=> r_s * u - t < 0 (one rounding),
 * where r_s is the top 24 bits of word 0 of Philox4x32-10 at counter
 * (s low 32 bits, 0x80000000 | s high bits, T, client) with key (seed low,
 * seed high), scaled by 2^-24 (the set top bit keeps these draws apart
 * from the per-parameter ones).  d_transmit[s] receives 1 or 0.
 *   seg        host int64 [S+1], 0 = seg[0] < seg[1] < ... < seg[S] = P
 *   S          >= 1 (1 = the whole parameter vector)
 *   d_transmit device uint8 [S]
 *   workspace  device scratch of bfasgd_segments_workspace_bytes(P, S)
 *              bytes, 256-byte aligned, contents irrelevant
 * The sums are fp64 in a fixed order, so the result is the same run to run.
 * Other arguments and errors as bfasgd_select_compact.
 */
size_t bfasgd_segments_workspace_bytes(int64_t P, int32_t S);
fasgd_status bfasgd_decide_segments(const fasgd_state* st, const int64_t* seg, int32_t S, float c, float eps_c,
                                    uint64_t seed, int64_t T, int32_t client, uint8_t* d_transmit,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Server side of a push decided per segment: the FASGD update of
 * fasgd_apply_updates, at timestamp T with staleness T - grad_ts, on the
 * segments with d_transmit[s] = 1 (their parameters get last_T = T) and
 * nothing on the others (Sec. 2.3 drops the push there); T advances by one.
 *   grad  device fp32 [P];  seg, S as bfasgd_decide_segments
 */
fasgd_status bfasgd_apply_segments(fasgd_state* st, const float* grad, const int64_t* seg, int32_t S,
                                   const uint8_t* d_transmit, int32_t client, int64_t grad_ts,
                                   hipStream_t stream);

/* Static text naming a status code. */
const char* fasgd_status_string(fasgd_status s);

/* Text describing the last error returned on the calling thread ("" if none). */
const char* fasgd_last_error(void);

/*
 * Diagnostics: the next FASGD pass kernel this thread launches (through
 * fasgd_apply_updates, fasgd_apply_with_push or
 * fasgd_apply_with_push_and_select) records `start` on its stream just
 * before the pass and `stop` just after it, so that the pass can be timed
 * alone within a call that launches more kernels.  One-shot: the events are
 * forgotten once recorded; a call rejected before its pass leaves the
 * request pending.  Both NULL clears a pending request; one NULL is
 * FASGD_ERR_NULL.  The events are the caller's (created, and destroyed only
 * after they are recorded or cleared).
 */
fasgd_status fasgd_record_next_pass(hipEvent_t start, hipEvent_t stop);

/*
 * Diagnostics: the bandwidth anchor, dst[0, n) = src[0, n) by a plain
 * streaming copy (one 16-byte vector per thread over an exact-cover grid,
 * non-temporal loads and stores, the access pattern of the passes above).
 * Its rate, 8 n bytes over its time, is what the machine's HBM sustains for one
 * read and one write stream, against which the passes' rates can be read.
 *   src, dst  device fp32 [n], 16-byte aligned, not overlapping
 * FASGD_ERR_NULL, FASGD_ERR_ALIGN, or FASGD_ERR_ARG for n < 1 or overlap.
 */
fasgd_status fasgd_copy_anchor(const float* src, float* dst, int64_t n, hipStream_t stream);

/*
 * Diagnostics: checks on the device that the IEEE mode's short sequences
 * give the correctly rounded results of the general ones, bit for bit.  In
 * IEEE mode every update computes sqrt(x) (x = max(n - b^2, 0) + eps),
 * 1 / sqrt(x) as two correctly rounded operations, and alpha / (v tau)
 * (Sec. 2.2's equations for v and the rate).  When eps >= 2^-96 (finite) and
 * 2^-20 <= |alpha| < 2^20 the kernels take shorter sequences (a hardware
 * estimate, then corrections by exact fma residuals); this call compares them
 * with the general sequences:
 *   d_mismatches[0]  sqrt over every float x >= 2^-96 (+inf and NaNs too);
 *   d_mismatches[1]  1 / sqrt(x) over the same x;
 *   d_mismatches[2]  alpha / d over all 2^32 bit patterns of d;
 *   d_mismatches[3]  n_updates whole updates in both readings of v, on
 *                    pseudo-random states drawn from `seed` (zeros,
 *                    subnormals, infinities and NaNs among them), with
 *                    gamma, beta, eps and alpha.
 * NaN results count as equal to NaN results.  d_mismatches: device, 4
 * counters (8-byte aligned), cleared by the call, read after the stream is
 * synchronised; all four are 0 when the sequences hold.  FASGD_ERR_ARG when
 * eps or alpha lie outside the range above (the kernels use the general
 * sequences there), gamma or beta outside [0, 1] or n_updates < 0;
 * FASGD_ERR_NULL / FASGD_ERR_ALIGN for d_mismatches.  Takes about 10 ms of
 * GPU time plus the updates.
 */
fasgd_status fasgd_check_ieee_sequences(float gamma, float beta, float eps, float alpha, uint64_t seed,
                                        int64_t n_updates, unsigned long long* d_mismatches, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* FASGD_H */
