/*
 * CPU oracle for the FASGD parameter-server update, its SASGD baseline mode and
 * the per-parameter B-FASGD send/skip selection with sparse apply.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The product path never
 * links, imports or calls it, and it shares no code with the GPU kernels.
 *
 * Plain, slow, single-threaded, fp64 (the paper fixes no precision).  Inputs
 * that the GPU path receives as fp32 (gradients, hyper-parameters, the B-FASGD
 * threshold inputs) are received here as the same fp32 values, widened exactly.
 *
 * Notation follows "Faster Asynchronous SGD" (Odena, arXiv:1601.04033):
 *   T      server timestamp, starts at 0, +1 per weight update    (Sec. 2.1)
 *   tau    step-staleness i - j of a gradient with timestamp j    (Sec. 2.1)
 *   n, b   moving averages of the squared gradient and gradient   (Sec. 2.2, eqs. for n_i, b_i)
 *   v      moving average of 1/sqrt(n - b^2 + eps)                (Sec. 2.2, eq. for v_i)
 *          or, in the prose reading (reading = 1), of sqrt(n - b^2 + eps), the
 *          moving average of the standard deviation the text of Sec. 2.2 describes
 *   step   alpha / (v * tau) * grad, theta <- theta - step         (Sec. 2.2, FASGD update rule)
 *
 * Readings where the paper is silent (each listed in the design notes):
 *   - tau = 0 (a fresh gradient) divides by 1, i.e. by max(tau, 1);
 *   - n - b^2 is clamped at 0 before eps is added (it is >= 0 in exact
 *     arithmetic; the clamp only guards rounding);
 *   - within one update the order is n, b, then v, then the step with the new v;
 *   - B-FASGD decides per parameter with that parameter's v (the paper's
 *     per-tensor/per-parameter direction, Sec. 5), and an untransmitted
 *     parameter is left untouched; a sparse apply still advances T by one.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>

/* ------------------------------------------------------------------------- */
/* Philox4x32-10, written from Salmon, Moraes, Dror & Shaw, "Parallel Random  */
/* Numbers: As Easy as 1, 2, 3" (SC'11): ten rounds of the 4x32 Philox        */
/* network; each round multiplies words 0 and 2 by the two round constants,  */
/* xors the high halves with the other two words and the round key, and the  */
/* key advances by the two Weyl constants between rounds.                    */
/* ------------------------------------------------------------------------- */
static const uint32_t PHILOX_M0 = 0xD2511F53u;
static const uint32_t PHILOX_M1 = 0xCD9E8D57u;
static const uint32_t PHILOX_W0 = 0x9E3779B9u;
static const uint32_t PHILOX_W1 = 0xBB67AE85u;

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += PHILOX_W0;
            k1 += PHILOX_W1;
        }
        uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)x0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)x2;
        uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
        uint32_t y1 = (uint32_t)p1;
        uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
        uint32_t y3 = (uint32_t)p0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* ------------------------------------------------------------------------- */
/* One parameter of one FASGD weight update (Sec. 2.2).                       */
/* ------------------------------------------------------------------------- */
static void fasgd_update_one(double *theta, double *n, double *b, double *v, double g,
                             double alpha, double gamma, double beta, double eps,
                             double tau_div, int reading)
{
    /* n_i = gamma n_{i-1} + (1 - gamma) (grad)^2, elementwise */
    *n = gamma * (*n) + (1.0 - gamma) * g * g;
    /* b_i = gamma b_{i-1} + (1 - gamma) grad */
    *b = gamma * (*b) + (1.0 - gamma) * g;
    /* v_i = beta v_{i-1} + (1 - beta) / sqrt(n_i - b_i^2 + eps) */
    double var = *n - (*b) * (*b);
    if (var < 0.0)
        var = 0.0;
    if (reading == 0)
        *v = beta * (*v) + (1.0 - beta) / sqrt(var + eps);
    else /* v averages the standard deviation sqrt(n_i - b_i^2 + eps) */
        *v = beta * (*v) + (1.0 - beta) * sqrt(var + eps);
    /* g_i = alpha / (v_i tau) * grad ;  theta_{i+1} = theta_i - g_i */
    double step = alpha / ((*v) * tau_div) * g;
    *theta = *theta - step;
}

/* tau = T - grad_ts must be >= 0 (Sec. 2.1); returns the divisor max(tau, 1). */
static int staleness_divisor(int64_t T, int64_t grad_ts, double *tau_div)
{
    if (grad_ts > T || grad_ts < 0)
        return -1;
    int64_t tau = T - grad_ts;
    *tau_div = tau > 0 ? (double)tau : 1.0;
    return 0;
}

/*
 * FASGD server apply-update for one client gradient (the lock serialises
 * arrivals, so several gradients are several calls in arrival order).
 * theta, n, b, v: fp64 [P]; last_T: int64 [P] or NULL; *T is advanced by one.
 * reading: 0 = v as in the equation for v_i, 1 = v as the text describes it.
 * Returns 0, or -1 if grad_ts is not in [0, *T] (negative staleness).
 */
int oracle_fasgd_apply(int64_t P, double *theta, double *n, double *b, double *v,
                       int64_t *last_T, int64_t *T, const float *grad, int64_t grad_ts,
                       double alpha, double gamma, double beta, double eps, int reading)
{
    double tau_div;
    if (staleness_divisor(*T, grad_ts, &tau_div) != 0)
        return -1;
    for (int64_t j = 0; j < P; ++j) {
        fasgd_update_one(&theta[j], &n[j], &b[j], &v[j], (double)grad[j],
                         alpha, gamma, beta, eps, tau_div, reading);
        if (last_T)
            last_T[j] = *T;
    }
    *T += 1;
    return 0;
}

/*
 * SASGD (staleness-aware ASGD, Sec. 1 and Sec. 2.1): the step-staleness
 * dependent rate alpha(tau) = alpha / tau, theta <- theta - alpha(tau) grad.
 */
int oracle_sasgd_apply(int64_t P, double *theta, int64_t *last_T, int64_t *T,
                       const float *grad, int64_t grad_ts, double alpha)
{
    double tau_div;
    if (staleness_divisor(*T, grad_ts, &tau_div) != 0)
        return -1;
    double rate = alpha / tau_div;
    for (int64_t j = 0; j < P; ++j) {
        theta[j] = theta[j] - rate * (double)grad[j];
        if (last_T)
            last_T[j] = *T;
    }
    *T += 1;
    return 0;
}

/* ------------------------------------------------------------------------- */
/* B-FASGD transmit rule (Sec. 2.3): transmit iff r < 1 / (1 + c / (v + eps)) */
/* with r uniform in [0, 1).  Decided in fp32 from the fp32 v:                 */
/*   t = v + eps and u = t + c are fp32 sums; since t > 0 the rule is          */
/*   r * u < t, and the product of two fp32 values is exact in fp64, so the    */
/*   comparison below takes no further rounding.                               */
/* r is the top 24 bits of Philox word (j mod 4) of the counter                */
/*   (j / 4 low, j / 4 high, T, client) under key (seed low, seed high).       */
/* ------------------------------------------------------------------------- */
int oracle_bfasgd_transmit(int64_t j, float v_j, float c, float eps_c, uint64_t seed,
                           int64_t T, int32_t client)
{
    uint64_t q = (uint64_t)j >> 2;
    uint32_t ctr[4] = {(uint32_t)q, (uint32_t)(q >> 32), (uint32_t)T, (uint32_t)client};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t w[4];
    oracle_philox4x32_10(ctr, key, w);
    float r = (float)(w[j & 3] >> 8) * 0x1p-24f;
    float t = v_j + eps_c;
    float u = t + c;
    return (double)r * (double)u < (double)t;
}

/* Decisions for a list of global indices js[0..ns) with their v values. */
void oracle_bfasgd_decide(int64_t ns, const int64_t *js, const float *v_at, float c,
                          float eps_c, uint64_t seed, int64_t T, int32_t client,
                          uint8_t *out)
{
    for (int64_t i = 0; i < ns; ++i)
        out[i] = (uint8_t)oracle_bfasgd_transmit(js[i], v_at[i], c, eps_c, seed, T, client);
}

/*
 * Select and compact one client's gradient: every transmitted index in
 * ascending order with its gradient value.  Writes at most `capacity` entries
 * and returns the number transmitted (which may exceed capacity).  The arrays
 * may be a slice of a larger parameter vector that starts at global index
 * index_base: decisions are keyed by the global index index_base + j, while
 * the listed indices are the slice's own j.
 */
int64_t oracle_bfasgd_select(int64_t P, const float *v, const float *grad, float c,
                             float eps_c, uint64_t seed, int64_t T, int32_t client,
                             int32_t *idx, float *val, int64_t capacity, int64_t index_base)
{
    int64_t m = 0;
    for (int64_t j = 0; j < P; ++j) {
        if (oracle_bfasgd_transmit(index_base + j, v[j], c, eps_c, seed, T, client)) {
            if (m < capacity) {
                idx[m] = (int32_t)j;
                val[m] = grad[j];
            }
            ++m;
        }
    }
    return m;
}

/*
 * Server side of a B-FASGD push: the FASGD update of Sec. 2.2 on the listed
 * parameters only, with the transmitted values as the gradient; every other
 * parameter keeps theta, n, b, v and last_T.  *T advances by one even for an
 * empty list (the push is one server update event).
 */
int oracle_bfasgd_apply_sparse(double *theta, double *n, double *b, double *v, int64_t *last_T,
                               int64_t *T, const int32_t *idx, const float *val, int64_t m,
                               int64_t grad_ts, double alpha, double gamma, double beta,
                               double eps, int reading)
{
    double tau_div;
    if (staleness_divisor(*T, grad_ts, &tau_div) != 0)
        return -1;
    for (int64_t i = 0; i < m; ++i) {
        int64_t j = idx[i];
        fasgd_update_one(&theta[j], &n[j], &b[j], &v[j], (double)val[i],
                         alpha, gamma, beta, eps, tau_div, reading);
        if (last_T)
            last_T[j] = *T;
    }
    *T += 1;
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Synchronous SGD server (the apply-update listing of Sec. 3): once all      */
/* lambda clients have pushed, every gradient is applied in client order as   */
/* p <- p - lr * (g / lambda); the timestamp then advances by one.            */
/* ------------------------------------------------------------------------- */
void oracle_sync_sgd_apply(int64_t P, double *theta, int64_t *last_T, int64_t *T,
                           const float *const *grads, int32_t lambda, double lr)
{
    for (int32_t k = 0; k < lambda; ++k) {
        for (int64_t j = 0; j < P; ++j) {
            double mod = (double)grads[k][j] / (double)lambda;
            theta[j] = theta[j] - lr * mod;
        }
    }
    if (last_T)
        for (int64_t j = 0; j < P; ++j)
            last_T[j] = *T;
    *T += 1;
}

/*
 * Dropped pushes re-apply the client's most recent gradient (Sec. 2.3),
 * per parameter: cache holds, for one client, the last value it transmitted
 * for each parameter (0 before the first).  The transmitted (index, value)
 * pairs overwrite the cache, and the whole cache is then applied as one
 * FASGD gradient (Sec. 2.2).
 */
int oracle_bfasgd_apply_cached(int64_t P, double *theta, double *n, double *b, double *v,
                               int64_t *last_T, int64_t *T, float *cache, const int32_t *idx,
                               const float *val, int64_t m, int64_t grad_ts, double alpha,
                               double gamma, double beta, double eps, int reading)
{
    for (int64_t i = 0; i < m; ++i)
        cache[idx[i]] = val[i];
    return oracle_fasgd_apply(P, theta, n, b, v, last_T, T, cache, grad_ts, alpha, gamma, beta, eps,
                              reading);
}

/* ------------------------------------------------------------------------- */
/* B-FASGD as the paper states it (Sec. 2.3): one decision per push or fetch  */
/* opportunity, from v averaged over all the parameters; per tensor (Sec. 5), */
/* one decision per segment [seg[s], seg[s+1]) from that segment's mean.      */
/* Decided in fp64: t = mean + eps, u = t + c, transmit iff r * u < t, with r */
/* the top 24 bits of word 0 of Philox4x32-10 at counter                      */
/* (s low, 0x80000000 | s high, T, client) (the set top bit keeps these draws */
/* apart from the per-parameter ones, whose second word is j / 2^34 = 0).     */
/* ------------------------------------------------------------------------- */
void oracle_bfasgd_decide_segments(int64_t S, const int64_t *seg, const float *v, float c,
                                   float eps_c, uint64_t seed, int64_t T, int32_t client,
                                   uint8_t *transmit, double *mean_out)
{
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    for (int64_t s = 0; s < S; ++s) {
        double sum = 0.0;
        for (int64_t j = seg[s]; j < seg[s + 1]; ++j)
            sum += (double)v[j];
        double mean = sum / (double)(seg[s + 1] - seg[s]);
        uint32_t ctr[4] = {(uint32_t)s, 0x80000000u | (uint32_t)((uint64_t)s >> 32), (uint32_t)T,
                           (uint32_t)client};
        uint32_t w[4];
        oracle_philox4x32_10(ctr, key, w);
        double r = (double)(w[0] >> 8) * 0x1p-24;
        double t = mean + (double)eps_c;
        double u = t + (double)c;
        transmit[s] = (uint8_t)(fma(r, u, -t) < 0.0);
        if (mean_out)
            mean_out[s] = mean;
    }
}

/*
 * Server side of a push decided per segment: the FASGD update (Sec. 2.2) on
 * the transmitted segments, nothing elsewhere; T advances by one.
 */
int oracle_bfasgd_apply_segments(int64_t S, const int64_t *seg, const uint8_t *transmit,
                                 double *theta, double *n, double *b, double *v, int64_t *last_T,
                                 int64_t *T, const float *grad, int64_t grad_ts, double alpha,
                                 double gamma, double beta, double eps, int reading)
{
    double tau_div;
    if (staleness_divisor(*T, grad_ts, &tau_div) != 0)
        return -1;
    for (int64_t s = 0; s < S; ++s) {
        if (!transmit[s])
            continue;
        for (int64_t j = seg[s]; j < seg[s + 1]; ++j) {
            fasgd_update_one(&theta[j], &n[j], &b[j], &v[j], (double)grad[j],
                             alpha, gamma, beta, eps, tau_div, reading);
            if (last_T)
                last_T[j] = *T;
        }
    }
    *T += 1;
    return 0;
}
