"""Pins for the oracle's synchronous-SGD server (Sec. 3 listing) and for
B-FASGD's dropped-push handling (Sec. 2.3: re-apply the client's most
recent gradient)."""
import numpy as np
import torch

import oracle
import workload


def _problem(P=513, lam=8, seed=4):
    w = workload.WORKLOADS["mlp"]
    theta0, m, s = workload.host_params(w, P, seed=seed)
    grads = [workload.host_gradient(w, m, s, t, seed=seed) for t in range(lam)]
    return theta0, grads


def test_sync_step_is_sgd_on_the_mean_gradient():
    """The listing applies lr * (g_k / lambda) for every client k, i.e. one SGD
    step with the mean of the lambda minibatch gradients (torch.optim.SGD)."""
    theta0, grads = _problem()
    lr = oracle.f32(0.04)
    st = oracle.init_state(theta0, alpha=0.01)
    oracle.sync_sgd_apply(st, grads, lr)
    p = torch.nn.Parameter(torch.from_numpy(theta0.astype(np.float64)))
    opt = torch.optim.SGD([p], lr=lr)
    p.grad = torch.from_numpy(np.mean([g.astype(np.float64) for g in grads], axis=0))
    opt.step()
    np.testing.assert_allclose(st.theta, p.detach().numpy(), rtol=1e-14, atol=1e-16)
    assert st.T == 1 and (st.last_T == 0).all()


def test_sync_step_identical_gradients_and_one_client():
    """lambda copies of one gradient move theta by exactly lr * g (power-of-two
    lambda makes g / lambda exact); lambda = 1 is plain SGD."""
    theta0, grads = _problem(lam=1)
    g = grads[0]
    for lam in (1, 4, 16):
        st = oracle.init_state(theta0, alpha=0.01)
        oracle.sync_sgd_apply(st, [g] * lam, 0.5)
        np.testing.assert_allclose(st.theta, theta0.astype(np.float64) - 0.5 * g.astype(np.float64),
                                   rtol=1e-15, atol=1e-17)


def test_sync_steps_advance_T_once_each():
    theta0, grads = _problem(lam=4)
    st = oracle.init_state(theta0, alpha=0.01)
    for _ in range(3):
        oracle.sync_sgd_apply(st, grads, 0.01)
    assert st.T == 3 and (st.last_T == 2).all()


def test_cached_push_with_everything_transmitted_is_dense_fasgd():
    theta0, grads = _problem(lam=6)
    a = oracle.init_state(theta0, alpha=0.005)
    b = oracle.init_state(theta0, alpha=0.005)
    cache = np.zeros_like(theta0)
    for t, g in enumerate(grads):
        oracle.fasgd_apply(a, g, max(t - 1, 0))
        oracle.bfasgd_apply_cached(b, cache, np.arange(g.size, dtype=np.int32), g, max(t - 1, 0))
        np.testing.assert_array_equal(cache, g)
    for name in ("theta", "n", "b", "v", "last_T"):
        np.testing.assert_array_equal(getattr(a, name), getattr(b, name))


def test_dropped_push_reapplies_the_most_recent_gradient():
    """An empty push applies the client's previous gradient again; a partial
    push applies new values where sent and the previous ones elsewhere."""
    theta0, grads = _problem(lam=3)
    g0, g1 = grads[0], grads[1]
    P = g0.size
    a = oracle.init_state(theta0, alpha=0.005)
    b = oracle.init_state(theta0, alpha=0.005)
    cache = np.zeros_like(theta0)
    all_idx = np.arange(P, dtype=np.int32)
    oracle.bfasgd_apply_cached(b, cache, all_idx, g0, 0)
    oracle.fasgd_apply(a, g0, 0)
    oracle.bfasgd_apply_cached(b, cache, np.zeros(0, np.int32), np.zeros(0, np.float32), 1)
    oracle.fasgd_apply(a, g0, 1)                      # dropped: g0 again
    sel = np.flatnonzero(np.arange(P) % 3 == 1).astype(np.int32)
    mixed = g0.copy()
    mixed[sel] = g1[sel]
    oracle.bfasgd_apply_cached(b, cache, sel, g1[sel], 2)
    oracle.fasgd_apply(a, mixed, 2)
    np.testing.assert_array_equal(cache, mixed)
    for name in ("theta", "n", "b", "v", "last_T"):
        np.testing.assert_array_equal(getattr(a, name), getattr(b, name))
    assert b.T == 3


# ------------------------------------------------ paper-literal mean-v decision
from fractions import Fraction  # noqa: E402


def _seg_r(s, seed, T, client):
    w = oracle.philox4x32_10([s & 0xFFFFFFFF, 0x80000000 | (s >> 32), T & 0xFFFFFFFF, client],
                             [seed & 0xFFFFFFFF, seed >> 32])[0]
    return Fraction(int(w) >> 8, 1 << 24)


def test_segment_decision_matches_exact_rule_with_exact_mean():
    """r < 1/(1 + c/(mean + eps)) with the mean of the fp32 v values taken
    exactly: the fp64 decision agrees outside a 2^-40 relative margin."""
    rng = np.random.default_rng(21)
    P = 3000
    v = np.exp(rng.uniform(np.log(1e-3), np.log(1e3), P)).astype(np.float32)
    seg = np.unique(np.concatenate([[0, P], rng.integers(1, P, 40)])).astype(np.int64)
    near = 0
    for T, client, c in [(0, 0, 1.0), (7, 3, 30.0), (123456, 11, 0.01), (2 ** 32 - 1, 5, 400.0)]:
        dec, mean = oracle.bfasgd_decide_segments(v, seg, c, 1e-8, 0xABCDEF, T, client)
        for s in range(seg.size - 1):
            lo, hi = seg[s], seg[s + 1]
            exact_mean = sum(Fraction(float(x)) for x in v[lo:hi]) / (hi - lo)
            assert abs(Fraction(mean[s]) - exact_mean) <= exact_mean * Fraction(1, 2 ** 44)
            t = exact_mean + Fraction(float(np.float32(1e-8)))
            p = t / (t + Fraction(float(np.float32(c))))
            r = _seg_r(s, 0xABCDEF, T, client)
            if abs(r - p) <= p * Fraction(1, 2 ** 40):
                near += 1
                continue
            assert dec[s] == (r < p), (T, s)
    assert near == 0


def test_segment_decision_constant_v_limits_and_independence():
    P = 4096
    seg = np.array([0, 1, 100, 4000, 4096], np.int64)
    v = np.full(P, 2.5, np.float32)
    dec, mean = oracle.bfasgd_decide_segments(v, seg, 1.0, 0.0, 9, 4, 1)
    assert (mean == 2.5).all()
    assert oracle.bfasgd_decide_segments(v, seg, 0.0, 1e-8, 9, 4, 1)[0].all()          # c = 0
    assert oracle.bfasgd_decide_segments(np.full(P, 1e30, np.float32), seg, 5.0, 1e-8, 9, 4, 1)[0].all()
    assert not oracle.bfasgd_decide_segments(np.zeros(P, np.float32), seg, 5.0, 1e-30, 9, 4, 1)[0].any()
    # a segment's decision depends on its own v only
    v2 = v.copy()
    v2[100:4000] = 1e-6
    d2, _ = oracle.bfasgd_decide_segments(v2, seg, 1.0, 0.0, 9, 4, 1)
    assert d2[0] == dec[0] and d2[1] == dec[1] and d2[3] == dec[3]


def test_segment_decision_rate():
    """Over many opportunities (timestamps) the transmit frequency is
    1/(1 + c/(mean + eps)) (binomial z-test)."""
    P = 64
    v = np.full(P, 3.0, np.float32)
    seg = np.array([0, P], np.int64)
    c = 7.0
    hits = sum(bool(oracle.bfasgd_decide_segments(v, seg, c, 0.0, 77, T, 2)[0][0]) for T in range(20000))
    p = 3.0 / (3.0 + c)
    z = (hits - 20000 * p) / np.sqrt(20000 * p * (1 - p))
    assert abs(z) < 5, (hits, z)


def test_apply_segments_all_and_none():
    theta0, grads = _problem(P=700, lam=3)
    seg = np.array([0, 10, 300, 700], np.int64)
    a = oracle.init_state(theta0, alpha=0.005)
    b = oracle.init_state(theta0, alpha=0.005)
    oracle.fasgd_apply(a, grads[0], 0)
    oracle.bfasgd_apply_segments(b, grads[0], seg, np.ones(3, bool), 0)
    for name in ("theta", "n", "b", "v", "last_T"):
        np.testing.assert_array_equal(getattr(a, name), getattr(b, name))
    before = b.copy()
    oracle.bfasgd_apply_segments(b, grads[1], seg, np.array([False, True, False]), 1)
    for name in ("theta", "n", "b", "v", "last_T"):
        np.testing.assert_array_equal(getattr(b, name)[:10], getattr(before, name)[:10])
        np.testing.assert_array_equal(getattr(b, name)[300:], getattr(before, name)[300:])
    assert (b.last_T[10:300] == 1).all() and b.T == 2
