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
