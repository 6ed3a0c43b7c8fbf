"""Pins for the CPU oracle: it is checked against facts the paper and the
mathematics fix, never against itself or against the GPU path.

 * a hand-computed 8-parameter trace (tests/golden/hand_trace_8.txt);
 * plain SGD (torch.optim.SGD) for one client, SASGD with the rate alpha/tau,
   and FASGD with a frozen v = 1 (Sec. 1, 2.1, 2.2);
 * closed forms for a constant gradient (geometric series of the moving averages);
 * exact metamorphic relations (gradient scaling, rate scaling);
 * invariants: n - b^2 >= 0 and 0 < v <= 1/sqrt(eps);
 * elementwise independence (a subsample evolves as inside the full vector).
"""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import workload

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


# ---------------------------------------------------------------- hand trace
def _parse_trace(path):
    theta0, grads, fasgd, sasgd = None, {}, [], None
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            tok = line.split()
            if tok[0] == "theta0":
                theta0 = [Fraction(x) for x in tok[1:]]
            elif tok[0] == "grad":
                grads[int(tok[1])] = [Fraction(x) for x in tok[2:]]
            elif tok[0] == "fasgd":
                fasgd.append((int(tok[1]), int(tok[2]), *[Fraction(x) for x in tok[3:]]))
            elif tok[0] == "sasgd":
                sasgd = (int(tok[1]), [Fraction(x) for x in tok[2:]])
    return theta0, grads, fasgd, sasgd


def _close(a, fr, rel=1e-14, abs_=1e-15):
    return abs(a - float(fr)) <= rel * abs(float(fr)) + abs_


def test_hand_trace_fasgd(golden_dir):
    theta0, grads, fasgd, _ = _parse_trace(os.path.join(golden_dir, "hand_trace_8.txt"))
    st = oracle.init_state(np.array([float(x) for x in theta0], dtype=np.float32),
                           alpha=0.25, gamma=0.5, beta=0.5, eps=9 / 16, v0=0.0)
    expect = {}
    for (i, j, n, b, v, th) in fasgd:
        expect[(i, j)] = (n, b, v, th)
    assert len(expect) == 32
    for i in range(1, 5):
        g = np.array([float(x) for x in grads[i]], dtype=np.float32)
        oracle.fasgd_apply(st, g, grad_ts=0)          # tau = T - 0 = 0, 1, 2, 3
        for j in range(8):
            n, b, v, th = expect[(i, j)]
            assert _close(st.n[j], n), (i, j, "n", st.n[j], n)
            assert _close(st.b[j], b), (i, j, "b", st.b[j], b)
            assert _close(st.v[j], v), (i, j, "v", st.v[j], v)
            assert _close(st.theta[j], th), (i, j, "theta", st.theta[j], th)
    assert st.T == 4
    assert (st.last_T == 3).all()


def test_hand_trace_sasgd(golden_dir):
    theta0, grads, _, (U, final) = _parse_trace(os.path.join(golden_dir, "hand_trace_8.txt"))
    st = oracle.init_state(np.array([float(x) for x in theta0], dtype=np.float32), alpha=0.25)
    for i in range(1, U + 1):
        oracle.sasgd_apply(st, np.array([float(x) for x in grads[i]], dtype=np.float32), grad_ts=0)
    for j in range(8):
        assert _close(st.theta[j], final[j]), (j, st.theta[j], final[j])


# ------------------------------------------------------- reductions to SGD
def _torch_sgd(theta0, grads, lrs):
    """Plain SGD with torch.optim.SGD (fp64, CPU): one step per gradient."""
    p = torch.nn.Parameter(torch.from_numpy(theta0.astype(np.float64)))
    opt = torch.optim.SGD([p], lr=1.0)
    for g, lr in zip(grads, lrs):
        for group in opt.param_groups:
            group["lr"] = lr
        p.grad = torch.from_numpy(g.astype(np.float64))
        opt.step()
    return p.detach().numpy()


def _random_problem(P=257, U=12, seed=3):
    w = workload.WORKLOADS["tiny"]
    theta0, m, s = workload.host_params(w, P, seed=seed)
    grads = [workload.host_gradient(w, m, s, t, seed=seed) for t in range(U)]
    return theta0, grads


def test_sasgd_one_client_is_plain_sgd():
    """One client: every gradient has tau = 0, SASGD is SGD with rate alpha."""
    theta0, grads = _random_problem()
    alpha = oracle.f32(0.01)
    st = oracle.init_state(theta0, alpha=alpha)
    for t, g in enumerate(grads):
        oracle.sasgd_apply(st, g, grad_ts=t)
    ref = _torch_sgd(theta0, grads, [alpha] * len(grads))
    np.testing.assert_allclose(st.theta, ref, rtol=1e-14, atol=1e-17)


def test_sasgd_divides_by_step_staleness():
    """SASGD: the rate is alpha / tau (tau >= 1); torch SGD with that rate per step."""
    theta0, grads = _random_problem(U=10)
    alpha = oracle.f32(0.04)
    ts = [0, 0, 0, 1, 4, 2, 6, 7, 0, 9]
    st = oracle.init_state(theta0, alpha=alpha)
    lrs = []
    for t, (g, j) in enumerate(zip(grads, ts)):
        oracle.sasgd_apply(st, g, grad_ts=j)
        lrs.append(alpha / max(t - j, 1))
    ref = _torch_sgd(theta0, grads, lrs)
    np.testing.assert_allclose(st.theta, ref, rtol=1e-14, atol=1e-17)
    # tau = 2 at t = 2 must halve the step relative to tau = 1
    st1 = oracle.init_state(theta0, alpha=alpha)
    oracle.sasgd_apply(st1, np.zeros_like(grads[0]), 0)
    oracle.sasgd_apply(st1, np.zeros_like(grads[0]), 1)
    before = st1.theta.copy()
    oracle.sasgd_apply(st1, grads[0], 0)
    # (before - after cancels against |theta| ~ 0.2: allow one ulp of theta)
    np.testing.assert_allclose(before - st1.theta, alpha / 2 * grads[0].astype(np.float64),
                               rtol=1e-15, atol=1e-16)


@pytest.mark.parametrize("reading", [0, 1])
def test_fasgd_with_frozen_v_is_sasgd_and_sgd(reading):
    """beta = 1 and v0 = 1 keep v = 1 (in either reading of v), so FASGD's
    rate alpha/(v tau) is SASGD's alpha/tau; with one client (tau = 0) both
    are plain SGD."""
    theta0, grads = _random_problem()
    alpha = oracle.f32(0.005)
    a = oracle.init_state(theta0, alpha=alpha, beta=1.0, v0=1.0, v_reading=reading)
    for t, g in enumerate(grads):
        oracle.fasgd_apply(a, g, grad_ts=t)
    assert (a.v == 1.0).all()
    ref = _torch_sgd(theta0, grads, [alpha] * len(grads))
    np.testing.assert_allclose(a.theta, ref, rtol=1e-14, atol=1e-17)
    # staleness > 0: torch SGD with rate alpha / tau
    b = oracle.init_state(theta0, alpha=alpha, beta=1.0, v0=1.0, v_reading=reading)
    ts = [0, 0, 1, 0, 2, 5, 3, 7, 8, 1, 10, 4]
    lrs = []
    for t, (g, j) in enumerate(zip(grads, ts)):
        oracle.fasgd_apply(b, g, grad_ts=j)
        lrs.append(alpha / max(t - j, 1))
    np.testing.assert_allclose(b.theta, _torch_sgd(theta0, grads, lrs), rtol=1e-14, atol=1e-17)


# -------------------------------------------------------------- closed forms
@pytest.mark.parametrize("reading", [0, 1])
@pytest.mark.parametrize("gamma,beta,eps", [(0.95, 0.9, 1e-4), (0.5, 0.25, 1e-8), (0.0, 0.9, 1e-4)])
def test_constant_gradient_closed_form(gamma, beta, eps, reading):
    """For a constant gradient g from n0 = b0 = 0: n_i = (1 - gamma^i) g^2,
    b_i = (1 - gamma^i) g and n_i - b_i^2 = gamma^i (1 - gamma^i) g^2; v_i is
    the beta-weighted sum of 1/sqrt(that + eps) (reading 0, the equation for
    v) or of sqrt(that + eps) (reading 1, the standard deviation of the text);
    theta moves by alpha g/(v_i tau_i)."""
    gamma, beta, eps = oracle.f32(gamma), oracle.f32(beta), oracle.f32(eps)
    gs = np.array([0.3, -1.25, 2e-3, 7.0], dtype=np.float32)
    alpha = oracle.f32(0.01)
    st = oracle.init_state(np.zeros(4, np.float32), alpha=alpha, gamma=gamma, beta=beta, eps=eps,
                           v_reading=reading)
    g = gs.astype(np.float64)
    v_ref = np.zeros(4)
    theta_ref = np.zeros(4)
    for i in range(1, 41):
        tau = (i * 7) % 5                    # staleness 2, 4, 1, 3, 0, ...
        oracle.fasgd_apply(st, gs, grad_ts=st.T - min(tau, st.T))
        tau = min(tau, i - 1)
        w = 1.0 - gamma ** i
        np.testing.assert_allclose(st.n, w * g * g, rtol=1e-13)
        np.testing.assert_allclose(st.b, w * g, rtol=1e-13)
        d = gamma ** i * w * g * g
        s_ref = np.sqrt(d + eps) if reading else 1.0 / np.sqrt(d + eps)
        v_ref = beta * v_ref + (1 - beta) * s_ref
        theta_ref = theta_ref - alpha * g / (v_ref * max(tau, 1))
        # n - b^2 is a cancellation: its fp64 error is a few ulp of n, which
        # is large relative to n - b^2 + eps when eps and gamma^i are tiny.
        cond = 1e-12 + 8 * 2.0 ** -52 * st.n / (d + eps)
        assert (np.abs(st.v - v_ref) <= cond * v_ref).all(), (i, st.v, v_ref)
        np.testing.assert_allclose(st.theta, theta_ref, rtol=i * cond.max(), atol=1e-18)


def test_prose_v_gamma0_closed_form():
    """Reading 1 with gamma = 0 and a constant gradient: n = g^2 and b = g
    after every update, so n - b^2 = 0 and v_i = (1 - beta^i) sqrt(eps)
    exactly as a geometric sum; theta_I = theta_0 - sum_i alpha g / v_i."""
    beta, eps, alpha = oracle.f32(0.75), oracle.f32(1e-4), oracle.f32(0.02)
    gs = np.array([0.5, -2.0, 1e-3, 3.0, 0.0], dtype=np.float32)
    st = oracle.init_state(np.zeros(5, np.float32), alpha=alpha, gamma=0.0, beta=beta, eps=eps, v_reading=1)
    theta_ref = np.zeros(5)
    for i in range(1, 31):
        oracle.fasgd_apply(st, gs, grad_ts=st.T)          # tau = 0: divisor 1
        v_i = (1.0 - beta ** i) * np.sqrt(eps)
        np.testing.assert_allclose(st.v, np.full(5, v_i), rtol=1e-14)
        theta_ref = theta_ref - alpha * gs.astype(np.float64) / v_i
        np.testing.assert_allclose(st.theta, theta_ref, rtol=1e-13, atol=1e-300)


def test_readings_reciprocal_at_beta0():
    """With beta = 0 each reading's v is its own term: 1/sqrt(n - b^2 + eps)
    for the equation and sqrt(n - b^2 + eps) for the text, so after every
    update the two states' v multiply to 1, and n, b (which v does not feed)
    agree exactly."""
    theta0, grads = _random_problem()
    a = oracle.init_state(theta0, alpha=0.01, beta=0.0, v_reading=0)
    b = oracle.init_state(theta0, alpha=0.01, beta=0.0, v_reading=1)
    for t, g in enumerate(grads):
        oracle.fasgd_apply(a, g, grad_ts=max(t - 2, 0))
        oracle.fasgd_apply(b, g, grad_ts=max(t - 2, 0))
        np.testing.assert_array_equal(a.n, b.n)
        np.testing.assert_array_equal(a.b, b.b)
        np.testing.assert_allclose(a.v * b.v, 1.0, rtol=4e-16)


def test_v_reading_rejected_unless_0_or_1():
    with pytest.raises(oracle.OracleError):
        oracle.init_state(np.zeros(3, np.float32), alpha=0.01, v_reading=2)


# ------------------------------------------------------ metamorphic relations
def test_gradient_scaling_is_exact():
    """Scaling every gradient by 2^k and eps by 4^k scales n - b^2 + eps by 4^k,
    v by 2^-k and therefore every step alpha g/(v tau) by 4^k -- exactly, since
    powers of two commute with IEEE rounding.  A misplaced eps, a wrong power or
    a transposed operand breaks this."""
    _, grads = _random_problem(P=64, U=9, seed=5)
    theta0 = np.zeros(64, np.float32)        # theta then holds minus the summed steps
    ts = [0, 0, 1, 1, 2, 0, 5, 3, 7]
    for k in (1, -3):
        a = oracle.init_state(theta0, alpha=0.01, gamma=0.75, beta=0.5, eps=2.0 ** -10)
        b = oracle.init_state(theta0, alpha=0.01, gamma=0.75, beta=0.5, eps=2.0 ** -10 * 4.0 ** k)
        for g, j in zip(grads, ts):
            oracle.fasgd_apply(a, g, j)
            oracle.fasgd_apply(b, (g * np.float32(2.0 ** k)).astype(np.float32), j)
        np.testing.assert_array_equal(b.n, a.n * 4.0 ** k)
        np.testing.assert_array_equal(b.b, a.b * 2.0 ** k)
        np.testing.assert_array_equal(b.v, a.v * 2.0 ** -k)
        np.testing.assert_array_equal(b.theta, a.theta * 4.0 ** k)


def test_rate_scaling_is_exact():
    """The statistics do not depend on alpha and each step is linear in it."""
    theta0, grads = _random_problem(P=64, U=6, seed=6)
    a = oracle.init_state(np.zeros_like(theta0), alpha=0.01)
    b = oracle.init_state(np.zeros_like(theta0), alpha=0.04)
    for t, g in enumerate(grads):
        oracle.fasgd_apply(a, g, max(t - 2, 0))
        oracle.fasgd_apply(b, g, max(t - 2, 0))
    np.testing.assert_array_equal(a.v, b.v)
    np.testing.assert_allclose(b.theta, 4.0 * a.theta, rtol=1e-14)


# ---------------------------------------------------------------- invariants
def test_variance_nonnegative_and_v_bounded():
    """n_i - b_i^2 >= 0 (the weights of the moving averages sum to at most 1,
    so by Cauchy-Schwarz b^2 <= n), and v, an average of values in
    (0, 1/sqrt(eps)], stays in (0, 1/sqrt(eps)]."""
    rng = np.random.default_rng(11)
    P = 2000
    eps = oracle.f32(1e-4)
    st = oracle.init_state(np.zeros(P, np.float32), alpha=0.01, eps=eps)
    for t in range(60):
        g = (rng.standard_normal(P) * rng.choice([1e-4, 1e-2, 1.0, 30.0], P)
             + rng.choice([0.0, 5.0], P)).astype(np.float32)
        oracle.fasgd_apply(st, g, t)
        d = st.n - st.b * st.b
        assert (d >= -1e-14 * st.n).all()
        assert (st.v > 0).all() and (st.v <= 1 / np.sqrt(eps) * (1 + 1e-12)).all()


def test_negative_staleness_rejected():
    st = oracle.init_state(np.zeros(3, np.float32), alpha=0.01)
    with pytest.raises(oracle.OracleError):
        oracle.fasgd_apply(st, np.ones(3, np.float32), grad_ts=1)   # T = 0 < 1
    with pytest.raises(oracle.OracleError):
        oracle.sasgd_apply(st, np.ones(3, np.float32), grad_ts=-1)
    assert st.T == 0 and (st.theta == 0).all() and (st.n == 0).all()


def test_subsample_evolves_like_full_vector():
    """Every rule is elementwise, so a gathered subsample run alone matches
    the same indices of the full run bit for bit (used for sampled parity at
    sizes the oracle cannot run in full)."""
    w = workload.WORKLOADS["tiny"]
    theta0, m, s = workload.host_params(w, 5000)
    clients, ts = workload.schedule(w, 20)
    full = oracle.init_state(theta0, alpha=0.01)
    js = np.array([0, 1, 17, 999, 2500, 4998, 4999])
    sub = full.take(js)
    for t in range(20):
        g = workload.host_gradient(w, m, s, t)
        oracle.fasgd_apply(full, g, ts[t])
        oracle.fasgd_apply(sub, g[js], ts[t])
    for name in ("theta", "n", "b", "v", "last_T"):
        np.testing.assert_array_equal(getattr(full, name)[js], getattr(sub, name))


def test_oracle_resume_is_exact():
    """The oracle's state is the whole state: a run split at T0 (state copied
    and the copy continued) ends where the unsplit run ends, and the
    selection after it is the same (draws are keyed by T)."""
    w = workload.WORKLOADS["tiny"]
    P = 1000
    theta0, m_, s_ = workload.host_params(w, P)
    clients, ts = workload.schedule(w, 40)
    grads = [workload.host_gradient(w, m_, s_, t) for t in range(40)]
    whole = oracle.init_state(theta0, alpha=0.01)
    for t in range(40):
        oracle.fasgd_apply(whole, grads[t], ts[t])
    first = oracle.init_state(theta0, alpha=0.01)
    for t in range(17):
        oracle.fasgd_apply(first, grads[t], ts[t])
    resumed = first.take(np.arange(P))
    for t in range(17, 40):
        oracle.fasgd_apply(resumed, grads[t], ts[t])
    for name in ("theta", "n", "b", "v", "last_T"):
        np.testing.assert_array_equal(getattr(resumed, name), getattr(whole, name), err_msg=name)
    assert resumed.T == whole.T == 40
    sel_a = oracle.bfasgd_select(whole.v.astype(np.float32), grads[0], 5.0, 1e-8, 3, whole.T, 1)
    sel_b = oracle.bfasgd_select(resumed.v.astype(np.float32), grads[0], 5.0, 1e-8, 3, resumed.T, 1)
    assert sel_a[2] == sel_b[2] and np.array_equal(sel_a[0], sel_b[0])
