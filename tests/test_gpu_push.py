"""GPU checks of a B-FASGD push applied inside the next dense pass
(fasgd_apply_with_push): the list index that bfasgd_select_compact writes,
bit-identity of theta, n, b, v with the two separate calls it stands for
(bfasgd_apply_sparse, then fasgd_apply_updates) and the same last update of
every parameter, and parity with the oracle applying the push and then the
K gradients one by one.  The same pass followed by the next push's selection
(fasgd_apply_with_push_and_select, whose pass takes the transmit decisions
itself) against fasgd_apply_with_push and then bfasgd_select_compact."""
import numpy as np
import pytest

import oracle
import paper_1601_04033_amd as fa
import workload
from helpers import RTOL_SEQ, assert_state_close, gpu, new_gpu_state, to_dev

pytestmark = pytest.mark.gpu
SEED = 0x9E1EC7


def _select(st, g, c, T, client, dev, cap=None):
    import torch
    P = st.P
    cap = P if cap is None else cap
    idx = torch.full((max(cap, 1),), -1, device=dev, dtype=torch.int32)[:cap]
    val = torch.zeros(max(cap, 1), device=dev)[:cap]
    cnt = torch.zeros(1, device=dev, dtype=torch.int64)
    seg = torch.full((fa.bfasgd_list_index_length(P),), -1, device=dev, dtype=torch.int32)
    fa.bfasgd_select_compact(st, g, c, 1e-8, SEED, T, client, idx, val, cnt, fa.allocate_workspace(P, dev),
                             seg_start=seg)
    return idx, val, cnt, seg


def _states(P, dev, mode, reading, seed, offset=0):
    """Two identical mid-run GPU states (the same synthetic n, b, v, theta,
    T = 5) and the oracle state holding the same values; offset = 1 places the
    arrays 4 bytes into their buffers (the scalar path)."""
    import torch
    w = workload.WORKLOADS["mlp_bfasgd" if P <= workload.MLP_P else "large"]
    theta0, m_, s_ = workload.host_params(w, P, seed=seed)
    b0 = m_ + s_ * np.float32(0.1)
    n0 = (b0 * b0 + s_ * s_).astype(np.float32)
    v0 = workload.synthetic_v(P, seed=seed, lo=5.0, hi=100.0)
    out = []
    for _ in range(2):
        bufs = fa.allocate_state(P + offset, dev)
        theta, n, b, v, last_T = (t[offset:] for t in bufs)
        st = fa.fasgd_init_state(theta, n, b, v, last_T, lam=w.lam, alpha=w.alpha_fasgd, math_mode=mode,
                                 v_reading=reading)
        for t, a in ((theta, theta0), (n, n0), (b, b0), (v, v0)):
            t.copy_(torch.from_numpy(a))
        st.c.T = 5
        out.append((st, bufs))
    ref = oracle.init_state(theta0, alpha=w.alpha_fasgd, v_reading=reading)
    ref.n, ref.b, ref.v = n0.astype(np.float64), b0.astype(np.float64), v0.astype(np.float64)
    ref.T = 5
    return out[0][0], out[1][0], ref, (m_, s_, w), (out[0][1], out[1][1])


def _assert_same(a, b):
    """theta, n, b, v bit for bit; the same T, dense_T and last update of
    every parameter (the fused pass leaves last_T alone: the dense updates
    after the push supersede it)."""
    import torch
    torch.cuda.synchronize()
    for name in ("theta", "n", "b", "v"):
        assert torch.equal(a.tensors[name], b.tensors[name]), name
    assert a.T == b.T and a.dense_T == b.dense_T
    assert torch.equal(a.last_update(), b.last_update())


@pytest.mark.parametrize("P", [1, 255, 257, 100_003, 1_000_003])
def test_list_index_points_at_each_segment(P):
    """seg_start[s] is the position of the first listed index >= 256 s and
    the last entry is the count, at fractions from nothing to everything."""
    import torch
    dev = gpu()
    v = workload.synthetic_v(P, seed=P % 97)
    st = new_gpu_state(np.zeros(P, np.float32), dev, 16, 0.005, fa.MATH_FAST)
    st.v.copy_(torch.from_numpy(v))
    g = torch.randn(P, device=dev)
    for c in (0.0, 40.0, 3e38):
        idx, val, cnt, seg = _select(st, g, c, 11, 2, dev)
        torch.cuda.synchronize()
        m = int(cnt.item())
        lst = idx[:m].cpu().numpy().astype(np.int64)
        want = np.searchsorted(lst, 256 * np.arange(fa.bfasgd_list_index_length(P) - 1))
        got = seg.cpu().numpy().astype(np.int64)
        np.testing.assert_array_equal(got[:-1], want)
        assert got[-1] == m


@pytest.mark.parametrize("reading", [fa.V_EQUATIONS, fa.V_PROSE])
@pytest.mark.parametrize("mode", [fa.MATH_FAST, fa.MATH_IEEE])
@pytest.mark.parametrize("P,K,offset", [(100_003, 8, 0), (1_000_003, 33, 0), (65_537, 1, 1), (1027, 64, 0)])
def test_push_inside_pass_is_bit_identical(P, K, offset, mode, reading):
    """A push at about 30 % followed by K gradients: one fused pass gives the
    state, last_T, T and dense_T of the two separate calls bit for bit
    (vector path with a ragged tail, and the scalar path for arrays 4 bytes
    off 16-byte alignment)."""
    dev = gpu()
    a, b, _, (m_, s_, w), keep = _states(P, dev, mode, reading, seed=P % 1000, offset=offset)
    g_push = to_dev(workload.host_gradient(w, m_, s_, 5, seed=3), dev)
    gs = [to_dev(workload.host_gradient(w, m_, s_, 6 + k, seed=3), dev) for k in range(K)]
    clients, ts = list(range(K)), [max(6 + k - 3, 0) for k in range(K)]
    idx, val, cnt, seg = _select(a, g_push, 100.0, 5, 1, dev)
    fa.bfasgd_apply_sparse(a, idx, val, cnt, 1, 4)
    fa.fasgd_apply_updates(a, gs, [c % w.lam for c in clients], ts)
    fa.fasgd_apply_with_push(b, idx, val, cnt, seg, 1, 4, gs, [c % w.lam for c in clients], ts)
    _assert_same(a, b)
    assert b.T == 5 + K + 1 and b.dense_T == 5 + K


@pytest.mark.parametrize("case", ["truncated", "empty", "all"])
def test_push_inside_pass_edge_lists(case):
    """A list cut by capacity, an empty push and a push of every parameter."""
    import torch
    dev = gpu()
    P, K = 200_003, 4
    a, b, _, (m_, s_, w), keep = _states(P, dev, fa.MATH_FAST, fa.V_EQUATIONS, seed=7)
    g_push = to_dev(workload.host_gradient(w, m_, s_, 5, seed=7), dev)
    gs = [to_dev(workload.host_gradient(w, m_, s_, 6 + k, seed=7), dev) for k in range(K)]
    c = {"truncated": 100.0, "empty": 3e38, "all": 0.0}[case]
    cap = 12_345 if case == "truncated" else None
    idx, val, cnt, seg = _select(a, g_push, c, 5, 1, dev, cap=cap)
    torch.cuda.synchronize()
    m = int(cnt.item())
    if case == "truncated":
        assert m > 12_345
    elif case == "all":
        assert m == P
    fa.bfasgd_apply_sparse(a, idx, val, cnt, 1, 5)
    fa.fasgd_apply_updates(a, gs, [0, 1, 2, 3], [6, 5, 4, 3])
    fa.fasgd_apply_with_push(b, idx, val, cnt, seg, 1, 5, gs, [0, 1, 2, 3], [6, 5, 4, 3])
    _assert_same(a, b)


def test_push_inside_pass_matches_oracle():
    """Against the oracle: the same list applied as a sparse push at T = 5,
    then 16 gradients one by one."""
    import torch
    dev = gpu()
    P, K = 300_007, 16
    _, st, ref, (m_, s_, w), keep = _states(P, dev, fa.MATH_FAST, fa.V_EQUATIONS, seed=12)
    g_push = workload.host_gradient(w, m_, s_, 5, seed=12)
    gs = [workload.host_gradient(w, m_, s_, 6 + k, seed=12) for k in range(K)]
    ts = [max(6 + k - 5, 0) for k in range(K)]
    clients = [k % w.lam for k in range(K)]
    idx, val, cnt, seg = _select(st, to_dev(g_push, dev), 100.0, 5, 3, dev)
    fa.fasgd_apply_with_push(st, idx, val, cnt, seg, 3, 2, [to_dev(g, dev) for g in gs], clients, ts)
    r_idx, r_val, r_m = oracle.bfasgd_select(ref.v.astype(np.float32), g_push, 100.0, 1e-8, SEED, 5, 3)
    oracle.bfasgd_apply_sparse(ref, r_idx, r_val, 2)
    for g, t in zip(gs, ts):
        oracle.fasgd_apply(ref, g, t)
    torch.cuda.synchronize()
    assert int(cnt.item()) == r_m
    assert_state_close(st, ref, RTOL_SEQ, what="push then 16 gradients")
    assert (st.last_T.cpu() == -1).all() and st.dense_T == 5 + K


def _selection_buffers(P, cap, dev):
    import torch
    return (torch.full((max(cap, 1),), -1, device=dev, dtype=torch.int32)[:cap],
            torch.zeros(max(cap, 1), device=dev)[:cap], torch.zeros(1, device=dev, dtype=torch.int64),
            torch.full((fa.bfasgd_list_index_length(P),), -1, device=dev, dtype=torch.int32),
            fa.allocate_workspace(P, dev))


@pytest.mark.parametrize("P,K,offset,cap_frac,base", [
    (1, 1, 0, 1.0, 0), (255, 3, 0, 1.0, 0), (257, 8, 0, 1.0, 0), (1027, 2, 0, 1.0, 4096),
    (100_003, 8, 0, 1.0, 0), (100_003, 8, 0, 0.03, 0), (262_144, 4, 0, 1.0, 0), (262_145, 4, 0, 1.0, 8),
    (1_000_003, 33, 0, 1.0, 0), (65_537, 5, 1, 1.0, 0), (12_000_003, 2, 0, 1.0, 0), (30_000_001, 2, 1, 0.5, 0),
    (67_108_869, 2, 0, 1.0, 0)])
@pytest.mark.parametrize("mode", [fa.MATH_FAST, fa.MATH_IEEE])
def test_push_pass_and_next_selection_are_bit_identical(P, K, offset, cap_frac, base, mode):
    """fasgd_apply_with_push_and_select against fasgd_apply_with_push, then
    bfasgd_select_compact at the timestamp after the pass: the state, T,
    dense_T, the next push's count, list and list index bit for bit.  The
    pass takes the next push's decisions itself at every size and alignment.
    Covers ragged tails (a last segment shorter than 256, a last tile whose
    later segments hold no parameter), P a multiple of 1024, a shard offset,
    a capacity cut, arrays 4 bytes off alignment, the selection after the
    pass in two launches with blocks of 8 tiles (12M) and of 16 (30M), and
    in three launches with more than 64 scan groups (67M)."""
    import torch
    dev = gpu()
    a, b, _, (m_, s_, w), keep = _states(P, dev, mode, fa.V_EQUATIONS, seed=P % 991, offset=offset)
    a.c.index_base = b.c.index_base = base
    g_push = to_dev(workload.host_gradient(w, m_, s_, 5, seed=2), dev)
    gs = [to_dev(workload.host_gradient(w, m_, s_, 6 + k, seed=2), dev) for k in range(K)]
    g_next = to_dev(workload.host_gradient(w, m_, s_, 6 + K, seed=2), dev)
    clients, ts = [k % w.lam for k in range(K)], [max(6 + k - 2, 0) for k in range(K)]
    idx, val, cnt, seg = _select(a, g_push, 100.0, 5, 1, dev)
    cap = max(1, int(P * cap_frac))
    A = _selection_buffers(P, cap, dev)
    B = _selection_buffers(P, cap, dev)
    fa.fasgd_apply_with_push(a, idx, val, cnt, seg, 1, 4, gs, clients, ts)
    fa.bfasgd_select_compact(a, g_next, 60.0, 1e-8, SEED, a.T, 2, A[0], A[1], A[2], A[4], seg_start=A[3])
    fa.fasgd_apply_with_push_and_select(b, idx, val, cnt, seg, 1, 4, gs, clients, ts, g_next, 2, 60.0, 1e-8, SEED,
                                        B[0], B[1], B[2], B[3], B[4])
    _assert_same(a, b)
    assert b.T == 5 + K + 1
    m = int(A[2].item())
    assert int(B[2].item()) == m
    u = min(m, cap)
    assert torch.equal(A[0][:u], B[0][:u])
    assert torch.equal(A[1][:u].view(torch.int32), B[1][:u].view(torch.int32))
    assert torch.equal(A[3], B[3])
    if cap_frac == 1.0:
        assert (B[0][u:] == -1).all()
        assert 0.02 * P < m < 0.6 * P or P < 300


def test_push_pass_and_next_selection_into_the_applied_lists():
    """The next push's list written into the buffers of the push the pass
    applies (the pipeline's use), against the two calls with separate buffers."""
    import torch
    dev = gpu()
    P, K = 300_007, 8
    a, b, _, (m_, s_, w), keep = _states(P, dev, fa.MATH_FAST, fa.V_EQUATIONS, seed=17)
    g_push = to_dev(workload.host_gradient(w, m_, s_, 5, seed=17), dev)
    gs = [to_dev(workload.host_gradient(w, m_, s_, 6 + k, seed=17), dev) for k in range(K)]
    g_next = to_dev(workload.host_gradient(w, m_, s_, 6 + K, seed=17), dev)
    clients, ts = [k % w.lam for k in range(K)], [6 + k - 1 for k in range(K)]
    ia, va, ca, sa = _select(a, g_push, 100.0, 5, 1, dev)
    ib, vb, cb, sb = (x.clone() for x in (ia, va, ca, sa))
    A = _selection_buffers(P, P, dev)
    fa.fasgd_apply_with_push(a, ia, va, ca, sa, 1, 4, gs, clients, ts)
    fa.bfasgd_select_compact(a, g_next, 60.0, 1e-8, SEED, a.T, 2, A[0], A[1], A[2], A[4], seg_start=A[3])
    ws = fa.allocate_workspace(P, dev)
    fa.fasgd_apply_with_push_and_select(b, ib, vb, cb, sb, 1, 4, gs, clients, ts, g_next, 2, 60.0, 1e-8, SEED,
                                        ib, vb, cb, sb, ws)
    _assert_same(a, b)
    m = int(A[2].item())
    assert int(cb.item()) == m
    assert torch.equal(A[0][:m], ib[:m]) and torch.equal(A[1][:m], vb[:m]) and torch.equal(A[3], sb)


@pytest.mark.parametrize("mode", [fa.MATH_FAST, fa.MATH_IEEE])
def test_push_pass_and_next_selection_prose_reading(mode):
    """The same bit-identity with the text's reading of v (the decisions use
    whichever v the state keeps)."""
    import torch
    dev = gpu()
    P, K = 200_003, 6
    a, b, _, (m_, s_, w), keep = _states(P, dev, mode, fa.V_PROSE, seed=29)
    g_push = to_dev(workload.host_gradient(w, m_, s_, 5, seed=29), dev)
    gs = [to_dev(workload.host_gradient(w, m_, s_, 6 + k, seed=29), dev) for k in range(K)]
    g_next = to_dev(workload.host_gradient(w, m_, s_, 6 + K, seed=29), dev)
    clients, ts = [k % w.lam for k in range(K)], [6 + k for k in range(K)]
    idx, val, cnt, seg = _select(a, g_push, 100.0, 5, 1, dev)
    A = _selection_buffers(P, P, dev)
    B = _selection_buffers(P, P, dev)
    fa.fasgd_apply_with_push(a, idx, val, cnt, seg, 1, 5, gs, clients, ts)
    fa.bfasgd_select_compact(a, g_next, 5.0, 1e-8, SEED, a.T, 3, A[0], A[1], A[2], A[4], seg_start=A[3])
    fa.fasgd_apply_with_push_and_select(b, idx, val, cnt, seg, 1, 5, gs, clients, ts, g_next, 3, 5.0, 1e-8, SEED,
                                        B[0], B[1], B[2], B[3], B[4])
    _assert_same(a, b)
    m = int(A[2].item())
    assert int(B[2].item()) == m and 0 < m < P
    assert torch.equal(A[0][:m], B[0][:m]) and torch.equal(A[3], B[3])



def test_resume_from_checkpoint_is_bit_exact():
    """Three pipelined server steps (each a push, 8 gradients and the next
    push's selection), a checkpoint to the host (the state and the pending
    push's list), a resume into new device buffers, and two more steps: the
    same state, T and list, bit for bit, as five steps without the stop
    (every draw is keyed by T, so the state and T are all a run needs)."""
    import torch
    dev = gpu()
    P, K = 300_007, 8
    a, b, _, (m_, s_, w), keep = _states(P, dev, fa.MATH_FAST, fa.V_EQUATIONS, seed=41)
    gs = [to_dev(workload.host_gradient(w, m_, s_, t, seed=41), dev) for t in range(K + 1)]
    clients, ts = workload.schedule(w, 5 + 6 * (K + 1) + 1)

    def lists():
        return _select(a, gs[K], 100.0, 5, 1, dev)

    def steps(st, L, n):
        idx, val, cnt, seg = L
        ws = fa.allocate_workspace(P, dev)
        for _ in range(n):
            T = st.T
            sl = slice(T + 1, T + 1 + K)
            fa.fasgd_apply_with_push_and_select(st, idx, val, cnt, seg, clients[T], ts[T], gs[:K], clients[sl],
                                                ts[sl], gs[K], clients[T + K + 1], 60.0, 1e-8, SEED,
                                                idx, val, cnt, seg, ws)

    La = lists()
    Lb = tuple(x.clone() for x in La)
    steps(a, La, 5)
    steps(b, Lb, 3)
    torch.cuda.synchronize()
    ck = fa.checkpoint(b)
    ck_lists = tuple(x.cpu() for x in Lb)
    del b, Lb
    r = fa.resume_state(ck, dev)
    Lr = tuple(x.to(dev) for x in ck_lists)
    steps(r, Lr, 2)
    _assert_same(a, r)
    m = int(La[2].item())
    assert int(Lr[2].item()) == m
    assert torch.equal(La[0][:m], Lr[0][:m]) and torch.equal(La[3], Lr[3])


@pytest.mark.parametrize("c,cap", [(0.0, None), (3e38, None), (60.0, 0)])
def test_push_pass_and_next_selection_edge_thresholds(c, cap):
    """The next push at a threshold that sends everything, one that sends
    nothing, and a capacity of zero (only the count is written): the same
    count, list and index as the two separate calls."""
    import torch
    dev = gpu()
    P, K = 123_457, 3
    a, b, _, (m_, s_, w), keep = _states(P, dev, fa.MATH_FAST, fa.V_EQUATIONS, seed=53)
    g_push = to_dev(workload.host_gradient(w, m_, s_, 5, seed=53), dev)
    gs = [to_dev(workload.host_gradient(w, m_, s_, 6 + k, seed=53), dev) for k in range(K)]
    g_next = to_dev(workload.host_gradient(w, m_, s_, 6 + K, seed=53), dev)
    clients, ts = [k % w.lam for k in range(K)], [6 + k for k in range(K)]
    idx, val, cnt, seg = _select(a, g_push, 100.0, 5, 1, dev)
    capacity = P if cap is None else cap
    A = _selection_buffers(P, capacity, dev)
    B = _selection_buffers(P, capacity, dev)
    fa.fasgd_apply_with_push(a, idx, val, cnt, seg, 1, 5, gs, clients, ts)
    fa.bfasgd_select_compact(a, g_next, c, 1e-8, SEED, a.T, 3, A[0], A[1], A[2], A[4], seg_start=A[3])
    fa.fasgd_apply_with_push_and_select(b, idx, val, cnt, seg, 1, 5, gs, clients, ts, g_next, 3, c, 1e-8, SEED,
                                        B[0], B[1], B[2], B[3], B[4])
    _assert_same(a, b)
    m = int(A[2].item())
    assert int(B[2].item()) == m
    assert m == {0.0: P, 3e38: 0}.get(c, m)
    u = min(m, capacity)
    assert torch.equal(A[0][:u], B[0][:u]) and torch.equal(A[3], B[3])


def test_record_next_pass_times_the_pass_once():
    """The events handed to fasgd_record_next_pass are recorded around the
    next pass kernel only (inside a call that also selects): the interval is
    positive and no longer than the whole call, and a later call leaves them
    alone."""
    import torch
    dev = gpu()
    P, K = 2_000_003, 8
    a, _, _, (m_, s_, w), keep = _states(P, dev, fa.MATH_FAST, fa.V_EQUATIONS, seed=61)
    gs = [to_dev(workload.host_gradient(w, m_, s_, 6 + k, seed=61), dev) for k in range(K + 1)]
    idx, val, cnt, seg = _select(a, gs[K], 100.0, 5, 1, dev)
    ws = fa.allocate_workspace(P, dev)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    p0, p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    fa.fasgd_record_next_pass(p0, p1)
    c0.record()
    fa.fasgd_apply_with_push_and_select(a, idx, val, cnt, seg, 1, 5, gs[:K], list(range(K)), [6 + k for k in range(K)],
                                        gs[K], 2, 60.0, 1e-8, SEED, idx, val, cnt, seg, ws)
    c1.record()
    torch.cuda.synchronize()
    t_pass, t_call = p0.elapsed_time(p1), c0.elapsed_time(c1)
    assert 0.0 < t_pass <= t_call
    fa.fasgd_apply_updates(a, gs[:K], list(range(K)), [a.T + k for k in range(K)])
    torch.cuda.synchronize()
    assert p0.elapsed_time(p1) == t_pass
