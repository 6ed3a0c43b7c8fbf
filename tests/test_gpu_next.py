"""GPU parity of the widened server paths: the synchronous-SGD server
(Sec. 3 listing), pushes with dropped values re-applied from the client's
cache (Sec. 2.3), and fetch-side selection of theta (Sec. 2.3)."""
import numpy as np
import pytest

import oracle
import paper_1601_04033_amd as fa
import workload
from helpers import RTOL_ONE, RTOL_SEQ, assert_close, assert_state_close, gpu, new_gpu_state, sample_indices, to_dev

pytestmark = pytest.mark.gpu
SEED = 0xF00D


@pytest.mark.parametrize("lam,P", [(16, workload.MLP_P), (1, 10_001), (100, 40_003)])
def test_sync_sgd_matches_oracle(lam, P):
    """Three synchronous steps; lambda = 100 exercises passes of 64 gradients."""
    import torch
    dev = gpu()
    w = workload.WORKLOADS["mlp"]
    theta0, m, s = workload.host_params(w, P)
    st = new_gpu_state(theta0, dev, lam, 0.04, fa.MATH_FAST, sasgd=True)
    ref = oracle.init_state(theta0, alpha=0.04)
    lr = 0.04
    for step in range(3):
        grads = [workload.host_gradient(w, m, s, step * lam + k) for k in range(lam)]
        fa.sgd_sync_apply(st, [to_dev(g, dev) for g in grads], lr)
        oracle.sync_sgd_apply(ref, grads, lr)
        if step == 0:
            torch.cuda.synchronize()
            assert_close(st.theta.cpu().numpy(), ref.theta, RTOL_ONE, what="after one step")
    torch.cuda.synchronize()
    assert_close(st.theta.cpu().numpy(), ref.theta, RTOL_SEQ, what="after three steps")
    assert st.T == ref.T == 3 and st.dense_T == 2
    np.testing.assert_array_equal(st.last_update().cpu().numpy(), ref.last_T)


def test_sync_sgd_rejects_a_missing_gradient_list():
    dev = gpu()
    st = new_gpu_state(np.zeros(100, np.float32), dev, 4, 0.01, fa.MATH_FAST, sasgd=True)
    import torch
    with pytest.raises(ValueError):
        fa.sgd_sync_apply(st, [torch.zeros(100, device=dev)] * 3, 0.1)


@pytest.mark.parametrize("mode", [fa.MATH_FAST, fa.MATH_IEEE])
def test_cached_pushes_match_oracle(mode):
    """MLP layout, lambda = 16, 40 pushes at about 20 %: every push writes its
    list into the client's cache and applies the whole cache.  Both sides get
    the same lists (the oracle's selection on its own v), so the comparison
    isolates the cached apply; the selection itself is tested elsewhere."""
    import torch
    dev = gpu()
    w = workload.WORKLOADS["mlp_bfasgd"]
    P, U = 300_007, 40
    theta0, m_, s_ = workload.host_params(w, P)
    clients, ts = workload.schedule(w, U)
    st = new_gpu_state(theta0, dev, w.lam, w.alpha_fasgd, mode)
    ref = oracle.init_state(theta0, alpha=w.alpha_fasgd)
    caches_gpu = torch.zeros(w.lam, P, device=dev)
    caches_ref = np.zeros((w.lam, P), np.float32)
    cnt = torch.zeros(1, device=dev, dtype=torch.int64)
    for t in range(U):
        g = workload.host_gradient(w, m_, s_, t)
        c = 0.0 if t < w.lam else 4.0 * float(np.median(ref.v))          # every client's first push is complete
        idx, val, mm = oracle.bfasgd_select(ref.v.astype(np.float32), g, c, 1e-8, SEED, ref.T, clients[t])
        cl = int(clients[t])
        cache_row = caches_ref[cl].copy()
        oracle.bfasgd_apply_cached(ref, cache_row, idx, val, ts[t])
        caches_ref[cl] = cache_row
        cnt.fill_(mm)
        fa.bfasgd_apply_cached(st, to_dev(idx, dev) if mm else torch.zeros(1, device=dev, dtype=torch.int32),
                               to_dev(val, dev) if mm else torch.zeros(1, device=dev), cnt, caches_gpu[cl], cl, ts[t])
        if t == 0:
            torch.cuda.synchronize()
            assert_state_close(st, ref, RTOL_ONE, what="after one push")
    torch.cuda.synchronize()
    assert_state_close(st, ref, RTOL_SEQ, what=f"after {U} pushes")
    np.testing.assert_array_equal(caches_gpu.cpu().numpy(), caches_ref)
    assert st.dense_T == U - 1


def test_fetch_selection_refreshes_client_copy_bit_exact():
    """A client's copy of theta refreshed where the fetch rule says so: the
    server's theta is the value array of the selection."""
    import torch
    dev = gpu()
    P = 1_000_003
    rng = np.random.default_rng(12)
    theta_srv = rng.standard_normal(P).astype(np.float32)
    v = workload.synthetic_v(P, seed=12)
    client = (theta_srv + rng.standard_normal(P).astype(np.float32)).astype(np.float32)
    st = new_gpu_state(theta_srv, dev, 8, 0.005, fa.MATH_FAST)
    st.v.copy_(torch.from_numpy(v))
    copy_gpu = to_dev(client, dev)
    idx = torch.empty(P, device=dev, dtype=torch.int32)
    val = torch.empty(P, device=dev)
    cnt = torch.zeros(1, device=dev, dtype=torch.int64)
    ws = fa.allocate_workspace(P, dev)
    fetch_seed = SEED ^ 0xFE7C000000000000
    fa.bfasgd_select_compact(st, st.theta, 30.0, 1e-8, fetch_seed, 5, 3, idx, val, cnt, ws)
    fa.bfasgd_apply_fetch(copy_gpu, idx, val, cnt)
    torch.cuda.synchronize()
    r_idx, r_val, r_m = oracle.bfasgd_select(v, theta_srv, 30.0, 1e-8, fetch_seed, 5, 3)
    expect = client.copy()
    expect[r_idx] = r_val
    assert int(cnt.item()) == r_m and 0 < r_m < P
    np.testing.assert_array_equal(copy_gpu.cpu().numpy().view(np.uint32), expect.view(np.uint32))
    # c = 0: the copy becomes the server's theta exactly
    fa.bfasgd_select_compact(st, st.theta, 0.0, 1e-8, fetch_seed, 6, 3, idx, val, cnt, ws)
    fa.bfasgd_apply_fetch(copy_gpu, idx, val, cnt)
    torch.cuda.synchronize()
    assert torch.equal(copy_gpu, st.theta)


# ------------------------------------------------ paper-literal mean-v decision
def _seg_r(s, seed, T, client):
    w = oracle.philox4x32_10([s & 0xFFFFFFFF, 0x80000000 | (s >> 32), T & 0xFFFFFFFF, client],
                             [seed & 0xFFFFFFFF, seed >> 32])[0]
    return (int(w) >> 8) * 2.0 ** -24


def _mlp_segments():
    offs = [0]
    for _, n, _ in workload.MLP_LAYOUT:
        offs.append(offs[-1] + n)
    return np.array(offs, np.int64)


def _check_decisions(got, want, mean, c, seed, T, client, eps_c=1e-8):
    """Equal, except where the fp64 threshold lies within 1e-12 of r (the two
    sides sum v in different orders)."""
    for s in np.flatnonzero(got != want):
        t = mean[s] + float(np.float32(eps_c))
        p = t / (t + c)
        assert abs(_seg_r(int(s), seed, T, client) - p) <= 1e-12 * p, (s, got[s], want[s])


@pytest.mark.parametrize("layout", ["whole", "mlp", "many"])
def test_segment_decisions_match_oracle(layout):
    import torch
    dev = gpu()
    if layout == "mlp":
        seg = _mlp_segments()
    elif layout == "whole":
        seg = np.array([0, 2_000_003], np.int64)
    else:                                   # 100 segments (four groups), ragged sizes down to 1
        rng = np.random.default_rng(5)
        seg = np.unique(np.concatenate([[0, 1, 2, 3, 999_999], rng.integers(4, 999_999, 95), [1_000_000]]))
        seg = seg.astype(np.int64)
    P = int(seg[-1])
    v = workload.synthetic_v(P, seed=P % 1000)
    st = new_gpu_state(np.zeros(P, np.float32), dev, 16, 0.005, fa.MATH_FAST)
    st.v.copy_(torch.from_numpy(v))
    S = seg.size - 1
    d = torch.zeros(S, device=dev, dtype=torch.uint8)
    ws = torch.empty(fa.bfasgd_segments_workspace_bytes(P, S), device=dev, dtype=torch.uint8)
    n_tx = 0
    for T, client, c in [(0, 0, 30.0), (17, 5, 100.0), (2 ** 32 - 1, 15, 3.0), (9, 2, 0.0)]:
        fa.bfasgd_decide_segments(st, seg, c, 1e-8, SEED, T, client, d, ws)
        torch.cuda.synchronize()
        got = d.cpu().numpy().astype(bool)
        want, mean = oracle.bfasgd_decide_segments(v, seg, c, 1e-8, SEED, T, client)
        _check_decisions(got, want, mean, c, SEED, T, client)
        n_tx += int(got.sum())
        if c == 0.0:
            assert got.all()
        again = [None] * 2
        for r in range(2):
            fa.bfasgd_decide_segments(st, seg, c, 1e-8, SEED, T, client, d, ws)
            torch.cuda.synchronize()
            again[r] = d.cpu().numpy().astype(bool)
        assert np.array_equal(again[0], got) and np.array_equal(again[1], got)
    assert 0 < n_tx


@pytest.mark.parametrize("mode", [fa.MATH_FAST, fa.MATH_IEEE])
def test_mlp_per_tensor_pushes_sequence(mode):
    """MLP layout, lambda = 16: 16 dense updates, then 200 pushes each decided
    per tensor from the tensors' mean v and applied on the transmitted
    tensors only."""
    import torch
    dev = gpu()
    w = workload.WORKLOADS["mlp_bfasgd"]
    P = w.P
    seg = _mlp_segments()
    S = seg.size - 1
    theta0, m_, s_ = workload.host_params(w)
    clients, ts = workload.schedule(w, 216)
    st = new_gpu_state(theta0, dev, w.lam, w.alpha_fasgd, mode)
    ref = oracle.init_state(theta0, alpha=w.alpha_fasgd)
    warm = [workload.host_gradient(w, m_, s_, k) for k in range(16)]
    fa.fasgd_apply_updates(st, [to_dev(g, dev) for g in warm], clients[:16], ts[:16])
    for k in range(16):
        oracle.fasgd_apply(ref, warm[k], ts[k])
    c = 3.0 * float(np.mean(ref.v))
    d = torch.zeros(S, device=dev, dtype=torch.uint8)
    ws = torch.empty(fa.bfasgd_segments_workspace_bytes(P, S), device=dev, dtype=torch.uint8)
    sent = 0
    for t in range(16, 216):
        g = workload.host_gradient(w, m_, s_, t)
        fa.bfasgd_decide_segments(st, seg, c, 1e-8, SEED, st.T, clients[t], d, ws)
        want, mean = oracle.bfasgd_decide_segments(ref.v.astype(np.float32), seg, c, 1e-8, SEED, ref.T, clients[t])
        fa.bfasgd_apply_segments(st, to_dev(g, dev), seg, d, clients[t], ts[t])
        oracle.bfasgd_apply_segments(ref, g, seg, want, ts[t])
        got = d.cpu().numpy().astype(bool)
        assert np.array_equal(got, want), (t, got, want)
        sent += int(want.sum())
    torch.cuda.synchronize()
    assert_state_close(st, ref, RTOL_SEQ, what="after 200 per-tensor pushes")
    assert 0 < sent < 200 * S


@pytest.mark.parametrize("reading", [fa.V_EQUATIONS, fa.V_PROSE])
@pytest.mark.parametrize("mode", [fa.MATH_FAST, fa.MATH_IEEE])
@pytest.mark.parametrize("P,c_mult,cap_frac,offset", [(100_003, 2.0, 1.0, 0), (1_000_003, 8.0, 1.0, 0),
                                                      (257, 0.0, 1.0, 0), (65_537, None, 1.0, 0),
                                                      (200_003, 4.0, 0.05, 0), (65_537, 3.0, 1.0, 1)])
def test_cached_push_in_one_pass_is_bit_identical(P, c_mult, cap_frac, offset, mode, reading):
    """With the list's index the list is merged into the cache inside the
    pass that applies it: the state, T, dense_T and the cache equal the list
    copy followed by the one-gradient pass, bit for bit (a ragged tail,
    everything sent, nothing sent, a capacity cut, and arrays 4 bytes off
    16-byte alignment, which take the two steps)."""
    import torch
    dev = gpu()
    rng = np.random.default_rng(P % 991)
    theta0 = rng.normal(0.0, 0.05, P).astype(np.float32)
    states, caches = [], []
    for _ in range(2):
        bufs = fa.allocate_state(P + offset, dev)
        theta, n, b, v, last_T = (t[offset:] for t in bufs)
        theta.copy_(torch.from_numpy(theta0))
        st = fa.fasgd_init_state(theta, n, b, v, last_T, lam=8, alpha=0.005, math_mode=mode, v_reading=reading)
        st.keep = bufs
        states.append(st)
        cb = torch.empty(P + offset, device=dev)
        cb[offset:].copy_(torch.from_numpy((0.01 * rng.standard_normal(P)).astype(np.float32)) if not caches
                          else caches[0])
        caches.append(cb[offset:])
    a, b = states
    g0 = to_dev((0.01 * rng.standard_normal(P)).astype(np.float32), dev)
    for st in (a, b):
        fa.fasgd_apply_updates(st, [g0], [0], [0])
    cap = max(1, int(P * cap_frac))
    idx = torch.full((cap,), -1, device=dev, dtype=torch.int32)
    val = torch.zeros(cap, device=dev)
    cnt = torch.zeros(1, device=dev, dtype=torch.int64)
    seg = torch.full((fa.bfasgd_list_index_length(P),), -1, device=dev, dtype=torch.int32)
    g = to_dev((0.01 * rng.standard_normal(P)).astype(np.float32), dev)
    # c as a multiple of the mean of v: about 1/(1 + c_mult) of the values are sent
    c = 3e38 if c_mult is None else float(np.float32(c_mult * a.v.double().mean().item()))
    fa.bfasgd_select_compact(a, g, c, 1e-8, SEED, a.T, 3, idx, val, cnt, fa.allocate_workspace(P, dev),
                             seg_start=seg)
    fa.bfasgd_apply_cached(a, idx, val, cnt, caches[0], 3, 0)
    fa.bfasgd_apply_cached(b, idx, val, cnt, caches[1], 3, 0, seg_start=seg)
    torch.cuda.synchronize()
    m = int(cnt.item())
    if c_mult == 0.0:
        assert m == P
    if c_mult is None:
        assert m < P // 1000
    if cap_frac < 1.0:
        assert m > cap
    if c_mult:
        assert 0.5 / (1 + c_mult) < m / P < 2.0 / (1 + c_mult)
    for name in ("theta", "n", "b", "v"):
        assert torch.equal(a.tensors[name], b.tensors[name]), name
    assert torch.equal(caches[0], caches[1])
    assert a.T == b.T == 2 and a.dense_T == b.dense_T == 1


@pytest.mark.parametrize("P,c,cap_frac,offset", [(1_000_003, 30.0, 1.0, 0), (257, 0.0, 1.0, 0),
                                                 (65_537, 3e38, 1.0, 0), (200_003, 5.0, 0.05, 0),
                                                 (100_003, 30.0, 1.0, 1), (3, 1.0, 1.0, 0)])
def test_fetch_copy_by_segments_equals_scattered_copy(P, c, cap_frac, offset):
    """With the list's index the fetch copy rewrites whole segments; the
    client's copy equals the scattered copy bit for bit (ragged tail,
    everything sent, nothing sent, a capacity cut, a copy 4 bytes off 16-byte
    alignment, which takes the scattered copy)."""
    import torch
    dev = gpu()
    rng = np.random.default_rng(P % 613)
    theta_srv = rng.standard_normal(P).astype(np.float32)
    st = new_gpu_state(theta_srv, dev, 8, 0.005, fa.MATH_FAST)
    st.v.copy_(torch.from_numpy(workload.synthetic_v(P, seed=P % 613)))
    client = rng.standard_normal(P).astype(np.float32)
    copies = []
    for _ in range(2):
        buf = torch.empty(P + offset, device=dev)
        buf[offset:].copy_(torch.from_numpy(client))
        copies.append(buf[offset:])
    cap = max(1, int(P * cap_frac))
    idx = torch.full((cap,), -1, device=dev, dtype=torch.int32)
    val = torch.zeros(cap, device=dev)
    cnt = torch.zeros(1, device=dev, dtype=torch.int64)
    seg = torch.full((fa.bfasgd_list_index_length(P),), -1, device=dev, dtype=torch.int32)
    fa.bfasgd_select_compact(st, st.theta, c, 1e-8, SEED ^ 0xFE7C, 4, 2, idx, val, cnt, fa.allocate_workspace(P, dev),
                             seg_start=seg)
    fa.bfasgd_apply_fetch(copies[0], idx, val, cnt)
    fa.bfasgd_apply_fetch(copies[1], idx, val, cnt, seg_start=seg)
    torch.cuda.synchronize()
    m = int(cnt.item())
    if c == 0.0:
        assert m == P
    if cap_frac < 1.0:
        assert m > cap
    assert torch.equal(copies[0].view(torch.int32), copies[1].view(torch.int32))
    if c == 0.0:
        assert torch.equal(copies[1], st.theta)
    expect = client.copy()
    r_idx, r_val, r_m = oracle.bfasgd_select(st.v.cpu().numpy(), theta_srv, c, 1e-8, SEED ^ 0xFE7C, 4, 2,
                                             capacity=cap)
    assert r_m == m
    expect[r_idx] = r_val
    np.testing.assert_array_equal(copies[1].cpu().numpy().view(np.uint32), expect.view(np.uint32))
