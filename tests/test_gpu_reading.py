"""GPU parity of the prose reading of v (v averages sqrt(n - b^2 + eps),
the moving average of the standard deviation that the text of Sec. 2.2
describes, instead of the 1/sqrt(...) of its equation) against the oracle in
the same reading, on every path that updates v: dense K = 1 and K-fused
passes, the sparse apply of a compacted push, the cached push and the
per-segment apply."""
import numpy as np
import pytest

import oracle
import paper_1601_04033_amd as fa
import workload
from helpers import RTOL_ONE, RTOL_SEQ, assert_state_close, gpu, new_gpu_state, to_dev

pytestmark = pytest.mark.gpu
MODES = [fa.MATH_FAST, fa.MATH_IEEE]
SEED = 0x0BAD5EED


@pytest.mark.parametrize("mode", MODES)
def test_tiny_trace_prose(mode):
    """The tiny trace (P = 100,000, 256 single updates) in the prose reading."""
    import torch
    dev = gpu()
    w = workload.WORKLOADS["tiny"]
    theta0, m, s = workload.host_params(w)
    clients, ts = workload.schedule(w)
    st = new_gpu_state(theta0, dev, w.lam, w.alpha_fasgd, mode, v_reading=fa.V_PROSE)
    ref = oracle.init_state(theta0, alpha=w.alpha_fasgd, v_reading=1)
    for t in range(w.updates):
        g = workload.host_gradient(w, m, s, t)
        fa.fasgd_apply_updates(st, [to_dev(g, dev)], [clients[t]], [ts[t]])
        oracle.fasgd_apply(ref, g, ts[t])
        if t == 0:
            torch.cuda.synchronize()
            assert_state_close(st, ref, RTOL_ONE, what="after one update")
    torch.cuda.synchronize()
    assert_state_close(st, ref, RTOL_SEQ, what="after 256 updates")


@pytest.mark.parametrize("mode", MODES)
def test_k_fused_prose(mode):
    """K = 8 gradients per pass over a ragged P (vector body and scalar tail),
    5 passes, against 40 single oracle updates."""
    import torch
    dev = gpu()
    w = workload.WORKLOADS["tiny"]
    P, K = 100_003, 8
    theta0, m, s = workload.host_params(w, P)
    clients, ts = workload.schedule(w, 5 * K)
    st = new_gpu_state(theta0, dev, w.lam, w.alpha_fasgd, mode, v_reading=fa.V_PROSE)
    ref = oracle.init_state(theta0, alpha=w.alpha_fasgd, v_reading=1)
    for p in range(5):
        gs = [workload.host_gradient(w, m, s, p * K + k) for k in range(K)]
        sl = slice(p * K, (p + 1) * K)
        fa.fasgd_apply_updates(st, [to_dev(g, dev) for g in gs], clients[sl], ts[sl])
        for k, g in enumerate(gs):
            oracle.fasgd_apply(ref, g, ts[p * K + k])
    torch.cuda.synchronize()
    assert_state_close(st, ref, RTOL_SEQ, what="after 5 passes of 8")


@pytest.mark.parametrize("mode", MODES)
def test_sparse_push_prose(mode):
    """A push at about 30 % from a synthetic mid-run state, both sides given
    the same list: listed parameters within 1e-5, the rest untouched."""
    import torch
    dev = gpu()
    w = workload.WORKLOADS["mlp_bfasgd"]
    P = 200_003
    theta0, m_, s_ = workload.host_params(w, P, seed=9)
    b0 = m_ + s_ * np.float32(0.1)
    n0 = (b0 * b0 + s_ * s_).astype(np.float32)
    v0 = workload.synthetic_v(P, seed=9, lo=1e-3, hi=0.1)      # a standard deviation's scale
    st = new_gpu_state(theta0, dev, w.lam, w.alpha_fasgd, mode, v_reading=fa.V_PROSE)
    for name, a in (("n", n0), ("b", b0), ("v", v0)):
        st.tensors[name].copy_(torch.from_numpy(a))
    st.c.T = 3
    ref = oracle.init_state(theta0, alpha=w.alpha_fasgd, v_reading=1)
    ref.n, ref.b, ref.v = n0.astype(np.float64), b0.astype(np.float64), v0.astype(np.float64)
    ref.T = 3
    g = workload.host_gradient(w, m_, s_, 3, seed=9)
    c = float(np.float32(2.0 * np.median(v0)))
    idx, val, m = oracle.bfasgd_select(v0, g, c, 1e-8, SEED, 3, 2)
    assert 0.1 * P < m < 0.6 * P
    cnt = torch.full((1,), m, device=dev, dtype=torch.int64)
    fa.bfasgd_apply_sparse(st, to_dev(idx, dev), to_dev(val, dev), cnt, 2, 1)
    oracle.bfasgd_apply_sparse(ref, idx, val, 1)
    torch.cuda.synchronize()
    assert_state_close(st, ref, RTOL_ONE, what="sparse push")
    rest = np.setdiff1d(np.arange(P), idx)
    np.testing.assert_array_equal(st.v.cpu().numpy()[rest], v0[rest])


@pytest.mark.parametrize("mode", MODES)
def test_cached_and_segment_pushes_prose(mode):
    """Cached pushes (list into the client's cache, whole cache applied) and
    per-segment pushes alternate, 12 of each, over the MLP layout's segments."""
    import torch
    dev = gpu()
    w = workload.WORKLOADS["mlp_bfasgd"]
    P = workload.MLP_P
    seg = np.concatenate([[0], np.cumsum([n for _, n, _ in workload.MLP_LAYOUT])]).astype(np.int64)
    assert seg[-1] == P
    theta0, m_, s_ = workload.host_params(w, P)
    clients, ts = workload.schedule(w, 24)
    st = new_gpu_state(theta0, dev, w.lam, w.alpha_fasgd, mode, v_reading=fa.V_PROSE)
    ref = oracle.init_state(theta0, alpha=w.alpha_fasgd, v_reading=1)
    cache_gpu = torch.zeros(P, device=dev)
    cache_ref = np.zeros(P, np.float32)
    cnt = torch.zeros(1, device=dev, dtype=torch.int64)
    rng = np.random.default_rng(4)
    for t in range(24):
        g = workload.host_gradient(w, m_, s_, t)
        if t % 2 == 0:
            c = 0.0 if t == 0 else 0.5 * float(np.median(ref.v))
            idx, val, m = oracle.bfasgd_select(ref.v.astype(np.float32), g, c, 1e-8, SEED, ref.T, 0)
            oracle.bfasgd_apply_cached(ref, cache_ref, idx, val, ts[t])
            cnt.fill_(m)
            fa.bfasgd_apply_cached(st, to_dev(idx, dev), to_dev(val, dev), cnt, cache_gpu, 0, ts[t])
        else:
            tx = rng.random(seg.size - 1) < 0.5
            oracle.bfasgd_apply_segments(ref, g, seg, tx, ts[t])
            fa.bfasgd_apply_segments(st, to_dev(g, dev), seg, to_dev(tx.astype(np.uint8), dev),
                                     int(clients[t]), ts[t])
        if t == 0:
            torch.cuda.synchronize()
            assert_state_close(st, ref, RTOL_ONE, what="after one push")
    torch.cuda.synchronize()
    assert_state_close(st, ref, RTOL_SEQ, what="after 24 pushes")
    np.testing.assert_array_equal(cache_gpu.cpu().numpy(), cache_ref)
