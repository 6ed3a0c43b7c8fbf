"""Calls on different streams, each with its own state, buffers and
workspace, are independent: work issued on two (default-priority) streams at
once gives what it gives issued alone.  Every call takes its stream through
the C ABI and no kernel shares memory with another call's."""
import numpy as np
import pytest

import oracle
import paper_1601_04033_amd as fa
import workload
from helpers import gpu, new_gpu_state, to_dev

pytestmark = pytest.mark.gpu


def _selection_case(P, seed, c, dev):
    import torch
    v = workload.synthetic_v(P, seed=seed)
    g = np.random.default_rng(seed).standard_normal(P).astype(np.float32)
    st = new_gpu_state(np.zeros(P, np.float32), dev, 16, 0.005, fa.MATH_FAST)
    st.v.copy_(torch.from_numpy(v))
    bufs = dict(g=to_dev(g, dev), idx=torch.full((P,), -7, device=dev, dtype=torch.int32),
                val=torch.zeros(P, device=dev), cnt=torch.full((1,), -1, device=dev, dtype=torch.int64),
                seg=torch.full((fa.bfasgd_list_index_length(P),), -1, device=dev, dtype=torch.int32),
                ws=fa.allocate_workspace(P, dev))
    bufs["ws"].fill_(seed % 256)
    return st, v, g, bufs


def test_selections_on_two_streams_match_the_oracle():
    """A two-launch selection (3M parameters) and a three-launch one (52M,
    whose scan counts arrivals in its workspace) repeated back to back on two
    streams at once: each list, count and list index is the oracle's."""
    import torch
    dev = gpu()
    cases = [(3_000_017, 11, 30.0), (52_000_003, 12, 60.0)]
    setups = [_selection_case(P, seed, c, dev) for P, seed, c in cases]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for _ in range(5):
        for (st, v, g, b), (P, seed, c), s in zip(setups, cases, streams):
            fa.bfasgd_select_compact(st, b["g"], c, 1e-8, seed, 40, 3, b["idx"], b["val"], b["cnt"], b["ws"],
                                     seg_start=b["seg"], stream=s)
    torch.cuda.synchronize()
    for (st, v, g, b), (P, seed, c) in zip(setups, cases):
        r_idx, r_val, r_m = oracle.bfasgd_select(v, g, c, 1e-8, seed, 40, 3)
        m = int(b["cnt"].item())
        assert m == r_m, P
        np.testing.assert_array_equal(b["idx"][:m].cpu().numpy(), r_idx)
        np.testing.assert_array_equal(b["val"][:m].cpu().numpy().view(np.uint32), r_val.view(np.uint32))
        want = np.searchsorted(r_idx.astype(np.int64), 256 * np.arange(fa.bfasgd_list_index_length(P) - 1))
        got = b["seg"].cpu().numpy().astype(np.int64)
        np.testing.assert_array_equal(got[:-1], want)
        assert got[-1] == m


def test_dense_passes_on_two_streams_equal_one_stream():
    """Two states updated at once on two streams (K = 8 passes, three each)
    hold, bit for bit, what the same calls give one after another on the
    default stream."""
    import torch
    dev = gpu()
    P, K = 2_000_003, 8
    w = workload.WORKLOADS["large"]
    thetas, grads = [], []
    for seed in (21, 22):
        theta0, m_, s_ = workload.host_params(w, P, seed=seed)
        thetas.append(theta0)
        grads.append([to_dev(workload.host_gradient(w, m_, s_, t, seed=seed), dev) for t in range(3 * K)])
    clients = [[(5 * t + k) % w.lam for t in range(3 * K)] for k in range(2)]

    def run(states, streams):
        for r in range(3):
            for k, (st, s) in enumerate(zip(states, streams)):
                T = st.T
                fa.fasgd_apply_updates(st, grads[k][r * K:(r + 1) * K], clients[k][r * K:(r + 1) * K],
                                       [max(0, T + i - 3) for i in range(K)], stream=s)
        torch.cuda.synchronize()

    apart = [new_gpu_state(t, dev, w.lam, w.alpha_fasgd, fa.MATH_FAST) for t in thetas]
    run(apart, [torch.cuda.Stream(), torch.cuda.Stream()])
    alone = [new_gpu_state(t, dev, w.lam, w.alpha_fasgd, fa.MATH_FAST) for t in thetas]
    run(alone, [None, None])
    for a, b in zip(apart, alone):
        assert a.T == b.T == 3 * K
        for f in ("theta", "n", "b", "v"):
            assert torch.equal(getattr(a, f).view(torch.int32), getattr(b, f).view(torch.int32)), f
