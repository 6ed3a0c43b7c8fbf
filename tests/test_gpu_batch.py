"""GPU checks of B-FASGD pushes handled in batches: bfasgd_select_compact_batch
(B selections in one set of launches) gives, push by push, the counts,
lists and list indexes of B single bfasgd_select_compact calls bit for bit
and the oracle's; fasgd_apply_pushes (B compacted pushes in one pass) gives
theta, n, b, v, last_T and T bit for bit as B bfasgd_apply_sparse calls in
order, and the oracle's state within the sequence tolerance."""
import numpy as np
import pytest

import oracle
import paper_1601_04033_amd as fa
import workload
from helpers import RTOL_SEQ, assert_state_close, gpu, new_gpu_state, philox_r, sample_indices, to_dev

pytestmark = pytest.mark.gpu
SEED = 0xBA7C4


def _mid_run_state(P, dev, mode=fa.MATH_FAST, reading=fa.V_EQUATIONS, seed=0, offset=0, T=40, copies=2):
    """`copies` identical mid-run GPU states (synthetic n, b, v, theta; T = 40,
    last_T partly set) and the oracle state holding the same values;
    offset = 1 places the arrays 4 bytes into their buffers (scalar paths)."""
    import torch
    w = workload.WORKLOADS["mlp_bfasgd" if P <= workload.MLP_P else "large"]
    theta0, m_, s_ = workload.host_params(w, P, seed=seed)
    b0 = m_ + s_ * np.float32(0.1)
    n0 = (b0 * b0 + s_ * s_).astype(np.float32)
    v0 = workload.synthetic_v(P, seed=seed, lo=5.0, hi=100.0)
    lt0 = np.where(np.arange(P) % 3 == 0, T - 7, -1).astype(np.int32)
    out = []
    for _ in range(copies):
        bufs = fa.allocate_state(P + offset, dev)
        theta, n, b, v, last_T = (t[offset:] for t in bufs)
        st = fa.fasgd_init_state(theta, n, b, v, last_T, lam=w.lam, alpha=w.alpha_fasgd, math_mode=mode,
                                 v_reading=reading)
        for t, a in ((theta, theta0), (n, n0), (b, b0), (v, v0), (last_T, lt0)):
            t.copy_(torch.from_numpy(a))
        st.c.T = T
        out.append((st, bufs))
    ref = oracle.init_state(theta0, alpha=w.alpha_fasgd, v_reading=reading)
    ref.n, ref.b, ref.v = n0.astype(np.float64), b0.astype(np.float64), v0.astype(np.float64)
    ref.last_T = lt0.astype(np.int64)
    ref.T = T
    return [o[0] for o in out], ref, (m_, s_, w), [o[1] for o in out]


def _gradients(B, P, m_, s_, w, dev, seed, offset=0):
    import torch
    out = []
    for k in range(B):
        g = workload.host_gradient(w, m_, s_, 100 + k, seed=seed)
        if offset:
            buf = torch.empty(P + offset, device=dev)
            buf[offset:].copy_(torch.from_numpy(g))
            out.append(buf[offset:])
        else:
            out.append(to_dev(g, dev))
    return out


def _batch_buffers(B, P, cap, dev):
    import torch
    idx = torch.full((B, cap), -1, device=dev, dtype=torch.int32)
    val = torch.zeros((B, cap), device=dev)
    cnt = torch.zeros(B, device=dev, dtype=torch.int64)
    seg = torch.full((B, fa.bfasgd_list_index_length(P)), -1, device=dev, dtype=torch.int32)
    ws = torch.empty(B * fa.bfasgd_workspace_bytes(P), device=dev, dtype=torch.uint8)
    return idx, val, cnt, seg, ws


@pytest.mark.parametrize("P,B,cap_frac,offset,base", [
    (1, 3, 1.0, 0, 0), (1027, 16, 1.0, 0, 0), (100_003, 16, 1.0, 0, 0), (100_003, 5, 0.05, 0, 0),
    (100_003, 6, 1.0, 0, 4 * 123_457), (1_000_003, 64, 1.0, 0, 0), (65_537, 7, 1.0, 1, 0),
    (17_000_003, 3, 1.0, 0, 0), (131_075, 64, 1.0, 0, 0), (4_194_308, 2, 0.5, 0, 0), (4_194_304, 2, 1.0, 1, 0),
    (30_000_001, 2, 0.5, 1, 0), (50_331_652, 2, 1.0, 0, 0)])
def test_batch_select_equals_single_selects(P, B, cap_frac, offset, base):
    """Push by push, the batch gives the count, list and list index of a
    single selection with the same gradient, T and client, bit for bit
    (including a capacity cut, a shard offset, the scalar path for gradients
    4 bytes off 16-byte alignment, 64 pushes, and 17M parameters).  The form
    of the selection depends on the parameters per push only (two launches
    with per-wave list positions up to 49,152 tiles, then three), so batch
    and single calls take the same form; 4,194,304 and 4,194,308 parameters
    sit either side of the scatter's first change of load count,
    30,000,001 takes blocks of 16 tiles (with misaligned gradients and a
    capacity cut), and 50,331,652 is the smallest size the three launches
    take."""
    import torch
    dev = gpu()
    (st,), _, (m_, s_, w), keep = _mid_run_state(P, dev, seed=P % 977, copies=1)
    st.c.index_base = base                   # a shard's global offset keys the draws
    grads = _gradients(B, P, m_, s_, w, dev, seed=5, offset=offset)
    Ts = [40 + 3 * k for k in range(B)]
    clients = [(5 * k + 1) % w.lam for k in range(B)]
    cap = max(1, int(P * cap_frac))
    idx, val, cnt, seg, ws = _batch_buffers(B, P, cap, dev)
    fa.bfasgd_select_compact_batch(st, grads, 60.0, 1e-8, SEED, Ts, clients, idx, val, cnt, ws, seg_start=seg)
    one_ws = fa.allocate_workspace(P, dev)
    for k in range(B):
        i1 = torch.full((cap,), -1, device=dev, dtype=torch.int32)
        v1 = torch.zeros(cap, device=dev)
        c1 = torch.zeros(1, device=dev, dtype=torch.int64)
        s1 = torch.full((fa.bfasgd_list_index_length(P),), -1, device=dev, dtype=torch.int32)
        fa.bfasgd_select_compact(st, grads[k], 60.0, 1e-8, SEED, Ts[k], clients[k], i1, v1, c1, one_ws,
                                 seg_start=s1)
        torch.cuda.synchronize()
        m = int(c1.item())
        assert int(cnt[k].item()) == m, k
        u = min(m, cap)
        assert torch.equal(idx[k, :u], i1[:u]), k
        assert torch.equal(val[k, :u].view(torch.int32), v1[:u].view(torch.int32)), k
        assert torch.equal(seg[k], s1), k
        if cap_frac == 1.0:
            assert (idx[k, u:] == -1).all(), "nothing is written past the count"


def test_batch_select_matches_oracle():
    """Every push of a batch against the oracle's selection from the same v."""
    import torch
    dev = gpu()
    P, B = 300_007, 8
    (st,), ref, (m_, s_, w), keep = _mid_run_state(P, dev, seed=31, copies=1)
    grads_h = [workload.host_gradient(w, m_, s_, 100 + k, seed=31) for k in range(B)]
    Ts, clients = [40 + k for k in range(B)], [k % w.lam for k in range(B)]
    idx, val, cnt, seg, ws = _batch_buffers(B, P, P, dev)
    fa.bfasgd_select_compact_batch(st, [to_dev(g, dev) for g in grads_h], 80.0, 1e-8, SEED, Ts, clients,
                                   idx, val, cnt, ws, seg_start=seg)
    torch.cuda.synchronize()
    v32 = ref.v.astype(np.float32)
    for k in range(B):
        r_idx, r_val, r_m = oracle.bfasgd_select(v32, grads_h[k], 80.0, 1e-8, SEED, Ts[k], clients[k])
        assert int(cnt[k].item()) == r_m
        np.testing.assert_array_equal(idx[k, :r_m].cpu().numpy(), r_idx)
        np.testing.assert_array_equal(val[k, :r_m].cpu().numpy().view(np.int32),
                                      np.asarray(r_val, np.float32).view(np.int32))
        assert 0.02 < r_m / P < 0.5


def _lists_from_singles(st, grads, cs, Ts, clients, cap, dev):
    """[B, cap] lists built from single selections with a threshold per push
    (the batched call shares one c)."""
    import torch
    B, P = len(grads), st.P
    idx, val, cnt, seg, _ = _batch_buffers(B, P, cap, dev)
    ws = fa.allocate_workspace(P, dev)
    for k in range(B):
        fa.bfasgd_select_compact(st, grads[k], cs[k], 1e-8, SEED, Ts[k], clients[k], idx[k], val[k],
                                 cnt[k:k + 1], ws, seg_start=seg[k])
    return idx, val, cnt, seg


def _assert_same(a, b):
    import torch
    torch.cuda.synchronize()
    for name in ("theta", "n", "b", "v", "last_T"):
        assert torch.equal(a.tensors[name].view(torch.int32), b.tensors[name].view(torch.int32)), name
    assert a.T == b.T and a.dense_T == b.dense_T


@pytest.mark.parametrize("reading", [fa.V_EQUATIONS, fa.V_PROSE])
@pytest.mark.parametrize("mode", [fa.MATH_FAST, fa.MATH_IEEE])
@pytest.mark.parametrize("P,B,offset", [(1, 2, 0), (255, 3, 0), (257, 9, 0), (100_003, 16, 0),
                                        (1_000_003, 64, 0), (65_537, 5, 1)])
def test_apply_pushes_is_bit_identical(P, B, offset, mode, reading):
    """B pushes at about 20 % from a batched selection: one fasgd_apply_pushes
    gives the state, last_T and T of B bfasgd_apply_sparse calls in order,
    bit for bit (vector path with a ragged tail, and the scalar path for
    arrays 4 bytes off 16-byte alignment)."""
    dev = gpu()
    (a, b), _, (m_, s_, w), keep = _mid_run_state(P, dev, mode, reading, seed=P % 1013, offset=offset)
    grads = _gradients(B, P, m_, s_, w, dev, seed=9)
    Ts = [40 + k for k in range(B)]
    clients = [k % w.lam for k in range(B)]
    grad_ts = [max(40 + k - (k % 5) - 1, 0) for k in range(B)]
    idx, val, cnt, seg, ws = _batch_buffers(B, P, P, dev)
    fa.bfasgd_select_compact_batch(a, grads, 60.0, 1e-8, SEED, Ts, clients, idx, val, cnt, ws, seg_start=seg)
    for k in range(B):
        fa.bfasgd_apply_sparse(a, idx[k], val[k], cnt[k:k + 1], clients[k], grad_ts[k])
    fa.fasgd_apply_pushes(b, idx, val, cnt, seg, clients, grad_ts)
    _assert_same(a, b)
    assert b.T == 40 + B


@pytest.mark.parametrize("case", ["mixed", "all_every_push", "truncated", "nothing"])
def test_apply_pushes_edge_lists(case):
    """Pushes of everything (more than 64 entries per 256 parameters), of
    nothing, lists cut by capacity, and a mix of these in one batch."""
    import torch
    dev = gpu()
    P, B = 200_003, 6
    (a, b), _, (m_, s_, w), keep = _mid_run_state(P, dev, seed=3)
    grads = _gradients(B, P, m_, s_, w, dev, seed=3)
    Ts, clients = [40 + k for k in range(B)], [k for k in range(B)]
    grad_ts = [38] * B
    cs = {"mixed": [0.0, 3e38, 60.0, 5.0, 0.0, 400.0], "all_every_push": [0.0] * B,
          "truncated": [20.0] * B, "nothing": [3e38] * B}[case]
    cap = 9_999 if case == "truncated" else P
    idx, val, cnt, seg = _lists_from_singles(a, grads, cs, Ts, clients, cap, dev)
    torch.cuda.synchronize()
    counts = cnt.cpu().numpy()
    if case == "truncated":
        assert (counts > cap).all()
    if case == "nothing":
        assert (counts == 0).all()
    for k in range(B):
        fa.bfasgd_apply_sparse(a, idx[k], val[k], cnt[k:k + 1], clients[k], grad_ts[k])
    fa.fasgd_apply_pushes(b, idx, val, cnt, seg, clients, grad_ts)
    _assert_same(a, b)


def test_apply_pushes_matches_oracle():
    """Against the oracle: B pushes selected from the batch's v, then applied
    one by one at T, T + 1, ..."""
    import torch
    dev = gpu()
    P, B = 300_007, 12
    (st,), ref, (m_, s_, w), keep = _mid_run_state(P, dev, seed=12, copies=1)
    grads_h = [workload.host_gradient(w, m_, s_, 100 + k, seed=12) for k in range(B)]
    Ts, clients = [40 + k for k in range(B)], [k % w.lam for k in range(B)]
    grad_ts = [max(40 + k - 3, 0) for k in range(B)]
    idx, val, cnt, seg, ws = _batch_buffers(B, P, P, dev)
    fa.bfasgd_select_compact_batch(st, [to_dev(g, dev) for g in grads_h], 60.0, 1e-8, SEED, Ts, clients,
                                   idx, val, cnt, ws, seg_start=seg)
    fa.fasgd_apply_pushes(st, idx, val, cnt, seg, clients, grad_ts)
    v32 = ref.v.astype(np.float32)
    lists = [oracle.bfasgd_select(v32, grads_h[k], 60.0, 1e-8, SEED, Ts[k], clients[k]) for k in range(B)]
    for k, (r_idx, r_val, r_m) in enumerate(lists):
        oracle.bfasgd_apply_sparse(ref, r_idx, r_val, grad_ts[k])
    torch.cuda.synchronize()
    assert [int(x) for x in cnt.cpu()] == [r[2] for r in lists]
    assert_state_close(st, ref, RTOL_SEQ, what=f"{B} pushes in one pass")
    assert st.T == ref.T == 40 + B


def test_mlp_bfasgd_batched_sequence_sampled():
    """MLP layout, lambda = 16: one dense pass of 16 updates, then 2,000
    pushes at about 20 % in 125 batches of 16, each batch selected from v at
    the batch's start and applied in one pass.  The oracle follows a sample of
    parameters, decides every push of a batch from its own v at that point
    and applies the pushes one by one.  A decision may differ only where the
    oracle's threshold lies within v's tolerance of r; such indices are
    dropped from later comparisons."""
    import torch
    dev = gpu()
    w = workload.WORKLOADS["mlp_bfasgd"]
    P, U, W, B = w.P, 2000, 16, 16
    theta0, m_, s_ = workload.host_params(w)
    clients, ts = workload.schedule(w, U + W)
    dm, ds = to_dev(m_, dev), to_dev(s_, dev)
    st = new_gpu_state(theta0, dev, w.lam, w.alpha_fasgd, fa.MATH_FAST)
    js = sample_indices(P, 3000, seed=7)
    jt = torch.from_numpy(js).to(dev)
    ref = oracle.init_state(theta0[js], alpha=w.alpha_fasgd)
    gb = [torch.empty(P, device=dev) for _ in range(B)]
    for k in range(W):
        workload.device_gradient(w, dm, ds, k, out=gb[k])
    fa.fasgd_apply_updates(st, gb[:W], clients[:W], ts[:W])
    for k in range(W):
        oracle.fasgd_apply(ref, gb[k][jt].cpu().numpy(), ts[k])
    vd = ref.v + 1e-8
    lo, hi = 0.0, 1e6
    for _ in range(80):
        c = 0.5 * (lo + hi)
        lo, hi = (c, hi) if (vd / (vd + c)).mean() > 0.2 else (lo, c)
    c = oracle.f32(c)
    idx, val, cnt, seg, ws = _batch_buffers(B, P, P, dev)
    mask = torch.zeros(P, device=dev, dtype=torch.bool)
    alive = np.ones(js.size, bool)
    flips = 0
    fractions = []
    for t0 in range(W, W + U, B):
        for k in range(B):
            workload.device_gradient(w, dm, ds, t0 + k, out=gb[k])
        T0 = st.T
        assert T0 == ref.T == t0
        fa.bfasgd_select_compact_batch(st, gb, c, 1e-8, SEED, list(range(T0, T0 + B)), clients[t0:t0 + B],
                                       idx, val, cnt, ws, seg_start=seg)
        v32 = ref.v.astype(np.float32)           # every push of the batch decides from this v
        counts = cnt.cpu().numpy()
        wants = []
        for k in range(B):
            m = int(counts[k])
            fractions.append(m / P)
            mask.zero_()
            mask[idx[k, :m].long()] = True
            got = mask[jt].cpu().numpy()
            want = oracle.bfasgd_decide(js, v32, c, 1e-8, SEED, T0 + k, clients[t0 + k])
            diff = alive & (got != want)
            if diff.any():
                tv = v32[diff].astype(np.float64) + 1e-8
                p = tv / (tv + c)
                r = philox_r(js[diff], SEED, T0 + k, int(clients[t0 + k]))
                assert (np.abs(r - p) <= 2 * RTOL_SEQ * p).all(), (r, p)
                flips += int(diff.sum())
                alive &= ~diff
            wants.append(want)
        g_at = [g[jt].cpu().numpy() for g in gb]
        for k in range(B):
            sel = np.flatnonzero(wants[k] & alive)
            oracle.bfasgd_apply_sparse(ref, sel.astype(np.int32), g_at[k][sel], ts[t0 + k])
        fa.fasgd_apply_pushes(st, idx, val, cnt, seg, clients[t0:t0 + B], ts[t0:t0 + B])
    torch.cuda.synchronize()
    assert flips <= js.size // 100, flips
    keep = np.flatnonzero(alive)
    assert_state_close(st, ref.take(keep), RTOL_SEQ, js=torch.from_numpy(js[keep]).to(dev),
                       what="after 2000 pushes in batches of 16")
    assert 0.15 < np.mean(fractions) < 0.35, np.mean(fractions)



def _host_list(P, dev, seed):
    """A list built on the host with its index: segment s (256 parameters)
    lists COUNTS[s mod len] distinct parameters (fewer in the ragged last
    segment), ascending, with random values."""
    import torch
    rng = np.random.default_rng(seed)
    counts = [0, 1, 7, 8, 9, 63, 64, 65, 128, 255, 256, 2, 0, 16]
    idx = []
    for s in range(-(-P // 256)):
        lo, hi = 256 * s, min(256 * s + 256, P)
        k = min(counts[s % len(counts)], hi - lo)
        idx.append(np.sort(rng.choice(np.arange(lo, hi), size=k, replace=False)))
    idx = np.concatenate(idx).astype(np.int32)
    val = (rng.standard_normal(idx.size) * 0.02).astype(np.float32)
    seg = np.searchsorted(idx.astype(np.int64), np.arange(0, P + 255, 256, dtype=np.int64)[:-(-P // 256)])
    seg = np.append(seg, idx.size).astype(np.int32)
    return idx, val, torch.from_numpy(seg).to(dev)


@pytest.mark.parametrize("reading", [fa.V_EQUATIONS, fa.V_PROSE])
@pytest.mark.parametrize("mode", [fa.MATH_FAST, fa.MATH_IEEE])
@pytest.mark.parametrize("offset", [0, 1])
@pytest.mark.parametrize("cut", ["none", "mid_segment", "half"])
def test_single_push_by_segments_equals_sparse_apply(cut, offset, mode, reading):
    """fasgd_apply_pushes with one push applies it segment by segment (whole
    segments from 8 entries on, listed parameters only below, empty ones
    skipped): theta, n, b, v, last_T (earlier values kept where nothing is
    listed) and T equal bfasgd_apply_sparse's bit for bit, at the threshold
    (7, 8, 9 entries), for full segments, a ragged last segment, misaligned
    arrays and lists cut by capacity."""
    import torch
    dev = gpu()
    P = 256 * 41 + 77
    (a, b), _, _, keep = _mid_run_state(P, dev, mode, reading, seed=5, offset=offset)
    idx_h, val_h, seg = _host_list(P, dev, seed=6)
    m = idx_h.size
    cap = {"none": m, "mid_segment": int(seg[20].item()) + 3, "half": m // 2}[cut]
    idx = torch.full((1, max(cap, 1)), -1, device=dev, dtype=torch.int32)
    val = torch.zeros((1, max(cap, 1)), device=dev)
    idx[0, :cap] = torch.from_numpy(idx_h[:cap]).to(dev)
    val[0, :cap] = torch.from_numpy(val_h[:cap]).to(dev)
    cnt = torch.tensor([m], device=dev, dtype=torch.int64)       # the count may exceed the capacity
    fa.bfasgd_apply_sparse(a, idx[0], val[0], cnt, 3, 38)
    fa.fasgd_apply_pushes(b, idx, val, cnt, seg.view(1, -1), [3], [38])
    _assert_same(a, b)
    assert b.T == 41
