"""Seeded random parity sweep through the C ABI: configurations drawn from a
fixed seed per case (sizes with ragged tails and sizes next to the vector,
segment and tile edges; thresholds, keys, shard offsets, capacity cuts and
misaligned views; both math modes and both readings of v; random K and
staleness), each held to the same bar as the enumerated tests:
 * the selection against the oracle, bit-exact, with the list index (also
   at sizes from 5M to 54M, one per form of the selection);
 * a K-update sequence against the oracle within the sequence tolerance;
 * the push applied inside the pass, and the server's step that also takes
   the next push's decisions, bit-identical to the separate calls;
 * a batch of pushes, selected and applied together, bit-identical to the
   single calls;
 * the widened paths: a synchronous SGD step, per-segment decisions and the
   segment apply, a cached push and a fetch refresh, against the oracle;
 * the cached push in one pass and the fetch copy by segments (with the
   list's index) bit-identical to their plain forms."""
import numpy as np
import pytest

import oracle
import paper_1601_04033_amd as fa
import workload
from helpers import RTOL_ONE, RTOL_SEQ, assert_close, assert_state_close, gpu, new_gpu_state, to_dev

pytestmark = pytest.mark.gpu
N_CASES = 64
EDGES = (4, 256, 1024, 4096, 16384, 65536, 262144)


def _size(rng, hi):
    kind = rng.integers(0, 3)
    if kind == 0:
        return int(rng.integers(1, 300))
    if kind == 1:
        e = int(rng.choice(EDGES)) * int(rng.integers(1, 9))
        return int(min(max(1, e + int(rng.integers(-5, 6))), hi))
    return int(np.exp(rng.uniform(np.log(300), np.log(hi))))


def _offset_view(host, dev, off):
    """A device copy of host starting `off` floats into its buffer."""
    import torch
    buf = torch.empty(host.shape[0] + off, device=dev, dtype=torch.float32)
    buf[off:].copy_(torch.from_numpy(host))
    return buf[off:]


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_selection_matches_oracle(case):
    rng = np.random.default_rng(1000 + case)
    _random_selection(rng, case, _size(rng, 3_000_000))


# one size near the middle of each load count of the two-launch form's
# scatter (2 to 6 loads with blocks of 8 tiles, 4 to 6 with blocks of 16)
# and one past it (three launches), jittered by up to 1M with a ragged tail
LARGE_SIZES = (6_300_000, 10_500_000, 14_700_000, 18_900_000, 23_100_000, 29_000_000, 37_700_000, 46_000_000,
               53_000_000)


@pytest.mark.parametrize("case", range(len(LARGE_SIZES)))
def test_random_large_selection_matches_oracle(case):
    """Every form of the selection from 4.2M to 55M parameters, to the same
    bar as the small random cases."""
    rng = np.random.default_rng(5000 + case)
    P = LARGE_SIZES[case] + int(rng.integers(-1_000_000, 1_000_000))
    _random_selection(rng, 100 + case, P)


def _random_selection(rng, case, P):
    import torch
    dev = gpu()
    v = workload.synthetic_v(P, seed=case, lo=float(rng.uniform(0.1, 10)), hi=float(rng.uniform(20, 400)))
    g = rng.standard_normal(P).astype(np.float32)
    c = float(np.float32(np.exp(rng.uniform(np.log(0.05), np.log(5e3)))))
    eps_c = float(rng.choice([0.0, 1e-8, 1e-3]))
    seed = int(rng.integers(0, 2 ** 63))
    T = int(rng.integers(0, 2 ** 32))
    lam = int(rng.integers(1, 300))
    client = int(rng.integers(0, lam))
    base = 4 * int(rng.integers(0, 2 ** 40)) if rng.random() < 0.5 else 0
    v_off, g_off = int(rng.random() < 0.25), int(rng.random() < 0.25)
    r_idx, r_val, r_m = oracle.bfasgd_select(v, g, c, eps_c, seed, T, client, index_base=base)
    cap = P if rng.random() < 0.7 else int(rng.integers(0, r_m + 2))
    print(f"case {case}: P={P} c={c:.4g} eps_c={eps_c} base={base} offsets={v_off},{g_off} cap={cap} m={r_m}",
          flush=True)

    st = new_gpu_state(np.zeros(P, np.float32), dev, lam, 0.005, fa.MATH_FAST)
    vd = _offset_view(v, dev, v_off)
    st.c.v = vd.data_ptr()
    st.tensors["v"] = vd
    st.c.index_base = base
    gd = _offset_view(g, dev, g_off)
    idx = torch.full((max(cap, 1),), -7, device=dev, dtype=torch.int32)[:cap]
    val = torch.zeros(max(cap, 1), device=dev)[:cap]
    cnt = torch.full((1,), -1, device=dev, dtype=torch.int64)
    seg = torch.full((fa.bfasgd_list_index_length(P),), -1, device=dev, dtype=torch.int32)
    ws = fa.allocate_workspace(P, dev)
    ws.fill_(int(rng.integers(0, 256)))
    fa.bfasgd_select_compact(st, gd, c, eps_c, seed, T, client, idx, val, cnt, ws, seg_start=seg)
    torch.cuda.synchronize()
    m = int(cnt.item())
    assert m == r_m
    u = min(m, cap)
    np.testing.assert_array_equal(idx[:u].cpu().numpy(), r_idx[:u])
    np.testing.assert_array_equal(val[:u].cpu().numpy().view(np.uint32), r_val[:u].view(np.uint32))
    assert (idx[u:] == -7).all()
    want = np.searchsorted(r_idx.astype(np.int64), 256 * np.arange(fa.bfasgd_list_index_length(P) - 1))
    got = seg.cpu().numpy().astype(np.int64)
    np.testing.assert_array_equal(got[:-1], want)
    assert got[-1] == m


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_dense_sequence_matches_oracle(case):
    rng = np.random.default_rng(2000 + case)
    dev = gpu()
    P = _size(rng, 400_000)
    mode = int(rng.choice([fa.MATH_FAST, fa.MATH_IEEE]))
    reading = int(rng.choice([fa.V_EQUATIONS, fa.V_PROSE]))
    lam = int(rng.integers(1, 65))
    gamma, beta = float(rng.uniform(0.5, 0.999)), float(rng.uniform(0.5, 0.999))
    eps = float(10 ** rng.uniform(-6, -2))
    alpha = float(10 ** rng.uniform(-4, -1.5))
    theta0 = rng.normal(0.0, 0.05, P).astype(np.float32)
    sd = float(10 ** rng.uniform(-3, 0))
    print(f"case {case}: P={P} mode={mode} reading={reading} lam={lam} gamma={gamma:.4f} beta={beta:.4f} "
          f"eps={eps:.3g} alpha={alpha:.3g} sd={sd:.3g}", flush=True)
    st = new_gpu_state(theta0, dev, lam, alpha, mode, gamma=gamma, beta=beta, eps=eps, v_reading=reading)
    ref = oracle.init_state(theta0, alpha=alpha, gamma=gamma, beta=beta, eps=eps, v_reading=reading)
    left = 64
    while left > 0:
        K = int(rng.integers(1, left + 1))
        left -= K
        grads = [(sd * rng.standard_normal(P)).astype(np.float32) for _ in range(K)]
        clients = [int(x) for x in rng.integers(0, lam, K)]
        ts = []
        for k in range(K):
            Tk = st.T + k
            ts.append(Tk - min(Tk, int(rng.integers(0, 2 * lam + 1))))
        fa.fasgd_apply_updates(st, [to_dev(x, dev) for x in grads], clients, ts)
        for k in range(K):
            oracle.fasgd_apply(ref, grads[k], ts[k])
    assert_state_close(st, ref, RTOL_SEQ, what=f"case {case}")


def _two_states(P, dev, rng, mode, reading, off):
    """Two identical mid-run GPU states (random n, b, v, theta; T = 9)."""
    import torch
    theta0 = rng.normal(0.0, 0.05, P).astype(np.float32)
    b0 = (1e-3 * rng.standard_normal(P)).astype(np.float32)
    n0 = (b0 * b0 + np.float32(1e-4) * rng.random(P).astype(np.float32)).astype(np.float32)
    v0 = workload.synthetic_v(P, seed=int(rng.integers(0, 1000)), lo=5.0, hi=100.0)
    out = []
    for _ in range(2):
        bufs = fa.allocate_state(P + off, dev)
        theta, n, b, v, last_T = (t[off:] for t in bufs)
        st = fa.fasgd_init_state(theta, n, b, v, last_T, lam=32, alpha=0.005, math_mode=mode, v_reading=reading)
        for t, a in ((theta, theta0), (n, n0), (b, b0), (v, v0)):
            t.copy_(torch.from_numpy(a))
        st.c.T = 9
        out.append((st, bufs))
    return out


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_push_pass_and_step_are_bit_identical(case):
    import torch
    rng = np.random.default_rng(3000 + case)
    dev = gpu()
    P = _size(rng, 2_000_000)
    mode = int(rng.choice([fa.MATH_FAST, fa.MATH_IEEE]))
    reading = int(rng.choice([fa.V_EQUATIONS, fa.V_PROSE]))
    off = int(rng.random() < 0.25)
    K = int(rng.integers(1, 65))
    c1, c2 = (float(np.float32(np.exp(rng.uniform(np.log(1.0), np.log(2e3))))) for _ in range(2))
    seed = int(rng.integers(0, 2 ** 63))
    print(f"case {case}: P={P} mode={mode} reading={reading} offset={off} K={K} c={c1:.4g},{c2:.4g}", flush=True)
    (a, keep_a), (b, keep_b) = _two_states(P, dev, rng, mode, reading, off)
    g_push = to_dev(rng.standard_normal(P).astype(np.float32), dev)
    gs = [to_dev((1e-2 * rng.standard_normal(P)).astype(np.float32), dev) for _ in range(K)]
    g_next = to_dev(rng.standard_normal(P).astype(np.float32), dev)
    clients = [int(x) for x in rng.integers(0, 32, K)]
    ts = [10 + k - int(rng.integers(0, 10)) for k in range(K)]
    pc, pts = int(rng.integers(0, 32)), 9 - int(rng.integers(0, 9))
    next_client = int(rng.integers(0, 32))
    L = fa.bfasgd_list_index_length(P)

    def lists():
        return (torch.full((P,), -1, device=dev, dtype=torch.int32), torch.zeros(P, device=dev),
                torch.zeros(1, device=dev, dtype=torch.int64), torch.full((L,), -1, device=dev, dtype=torch.int32))

    idx, val, cnt, seg = lists()
    fa.bfasgd_select_compact(a, g_push, c1, 1e-8, seed, 9, pc, idx, val, cnt, fa.allocate_workspace(P, dev),
                             seg_start=seg)
    # separate calls on a: the push, the K gradients, then the next push's selection
    fa.bfasgd_apply_sparse(a, idx, val, cnt, pc, pts)
    fa.fasgd_apply_updates(a, gs, clients, ts)
    n_idx, n_val, n_cnt, n_seg = lists()
    fa.bfasgd_select_compact(a, g_next, c2, 1e-8, seed, a.T, next_client, n_idx, n_val, n_cnt,
                             fa.allocate_workspace(P, dev), seg_start=n_seg)
    # the server's step on b: one call
    o_idx, o_val, o_cnt, o_seg = lists()
    fa.fasgd_apply_with_push_and_select(b, idx, val, cnt, seg, pc, pts, gs, clients, ts, g_next, next_client,
                                        c2, 1e-8, seed, o_idx, o_val, o_cnt, o_seg, fa.allocate_workspace(P, dev))
    torch.cuda.synchronize()
    for name in ("theta", "n", "b", "v"):
        assert torch.equal(a.tensors[name], b.tensors[name]), name
    assert a.T == b.T
    assert torch.equal(a.last_update(), b.last_update())
    m = int(n_cnt.item())
    assert int(o_cnt.item()) == m
    assert torch.equal(o_idx[:m], n_idx[:m])
    assert torch.equal(o_val[:m].view(torch.int32), n_val[:m].view(torch.int32))
    assert torch.equal(o_seg, n_seg)


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_batches_equal_single_calls(case):
    """A batch of B pushes: the batched selection equals B single selections
    (count, list, list index) and the batched apply equals B sparse applies
    in order (theta, n, b, v, last_T, T), bit for bit."""
    import torch
    rng = np.random.default_rng(4000 + case)
    dev = gpu()
    P = _size(rng, 1_000_000)
    B = int(rng.integers(1, 65))
    while B > 1 and B * P > 16_000_000:
        B //= 2
    mode = int(rng.choice([fa.MATH_FAST, fa.MATH_IEEE]))
    reading = int(rng.choice([fa.V_EQUATIONS, fa.V_PROSE]))
    off = int(rng.random() < 0.25)
    c = float(rng.choice([0.0, 3e38, float(np.float32(np.exp(rng.uniform(np.log(0.05), np.log(5e3)))))],
                         p=[0.1, 0.1, 0.8]))
    eps_c = float(rng.choice([0.0, 1e-8]))
    seed = int(rng.integers(0, 2 ** 63))
    cap = P if rng.random() < 0.7 else int(rng.integers(0, P // 4 + 2))
    print(f"case {case}: P={P} B={B} mode={mode} reading={reading} offset={off} c={c:.4g} cap={cap}", flush=True)
    (a, keep_a), (b, keep_b) = _two_states(P, dev, rng, mode, reading, off)
    grads = [to_dev(rng.standard_normal(P).astype(np.float32), dev) for _ in range(B)]
    Ts = [9 + k for k in range(B)]
    clients = [int(x) for x in rng.integers(0, 32, B)]
    grad_ts = [9 + k - int(rng.integers(0, 10 + k)) for k in range(B)]
    L = fa.bfasgd_list_index_length(P)
    idx = torch.full((B, max(cap, 1)), -1, device=dev, dtype=torch.int32)[:, :cap]
    val = torch.zeros((B, max(cap, 1)), device=dev)[:, :cap]
    cnt = torch.zeros(B, device=dev, dtype=torch.int64)
    seg = torch.full((B, L), -1, device=dev, dtype=torch.int32)
    ws = torch.empty(B * fa.bfasgd_workspace_bytes(P), device=dev, dtype=torch.uint8)
    if cap == 0:
        idx = torch.empty((B, 0), device=dev, dtype=torch.int32)
        val = torch.empty((B, 0), device=dev)
    fa.bfasgd_select_compact_batch(a, grads, c, eps_c, seed, Ts, clients, idx, val, cnt, ws, seg_start=seg)
    ws1 = fa.allocate_workspace(P, dev)
    for k in range(B):
        i1 = torch.full((max(cap, 1),), -1, device=dev, dtype=torch.int32)[:cap]
        v1 = torch.zeros(max(cap, 1), device=dev)[:cap]
        c1 = torch.zeros(1, device=dev, dtype=torch.int64)
        s1 = torch.full((L,), -1, device=dev, dtype=torch.int32)
        fa.bfasgd_select_compact(a, grads[k], c, eps_c, seed, Ts[k], clients[k], i1, v1, c1, ws1, seg_start=s1)
        torch.cuda.synchronize()
        m = int(c1.item())
        assert int(cnt[k].item()) == m, k
        u = min(m, cap)
        assert torch.equal(idx[k, :u], i1[:u]), k
        assert torch.equal(val[k, :u].view(torch.int32), v1[:u].view(torch.int32)), k
        assert torch.equal(seg[k], s1), k
    for k in range(B):
        fa.bfasgd_apply_sparse(a, idx[k], val[k], cnt[k:k + 1], clients[k], grad_ts[k])
    fa.fasgd_apply_pushes(b, idx, val, cnt, seg, clients, grad_ts)
    torch.cuda.synchronize()
    for name in ("theta", "n", "b", "v", "last_T"):
        assert torch.equal(a.tensors[name].view(torch.int32), b.tensors[name].view(torch.int32)), name
    assert a.T == b.T == 9 + B and a.dense_T == b.dense_T


def _near_tie(got, want, mean, c, eps_c, seed, T, client):
    """Segment decisions equal, except where r lies within 1e-12 of the fp64
    threshold (the two sides sum v in different orders)."""
    for s in np.flatnonzero(got != want):
        w = oracle.philox4x32_10([s & 0xFFFFFFFF, 0x80000000 | (s >> 32), T & 0xFFFFFFFF, client],
                                 [seed & 0xFFFFFFFF, seed >> 32])[0]
        t = mean[s] + float(np.float32(eps_c))
        p = t / (t + c)
        assert abs((int(w) >> 8) * 2.0 ** -24 - p) <= 1e-12 * p, (s, got[s], want[s])


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_widened_paths_match_oracle(case):
    """The widened server paths on random sizes and settings: a synchronous
    SGD step, per-segment decisions and the segment apply, a push with its
    dropped values taken from the client's cache, and a fetch refresh."""
    import torch
    rng = np.random.default_rng(5000 + case)
    dev = gpu()
    P = _size(rng, 300_000)
    lam = int(rng.integers(1, 40))
    mode = int(rng.choice([fa.MATH_FAST, fa.MATH_IEEE]))
    reading = int(rng.choice([fa.V_EQUATIONS, fa.V_PROSE]))
    seed = int(rng.integers(0, 2 ** 63))
    print(f"case {case}: P={P} lam={lam} mode={mode} reading={reading}", flush=True)
    theta0 = rng.normal(0.0, 0.05, P).astype(np.float32)

    # synchronous SGD: lambda gradients, one step
    st = new_gpu_state(theta0, dev, lam, 0.04, fa.MATH_FAST, sasgd=True)
    ref = oracle.init_state(theta0, alpha=0.04)
    lr = float(10 ** rng.uniform(-3, -1))
    grads = [(0.1 * rng.standard_normal(P)).astype(np.float32) for _ in range(lam)]
    fa.sgd_sync_apply(st, [to_dev(g, dev) for g in grads], lr)
    oracle.sync_sgd_apply(ref, grads, lr)
    torch.cuda.synchronize()
    assert_close(st.theta.cpu().numpy(), ref.theta, RTOL_ONE, what="sync step")
    assert st.T == ref.T == 1

    # a FASGD state after a few dense updates, then per-segment pushes, a
    # cached push and a fetch
    st = new_gpu_state(theta0, dev, lam, 0.005, mode, v_reading=reading)
    ref = oracle.init_state(theta0, alpha=0.005, v_reading=reading)
    for t in range(3):
        g = (0.01 * rng.standard_normal(P)).astype(np.float32)
        fa.fasgd_apply_updates(st, [to_dev(g, dev)], [t % lam], [t])
        oracle.fasgd_apply(ref, g, t)
    S = int(rng.integers(1, min(P, 50) + 1))
    seg = np.unique(np.concatenate([[0, P], rng.integers(1, P, S - 1) if P > 1 else []])).astype(np.int64)
    S = seg.size - 1
    c = float(np.float32(np.exp(rng.uniform(np.log(0.1), np.log(1e3)))))
    T, client = st.T, int(rng.integers(0, lam))
    d = torch.zeros(S, device=dev, dtype=torch.uint8)
    ws = torch.empty(fa.bfasgd_segments_workspace_bytes(P, S), device=dev, dtype=torch.uint8)
    fa.bfasgd_decide_segments(st, seg, c, 1e-8, seed, T, client, d, ws)
    torch.cuda.synchronize()
    got = d.cpu().numpy().astype(bool)
    v32 = st.v.cpu().numpy()
    want, mean = oracle.bfasgd_decide_segments(v32, seg, c, 1e-8, seed, T, client)
    _near_tie(got, want, mean, c, 1e-8, seed, T, client)
    g = (0.01 * rng.standard_normal(P)).astype(np.float32)
    fa.bfasgd_apply_segments(st, to_dev(g, dev), seg, d, client, T - 1)
    oracle.bfasgd_apply_segments(ref, g, seg, got.astype(np.uint8), T - 1)
    torch.cuda.synchronize()
    assert_state_close(st, ref, RTOL_SEQ, what="after the segment push")

    cl = int(rng.integers(0, lam))
    cache_h = (0.01 * rng.standard_normal(P)).astype(np.float32)
    cache_d = to_dev(cache_h, dev)
    g = (0.01 * rng.standard_normal(P)).astype(np.float32)
    idx, val, mm = oracle.bfasgd_select(st.v.cpu().numpy(), g, c, 1e-8, seed, st.T, cl)
    cnt = torch.full((1,), mm, device=dev, dtype=torch.int64)
    fa.bfasgd_apply_cached(st, to_dev(idx, dev) if mm else torch.zeros(1, device=dev, dtype=torch.int32),
                           to_dev(val, dev) if mm else torch.zeros(1, device=dev), cnt, cache_d, cl, st.T - 1)
    oracle.bfasgd_apply_cached(ref, cache_h, idx, val, ref.T - 1)
    torch.cuda.synchronize()
    assert_state_close(st, ref, RTOL_SEQ, what="after the cached push")
    np.testing.assert_array_equal(cache_d.cpu().numpy().view(np.uint32), cache_h.view(np.uint32))

    copy_h = rng.standard_normal(P).astype(np.float32)
    copy_d = to_dev(copy_h, dev)
    theta_now = st.theta.cpu().numpy()
    fi, fv, fm = oracle.bfasgd_select(st.v.cpu().numpy(), theta_now, c, 1e-8, seed ^ 1, st.T, cl)
    i_d = torch.empty(P, device=dev, dtype=torch.int32)
    v_d = torch.empty(P, device=dev)
    c_d = torch.zeros(1, device=dev, dtype=torch.int64)
    fa.bfasgd_select_compact(st, st.theta, c, 1e-8, seed ^ 1, st.T, cl, i_d, v_d, c_d, fa.allocate_workspace(P, dev))
    fa.bfasgd_apply_fetch(copy_d, i_d, v_d, c_d)
    torch.cuda.synchronize()
    assert int(c_d.item()) == fm
    copy_h[fi] = fv
    np.testing.assert_array_equal(copy_d.cpu().numpy().view(np.uint32), copy_h.view(np.uint32))


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_indexed_copies_equal_plain_ones(case):
    """Given the list's index, the cached push runs in one pass and the fetch
    copy goes segment by segment: states, caches and copies equal those of
    the plain forms bit for bit."""
    import torch
    rng = np.random.default_rng(6000 + case)
    dev = gpu()
    P = _size(rng, 2_000_000)
    mode = int(rng.choice([fa.MATH_FAST, fa.MATH_IEEE]))
    reading = int(rng.choice([fa.V_EQUATIONS, fa.V_PROSE]))
    off = int(rng.random() < 0.2)
    c_mult = float(rng.choice([0.0, 0.5, 2.0, 9.0, 50.0]))
    seed = int(rng.integers(0, 2 ** 63))
    print(f"case {case}: P={P} mode={mode} reading={reading} offset={off} c_mult={c_mult}", flush=True)
    (a, keep_a), (b, keep_b) = _two_states(P, dev, rng, mode, reading, off)
    cache_h = (0.01 * rng.standard_normal(P)).astype(np.float32)
    caches = [_offset_view(cache_h, dev, off) for _ in range(2)]
    c = float(np.float32(c_mult * a.v.double().mean().item()))
    cap = P if rng.random() < 0.75 else int(rng.integers(1, P // 8 + 2))
    L = fa.bfasgd_list_index_length(P)
    idx = torch.full((cap,), -1, device=dev, dtype=torch.int32)
    val = torch.zeros(cap, device=dev)
    cnt = torch.zeros(1, device=dev, dtype=torch.int64)
    seg = torch.full((L,), -1, device=dev, dtype=torch.int32)
    g = to_dev(rng.standard_normal(P).astype(np.float32), dev)
    client = int(rng.integers(0, 32))
    fa.bfasgd_select_compact(a, g, c, 1e-8, seed, a.T, client, idx, val, cnt, fa.allocate_workspace(P, dev),
                             seg_start=seg)
    fa.bfasgd_apply_cached(a, idx, val, cnt, caches[0], client, 8)
    fa.bfasgd_apply_cached(b, idx, val, cnt, caches[1], client, 8, seg_start=seg)
    copy_h = rng.standard_normal(P).astype(np.float32)
    copies = [_offset_view(copy_h, dev, off) for _ in range(2)]
    fa.bfasgd_apply_fetch(copies[0], idx, val, cnt)
    fa.bfasgd_apply_fetch(copies[1], idx, val, cnt, seg_start=seg)
    torch.cuda.synchronize()
    for name in ("theta", "n", "b", "v"):
        assert torch.equal(a.tensors[name].view(torch.int32), b.tensors[name].view(torch.int32)), name
    assert a.T == b.T == 10 and a.dense_T == b.dense_T == 9
    assert torch.equal(caches[0].view(torch.int32), caches[1].view(torch.int32))
    assert torch.equal(copies[0].view(torch.int32), copies[1].view(torch.int32))
