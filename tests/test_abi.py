"""The C ABI without a GPU: the library loads, exports every function the
header declares, and its host-side checks reject bad arguments before any
launch (so these calls never touch a device)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_1601_04033_amd as fa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fasgd.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fa.LIB_PATH):
        from paper_1601_04033_amd import _build
        _build.build()
    return fa.load_library()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(", text, flags=re.M)))


def test_header_and_binding_agree():
    assert sorted(fa.ABI_FUNCTIONS) == _declared_functions()


def test_every_declared_symbol_is_exported(lib):
    for name in _declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code in range(8):
        assert lib.fasgd_status_string(code)
    assert lib.fasgd_status_string(99) == b"unknown status"


def test_workspace_bytes(lib):
    assert fa.bfasgd_workspace_bytes(0) == 0
    small = fa.bfasgd_workspace_bytes(1)
    assert small > 0 and small % 256 == 0
    big = fa.bfasgd_workspace_bytes(1_000_000_000)
    # 1 bit of ballot per parameter, padded to whole tiles, plus two 4-byte
    # words per tile of 1024 parameters: under 0.14 bytes per parameter
    assert 1_000_000_000 / 8 <= big < 1_000_000_000 * 0.14


class _Fake:
    """16-byte aligned host buffers standing in for device pointers; the
    calls below fail validation before any kernel could read them."""

    def __init__(self, P):
        self.bufs = [np.zeros(P + 8, np.float32) for _ in range(6)]

    def ptr(self, i, misalign=0):
        a = self.bufs[i]
        p = a.ctypes.data
        p = (p + 15) & ~15
        return p + misalign


def _state(P=16, lam=4, T=0):
    f = _Fake(P)
    st = fa.fasgd_state()
    st.P, st.lambda_, st.mu = P, lam, 1
    st.alpha, st.gamma, st.beta, st.eps = 0.01, 0.95, 0.9, 1e-4
    st.math_mode, st.T, st.dense_T = 1, T, -1
    st.theta, st.n, st.b, st.v, st.last_T = f.ptr(0), f.ptr(1), f.ptr(2), f.ptr(3), f.ptr(4)
    return st, f


def _call_dense(lib, fn, st, ts, clients=None, K=None, grads=None, fake=None):
    K = len(ts) if K is None else K
    g = (ctypes.c_void_p * max(K, 1))(*([fake.ptr(5)] * max(K, 1))) if grads is None else grads
    c = (ctypes.c_int32 * max(K, 1))(*(clients or [0] * max(K, 1)))
    t = (ctypes.c_int64 * max(K, 1))(*(ts or [0]))
    return getattr(lib, fn)(ctypes.byref(st), g, c, t, K, None)


@pytest.mark.parametrize("fn", ["fasgd_apply_updates", "sasgd_apply_updates"])
def test_dense_rejects_bad_arguments(lib, fn):
    st, f = _state(T=3)
    # negative staleness: gradient timestamp after the update it is applied at
    assert _call_dense(lib, fn, st, [4], fake=f) == 3
    assert b"grad_ts[0]" in lib.fasgd_last_error()
    assert _call_dense(lib, fn, st, [3, 5], fake=f) == 3          # T + 1 = 4 < 5
    assert _call_dense(lib, fn, st, [-1], fake=f) == 3
    # client outside [0, lambda)
    assert _call_dense(lib, fn, st, [0], clients=[4], fake=f) == 4
    assert _call_dense(lib, fn, st, [0], clients=[-1], fake=f) == 4
    # K out of range
    assert _call_dense(lib, fn, st, [0], K=0, fake=f) == 2
    assert _call_dense(lib, fn, st, [0] * 65, K=65, fake=f) == 2
    # null gradient pointer, null state arrays, misalignment
    nullg = (ctypes.c_void_p * 1)(None)
    assert _call_dense(lib, fn, st, [0], grads=nullg, fake=f) == 1
    assert lib.fasgd_apply_updates(None, nullg, None, None, 1, None) == 1
    bad, f2 = _state()
    bad.theta = None
    assert _call_dense(lib, fn, bad, [0], fake=f2) == 1
    mis, f3 = _state()
    mis.theta = f3.ptr(0, misalign=2)
    assert _call_dense(lib, fn, mis, [0], fake=f3) == 5
    # dense_T must lie in [-1, T)
    dt, f5 = _state(T=3)
    dt.dense_T = 3
    assert _call_dense(lib, fn, dt, [0], fake=f5) == 2
    dt.dense_T = -2
    assert _call_dense(lib, fn, dt, [0], fake=f5) == 2
    # timestamps stay in the int32 range of last_T: T + K - 1 must fit
    big, f4 = _state(T=2 ** 31 - 2)
    assert _call_dense(lib, fn, big, [0, 0, 0], fake=f4) == 2
    # nothing was applied
    assert st.T == 3


def test_v_reading_validated_by_fasgd_not_by_sasgd(lib):
    """v_reading must be a fasgd_v_reading value for the updates that keep v;
    SASGD never reads v, so it does not look at the field."""
    st, f = _state(T=1)
    assert st.v_reading == fa.V_EQUATIONS
    st.v_reading = 2
    assert _call_dense(lib, "fasgd_apply_updates", st, [0], fake=f) == 2
    assert b"v_reading" in lib.fasgd_last_error()
    st.v_reading = -1
    assert _call_dense(lib, "fasgd_apply_updates", st, [0], fake=f) == 2
    assert _call_dense(lib, "sasgd_apply_updates", st, [7], fake=f) == 3   # reaches the staleness check
    assert st.T == 1


def test_fasgd_needs_statistics_but_sasgd_does_not_validate_them(lib):
    st, f = _state(T=1)
    st.n = None
    assert _call_dense(lib, "fasgd_apply_updates", st, [5], fake=f) == 1   # n missing is checked first
    assert _call_dense(lib, "sasgd_apply_updates", st, [5], fake=f) == 3   # n unused by SASGD
    st.n = f.ptr(1)
    st.math_mode = 7
    assert _call_dense(lib, "fasgd_apply_updates", st, [0], fake=f) == 2


def test_init_rejects_bad_arguments(lib):
    f = _Fake(16)
    st = fa.fasgd_state()
    P4 = [f.ptr(i) for i in range(5)]

    def init(P=16, lam=4, mu=1, alpha=0.01, gamma=0.95, beta=0.9, eps=1e-4, mode=1, ptrs=P4):
        return lib.fasgd_init_state(ctypes.byref(st), P, lam, mu, alpha, gamma, beta, eps, mode,
                                    0.0, 0.0, 0.0, *ptrs, None)

    assert init(P=0) == 2
    assert init(lam=0) == 2
    assert init(alpha=0.0) == 2
    assert init(alpha=float("nan")) == 2
    assert init(gamma=1.5) == 2
    assert init(beta=-0.1) == 2
    assert init(eps=0.0) == 2
    assert init(mode=2) == 2
    assert init(ptrs=[None] + P4[1:]) == 1
    assert init(ptrs=[P4[0], None, P4[2], P4[3], P4[4]]) == 1     # n, b, v all or none
    assert init(ptrs=[P4[0] + 2] + P4[1:]) == 5
    assert lib.fasgd_init_state(None, 16, 4, 1, 0.01, 0.95, 0.9, 1e-4, 1, 0.0, 0.0, 0.0, *P4, None) == 1


def test_select_rejects_bad_arguments(lib):
    st, f = _state(P=16)
    ws_need = fa.bfasgd_workspace_bytes(16)
    ws = np.zeros(ws_need + 512, np.uint8)
    wsp = (ws.ctypes.data + 255) & ~255
    cnt = np.zeros(2, np.int64)
    cntp = (cnt.ctypes.data + 7) & ~7

    def sel(c=1.0, eps_c=1e-8, T=0, client=0, cap=16, ws_ptr=wsp, ws_bytes=ws_need, grad=None, s=st, seg=None):
        return lib.bfasgd_select_compact(ctypes.byref(s), grad or f.ptr(5), c, eps_c, 7, T, client,
                                         f.ptr(0), f.ptr(1), cap, cntp, seg, ws_ptr, ws_bytes, None)

    assert sel(c=-1.0) == 2
    assert sel(c=float("inf")) == 2
    assert sel(eps_c=float("nan")) == 2
    assert sel(T=-1) == 2
    assert sel(T=2 ** 32) == 2
    assert sel(client=4) == 4
    assert sel(cap=-1) == 2
    assert sel(ws_bytes=ws_need - 1) == 6
    assert sel(ws_ptr=wsp + 8) == 5
    assert sel(grad=f.ptr(5, misalign=1)) == 5
    big, f2 = _state(P=2 ** 31)
    assert sel(s=big) == 2
    assert sel(seg=f.ptr(2, misalign=2)) == 5                        # the list index is uint32
    # a slice's global offset: a multiple of 4, >= 0, index_base + P <= 2^62
    for base in (-4, 2, 2 ** 62 - 12):
        st.index_base = base
        assert sel() == 2
        assert b"index_base" in lib.fasgd_last_error()
    st.index_base = 0


def test_noalloc_select_rejects_sizes_beyond_its_scratch(lib):
    # checked before the device is touched: no GPU needed
    st, f = _state(P=fa.FASGD_NOALLOC_MAX_P + 1)
    cnt = np.zeros(2, np.int64)
    cntp = (cnt.ctypes.data + 7) & ~7
    rc = lib.bfasgd_select_compact_noalloc(ctypes.byref(st), f.ptr(5), 1.0, 1e-8, 7, 0, 0, f.ptr(0), f.ptr(1),
                                           16, cntp, None, None)
    assert rc == 6
    assert b"exceeds" in lib.fasgd_last_error()
    assert lib.bfasgd_select_compact_noalloc(None, f.ptr(5), 1.0, 1e-8, 7, 0, 0, f.ptr(0), f.ptr(1), 16, cntp,
                                             None, None) == 1
    # the header's figures are the library's
    text = open(HEADER).read()
    assert f"FASGD_NOALLOC_MAX_P {fa.FASGD_NOALLOC_MAX_P}LL" in text
    assert f"FASGD_NOALLOC_SCRATCH_BYTES {fa.bfasgd_workspace_bytes(fa.FASGD_NOALLOC_MAX_P)}ULL" in text


def test_fused_push_rejects_bad_arguments(lib):
    st, f = _state(P=16, T=2)
    cnt = np.zeros(2, np.int64)
    cntp = (cnt.ctypes.data + 7) & ~7

    def fp(pc=0, pts=0, cap=16, count=cntp, seg="ok", ts=(0,), clients=None, K=None):
        K = len(ts) if K is None else K
        g = (ctypes.c_void_p * max(K, 1))(*([f.ptr(5)] * max(K, 1)))
        c = (ctypes.c_int32 * max(K, 1))(*(clients or [0] * max(K, 1)))
        t = (ctypes.c_int64 * max(K, 1))(*ts)
        segp = f.ptr(3) if seg == "ok" else seg
        return lib.fasgd_apply_with_push(ctypes.byref(st), f.ptr(0), f.ptr(1), count, segp, cap, pc, pts,
                                         g, c, t, K, None)

    assert fp(count=None) == 1
    assert fp(seg=None) == 1
    assert fp(seg=f.ptr(3, misalign=2)) == 5
    assert fp(cap=-1) == 2
    assert fp(pc=4) == 4                    # push client outside [0, lambda)
    assert fp(pts=3) == 3                   # the push is applied at T = 2
    assert fp(ts=(4,)) == 3                 # the first gradient is applied at T + 1 = 3
    assert fp(ts=(0,), K=0) == 2
    assert fp(ts=(0,), clients=[7]) == 4
    assert st.T == 2 and st.dense_T == -1


def test_batch_select_rejects_bad_arguments(lib):
    """The batched selection checks every push's arguments and the workspace
    for all B pushes; B is in 1 .. FASGD_MAX_BATCH."""
    st, f = _state(P=16)
    ws_need = fa.bfasgd_workspace_bytes(16)
    ws = np.zeros(3 * ws_need + 512, np.uint8)
    wsp = (ws.ctypes.data + 255) & ~255
    cnt = np.zeros(4, np.int64)
    cntp = (cnt.ctypes.data + 7) & ~7

    def sel(B=3, T=(0, 1, 2), clients=(0, 1, 2), grads=None, ws_bytes=3 * ws_need, cap=16):
        n = max(B, 1)
        g = (ctypes.c_void_p * n)(*(grads or [f.ptr(5)] * n))
        t = (ctypes.c_int64 * n)(*(list(T) + [0] * n)[:n])
        c = (ctypes.c_int32 * n)(*(list(clients) + [0] * n)[:n])
        return lib.bfasgd_select_compact_batch(ctypes.byref(st), B, g, 1.0, 1e-8, 7, t, c, f.ptr(0), f.ptr(1),
                                               cap, cntp, None, wsp, ws_bytes, None)

    assert sel(B=0) == 2
    assert sel(B=fa.FASGD_MAX_BATCH + 1) == 2
    assert sel(T=(0, -1, 2)) == 2
    assert sel(clients=(0, 1, 4)) == 4
    assert sel(grads=[f.ptr(5), None, f.ptr(5)]) == 1
    assert sel(grads=[f.ptr(5), f.ptr(5), f.ptr(5, misalign=2)]) == 5
    assert sel(ws_bytes=3 * ws_need - 1) == 6
    assert sel(cap=-1) == 2
    assert lib.bfasgd_select_compact_batch(ctypes.byref(st), 1, None, 1.0, 1e-8, 7, None, None, f.ptr(0),
                                           f.ptr(1), 16, cntp, None, wsp, ws_need, None) == 1


def test_apply_pushes_rejects_bad_arguments(lib):
    """The batched apply: push b is applied at T + b, so grad_ts[b] may be
    at most T + b; a rejected call leaves T alone."""
    st, f = _state(P=16, T=2)
    cnt = np.zeros(4, np.int64)
    cntp = (cnt.ctypes.data + 7) & ~7

    def ap(B=2, ts=(2, 3), clients=(0, 1), cap=16, count=cntp, seg="ok"):
        n = max(B, 1)
        t = (ctypes.c_int64 * n)(*(list(ts) + [0] * n)[:n])
        c = (ctypes.c_int32 * n)(*(list(clients) + [0] * n)[:n])
        segp = f.ptr(3) if seg == "ok" else seg
        return lib.fasgd_apply_pushes(ctypes.byref(st), B, f.ptr(0), f.ptr(1), count, segp, cap, c, t, None)

    assert ap(B=0) == 2
    assert ap(B=fa.FASGD_MAX_BATCH + 1) == 2
    assert ap(ts=(3, 3)) == 3            # push 0 is applied at T = 2
    assert ap(ts=(2, 4)) == 3            # push 1 at T + 1 = 3
    assert ap(clients=(0, 4)) == 4
    assert ap(count=None) == 1
    assert ap(seg=None) == 1
    assert ap(seg=f.ptr(3, misalign=2)) == 5
    assert ap(count=cntp + 4) == 5
    assert ap(cap=-1) == 2
    st.T = 2 ** 31 - 1
    assert ap(ts=(0, 0), cap=0) == 2     # T + B - 1 beyond INT32_MAX
    assert st.T == 2 ** 31 - 1
    st.T = 2
    assert ap(cap=0) == 0 and st.T == 4  # nothing to apply: T still advances by B


def test_push_and_select_rejects_bad_arguments(lib):
    """The pass-and-select call checks the pass's arguments and the next
    selection's (at the timestamp after the pass) before enqueueing anything."""
    st, f = _state(P=16, T=2)
    cnt = np.zeros(4, np.int64)
    cntp = (cnt.ctypes.data + 7) & ~7
    ws_need = fa.bfasgd_workspace_bytes(16)
    ws = np.zeros(ws_need + 512, np.uint8)
    wsp = (ws.ctypes.data + 255) & ~255

    def ps(pts=0, ts=(0,), nc=0, c=1.0, ws_bytes=ws_need, next_grad="ok", out_count=cntp + 8):
        K = len(ts)
        g = (ctypes.c_void_p * K)(*([f.ptr(5)] * K))
        cl = (ctypes.c_int32 * K)(*([0] * K))
        t = (ctypes.c_int64 * K)(*ts)
        ng = f.ptr(5) if next_grad == "ok" else next_grad
        return lib.fasgd_apply_with_push_and_select(ctypes.byref(st), f.ptr(0), f.ptr(1), cntp, f.ptr(3), 16, 0,
                                                    pts, g, cl, t, K, ng, nc, c, 1e-8, 7, f.ptr(2), f.ptr(4), 16,
                                                    out_count, None, wsp, ws_bytes, None)

    assert ps(pts=3) == 3                  # the push is applied at T = 2
    assert ps(ts=(4,)) == 3                # the gradient at T + 1 = 3
    assert ps(nc=4) == 4                   # next client outside [0, lambda)
    assert ps(c=-1.0) == 2
    assert ps(ws_bytes=ws_need - 1) == 6
    assert ps(next_grad=None) == 1
    assert ps(out_count=cntp + 4) == 5
    assert st.T == 2 and st.dense_T == -1


def test_record_next_pass_takes_both_events_or_none(lib):
    fake = np.zeros(4, np.int64)
    assert lib.fasgd_record_next_pass(fake.ctypes.data, None) == 1
    assert lib.fasgd_record_next_pass(None, fake.ctypes.data) == 1
    assert lib.fasgd_record_next_pass(None, None) == 0


def test_ieee_sequence_check_rejects_bad_arguments(lib):
    """fasgd_check_ieee_sequences accepts exactly the eps and alpha for which
    the kernels take the short sequences (eps >= 2^-96, 2^-20 <= |alpha| <
    2^20); every rejection happens before a launch."""
    counts = np.zeros(5, np.int64)
    ptr = counts.ctypes.data
    call = lib.fasgd_check_ieee_sequences
    assert call(0.95, 0.9, 1e-4, 0.005, 0, 16, None, None) == 1
    assert call(0.95, 0.9, 1e-4, 0.005, 0, 16, ptr + 4, None) == 5
    for eps, alpha in ((2.0 ** -97, 0.005), (float("inf"), 0.005), (float("nan"), 0.005), (0.0, 0.005),
                       (1e-4, 2.0 ** -21), (1e-4, 2.0 ** 20), (1e-4, float("nan")), (1e-4, 0.0)):
        assert call(0.95, 0.9, eps, alpha, 0, 16, ptr, None) == 2, (eps, alpha)
    assert "2^-96" in lib.fasgd_last_error().decode()
    assert call(1.5, 0.9, 1e-4, 0.005, 0, 16, ptr, None) == 2
    assert call(0.95, -0.1, 1e-4, 0.005, 0, 16, ptr, None) == 2
    assert call(0.95, 0.9, 1e-4, 0.005, 0, -1, ptr, None) == 2
    assert (counts == 0).all()


def test_copy_anchor_rejects_bad_arguments(lib):
    buf = np.zeros(64, np.float32)
    base = buf.ctypes.data
    a = base + (-base) % 16                      # a 16-byte aligned address inside buf
    assert lib.fasgd_copy_anchor(None, a, 4, None) == 1
    assert lib.fasgd_copy_anchor(a, None, 4, None) == 1
    assert lib.fasgd_copy_anchor(a, a + 64, 0, None) == 2
    assert lib.fasgd_copy_anchor(a + 4, a + 64, 4, None) == 5
    assert lib.fasgd_copy_anchor(a, a + 68, 4, None) == 5
    assert lib.fasgd_copy_anchor(a, a + 16, 8, None) == 2        # overlapping ranges
    assert "overlap" in lib.fasgd_last_error().decode()


def test_sparse_rejects_bad_arguments(lib):
    st, f = _state(P=16, T=2)
    cnt = np.zeros(2, np.int64)
    cntp = (cnt.ctypes.data + 7) & ~7

    def sp(client=0, ts=0, cap=16, count=cntp):
        return lib.bfasgd_apply_sparse(ctypes.byref(st), f.ptr(0), f.ptr(1), count, cap, client, ts, None)

    assert sp(ts=3) == 3
    assert sp(client=9) == 4
    assert sp(cap=-5) == 2
    assert sp(count=None) == 1
    assert sp(count=cntp + 4) == 5
    assert st.T == 2


def test_next_entry_points_reject_bad_arguments(lib):
    st, f = _state(P=16, lam=3, T=2)
    g = (ctypes.c_void_p * 3)(f.ptr(5), f.ptr(5), f.ptr(5))
    assert lib.sgd_sync_apply(ctypes.byref(st), None, 0.1, None) == 1
    assert lib.sgd_sync_apply(ctypes.byref(st), g, 0.0, None) == 2
    assert lib.sgd_sync_apply(ctypes.byref(st), g, float("inf"), None) == 2
    gnull = (ctypes.c_void_p * 3)(f.ptr(5), None, f.ptr(5))
    assert lib.sgd_sync_apply(ctypes.byref(st), gnull, 0.1, None) == 1
    gmis = (ctypes.c_void_p * 3)(f.ptr(5), f.ptr(5, misalign=2), f.ptr(5))
    assert lib.sgd_sync_apply(ctypes.byref(st), gmis, 0.1, None) == 5
    cnt = np.zeros(2, np.int64)
    cntp = (cnt.ctypes.data + 7) & ~7

    def cached(cache=f.ptr(5), client=0, ts=0, cap=16, seg=None):
        return lib.bfasgd_apply_cached(ctypes.byref(st), f.ptr(0), f.ptr(1), cntp, seg, cap, cache, client, ts, None)

    assert cached(cache=None) == 1
    assert cached(ts=3) == 3
    assert cached(client=3) == 4
    assert cached(cap=-1) == 2
    assert cached(cache=f.ptr(5, misalign=1)) == 5
    assert cached(seg=f.ptr(4, misalign=2)) == 5          # the list index must be 4-byte aligned

    def fetch(dst=f.ptr(2), P=16, cap=16, count=cntp, seg=None):
        return lib.bfasgd_apply_fetch(dst, P, f.ptr(0), f.ptr(1), count, seg, cap, None)

    assert fetch(dst=None) == 1
    assert fetch(P=0) == 2
    assert fetch(cap=-3) == 2
    assert fetch(count=None) == 1
    assert fetch(dst=f.ptr(2, misalign=2)) == 5
    assert fetch(seg=f.ptr(4, misalign=1)) == 5
    assert st.T == 2


def test_segment_entry_points_reject_bad_arguments(lib):
    st, f = _state(P=16, lam=3, T=2)
    ws_need = fa.bfasgd_segments_workspace_bytes(16, 2)
    assert ws_need > 0 and fa.bfasgd_segments_workspace_bytes(16, 0) == 0
    ws = np.zeros(ws_need + 512, np.uint8)
    wsp = (ws.ctypes.data + 255) & ~255
    out = np.zeros(8, np.uint8)

    def decide(seg=(0, 5, 16), c=1.0, T=0, client=0, ws_ptr=wsp, ws_bytes=ws_need):
        a = np.array(seg, np.int64)
        return lib.bfasgd_decide_segments(ctypes.byref(st), a.ctypes.data, a.size - 1, c, 1e-8, 7, T, client,
                                          out.ctypes.data, ws_ptr, ws_bytes, None)

    assert decide(seg=(0, 5, 15)) == 2          # does not end at P
    assert decide(seg=(1, 5, 16)) == 2          # does not start at 0
    assert decide(seg=(0, 5, 5, 16)) == 2       # empty segment
    assert decide(seg=(0,)) == 2                # S = 0
    assert decide(c=-1.0) == 2
    assert decide(T=2 ** 32) == 2
    assert decide(client=3) == 4
    assert decide(ws_bytes=ws_need - 1) == 6
    assert decide(ws_ptr=wsp + 16) == 5
    assert lib.bfasgd_decide_segments(ctypes.byref(st), None, 1, 1.0, 0.0, 7, 0, 0, out.ctypes.data, wsp,
                                      ws_need, None) == 1

    def apply(seg=(0, 5, 16), client=0, ts=0):
        a = np.array(seg, np.int64)
        return lib.bfasgd_apply_segments(ctypes.byref(st), f.ptr(5), a.ctypes.data, a.size - 1, out.ctypes.data,
                                         client, ts, None)

    assert apply(seg=(0, 16, 16)) == 2
    assert apply(ts=3) == 3
    assert apply(client=-1) == 4
    assert st.T == 2


def test_header_is_c_and_state_layout_matches_binding(tmp_path):
    """include/fasgd.h compiles as C11, and the binding's ctypes fasgd_state
    has the C struct's size and field offsets."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    hip_inc = "/opt/rocm/include"
    if gcc is None or not os.path.isdir(os.path.join(hip_inc, "hip")):
        pytest.skip("gcc or the HIP headers are not available")
    fields = [name for name, _ in fa.fasgd_state._fields_]
    c_names = ["lambda" if n == "lambda_" else n for n in fields]
    src = tmp_path / "layout.c"
    src.write_text("#include <stddef.h>\n#include <stdio.h>\n#include \"fasgd.h\"\nint main(void) {\n"
                   "    printf(\"%zu\\n\", sizeof(fasgd_state));\n" +
                   "".join(f"    printf(\"%zu\\n\", offsetof(fasgd_state, {n}));\n" for n in c_names) +
                   "    return 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run([gcc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I", hip_inc,
                    "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()]
    want = [ctypes.sizeof(fa.fasgd_state)] + [getattr(fa.fasgd_state, n).offset for n in fields]
    assert got == want
