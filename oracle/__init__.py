"""CPU oracle for FASGD / SASGD / B-FASGD (arXiv:1601.04033) -- test infrastructure.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It wraps ``liboracle.so`` (plain C,
fp64, single-threaded; see ``fasgd_oracle.c``) with numpy arrays and shares no
code with the GPU library.

State is fp64.  Values the GPU path receives in fp32 (gradients, the
hyper-parameters alpha, gamma, beta, eps, and the B-FASGD inputs) are passed
here as the same fp32 values: every scalar goes through ``f32()`` first.
"""
import ctypes
import os
from dataclasses import dataclass, field

import numpy as np

from . import build as _build

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_build.LIB):
        _build.build()
    lib = ctypes.CDLL(_build.LIB)
    P = ctypes.POINTER
    dp, fp, i64p, i32p = P(ctypes.c_double), P(ctypes.c_float), P(ctypes.c_int64), P(ctypes.c_int32)
    u32p, u8p = P(ctypes.c_uint32), P(ctypes.c_uint8)
    d, f, i64, i32, u64 = ctypes.c_double, ctypes.c_float, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64
    lib.oracle_philox4x32_10.argtypes = [u32p, u32p, u32p]
    lib.oracle_philox4x32_10.restype = None
    lib.oracle_fasgd_apply.argtypes = [i64, dp, dp, dp, dp, i64p, i64p, fp, i64, d, d, d, d, i32]
    lib.oracle_fasgd_apply.restype = ctypes.c_int
    lib.oracle_sasgd_apply.argtypes = [i64, dp, i64p, i64p, fp, i64, d]
    lib.oracle_sasgd_apply.restype = ctypes.c_int
    lib.oracle_bfasgd_transmit.argtypes = [i64, f, f, f, u64, i64, i32]
    lib.oracle_bfasgd_transmit.restype = ctypes.c_int
    lib.oracle_bfasgd_decide.argtypes = [i64, i64p, fp, f, f, u64, i64, i32, u8p]
    lib.oracle_bfasgd_decide.restype = None
    lib.oracle_bfasgd_select.argtypes = [i64, fp, fp, f, f, u64, i64, i32, i32p, fp, i64, i64]
    lib.oracle_bfasgd_select.restype = ctypes.c_int64
    lib.oracle_bfasgd_apply_sparse.argtypes = [dp, dp, dp, dp, i64p, i64p, i32p, fp, i64, i64, d, d, d, d, i32]
    lib.oracle_bfasgd_apply_sparse.restype = ctypes.c_int
    lib.oracle_sync_sgd_apply.argtypes = [i64, dp, i64p, i64p, P(fp), i32, d]
    lib.oracle_sync_sgd_apply.restype = None
    lib.oracle_bfasgd_apply_cached.argtypes = [i64, dp, dp, dp, dp, i64p, i64p, fp, i32p, fp, i64, i64, d, d, d, d, i32]
    lib.oracle_bfasgd_apply_cached.restype = ctypes.c_int
    lib.oracle_bfasgd_decide_segments.argtypes = [i64, i64p, fp, f, f, u64, i64, i32, u8p, dp]
    lib.oracle_bfasgd_decide_segments.restype = None
    lib.oracle_bfasgd_apply_segments.argtypes = [i64, i64p, u8p, dp, dp, dp, dp, i64p, i64p, fp, i64, d, d, d, d, i32]
    lib.oracle_bfasgd_apply_segments.restype = ctypes.c_int
    _lib = lib
    return lib


def f32(x) -> float:
    """The fp32 value nearest to x, as a Python float (exact widening)."""
    return float(np.float32(x))


def _ptr(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _check(a, dtype, name):
    if not isinstance(a, np.ndarray) or a.dtype != dtype or not a.flags.c_contiguous:
        raise TypeError(f"{name} must be a C-contiguous numpy {np.dtype(dtype).name} array")


class OracleError(ValueError):
    pass


@dataclass
class State:
    """Server state: theta, n, b, v (fp64 [P]), last_T (int64 [P], -1 = never), T."""
    theta: np.ndarray
    n: np.ndarray
    b: np.ndarray
    v: np.ndarray
    last_T: np.ndarray
    T: int = 0
    hyper: dict = field(default_factory=dict)

    @property
    def P(self) -> int:
        return int(self.theta.shape[0])

    def copy(self) -> "State":
        return State(self.theta.copy(), self.n.copy(), self.b.copy(), self.v.copy(),
                     self.last_T.copy(), self.T, dict(self.hyper))

    def take(self, js) -> "State":
        """The state of the parameters js (updates are elementwise, so a
        subsample evolves exactly as it does inside the full vector)."""
        js = np.asarray(js)
        return State(self.theta[js].copy(), self.n[js].copy(), self.b[js].copy(),
                     self.v[js].copy(), self.last_T[js].copy(), self.T, dict(self.hyper))


def init_state(theta0, alpha, gamma=0.95, beta=0.9, eps=1e-4, n0=0.0, b0=0.0, v0=0.0, v_reading=0) -> State:
    """Server initialisation: theta from theta0 (fp32 values), n, b, v constant,
    last_T = -1, T = 0 (the timestamp starts at 0, Sec. 2.1).  v_reading 0: v
    follows the equation for v (average of 1/sqrt(n - b^2 + eps)); 1: v is
    the moving average of the standard deviation the text describes."""
    theta0 = np.asarray(theta0)
    P = theta0.shape[0]
    st = State(theta=theta0.astype(np.float32).astype(np.float64),
               n=np.full(P, f32(n0)), b=np.full(P, f32(b0)), v=np.full(P, f32(v0)),
               last_T=np.full(P, -1, dtype=np.int64), T=0)
    if v_reading not in (0, 1):
        raise OracleError("v_reading must be 0 or 1")
    st.hyper = dict(alpha=f32(alpha), gamma=f32(gamma), beta=f32(beta), eps=f32(eps), reading=int(v_reading))
    return st


def fasgd_apply(st: State, grad, grad_ts: int) -> None:
    """One FASGD weight update with one client gradient (Sec. 2.2)."""
    lib = _load()
    grad = np.ascontiguousarray(grad, dtype=np.float32)
    if grad.shape != (st.P,):
        raise OracleError("gradient length differs from P")
    T = ctypes.c_int64(st.T)
    h = st.hyper
    rc = lib.oracle_fasgd_apply(st.P, _ptr(st.theta, ctypes.c_double), _ptr(st.n, ctypes.c_double),
                                _ptr(st.b, ctypes.c_double), _ptr(st.v, ctypes.c_double),
                                _ptr(st.last_T, ctypes.c_int64), ctypes.byref(T),
                                _ptr(grad, ctypes.c_float), int(grad_ts),
                                h["alpha"], h["gamma"], h["beta"], h["eps"], h.get("reading", 0))
    if rc != 0:
        raise OracleError(f"negative staleness: grad_ts={grad_ts} > T={st.T}")
    st.T = T.value


def sasgd_apply(st: State, grad, grad_ts: int) -> None:
    """One SASGD weight update: theta -= (alpha / max(tau, 1)) * grad."""
    lib = _load()
    grad = np.ascontiguousarray(grad, dtype=np.float32)
    if grad.shape != (st.P,):
        raise OracleError("gradient length differs from P")
    T = ctypes.c_int64(st.T)
    rc = lib.oracle_sasgd_apply(st.P, _ptr(st.theta, ctypes.c_double), _ptr(st.last_T, ctypes.c_int64),
                                ctypes.byref(T), _ptr(grad, ctypes.c_float), int(grad_ts),
                                st.hyper["alpha"])
    if rc != 0:
        raise OracleError(f"negative staleness: grad_ts={grad_ts} > T={st.T}")
    st.T = T.value


def philox4x32_10(ctr, key) -> np.ndarray:
    lib = _load()
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib.oracle_philox4x32_10(_ptr(c, ctypes.c_uint32), _ptr(k, ctypes.c_uint32), _ptr(out, ctypes.c_uint32))
    return out


def bfasgd_decide(js, v_at, c, eps_c, seed, T, client) -> np.ndarray:
    """Transmit decisions (bool) for global indices js with fp32 v values v_at."""
    lib = _load()
    js = np.ascontiguousarray(js, dtype=np.int64)
    v_at = np.ascontiguousarray(v_at, dtype=np.float32)
    if js.shape != v_at.shape:
        raise OracleError("js and v_at differ in shape")
    out = np.zeros(js.shape[0], dtype=np.uint8)
    lib.oracle_bfasgd_decide(js.shape[0], _ptr(js, ctypes.c_int64), _ptr(v_at, ctypes.c_float),
                             f32(c), f32(eps_c), int(seed) & (2**64 - 1), int(T), int(client),
                             _ptr(out, ctypes.c_uint8))
    return out.astype(bool)


def bfasgd_select(v, grad, c, eps_c, seed, T, client, capacity=None, index_base=0):
    """(idx int32 ascending, val fp32, count) for one client's push.  v and
    grad may be the slice of a larger vector that starts at global index
    index_base: decisions use the global index, the list the slice's own."""
    lib = _load()
    v = np.ascontiguousarray(v, dtype=np.float32)
    grad = np.ascontiguousarray(grad, dtype=np.float32)
    if v.shape != grad.shape:
        raise OracleError("v and grad differ in shape")
    P = v.shape[0]
    cap = P if capacity is None else int(capacity)
    idx = np.zeros(max(cap, 1), dtype=np.int32)
    val = np.zeros(max(cap, 1), dtype=np.float32)
    m = lib.oracle_bfasgd_select(P, _ptr(v, ctypes.c_float), _ptr(grad, ctypes.c_float), f32(c), f32(eps_c),
                                 int(seed) & (2**64 - 1), int(T), int(client),
                                 _ptr(idx, ctypes.c_int32), _ptr(val, ctypes.c_float), cap, int(index_base))
    k = min(m, cap)
    return idx[:k].copy(), val[:k].copy(), int(m)


def bfasgd_apply_sparse(st: State, idx, val, grad_ts: int) -> None:
    """FASGD update on the listed parameters only; T advances by one."""
    lib = _load()
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    val = np.ascontiguousarray(val, dtype=np.float32)
    if idx.shape != val.shape:
        raise OracleError("idx and val differ in shape")
    if idx.size and (idx.min() < 0 or idx.max() >= st.P):
        raise OracleError("index out of range")
    T = ctypes.c_int64(st.T)
    h = st.hyper
    rc = lib.oracle_bfasgd_apply_sparse(_ptr(st.theta, ctypes.c_double), _ptr(st.n, ctypes.c_double),
                                        _ptr(st.b, ctypes.c_double), _ptr(st.v, ctypes.c_double),
                                        _ptr(st.last_T, ctypes.c_int64), ctypes.byref(T),
                                        _ptr(idx, ctypes.c_int32), _ptr(val, ctypes.c_float), idx.shape[0],
                                        int(grad_ts), h["alpha"], h["gamma"], h["beta"], h["eps"], h.get("reading", 0))
    if rc != 0:
        raise OracleError(f"negative staleness: grad_ts={grad_ts} > T={st.T}")
    st.T = T.value


def sync_sgd_apply(st: State, grads, lr) -> None:
    """Synchronous SGD step (Sec. 3 listing): every one of the lambda
    gradients applied as theta -= lr * (g / lambda) in client order; T += 1."""
    lib = _load()
    gs = [np.ascontiguousarray(g, dtype=np.float32) for g in grads]
    for g in gs:
        if g.shape != (st.P,):
            raise OracleError("gradient length differs from P")
    arr = (ctypes.POINTER(ctypes.c_float) * len(gs))(*[_ptr(g, ctypes.c_float) for g in gs])
    T = ctypes.c_int64(st.T)
    lib.oracle_sync_sgd_apply(st.P, _ptr(st.theta, ctypes.c_double), _ptr(st.last_T, ctypes.c_int64),
                              ctypes.byref(T), arr, len(gs), f32(lr))
    st.T = T.value


def bfasgd_apply_cached(st: State, cache, idx, val, grad_ts: int) -> None:
    """Push with dropped values re-applied from the client's cache (Sec. 2.3):
    cache[idx] = val, then a FASGD update with the whole cache.  cache
    (float32 [P]) is updated in place."""
    lib = _load()
    _check(cache, np.float32, "cache")
    if cache.shape != (st.P,):
        raise OracleError("cache length differs from P")
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    val = np.ascontiguousarray(val, dtype=np.float32)
    if idx.shape != val.shape:
        raise OracleError("idx and val differ in shape")
    if idx.size and (idx.min() < 0 or idx.max() >= st.P):
        raise OracleError("index out of range")
    T = ctypes.c_int64(st.T)
    h = st.hyper
    rc = lib.oracle_bfasgd_apply_cached(st.P, _ptr(st.theta, ctypes.c_double), _ptr(st.n, ctypes.c_double),
                                        _ptr(st.b, ctypes.c_double), _ptr(st.v, ctypes.c_double),
                                        _ptr(st.last_T, ctypes.c_int64), ctypes.byref(T),
                                        _ptr(cache, ctypes.c_float), _ptr(idx, ctypes.c_int32),
                                        _ptr(val, ctypes.c_float), idx.shape[0], int(grad_ts),
                                        h["alpha"], h["gamma"], h["beta"], h["eps"], h.get("reading", 0))
    if rc != 0:
        raise OracleError(f"negative staleness: grad_ts={grad_ts} > T={st.T}")
    st.T = T.value


def _segments(seg, P):
    seg = np.ascontiguousarray(seg, dtype=np.int64)
    if seg.ndim != 1 or seg.size < 2 or seg[0] != 0 or seg[-1] != P or (np.diff(seg) <= 0).any():
        raise OracleError("segments must be 0 = seg[0] < seg[1] < ... < seg[S] = P")
    return seg


def bfasgd_decide_segments(v, seg, c, eps_c, seed, T, client):
    """Paper-literal decisions (Sec. 2.3 / Sec. 5): one per segment from the
    segment's mean of v (fp32 values, summed in fp64).  Returns (bool [S],
    mean fp64 [S])."""
    lib = _load()
    v = np.ascontiguousarray(v, dtype=np.float32)
    seg = _segments(seg, v.shape[0])
    S = seg.size - 1
    out = np.zeros(S, np.uint8)
    mean = np.zeros(S, np.float64)
    lib.oracle_bfasgd_decide_segments(S, _ptr(seg, ctypes.c_int64), _ptr(v, ctypes.c_float), f32(c), f32(eps_c),
                                      int(seed) & (2**64 - 1), int(T), int(client), _ptr(out, ctypes.c_uint8),
                                      _ptr(mean, ctypes.c_double))
    return out.astype(bool), mean


def bfasgd_apply_segments(st: State, grad, seg, transmit, grad_ts: int) -> None:
    """FASGD update on the transmitted segments only; T advances by one."""
    lib = _load()
    grad = np.ascontiguousarray(grad, dtype=np.float32)
    seg = _segments(seg, st.P)
    tr = np.ascontiguousarray(transmit, dtype=np.uint8)
    if tr.size != seg.size - 1 or grad.shape != (st.P,):
        raise OracleError("shape mismatch")
    T = ctypes.c_int64(st.T)
    h = st.hyper
    rc = lib.oracle_bfasgd_apply_segments(seg.size - 1, _ptr(seg, ctypes.c_int64), _ptr(tr, ctypes.c_uint8),
                                          _ptr(st.theta, ctypes.c_double), _ptr(st.n, ctypes.c_double),
                                          _ptr(st.b, ctypes.c_double), _ptr(st.v, ctypes.c_double),
                                          _ptr(st.last_T, ctypes.c_int64), ctypes.byref(T),
                                          _ptr(grad, ctypes.c_float), int(grad_ts),
                                          h["alpha"], h["gamma"], h["beta"], h["eps"], h.get("reading", 0))
    if rc != 0:
        raise OracleError(f"negative staleness: grad_ts={grad_ts} > T={st.T}")
    st.T = T.value
