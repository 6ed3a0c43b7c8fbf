"""Python binding of libfasgd.so: the FASGD parameter-server hot path of
"Faster Asynchronous SGD" (arXiv:1601.04033) on an MI355X.

Argument marshalling only.  Every step runs in the HIP kernels of
libfasgd.so; torch provides device memory and the stream.  The functions
keep the C ABI's names (include/fasgd.h):

    fasgd_init_state, fasgd_apply_updates, sasgd_apply_updates,
    bfasgd_workspace_bytes, bfasgd_select_compact, bfasgd_apply_sparse,
    sgd_sync_apply, bfasgd_apply_cached, bfasgd_apply_fetch

There is no fallback: if libfasgd.so is missing or cannot be loaded, every
call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfasgd.so")

FASGD_MAX_K = 64
FASGD_MAX_BATCH = 64
MATH_IEEE = 0
MATH_FAST = 1
V_EQUATIONS = 0     # v averages 1/sqrt(n - b^2 + eps) (Sec. 2.2's equation)
V_PROSE = 1         # v averages sqrt(n - b^2 + eps) (Sec. 2.2's text)

STATUS = {0: "FASGD_OK", 1: "FASGD_ERR_NULL", 2: "FASGD_ERR_ARG", 3: "FASGD_ERR_STALENESS",
          4: "FASGD_ERR_CLIENT", 5: "FASGD_ERR_ALIGN", 6: "FASGD_ERR_CAPACITY", 7: "FASGD_ERR_HIP"}

# every function include/fasgd.h declares
ABI_FUNCTIONS = ("fasgd_init_state", "fasgd_apply_updates", "sasgd_apply_updates",
                 "bfasgd_workspace_bytes", "bfasgd_select_compact", "bfasgd_apply_sparse",
                 "sgd_sync_apply", "bfasgd_apply_cached", "bfasgd_apply_fetch",
                 "bfasgd_segments_workspace_bytes", "bfasgd_decide_segments", "bfasgd_apply_segments",
                 "bfasgd_list_index_length", "fasgd_apply_with_push",
                 "bfasgd_select_compact_batch", "fasgd_apply_pushes", "fasgd_apply_with_push_and_select",
                 "fasgd_record_next_pass", "bfasgd_select_compact_noalloc", "fasgd_check_ieee_sequences", "fasgd_copy_anchor",
                 "fasgd_status_string", "fasgd_last_error")

# bfasgd_select_compact_noalloc: the largest P its built-in scratch holds
FASGD_NOALLOC_MAX_P = 1 << 26


class FasgdError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class fasgd_state(ctypes.Structure):
    """Mirror of the C struct fasgd_state."""
    _fields_ = [("P", ctypes.c_int64), ("lambda_", ctypes.c_int32), ("mu", ctypes.c_int32),
                ("alpha", ctypes.c_float), ("gamma", ctypes.c_float), ("beta", ctypes.c_float),
                ("eps", ctypes.c_float), ("math_mode", ctypes.c_int32), ("v_reading", ctypes.c_int32),
                ("T", ctypes.c_int64), ("dense_T", ctypes.c_int64),
                ("theta", ctypes.c_void_p), ("n", ctypes.c_void_p), ("b", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("last_T", ctypes.c_void_p), ("index_base", ctypes.c_int64)]


_lib = None


def load_library(path: Optional[str] = None):
    """Load libfasgd.so (raises OSError if it is missing: no fallback)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise OSError(f"{p} is not built; run __graft_entry__.build() (hipcc, gfx950)")
    lib = ctypes.CDLL(p)
    S, P = ctypes.POINTER(fasgd_state), ctypes.c_void_p
    i32, i64, f, u64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_uint64, ctypes.c_size_t
    lib.fasgd_init_state.argtypes = [S, i64, i32, i32, f, f, f, f, i32, f, f, f, P, P, P, P, P, P]
    lib.fasgd_apply_updates.argtypes = [S, P, P, P, i32, P]
    lib.sasgd_apply_updates.argtypes = [S, P, P, P, i32, P]
    lib.bfasgd_workspace_bytes.argtypes = [i64]
    lib.bfasgd_workspace_bytes.restype = sz
    lib.bfasgd_select_compact.argtypes = [S, P, f, f, u64, i64, i32, P, P, i64, P, P, P, sz, P]
    lib.bfasgd_select_compact_noalloc.argtypes = [S, P, f, f, u64, i64, i32, P, P, i64, P, P, P]
    lib.bfasgd_list_index_length.argtypes = [i64]
    lib.bfasgd_list_index_length.restype = i64
    lib.fasgd_apply_with_push.argtypes = [S, P, P, P, P, i64, i32, i64, P, P, P, i32, P]
    lib.fasgd_apply_with_push_and_select.argtypes = [S, P, P, P, P, i64, i32, i64, P, P, P, i32,
                                                     P, i32, f, f, u64, P, P, i64, P, P, P, sz, P]
    lib.bfasgd_apply_sparse.argtypes = [S, P, P, P, i64, i32, i64, P]
    lib.bfasgd_select_compact_batch.argtypes = [S, i32, P, f, f, u64, P, P, P, P, i64, P, P, P, sz, P]
    lib.fasgd_apply_pushes.argtypes = [S, i32, P, P, P, P, i64, P, P, P]
    lib.sgd_sync_apply.argtypes = [S, P, f, P]
    lib.bfasgd_apply_cached.argtypes = [S, P, P, P, P, i64, P, i32, i64, P]
    lib.bfasgd_apply_fetch.argtypes = [P, i64, P, P, P, P, i64, P]
    lib.bfasgd_segments_workspace_bytes.argtypes = [i64, i32]
    lib.bfasgd_segments_workspace_bytes.restype = sz
    lib.bfasgd_decide_segments.argtypes = [S, P, i32, f, f, u64, i64, i32, P, P, sz, P]
    lib.bfasgd_apply_segments.argtypes = [S, P, P, i32, P, i32, i64, P]
    for name in ("fasgd_init_state", "fasgd_apply_updates", "sasgd_apply_updates",
                 "bfasgd_select_compact", "bfasgd_apply_sparse", "sgd_sync_apply",
                 "bfasgd_apply_cached", "bfasgd_apply_fetch", "bfasgd_decide_segments",
                 "bfasgd_apply_segments", "fasgd_apply_with_push", "bfasgd_select_compact_noalloc"):
        getattr(lib, name).restype = ctypes.c_int
    lib.fasgd_record_next_pass.argtypes = [P, P]
    lib.fasgd_check_ieee_sequences.argtypes = [f, f, f, f, u64, i64, P, P]
    lib.fasgd_copy_anchor.argtypes = [P, P, i64, P]
    lib.fasgd_copy_anchor.restype = ctypes.c_int
    lib.fasgd_check_ieee_sequences.restype = ctypes.c_int
    lib.fasgd_status_string.argtypes = [ctypes.c_int]
    lib.fasgd_status_string.restype = ctypes.c_char_p
    lib.fasgd_last_error.argtypes = []
    lib.fasgd_last_error.restype = ctypes.c_char_p
    if path is None:
        _lib = lib
    return lib


def _check(rc: int):
    if rc != 0:
        raise FasgdError(rc, load_library().fasgd_last_error().decode())


def _stream(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def _dev_ptr(t, dtype, name, allow_none=False):
    import torch
    if t is None:
        if allow_none:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous {dtype} tensor")
    return t.data_ptr()


class State:
    """A server state: the C struct plus the tensors it points to (kept alive here)."""

    def __init__(self, c: fasgd_state, tensors: dict):
        self.c = c
        self.tensors = tensors

    @property
    def T(self) -> int:
        return int(self.c.T)

    @property
    def P(self) -> int:
        return int(self.c.P)

    @property
    def dense_T(self) -> int:
        return int(self.c.dense_T)

    def last_update(self):
        """Device int32 [P]: timestamp of the last update of each parameter,
        max(last_T, dense_T) (-1: never updated)."""
        import torch
        return torch.clamp(self.tensors["last_T"], min=int(self.c.dense_T))

    def __getattr__(self, name):
        t = self.__dict__.get("tensors", {})
        if name in t:
            return t[name]
        raise AttributeError(name)


def fasgd_init_state(theta, n, b, v, last_T, *, lam: int, mu: int = 1, alpha: float,
                     gamma: float = 0.95, beta: float = 0.9, eps: float = 1e-4,
                     math_mode: int = MATH_FAST, n0: float = 0.0, b0: float = 0.0, v0: float = 0.0,
                     v_reading: int = V_EQUATIONS, stream=None) -> State:
    """theta (holding theta0), n, b, v: fp32 [P]; last_T: int32 [P].  n, b, v may be None (SASGD only).
    v_reading selects which average v keeps (V_EQUATIONS or V_PROSE); it is a
    field of the state that the apply calls validate."""
    import torch
    P = theta.numel()
    for name, t in (("n", n), ("b", b), ("v", v), ("last_T", last_T)):
        if t is not None and t.numel() != P:
            raise ValueError(f"{name} has {t.numel()} elements, theta has {P}")
    st = fasgd_state()
    rc = load_library().fasgd_init_state(
        ctypes.byref(st), P, lam, mu, alpha, gamma, beta, eps, math_mode, n0, b0, v0,
        _dev_ptr(theta, torch.float32, "theta"), _dev_ptr(n, torch.float32, "n", True),
        _dev_ptr(b, torch.float32, "b", True), _dev_ptr(v, torch.float32, "v", True),
        _dev_ptr(last_T, torch.int32, "last_T"), _stream(stream))
    _check(rc)
    st.v_reading = v_reading
    return State(st, dict(theta=theta, n=n, b=b, v=v, last_T=last_T))


def checkpoint(state: State) -> dict:
    """The whole server state on the host: the struct's scalars and copies of
    its arrays (every random draw is keyed by T, so this is all a resumed run
    needs)."""
    c = state.c
    out = {name: getattr(c, name) for name, _ in fasgd_state._fields_
           if name not in ("theta", "n", "b", "v", "last_T")}
    out["arrays"] = {k: (t.cpu().clone() if t is not None else None) for k, t in state.tensors.items()}
    return out


def resume_state(ckpt: dict, device="cuda") -> State:
    """A state rebuilt from checkpoint() into new device arrays; no array is
    re-initialised (fasgd_init_state would reset n, b, v and last_T)."""
    import torch
    tensors = {k: (t.to(device) if t is not None else None) for k, t in ckpt["arrays"].items()}
    c = fasgd_state()
    for name, _ in fasgd_state._fields_:
        if name in ("theta", "n", "b", "v", "last_T"):
            t = tensors[name]
            setattr(c, name, _dev_ptr(t, torch.int32 if name == "last_T" else torch.float32, name, True))
        else:
            setattr(c, name, ckpt[name])
    return State(c, tensors)


def _dense_args(state: State, grads: Sequence, clients: Sequence[int], grad_ts: Sequence[int]):
    import torch
    K = len(grads)
    if len(clients) != K or len(grad_ts) != K:
        raise ValueError("grads, clients and grad_ts must have the same length")
    if not 1 <= K <= FASGD_MAX_K:
        raise ValueError(f"K = {K} is not in [1, {FASGD_MAX_K}]")
    ptrs = (ctypes.c_void_p * K)()
    for k, g in enumerate(grads):
        if g.numel() != state.P:
            raise ValueError(f"grads[{k}] has {g.numel()} elements, P = {state.P}")
        ptrs[k] = _dev_ptr(g, torch.float32, f"grads[{k}]")
    c = (ctypes.c_int32 * K)(*[int(x) for x in clients])
    ts = (ctypes.c_int64 * K)(*[int(x) for x in grad_ts])
    return ptrs, c, ts, K


def fasgd_apply_updates(state: State, grads: Sequence, clients: Sequence[int], grad_ts: Sequence[int],
                        stream=None) -> None:
    """Apply K gradients (arrival order) with the FASGD rule; T advances by K."""
    ptrs, c, ts, K = _dense_args(state, grads, clients, grad_ts)
    _check(load_library().fasgd_apply_updates(ctypes.byref(state.c), ptrs, c, ts, K, _stream(stream)))


def sasgd_apply_updates(state: State, grads: Sequence, clients: Sequence[int], grad_ts: Sequence[int],
                        stream=None) -> None:
    """Apply K gradients with the SASGD rate alpha / max(tau, 1); T advances by K."""
    ptrs, c, ts, K = _dense_args(state, grads, clients, grad_ts)
    _check(load_library().sasgd_apply_updates(ctypes.byref(state.c), ptrs, c, ts, K, _stream(stream)))


def bfasgd_workspace_bytes(P: int) -> int:
    return int(load_library().bfasgd_workspace_bytes(int(P)))


def bfasgd_list_index_length(P: int) -> int:
    return int(load_library().bfasgd_list_index_length(int(P)))


def bfasgd_select_compact(state: State, grad, c: float, eps_c: float, seed: int, T: int, client: int,
                          out_idx, out_val, d_count, workspace, seg_start=None, stream=None) -> None:
    """Per-parameter send/skip selection of one client gradient, compacted
    into out_idx (int32) / out_val (fp32) in ascending index order; the
    number transmitted goes to d_count (int64 [1], device).  seg_start
    (optional, int32 [bfasgd_list_index_length(P)], values < 2^31) receives
    the list's index: the position of each 256-parameter segment's first entry."""
    import torch
    cap = out_idx.numel()
    if out_val.numel() != cap:
        raise ValueError("out_idx and out_val must have the same capacity")
    if grad.numel() != state.P:
        raise ValueError("grad length differs from P")
    rc = load_library().bfasgd_select_compact(
        ctypes.byref(state.c), _dev_ptr(grad, torch.float32, "grad"), c, eps_c,
        int(seed) & (2 ** 64 - 1), int(T), int(client),
        _dev_ptr(out_idx, torch.int32, "out_idx"), _dev_ptr(out_val, torch.float32, "out_val"), cap,
        _dev_ptr(d_count, torch.int64, "d_count"), _seg_start_ptr(seg_start, state.P),
        _dev_ptr(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream))
    _check(rc)


def bfasgd_select_compact_noalloc(state: State, grad, c: float, eps_c: float, seed: int, T: int, client: int,
                                  out_idx, out_val, d_count, seg_start=None, stream=None) -> None:
    """bfasgd_select_compact with the library's built-in per-device scratch
    instead of a workspace (P <= FASGD_NOALLOC_MAX_P): for callers that
    cannot allocate.  Calls that overlap on one GPU race on that scratch."""
    import torch
    cap = out_idx.numel()
    if out_val.numel() != cap:
        raise ValueError("out_idx and out_val must have the same capacity")
    if grad.numel() != state.P:
        raise ValueError("grad length differs from P")
    rc = load_library().bfasgd_select_compact_noalloc(
        ctypes.byref(state.c), _dev_ptr(grad, torch.float32, "grad"), c, eps_c,
        int(seed) & (2 ** 64 - 1), int(T), int(client),
        _dev_ptr(out_idx, torch.int32, "out_idx"), _dev_ptr(out_val, torch.float32, "out_val"), cap,
        _dev_ptr(d_count, torch.int64, "d_count"), _seg_start_ptr(seg_start, state.P), _stream(stream))
    _check(rc)


def _seg_start_ptr(seg_start, P, required=False):
    import torch
    if seg_start is None and not required:
        return None
    if seg_start is None or seg_start.numel() < bfasgd_list_index_length(P):
        raise ValueError(f"seg_start needs bfasgd_list_index_length(P) = {bfasgd_list_index_length(P)} entries")
    return _dev_ptr(seg_start, torch.int32, "seg_start")


def fasgd_apply_with_push(state: State, push_idx, push_val, push_count, push_seg_start, push_client: int,
                          push_grad_ts: int, grads: Sequence, clients: Sequence[int], grad_ts: Sequence[int],
                          stream=None) -> None:
    """One pass: the compacted push (at T, as bfasgd_apply_sparse) and then the K
    gradients (at T + 1 ... T + K, as fasgd_apply_updates).  T advances by K + 1."""
    import torch
    cap = push_idx.numel()
    if push_val.numel() != cap:
        raise ValueError("push_idx and push_val must have the same capacity")
    ptrs, c, t, K = _dense_args(state, grads, clients, grad_ts)
    rc = load_library().fasgd_apply_with_push(
        ctypes.byref(state.c), _dev_ptr(push_idx, torch.int32, "push_idx"),
        _dev_ptr(push_val, torch.float32, "push_val"), _dev_ptr(push_count, torch.int64, "push_count"),
        _seg_start_ptr(push_seg_start, state.P, required=True), cap, int(push_client), int(push_grad_ts),
        ptrs, c, t, K, _stream(stream))
    _check(rc)


def _batch_lists(B, out_idx, out_val, d_count):
    """(capacity, B) of [B, capacity] list tensors and a [B] count tensor."""
    if out_idx.dim() != 2 or out_idx.shape[0] != B or tuple(out_val.shape) != tuple(out_idx.shape):
        raise ValueError(f"idx and val must both be [B = {B}, capacity]")
    if d_count.numel() != B:
        raise ValueError(f"d_count must have B = {B} entries")
    return int(out_idx.shape[1])


def _batch_seg(seg_start, B, P, required):
    import torch
    if seg_start is None and not required:
        return None
    L = bfasgd_list_index_length(P)
    if seg_start is None or tuple(seg_start.shape) != (B, L):
        raise ValueError(f"seg_start must be [B = {B}, bfasgd_list_index_length(P) = {L}]")
    return _dev_ptr(seg_start, torch.int32, "seg_start")


def bfasgd_select_compact_batch(state: State, grads: Sequence, c: float, eps_c: float, seed: int,
                                T: Sequence[int], clients: Sequence[int], out_idx, out_val, d_count, workspace,
                                seg_start=None, stream=None) -> None:
    """B pushes selected in one set of launches, each exactly as
    bfasgd_select_compact with its own gradient, T and client, all decided
    from v as it stands now.  out_idx / out_val: [B, capacity]; d_count: [B];
    seg_start (optional): int32 [B, bfasgd_list_index_length(P)]; workspace:
    at least B * bfasgd_workspace_bytes(P) bytes."""
    import torch
    B = len(grads)
    if len(T) != B or len(clients) != B:
        raise ValueError("grads, T and clients must have the same length")
    if not 1 <= B <= FASGD_MAX_BATCH:
        raise ValueError(f"B = {B} is not in [1, {FASGD_MAX_BATCH}]")
    cap = _batch_lists(B, out_idx, out_val, d_count)
    ptrs = (ctypes.c_void_p * B)()
    for k, g in enumerate(grads):
        if g.numel() != state.P:
            raise ValueError(f"grads[{k}] has {g.numel()} elements, P = {state.P}")
        ptrs[k] = _dev_ptr(g, torch.float32, f"grads[{k}]")
    ts = (ctypes.c_int64 * B)(*[int(x) for x in T])
    cl = (ctypes.c_int32 * B)(*[int(x) for x in clients])
    rc = load_library().bfasgd_select_compact_batch(
        ctypes.byref(state.c), B, ptrs, c, eps_c, int(seed) & (2 ** 64 - 1), ts, cl,
        _dev_ptr(out_idx, torch.int32, "out_idx"), _dev_ptr(out_val, torch.float32, "out_val"), cap,
        _dev_ptr(d_count, torch.int64, "d_count"), _batch_seg(seg_start, B, state.P, False),
        _dev_ptr(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream))
    _check(rc)


def fasgd_apply_pushes(state: State, idx, val, d_count, seg_start, clients: Sequence[int], grad_ts: Sequence[int],
                       stream=None) -> None:
    """B compacted pushes ([B, capacity] lists with their [B, L] index) in one
    pass, as B bfasgd_apply_sparse calls in order; T advances by B."""
    import torch
    B = len(clients)
    if len(grad_ts) != B:
        raise ValueError("clients and grad_ts must have the same length")
    if not 1 <= B <= FASGD_MAX_BATCH:
        raise ValueError(f"B = {B} is not in [1, {FASGD_MAX_BATCH}]")
    cap = _batch_lists(B, idx, val, d_count)
    cl = (ctypes.c_int32 * B)(*[int(x) for x in clients])
    ts = (ctypes.c_int64 * B)(*[int(x) for x in grad_ts])
    rc = load_library().fasgd_apply_pushes(
        ctypes.byref(state.c), B, _dev_ptr(idx, torch.int32, "idx"), _dev_ptr(val, torch.float32, "val"),
        _dev_ptr(d_count, torch.int64, "d_count"), _batch_seg(seg_start, B, state.P, True), cap, cl, ts,
        _stream(stream))
    _check(rc)


def fasgd_apply_with_push_and_select(state: State, push_idx, push_val, push_count, push_seg_start,
                                     push_client: int, push_grad_ts: int, grads: Sequence, clients: Sequence[int],
                                     grad_ts: Sequence[int], next_grad, next_client: int, c: float, eps_c: float,
                                     seed: int, out_idx, out_val, out_count, out_seg_start, workspace,
                                     stream=None) -> None:
    """fasgd_apply_with_push, then the next push's selection (as
    bfasgd_select_compact at the timestamp after the pass, from the v the
    pass leaves) in one call; the output list may be the input push's
    buffers.  T advances by K + 1."""
    import torch
    cap = push_idx.numel()
    if push_val.numel() != cap:
        raise ValueError("push_idx and push_val must have the same capacity")
    out_cap = out_idx.numel()
    if out_val.numel() != out_cap:
        raise ValueError("out_idx and out_val must have the same capacity")
    if next_grad.numel() != state.P:
        raise ValueError("next_grad length differs from P")
    ptrs, cl, t, K = _dense_args(state, grads, clients, grad_ts)
    rc = load_library().fasgd_apply_with_push_and_select(
        ctypes.byref(state.c), _dev_ptr(push_idx, torch.int32, "push_idx"),
        _dev_ptr(push_val, torch.float32, "push_val"), _dev_ptr(push_count, torch.int64, "push_count"),
        _seg_start_ptr(push_seg_start, state.P, required=True), cap, int(push_client), int(push_grad_ts),
        ptrs, cl, t, K, _dev_ptr(next_grad, torch.float32, "next_grad"), int(next_client), c, eps_c,
        int(seed) & (2 ** 64 - 1), _dev_ptr(out_idx, torch.int32, "out_idx"),
        _dev_ptr(out_val, torch.float32, "out_val"), out_cap, _dev_ptr(out_count, torch.int64, "out_count"),
        _seg_start_ptr(out_seg_start, state.P), _dev_ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
        _stream(stream))
    _check(rc)


def fasgd_record_next_pass(start, stop) -> None:
    """Record two events around the next FASGD pass kernel this thread
    launches (diagnostics; both None clears): torch.cuda.Events (recorded
    once here first, so that torch has created them) or raw hipEvent_t
    handles (anything int() gives the handle of)."""
    if start is None and stop is None:
        _check(load_library().fasgd_record_next_pass(None, None))
        return
    if hasattr(start, "cuda_event"):
        start.record()
        stop.record()
        start, stop = start.cuda_event, stop.cuda_event
    _check(load_library().fasgd_record_next_pass(int(start), int(stop)))


def fasgd_copy_anchor(src, dst, stream=None) -> None:
    """Diagnostics: dst[:] = src[:] by the library's plain streaming copy
    (the bandwidth anchor); float32 tensors of one length, 16-byte aligned."""
    import torch
    if src.numel() != dst.numel():
        raise ValueError("src and dst differ in length")
    _check(load_library().fasgd_copy_anchor(_dev_ptr(src, torch.float32, "src"), _dev_ptr(dst, torch.float32, "dst"),
                                            src.numel(), _stream(stream)))


def fasgd_check_ieee_sequences(gamma: float, beta: float, eps: float, alpha: float, seed: int, n_updates: int,
                               mismatches, stream=None) -> None:
    """Diagnostics: compare, on the device, the IEEE update's short correctly
    rounded sequences with the general ones, bit for bit; the four mismatch
    counts go to `mismatches` (int64 [4], device): square root, 1/sqrt, the
    division alpha / d over every d, and n_updates whole updates."""
    import torch
    if mismatches.numel() < 4:
        raise ValueError("mismatches needs 4 counters")
    _check(load_library().fasgd_check_ieee_sequences(gamma, beta, eps, alpha, int(seed) & (2 ** 64 - 1),
                                                      int(n_updates),
                                                      _dev_ptr(mismatches, torch.int64, "mismatches"),
                                                      _stream(stream)))


def bfasgd_apply_sparse(state: State, idx, val, d_count, client: int, grad_ts: int, stream=None) -> None:
    """FASGD update of the listed parameters (first *d_count entries); T advances by one."""
    import torch
    cap = idx.numel()
    if val.numel() != cap:
        raise ValueError("idx and val must have the same capacity")
    rc = load_library().bfasgd_apply_sparse(
        ctypes.byref(state.c), _dev_ptr(idx, torch.int32, "idx"), _dev_ptr(val, torch.float32, "val"),
        _dev_ptr(d_count, torch.int64, "d_count"), cap, int(client), int(grad_ts), _stream(stream))
    _check(rc)


def sgd_sync_apply(state: State, grads: Sequence, lr: float, stream=None) -> None:
    """Synchronous SGD step with the gradients of all lambda clients; T advances by one."""
    import torch
    if len(grads) != int(state.c.lambda_):
        raise ValueError(f"{len(grads)} gradients for lambda = {state.c.lambda_} clients")
    ptrs = (ctypes.c_void_p * len(grads))()
    for k, g in enumerate(grads):
        if g.numel() != state.P:
            raise ValueError(f"grads[{k}] has {g.numel()} elements, P = {state.P}")
        ptrs[k] = _dev_ptr(g, torch.float32, f"grads[{k}]")
    _check(load_library().sgd_sync_apply(ctypes.byref(state.c), ptrs, lr, _stream(stream)))


def bfasgd_apply_cached(state: State, idx, val, d_count, cache, client: int, grad_ts: int, seg_start=None,
                        stream=None) -> None:
    """Push with dropped values re-applied from the client's cache (updated in
    place).  seg_start (optional): the list's index from the selection, with
    which the list is merged into the cache inside the one pass."""
    import torch
    cap = idx.numel()
    if val.numel() != cap:
        raise ValueError("idx and val must have the same capacity")
    if cache.numel() != state.P:
        raise ValueError("cache length differs from P")
    rc = load_library().bfasgd_apply_cached(
        ctypes.byref(state.c), _dev_ptr(idx, torch.int32, "idx"), _dev_ptr(val, torch.float32, "val"),
        _dev_ptr(d_count, torch.int64, "d_count"), _seg_start_ptr(seg_start, state.P), cap,
        _dev_ptr(cache, torch.float32, "cache"), int(client), int(grad_ts), _stream(stream))
    _check(rc)


def bfasgd_apply_fetch(theta_client, idx, val, d_count, seg_start=None, stream=None) -> None:
    """Copy the listed values into a client's copy of theta.  seg_start
    (optional): the list's index, with which segments holding an entry are
    rewritten whole (faster when most segments hold one)."""
    import torch
    cap = idx.numel()
    if val.numel() != cap:
        raise ValueError("idx and val must have the same capacity")
    rc = load_library().bfasgd_apply_fetch(
        _dev_ptr(theta_client, torch.float32, "theta_client"), theta_client.numel(),
        _dev_ptr(idx, torch.int32, "idx"), _dev_ptr(val, torch.float32, "val"),
        _dev_ptr(d_count, torch.int64, "d_count"), _seg_start_ptr(seg_start, theta_client.numel()), cap,
        _stream(stream))
    _check(rc)


def _seg_array(seg):
    import numpy as np
    a = np.ascontiguousarray(seg, dtype=np.int64)
    return a, a.ctypes.data_as(ctypes.c_void_p), a.size - 1


def bfasgd_segments_workspace_bytes(P: int, S: int) -> int:
    return int(load_library().bfasgd_segments_workspace_bytes(int(P), int(S)))


def bfasgd_decide_segments(state: State, seg, c: float, eps_c: float, seed: int, T: int, client: int,
                           d_transmit, workspace, stream=None) -> None:
    """Paper-literal decisions, one per segment of `seg` (host offsets, S + 1
    of them), into d_transmit (device uint8 [S])."""
    import torch
    arr, ptr, S = _seg_array(seg)
    if d_transmit.numel() != S:
        raise ValueError("d_transmit needs one entry per segment")
    rc = load_library().bfasgd_decide_segments(
        ctypes.byref(state.c), ptr, S, c, eps_c, int(seed) & (2 ** 64 - 1), int(T), int(client),
        _dev_ptr(d_transmit, torch.uint8, "d_transmit"), _dev_ptr(workspace, torch.uint8, "workspace"),
        workspace.numel(), _stream(stream))
    _check(rc)


def bfasgd_apply_segments(state: State, grad, seg, d_transmit, client: int, grad_ts: int, stream=None) -> None:
    """FASGD update on the transmitted segments; T advances by one."""
    import torch
    arr, ptr, S = _seg_array(seg)
    if grad.numel() != state.P:
        raise ValueError("grad length differs from P")
    rc = load_library().bfasgd_apply_segments(
        ctypes.byref(state.c), _dev_ptr(grad, torch.float32, "grad"), ptr, S,
        _dev_ptr(d_transmit, torch.uint8, "d_transmit"), int(client), int(grad_ts), _stream(stream))
    _check(rc)


def allocate_state(P: int, device="cuda", with_stats: bool = True):
    """Device tensors for a state of P parameters (torch allocations are
    256-byte aligned, so the vectorised kernels are used)."""
    import torch
    f = dict(device=device, dtype=torch.float32)
    theta = torch.empty(P, **f)
    n = torch.empty(P, **f) if with_stats else None
    b = torch.empty(P, **f) if with_stats else None
    v = torch.empty(P, **f) if with_stats else None
    last_T = torch.empty(P, device=device, dtype=torch.int32)
    return theta, n, b, v, last_T


def allocate_workspace(P: int, device="cuda"):
    import torch
    return torch.empty(bfasgd_workspace_bytes(P), device=device, dtype=torch.uint8)
