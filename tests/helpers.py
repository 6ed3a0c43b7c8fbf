"""Shared helpers for the GPU parity tests (GPU path through the C ABI vs the CPU oracle)."""
import numpy as np
import pytest

import paper_1601_04033_amd as fa

# Tolerances fixed for this path: after one update, relative 1e-5 with an
# absolute floor of 1e-6; after a whole update sequence, relative 1e-4 with
# the same floor.
RTOL_ONE, ATOL = 1e-5, 1e-6
RTOL_SEQ = 1e-4

STATE_FIELDS = ("theta", "n", "b", "v")


def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    fa.load_library()          # raises if the HIP library is not built
    return torch.device("cuda:0")


def to_dev(a, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def assert_close(got, want, rtol, atol=ATOL, what=""):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    err = np.abs(got - want)
    bound = atol + rtol * np.abs(want)
    bad = np.flatnonzero(~(err <= bound))
    if bad.size:
        i = bad[np.argmax((err - bound)[bad])]
        raise AssertionError(f"{what}: {bad.size}/{got.size} outside rtol={rtol} atol={atol}; "
                             f"worst index {i}: got {got[i]!r} want {want[i]!r}")


def assert_state_close(st_gpu, ref, rtol, js=None, what=""):
    """Compare theta, n, b, v (and last_T exactly) of a GPU state with an
    oracle state; js selects the compared indices of the GPU state."""
    for name in STATE_FIELDS:
        t = st_gpu.tensors[name]
        got = (t[js] if js is not None else t).cpu().numpy()
        assert_close(got, getattr(ref, name), rtol, ATOL, f"{what} {name}")
    lt = st_gpu.last_update()            # max(last_T, dense_T)
    got = (lt[js] if js is not None else lt).cpu().numpy()
    np.testing.assert_array_equal(got.astype(np.int64), ref.last_T, err_msg=f"{what} last update")
    assert st_gpu.T == ref.T


def new_gpu_state(theta0, dev, lam, alpha, mode, gamma=0.95, beta=0.9, eps=1e-4, v0=0.0, sasgd=False,
                  v_reading=0):
    import torch
    P = theta0.shape[0] if hasattr(theta0, "shape") else theta0.numel()
    theta, n, b, v, last_T = fa.allocate_state(P, dev, with_stats=not sasgd)
    if isinstance(theta0, np.ndarray):
        theta.copy_(torch.from_numpy(theta0))
    else:
        theta.copy_(theta0)
    return fa.fasgd_init_state(theta, n, b, v, last_T, lam=lam, alpha=alpha, gamma=gamma, beta=beta,
                               eps=eps, math_mode=mode, v0=v0, v_reading=v_reading)


def sample_indices(P, k=4096, seed=0):
    """Sorted sample: the first and last 64 indices plus k random ones."""
    rng = np.random.default_rng(seed)
    js = np.concatenate([np.arange(min(64, P)), np.arange(max(P - 64, 0), P),
                         rng.integers(0, P, size=k)])
    return np.unique(js)


def philox_r(js, seed, T, client):
    """r_j of the oracle's Philox stream for the given indices."""
    import oracle
    out = np.empty(len(js))
    for i, j in enumerate(js):
        j = int(j)
        q = j >> 2
        w = oracle.philox4x32_10([q & 0xFFFFFFFF, q >> 32, T & 0xFFFFFFFF, client],
                                 [seed & 0xFFFFFFFF, seed >> 32])[j & 3]
        out[i] = (int(w) >> 8) * 2.0 ** -24
    return out
