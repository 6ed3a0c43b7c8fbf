"""GPU: bfasgd_select_compact_noalloc (the selection with the library's
built-in per-device scratch, for callers that cannot allocate) gives the
same list, count and list index, bit for bit, as bfasgd_select_compact with
a caller workspace.  Several calls in a row share the scratch, each smaller
than the one before, so a call that depended on what the previous call left
there would show it."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_1601_04033_amd as fa
import workload
from helpers import gpu, new_gpu_state, to_dev

pytestmark = pytest.mark.gpu

SEED = 0x5EED0F5C7A7C4


def _outputs(P, cap, dev):
    import torch
    idx = torch.full((max(cap, 1),), -7, device=dev, dtype=torch.int32)[:cap]
    val = torch.full((max(cap, 1),), -7.0, device=dev)[:cap]
    cnt = torch.full((1,), -1, device=dev, dtype=torch.int64)
    seg = torch.full((fa.bfasgd_list_index_length(P),), -7, device=dev, dtype=torch.int32)
    return idx, val, cnt, seg


def _host(idx, val, cnt, seg, cap):
    import torch
    torch.cuda.synchronize()
    m = int(cnt.item())
    k = min(m, cap)
    return m, idx[:k].cpu().numpy(), val[:k].cpu().numpy().view(np.uint32), seg.cpu().numpy()


def _state(P, dev, seed):
    import torch
    st = new_gpu_state(np.zeros(P, np.float32), dev, 16, 0.005, fa.MATH_FAST)
    st.v.copy_(torch.from_numpy(workload.synthetic_v(P, seed=seed)))
    return st


# (P, threshold c, capacity as a fraction of P): the largest P the scratch
# holds, then smaller calls (a ragged size, a capacity cut, a tiny one).
CASES = [(fa.FASGD_NOALLOC_MAX_P, 60.0, 1.0), (1_796_010, 40.0, 1.0), (100_003, 40.0, 0.02), (5, 0.0, 1.0)]


def test_noalloc_selection_equals_workspace_selection():
    import torch
    dev = gpu()
    for i, (P, c, capf) in enumerate(CASES):
        print(f"noalloc case {i}: P={P} c={c} capacity={capf}", flush=True)
        st = _state(P, dev, seed=P)
        g = torch.randn(P, device=dev, generator=torch.Generator(device=dev).manual_seed(P))
        cap = max(int(P * capf), 1)
        T, client = 3 + i, i % 16
        a = _outputs(P, cap, dev)
        ws = fa.allocate_workspace(P, dev)
        fa.bfasgd_select_compact(st, g, c, 1e-8, SEED, T, client, a[0], a[1], a[2], ws, seg_start=a[3])
        want = _host(*a, cap)
        b = _outputs(P, cap, dev)
        fa.bfasgd_select_compact_noalloc(st, g, c, 1e-8, SEED, T, client, b[0], b[1], b[2], seg_start=b[3])
        got = _host(*b, cap)
        assert got[0] == want[0], (P, got[0], want[0])
        for x, y, what in zip(got[1:], want[1:], ("idx", "val bits", "list index")):
            np.testing.assert_array_equal(x, y, err_msg=f"P={P} {what}")
        if P <= 2_000_000:
            # and the oracle's list, from the same v and gradient
            r_idx, r_val, r_m = oracle.bfasgd_select(st.v.cpu().numpy(), g.cpu().numpy(), c, 1e-8, SEED, T,
                                                     client, capacity=cap)
            assert got[0] == r_m
            np.testing.assert_array_equal(got[1], r_idx)
            np.testing.assert_array_equal(got[2], r_val.view(np.uint32))
        if c == 0.0:
            assert got[0] == P
        del ws


def test_noalloc_rejects_more_than_its_scratch_holds():
    import torch
    dev = gpu()
    P = fa.FASGD_NOALLOC_MAX_P + 1
    st = _state(8, dev, seed=1)
    st.c.P = P                  # only the size check runs: nothing is launched
    idx, val, cnt, seg = _outputs(8, 8, dev)
    g = torch.zeros(8, device=dev)
    rc = fa.load_library().bfasgd_select_compact_noalloc(
        ctypes.byref(st.c), g.data_ptr(), 1.0, 1e-8, 1, 0, 0, idx.data_ptr(), val.data_ptr(), 8,
        cnt.data_ptr(), None, None)
    assert rc == 6 and b"exceeds" in fa.load_library().fasgd_last_error()
    torch.cuda.synchronize()
    assert int(cnt.item()) == -1
