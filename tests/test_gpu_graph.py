"""The library's calls captured in a HIP graph: every replay gives what the
same calls give eagerly, bit for bit (the calls enqueue kernels only: no
allocation, no host synchronisation, no memset node).  Each replay is
followed by eager work of the program's own and a synchronisation, and is
checked against eager calls made with the same arguments."""
import numpy as np
import pytest

import paper_1601_04033_amd as fa
import workload
from helpers import gpu

pytestmark = pytest.mark.gpu
SEED = 0x6EA9


def _pair(P, dev, seed):
    """Two identical mid-run states (T = 30)."""
    import torch
    w = workload.WORKLOADS["mlp_bfasgd"]
    theta0, m_, s_ = workload.host_params(w, P, seed=seed)
    v0 = workload.synthetic_v(P, seed=seed, lo=5.0, hi=100.0)
    out = []
    for _ in range(2):
        theta, n, b, v, last_T = fa.allocate_state(P, dev)
        st = fa.fasgd_init_state(theta, n, b, v, last_T, lam=w.lam, alpha=w.alpha_fasgd)
        theta.copy_(torch.from_numpy(theta0))
        n.copy_(torch.from_numpy((m_ * m_ + s_ * s_).astype(np.float32)))
        b.copy_(torch.from_numpy(m_))
        v.copy_(torch.from_numpy(v0))
        st.c.T = 30
        out.append(st)
    grads = [torch.from_numpy(workload.host_gradient(w, m_, s_, t, seed=seed)).to(dev) for t in range(8)]
    return out[0], out[1], grads, w


def _same(a, b, what):
    import torch
    for name in ("theta", "n", "b", "v", "last_T"):
        assert torch.equal(a.tensors[name].view(torch.int32), b.tensors[name].view(torch.int32)), f"{what}: {name}"


def test_replayed_push_batches_and_dense_passes_match_eager():
    """One graph holding a batched selection, the batched apply, a K = 4
    FASGD pass, a selection with its list index, the pass that applies that
    push before 2 more gradients, and the pass that applies the same list
    before 3 more and selects the next push into those buffers; replayed
    three times."""
    import torch
    dev = gpu()
    P, B = 200_003, 4
    gs, es, grads, w = _pair(P, dev, seed=4)
    L = fa.bfasgd_list_index_length(P)

    def buffers():
        return dict(idx=torch.zeros((B, P), device=dev, dtype=torch.int32), val=torch.zeros((B, P), device=dev),
                    cnt=torch.zeros(B, device=dev, dtype=torch.int64),
                    seg=torch.zeros((B, L), device=dev, dtype=torch.int32),
                    ws=torch.empty(B * fa.bfasgd_workspace_bytes(P), device=dev, dtype=torch.uint8))
    gb, eb = buffers(), buffers()
    clients = [k % w.lam for k in range(B)]

    def calls(st, bf, T0):
        """The calls, at timestamps from T0 (the host state's T and dense_T
        reset first, so every eager round repeats the captured arguments)."""
        st.c.T = T0
        st.c.dense_T = -1
        fa.bfasgd_select_compact_batch(st, grads[:B], 80.0, 1e-8, SEED, [T0 + k for k in range(B)], clients,
                                       bf["idx"], bf["val"], bf["cnt"], bf["ws"], seg_start=bf["seg"])
        fa.fasgd_apply_pushes(st, bf["idx"], bf["val"], bf["cnt"], bf["seg"], clients, [T0 - 2] * B)
        T = st.T
        fa.fasgd_apply_updates(st, grads[4:8], [0, 1, 2, 3], [T - 1, T - 3, T, T - 2])
        T = st.T
        fa.bfasgd_select_compact(st, grads[0], 40.0, 1e-8, SEED, T, 5, bf["idx"][0], bf["val"][0],
                                 bf["cnt"][0:1], bf["ws"], seg_start=bf["seg"][0])
        fa.fasgd_apply_with_push(st, bf["idx"][0], bf["val"][0], bf["cnt"][0:1], bf["seg"][0], 5, T - 1,
                                 grads[1:3], [6, 7], [T, T - 1])
        T = st.T
        fa.fasgd_apply_with_push_and_select(st, bf["idx"][0], bf["val"][0], bf["cnt"][0:1], bf["seg"][0], 8, T - 3,
                                            grads[3:6], [1, 2, 3], [T, T, T - 2], grads[6], 9, 40.0, 1e-8, SEED,
                                            bf["idx"][0], bf["val"][0], bf["cnt"][0:1], bf["seg"][0], bf["ws"])

    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        calls(gs, gb, 30)
    T_after = gs.T
    torch.cuda.synchronize()
    scratch = torch.randn(1 << 20, device=dev)
    for r in range(3):
        graph.replay()
        scratch.mul_(1.0001).add_(1.0)           # the program's own eager work between replays
        torch.cuda.synchronize()
        calls(es, eb, 30)
        torch.cuda.synchronize()
        assert es.T == T_after
        _same(gs, es, f"replay {r}")
        for key in ("cnt", "seg"):
            assert torch.equal(gb[key], eb[key]), f"replay {r}: {key}"
        for k in (0, 1):
            m = int(eb["cnt"][k].item())
            assert torch.equal(gb["idx"][k, :m], eb["idx"][k, :m]), f"replay {r}: list {k}"
