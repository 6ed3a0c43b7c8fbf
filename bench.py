"""Benchmark of the FASGD parameter-server step on one MI355X.

One step = the whole server path over one batch of client gradients:
  1. fasgd_apply_with_push  one pass that applies the B-FASGD push selected
                            in the previous step (Sec. 2.3) and then K client
                            gradients (dense FASGD, eqs. of Sec. 2.2, K-fold
                            state reuse);
  2. bfasgd_select_compact  the next client's push: per-parameter send/skip
                            and compaction into (index, value) lists.
Inputs (state and a pool of K + 1 distinct synthetic gradients) are resident
in HBM before timing; every step uses fresh (client, timestamp) pairs.

Prints ONE JSON line.  value = parameter updates applied per second
(P*K dense + m sparse per step).  roofline = the fused pass's algorithmic
HBM bytes per launch over its average event-timed duration.  Further legs,
timed after the step, cover the other entry points and the small workloads
(100k parameters; the 784-1000-1000-10 MLP's 1.8M, with B-FASGD pushes
handled one by one or in batches), eagerly and as replayed HIP graphs.
"""
import argparse
import ctypes
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "param-updates/sec and achieved HBM GB/s (% of peak), FASGD apply at 25M/1B params"
HBM_PEAK_GBS = 8000.0
EPS_C = 1e-8
SEED = 0x5EED
# rocprofv3 counter summaries of the step's pass, per workload
PMC_SUMMARIES = {"memscale": os.path.join(ROOT, "profiles", "fasgd_dense_push_k32_memscale_1e9_pmc.txt"),
                 "large": os.path.join(ROOT, "profiles", "fasgd_dense_push_k32_large_25m_pmc.txt")}
DENSE_SOURCES = [os.path.join(ROOT, "paper_1601_04033_amd", "csrc", f)
                 for f in ("dense.hip", "device_math.hpp", "kernels.hpp")]


def dense_source_hash():
    """Hash of the code of the profiled pass (its sources with comments and
    whitespace removed, so that an edited comment keeps the counters valid)."""
    h = hashlib.sha256()
    for f in DENSE_SOURCES:
        with open(f) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update("".join(text.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload_name, P, K, math="fast"):
    """HBM bytes per launch of the step's pass from the committed rocprofv3
    counter summary of the workload, or None when it is absent, of another
    shape or math mode (the counters were taken in fast math), or the kernel
    changed since."""
    if math != "fast":
        return None
    path = PMC_SUMMARIES.get(workload_name)
    if path is None or not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"source_hash:\s*([0-9a-f]+)", text)
    m_bytes = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    m_shape = re.search(r"shape:\s*P=(\d+)\s+K=(\d+)", text)
    if not (m_hash and m_bytes and m_shape) or m_hash.group(1) != dense_source_hash():
        return None
    if int(m_shape.group(1)) != P or int(m_shape.group(2)) != K:
        return None
    return float(m_bytes.group(1))


def calibrate_c(v, target, n=1 << 20):
    """Threshold c with mean_j t_j/(t_j + c) = target over a sample of v."""
    import numpy as np
    import torch
    P = v.numel()
    g = torch.Generator(device=v.device)
    g.manual_seed(1)
    sample = v[torch.randint(0, P, (min(n, P),), device=v.device, generator=g)]
    t = sample.double().cpu().numpy() + EPS_C
    lo, hi = 0.0, 1e9
    for _ in range(200):
        c = 0.5 * (lo + hi)
        lo, hi = (c, hi) if (t / (t + c)).mean() > target else (lo, c)
    return float(np.float32(c))


def fetch_copy_by_segments(P, m):
    """The rule bfasgd_apply_fetch's header states for its optional list
    index: copy by segments when the client's copy does not fit the 256 MB
    Infinity Cache and the transmitted fraction is above a few percent (most
    segments then hold an entry), otherwise scatter one value per entry."""
    return 4 * P > 256 * 2 ** 20 and m >= 0.05 * P


def host_cpu():
    """The host's CPU model (from /proc/cpuinfo), its logical CPU count and
    the CPUs this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, os.cpu_count(), sorted(os.sched_getaffinity(0))


def _oracle_step(theta0, grads, clients, ts, c, w, K, index_base=0):
    """One step of the oracle on a slice: K dense updates, the selection of
    one push (decided from the slice's global indices), its sparse apply."""
    import numpy as np
    import oracle
    st = oracle.init_state(theta0, alpha=w.alpha_fasgd)
    for k in range(K):
        oracle.fasgd_apply(st, grads[k], ts[k])
    idx, val, m = oracle.bfasgd_select(st.v.astype(np.float32), grads[K], c, EPS_C, SEED, st.T, clients[K],
                                       index_base=index_base)
    oracle.bfasgd_apply_sparse(st, idx, val, ts[K])
    return m


def cpu_baseline(pool, theta0_host, clients, ts, c, w, K, P_s):
    """The oracle (single-threaded C, fp64) on the first P_s parameters of the
    same step (K dense updates, one selection, one sparse apply), with the
    calling thread pinned to one CPU; then the same function on all the CPUs
    this process may use, each thread on its own slice of the index range (the
    updates are elementwise and the decisions keyed by the global index, so
    the slices together do exactly the work of the whole)."""
    from concurrent.futures import ThreadPoolExecutor
    model, n_cpu, allowed = host_cpu()
    grads = [g[:P_s].cpu().numpy() for g in pool]
    theta0 = theta0_host[:P_s]
    core = allowed[-1]
    os.sched_setaffinity(0, {core})          # this thread only: the oracle runs on it
    try:
        t0 = time.perf_counter()
        m = _oracle_step(theta0, grads, clients, ts, c, w, K)
        dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, set(allowed))
    n_thr = len(allowed)
    bounds = [(P_s * i // n_thr) & ~3 for i in range(n_thr)] + [P_s]

    def part(i):
        a, b = bounds[i], bounds[i + 1]
        return _oracle_step(theta0[a:b], [g[a:b] for g in grads], clients, ts, c, w, K, index_base=a)

    t0 = time.perf_counter()
    with ThreadPoolExecutor(n_thr) as ex:
        m_all = sum(ex.map(part, range(n_thr)))
    dt_all = time.perf_counter() - t0
    assert m_all == m, (m_all, m)
    return {"value": (P_s * K + m) / dt, "seconds": dt, "transmitted": m, "pinned_core": core,
            "host_logical_cpus": n_cpu, "cpus_available": n_thr, "cpu_model": model,
            "all_cores": {"value": (P_s * K + m) / dt_all, "threads": n_thr, "seconds": dt_all}}


HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000   # hipEventDisableSystemFence


class TimingEvent:
    """A HIP event for timing only, created with hipEventDisableSystemFence:
    recording it writes a timestamp without the system-scope cache writeback
    and invalidation that a default event (torch.cuda.Event) performs, which
    between back-to-back kernels costs several microseconds per record.  Used
    for the per-step events inside the timed loop; the timed region itself
    is bracketed by default events and synchronisations.  The HIP runtime is
    the one libfasgd.so runs on (its symbols are looked up through the
    library's handle)."""
    _hip = None

    def __init__(self, fa):
        if TimingEvent._hip is None:
            hip = fa.load_library()
            vp = ctypes.c_void_p
            hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp), ctypes.c_uint]
            hip.hipEventRecord.argtypes = [vp, vp]
            hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
            hip.hipEventDestroy.argtypes = [vp]
            TimingEvent._hip = hip
        self.handle = ctypes.c_void_p()
        rc = TimingEvent._hip.hipEventCreateWithFlags(ctypes.byref(self.handle), HIP_EVENT_DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")

    def __int__(self):
        return int(self.handle.value)

    def record(self):
        import torch
        rc = TimingEvent._hip.hipEventRecord(self.handle, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_time(self, end):
        ms = ctypes.c_float()
        rc = TimingEvent._hip.hipEventElapsedTime(ctypes.byref(ms), self.handle, end.handle)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(ms.value)

    def __del__(self):
        if TimingEvent._hip is not None and self.handle:
            TimingEvent._hip.hipEventDestroy(self.handle)


GROUPS = 5   # back-to-back groups per figure; the median of their per-call means is reported


def grouped_b2b(torch, fn, count, groups=GROUPS):
    """Per-call ms of `groups` groups of `count` back-to-back calls, each
    group between two events (after one untimed call): the median of the
    groups' per-call means, and their range."""
    fn()
    means = []
    for _ in range(groups):
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(count):
            fn()
        e.record()
        torch.cuda.synchronize()
        means.append(a.elapsed_time(e) / count)
    return float(statistics.median(means)), [float(min(means)), float(max(means))]


# Calls per back-to-back group at 25M parameters, so that every group holds
# 5 ms or more of GPU work: the two events around a group (each a
# system-scope cache writeback) and the first call's ramp then add well
# under 1 % per call.  With 20 selections (0.8 ms) per group they added
# about 0.5 us to each 38 us call.
DENSE_25M_CALLS = {1: 40, 8: 20, 32: 10}
SELECT_25M_CALLS = 128


def large_25m(fa, workload, dev, mode, K=32, reps=20):
    """The 25M-parameter workload (50 blocks of 500k, lambda = 64) beside the
    main one: the dense pass at K = 1, 8, 32, the server's step (one
    fasgd_apply_with_push_and_select call: a 10 % push and K gradients in one
    pass that also takes the next push's decisions, then its compaction) and
    the selection on its own, each over calls issued back to back.  Fractions
    are algorithmic bytes over time against 8 TB/s."""
    import torch
    w = workload.WORKLOADS["large"]
    P = w.P
    theta0, m, s = workload.device_params(w, dev)
    pool = [workload.device_gradient(w, m, s, t) for t in range(K + 1)]
    del m, s
    theta, n, b, v, last_T = fa.allocate_state(P, dev)
    theta.copy_(theta0)
    del theta0
    st = fa.fasgd_init_state(theta, n, b, v, last_T, lam=w.lam, alpha=w.alpha_fasgd, math_mode=mode)
    dense_updates = sum((GROUPS * n_calls + 1) * k for k, n_calls in DENSE_25M_CALLS.items())
    clients, ts = workload.schedule(w, K + dense_updates + (GROUPS * reps + 4) * (K + 1) + 64)
    idx = torch.empty(P, device=dev, dtype=torch.int32)
    val = torch.empty(P, device=dev)
    cnt = torch.zeros(1, device=dev, dtype=torch.int64)
    seg = torch.empty(fa.bfasgd_list_index_length(P), device=dev, dtype=torch.int32)
    ws = fa.allocate_workspace(P, dev)
    fa.fasgd_apply_updates(st, pool[:K], clients[:K], ts[:K])
    torch.cuda.synchronize()
    c = calibrate_c(v, w.transmit_fraction or 0.1)

    def b2b(fn, count):
        return grouped_b2b(torch, fn, count)

    out = {"P": P, "lambda": w.lam, "dense": {}}
    for k, n_calls in DENSE_25M_CALLS.items():
        def dense(k=k):
            T = st.T
            fa.fasgd_apply_updates(st, pool[:k], clients[T:T + k], ts[T:T + k])
        ms, spread = b2b(dense, n_calls)
        out["dense"][f"K={k}"] = {"ms": ms, "frac": P * (32 + 4 * k) / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                                  "ms_range": spread}
    # the server's step, its pass timed alone with events around the kernel
    T = st.T
    fa.bfasgd_select_compact(st, pool[K], c, EPS_C, SEED, T, clients[T], idx, val, cnt, ws, seg_start=seg)
    passes = []

    def step():
        T = st.T
        p0, p1 = TimingEvent(fa), TimingEvent(fa)
        fa.fasgd_record_next_pass(p0, p1)
        fa.fasgd_apply_with_push_and_select(st, idx, val, cnt, seg, clients[T], ts[T], pool[:K],
                                            clients[T + 1:T + 1 + K], ts[T + 1:T + 1 + K], pool[K],
                                            clients[T + K + 1], c, EPS_C, SEED, idx, val, cnt, seg, ws)
        passes.append((p0, p1))
    step_ms, step_spread = b2b(step, reps)
    torch.cuda.synchronize()
    pass_ms = sum(a.elapsed_time(e) for a, e in passes[1:]) / len(passes[1:])
    m = int(cnt.item())
    pass_bytes = P * (32 + 4 * K) + 8 * m + 4 * fa.bfasgd_list_index_length(P) + P / 8
    out["step"] = {"ms": step_ms, "ms_range": step_spread, "param_updates_per_s": (P * K + m) / (step_ms * 1e-3),
                   "pass_ms": pass_ms, "pass_frac": pass_bytes / (pass_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                   "transmitted_fraction": m / P}
    T = st.T
    fa.bfasgd_apply_sparse(st, idx, val, cnt, clients[T], ts[T])
    sel_ms, sel_spread = b2b(lambda: fa.bfasgd_select_compact(st, pool[K], c, EPS_C, SEED, st.T, clients[st.T], idx,
                                                              val, cnt, ws), SELECT_25M_CALLS)
    m = int(cnt.item())
    out["bfasgd_select_compact"] = {"ms": sel_ms, "frac": (8 * P + 8 * m) / (sel_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                                    "ms_range": sel_spread}
    return out


def small_configs(fa, workload, dev, mode, B=16, reps=20):
    """The small workloads, whose state fits the 256 MB Infinity Cache (so
    their GB/s are 'effective', not HBM): the tiny trace (100k parameters,
    K = 1, FASGD and SASGD), the MLP-shaped FASGD pass (1.8M parameters,
    K = 16) and MLP-sized B-FASGD (about 20 % per push), with B pushes handled
    one by one (a selection and a sparse apply each) or batched
    (bfasgd_select_compact_batch, then fasgd_apply_pushes; the same state).
    Each operation is timed over `reps` calls issued back to back by the host
    and over the same calls captured in one HIP graph and replayed, which
    takes the host's per-call work and most launch gaps out."""
    import torch

    def eager_ms(fn):
        fn()
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        e.record()
        torch.cuda.synchronize()
        return a.elapsed_time(e) / reps

    def graph_ms(fn):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                fn()
        g.replay()
        torch.cuda.synchronize()
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        g.replay()
        e.record()
        torch.cuda.synchronize()
        return a.elapsed_time(e) / reps

    def measure(fn, nbytes, updates):
        ea, gr = eager_ms(fn), graph_ms(fn)
        return {"us_eager": ea * 1e3, "us_graph": gr * 1e3, "GB/s_effective": nbytes / (gr * 1e-3) / 1e9,
                "param_updates_per_s": updates / (gr * 1e-3)}

    def new_state(w, sasgd=False):
        theta0, m_, s_ = workload.host_params(w)
        theta, n, b, v, last_T = fa.allocate_state(w.P, dev, with_stats=not sasgd)
        theta.copy_(torch.from_numpy(theta0))
        st = fa.fasgd_init_state(theta, n, b, v, last_T, lam=w.lam,
                                 alpha=w.alpha_sasgd if sasgd else w.alpha_fasgd, math_mode=mode)
        return st, m_, s_

    out = {}
    # tiny trace: K = 1 passes
    w = workload.WORKLOADS["tiny"]
    n_calls = 2 * reps + 4
    for name, sasgd in (("tiny_fasgd_k1", False), ("tiny_sasgd_k1", True)):
        st, m_, s_ = new_state(w, sasgd)
        g1 = torch.from_numpy(workload.host_gradient(w, m_, s_, 0)).to(dev)
        clients, ts = workload.schedule(w, n_calls)
        call = fa.sasgd_apply_updates if sasgd else fa.fasgd_apply_updates

        def one(st=st, g1=g1, clients=clients, ts=ts, call=call):
            T = st.T
            call(st, [g1], clients[T:T + 1], ts[T:T + 1])
        out[name] = measure(one, w.P * (12 if sasgd else 36), w.P)
        out[name]["P"] = w.P

    # MLP-shaped FASGD: K = 16 gradients per pass
    w = workload.WORKLOADS["mlp"]
    K = 16
    st, m_, s_ = new_state(w)
    grads = [torch.from_numpy(workload.host_gradient(w, m_, s_, t)).to(dev) for t in range(K)]
    clients, ts = workload.schedule(w, K * (2 * reps + 4))

    def mlp_pass():
        T = st.T
        fa.fasgd_apply_updates(st, grads, clients[T:T + K], ts[T:T + K])
    out["mlp_fasgd_k16"] = measure(mlp_pass, w.P * (32 + 4 * K), w.P * K)
    out["mlp_fasgd_k16"].update({"P": w.P, "K": K})

    # MLP-sized B-FASGD: B pushes one by one or batched
    w = workload.WORKLOADS["mlp_bfasgd"]
    P = w.P
    st, m_, s_ = new_state(w)
    grads = [torch.from_numpy(workload.host_gradient(w, m_, s_, t)).to(dev) for t in range(B)]
    clients, ts = workload.schedule(w, B + 8 * (reps + 2) * B)
    fa.fasgd_apply_updates(st, grads, clients[:B], ts[:B])     # gives v its scale
    torch.cuda.synchronize()
    c = calibrate_c(st.v, w.transmit_fraction or 0.2)
    L = fa.bfasgd_list_index_length(P)
    idx = torch.empty((B, P), device=dev, dtype=torch.int32)
    val = torch.empty((B, P), device=dev)
    cnt = torch.zeros(B, device=dev, dtype=torch.int64)
    seg = torch.empty((B, L), device=dev, dtype=torch.int32)
    ws = torch.empty(B * fa.bfasgd_workspace_bytes(P), device=dev, dtype=torch.uint8)
    ws1 = fa.allocate_workspace(P, dev)

    def one_by_one():
        for k in range(B):
            T = st.T
            fa.bfasgd_select_compact(st, grads[k], c, EPS_C, SEED, T, clients[T], idx[k], val[k],
                                     cnt[k:k + 1], ws1)
            fa.bfasgd_apply_sparse(st, idx[k], val[k], cnt[k:k + 1], clients[T], ts[T])

    def batched_select():
        T = st.T
        fa.bfasgd_select_compact_batch(st, grads, c, EPS_C, SEED, list(range(T, T + B)), clients[T:T + B],
                                       idx, val, cnt, ws, seg_start=seg)

    def batched_apply():
        T = st.T
        fa.fasgd_apply_pushes(st, idx, val, cnt, seg, clients[T:T + B], ts[T:T + B])

    def batched():
        batched_select()
        batched_apply()

    seq = measure(one_by_one, 0, 0)
    bat = measure(batched, 0, 0)
    sel = measure(batched_select, 0, 0)
    m_avg = float(cnt.double().mean().item())
    app = measure(batched_apply, 0, 0)
    # algorithmic bytes: each selection reads v and g and writes (idx, val)
    # and its list index; the batched apply reads and writes the state once
    # (plus last_T of the listed parameters) and reads every list
    sel_bytes = B * (8 * P + 8 * m_avg + 4 * L)
    touched = P * (1.0 - (1.0 - m_avg / P) ** B)
    app_bytes = 32 * P + 4 * touched + B * (8 * m_avg + 8 * L)
    for d, nb in ((sel, sel_bytes), (app, app_bytes)):
        d["GB/s_effective"] = nb / (d["us_graph"] * 1e-6) / 1e9
    for d in (seq, bat):
        d.pop("GB/s_effective")
        d["param_updates_per_s"] = B * m_avg / (d["us_graph"] * 1e-6)
    for d in (sel, app):
        d.pop("param_updates_per_s")
    out["mlp_bfasgd_pushes"] = {
        "P": P, "B": B, "lambda": w.lam, "c": c, "transmitted_fraction": m_avg / P,
        "one_by_one": seq, "batched": bat,
        "speedup_eager": seq["us_eager"] / bat["us_eager"], "speedup_graph": seq["us_graph"] / bat["us_graph"],
        "bfasgd_select_compact_batch": sel, "fasgd_apply_pushes": app}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="memscale", choices=["memscale", "large"])
    ap.add_argument("--K", type=int, default=32)
    ap.add_argument("--math", default="fast", choices=["fast", "ieee"])
    ap.add_argument("--cpu-params", type=int, default=100_000_000,
                    help="parameters in the oracle's CPU-baseline sample (0 = skip)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this library runs on one GPU: the server update is elementwise and "
                                   "would shard by parameter range with no exchange, but no multi-GPU "
                                   "path is built; run with --gpus 1"}), flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_1601_04033_amd as fa
    import workload

    fa.load_library()
    dev = torch.device("cuda:0")
    w = workload.WORKLOADS[args.workload]
    P, K = w.P, args.K
    f = w.transmit_fraction or 0.1
    mode = fa.MATH_FAST if args.math == "fast" else fa.MATH_IEEE
    steps, warm = args.steps, args.warmup

    print(f"# setup: workload={args.workload} P={P} K={K} math={args.math}", file=sys.stderr, flush=True)
    theta0, m, s = workload.device_params(w, dev)
    theta0_host = theta0[: args.cpu_params].cpu().numpy() if args.cpu_params else None
    pool = [workload.device_gradient(w, m, s, t) for t in range(K + 1)]
    del m, s
    theta, n, b, v, last_T = fa.allocate_state(P, dev)
    theta.copy_(theta0)
    del theta0
    st = fa.fasgd_init_state(theta, n, b, v, last_T, lam=w.lam, alpha=w.alpha_fasgd, math_mode=mode)
    cap = P
    idx = torch.empty(cap, device=dev, dtype=torch.int32)
    val = torch.empty(cap, device=dev)
    cnt = torch.zeros(1, device=dev, dtype=torch.int64)
    ws = fa.allocate_workspace(P, dev)
    seg = torch.empty(fa.bfasgd_list_index_length(P), device=dev, dtype=torch.int32)
    per_step = K + 1
    # timestamps used: K (first pass) + (K + 1) per step + 1 (the last push),
    # then the legs after the timed region: 3 steps of separate calls, 3 of
    # two calls (+ 1 push), 3 SASGD passes of K, 3 cached pushes, 3 segment
    # pushes, 3 synchronous steps and the dense passes at K = 1, 8, 32 (11
    # calls each)
    KS = (1, 8, 32)
    clients, ts = workload.schedule(w, K + (warm + steps + 6) * per_step + 2 + 3 * K + 9 + 16
                                    + (GROUPS * 10 + 1) * sum(KS))
    torch.cuda.synchronize()

    # One step: one call (fasgd_apply_with_push_and_select) whose pass
    # applies the push selected in the previous step (at its timestamp T) and
    # then K client gradients (T + 1 ... T + K), taking the transmit decisions
    # of this step's push from the v it leaves, followed by that selection's
    # scan and scatter (the push is applied at T + K + 1 by the next pass).
    # That is the order in which the server lock serialises the arrivals,
    # and per step the work is K dense updates, one push selected and one
    # push applied.  The first step of the warm-up has no push to apply; the
    # push selected by the last timed step is applied after the timed
    # region.  Each step's count goes to its own buffer, so the count of the
    # push a pass applies stays readable.
    ev = {name: [] for name in ("pass", "select")}
    counts = []
    n_steps_all = warm + steps
    cnts = torch.zeros(n_steps_all + 1, device=dev, dtype=torch.int64)
    pending = []                              # (client, grad_ts, step) of the selected, unapplied push

    def step(i, timed, c):
        base = st.T                          # the schedule is indexed by server timestamp
        p0, p1, e2 = TimingEvent(fa), TimingEvent(fa), TimingEvent(fa)
        out_cnt = cnts[i + 1:i + 2]
        if pending:
            pc, pts, j = pending.pop()
            sl = slice(base + 1, base + 1 + K)
            T_sel = base + K + 1
            fa.fasgd_record_next_pass(p0, p1)
            fa.fasgd_apply_with_push_and_select(st, idx, val, cnts[j + 1:j + 2], seg, pc, pts, pool[:K],
                                                clients[sl], ts[sl], pool[K], clients[T_sel], c, EPS_C, SEED,
                                                idx, val, out_cnt, seg, ws)
            applied = j + 1
        else:
            sl = slice(base, base + K)
            fa.fasgd_apply_updates(st, pool[:K], clients[sl], ts[sl])
            p1.record()
            T_sel = st.T
            fa.bfasgd_select_compact(st, pool[K], c, EPS_C, SEED, T_sel, clients[T_sel], idx, val, out_cnt, ws,
                                     seg_start=seg)
            applied = None
        e2.record()
        assert st.T == T_sel
        pending.append((clients[T_sel], ts[T_sel], i))
        if timed:
            ev["select"].append((p1, e2))
            if applied is not None:
                ev["pass"].append((p0, p1))
                counts.append(applied)

    # the first dense pass gives v its scale; c is then fixed for the run
    fa.fasgd_apply_updates(st, pool[:K], clients[:K], ts[:K])
    torch.cuda.synchronize()
    c = calibrate_c(v, f)
    print(f"# c = {c:.6g} for transmit fraction {f}", file=sys.stderr, flush=True)
    for i in range(warm):
        step(i, False, c)
    torch.cuda.synchronize()
    print(f"# warmup done ({warm} steps)", file=sys.stderr, flush=True)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(warm + i, True, c)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    print(f"# timed {steps} steps in {wall:.3f} s", file=sys.stderr, flush=True)
    # the last push is applied after the timed region
    pc, pts, j = pending.pop()
    fa.bfasgd_apply_sparse(st, idx, val, cnts[j + 1:j + 2], pc, pts)
    cnt.copy_(cnts[j + 1:j + 2])

    ms = {k: [a.elapsed_time(b_) for a, b_ in pairs] for k, pairs in ev.items()}
    cnt_host = cnts.cpu().numpy()
    m_list = [int(cnt_host[k]) for k in counts]
    m_avg = float(np.mean(m_list)) if m_list else 0.0
    updates = steps * P * K + sum(m_list)
    value = updates / wall
    pass_ms = float(np.mean(ms["pass"])) if ms["pass"] else float("nan")
    # per launch: state 16 B read + 16 B write, 4 B per gradient, for the
    # push 4 B index + 4 B value per entry and its list index, and the next
    # push's decisions (1 bit per parameter)
    pass_bytes = P * (32 + 4 * K) + 8 * m_avg + 4 * fa.bfasgd_list_index_length(P) + P / 8
    achieved = pass_bytes / (pass_ms * 1e-3) / 1e9
    traffic = measured_traffic(args.workload, P, K, args.math)
    sel_ms = float(np.mean(ms["select"]))
    # after the pass took the decisions: ballots and g read, (idx, val) written
    sel_bytes = P * 4 + P / 8 + m_avg * 8

    # the same steps as three separate calls (dense pass, selection, sparse
    # apply), for comparison
    sep_ms, sp_ms = [], []
    for r in range(3):
        base = st.T
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        e[0].record()
        fa.fasgd_apply_updates(st, pool[:K], clients[base:base + K], ts[base:base + K])
        e[1].record()
        fa.bfasgd_select_compact(st, pool[K], c, EPS_C, SEED, st.T, clients[base + K], idx, val, cnt, ws)
        e[2].record()
        fa.bfasgd_apply_sparse(st, idx, val, cnt, clients[base + K], ts[base + K])
        e[3].record()
        torch.cuda.synchronize()
        sep_ms.append(e[0].elapsed_time(e[3]))
        sp_ms.append(e[2].elapsed_time(e[3]))
    sep_ms_avg = float(np.mean(sep_ms[1:]))
    sp_ms = float(np.mean(sp_ms[1:]))
    # the same push applied segment by segment with its list index
    # (fasgd_apply_pushes with one push)
    seg_ms = []
    for r in range(3):
        base = st.T
        fa.bfasgd_select_compact(st, pool[K], c, EPS_C, SEED, st.T, clients[base], idx, val, cnt, ws, seg_start=seg)
        a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fa.fasgd_apply_pushes(st, idx.view(1, -1), val.view(1, -1), cnt, seg.view(1, -1), [clients[base]], [ts[base]])
        b_.record()
        torch.cuda.synchronize()
        seg_ms.append(a.elapsed_time(b_))
    sp_seg_ms = float(np.mean(seg_ms[1:]))
    # and as two calls: the pass with the queued push, then the full
    # selection (which reads v again)
    two_ms = []
    fa.bfasgd_select_compact(st, pool[K], c, EPS_C, SEED, st.T, clients[st.T], idx, val, cnt, ws, seg_start=seg)
    for r in range(3):
        base = st.T
        a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fa.fasgd_apply_with_push(st, idx, val, cnt, seg, clients[base], ts[base], pool[:K],
                                 clients[base + 1:base + 1 + K], ts[base + 1:base + 1 + K])
        fa.bfasgd_select_compact(st, pool[K], c, EPS_C, SEED, st.T, clients[st.T], idx, val, cnt, ws,
                                 seg_start=seg)
        b_.record()
        torch.cuda.synchronize()
        two_ms.append(a.elapsed_time(b_))
    fa.bfasgd_apply_sparse(st, idx, val, cnt, clients[st.T], ts[st.T])
    two_ms_avg = float(np.mean(two_ms[1:]))
    sp_bytes = m_avg * 44                           # idx, val + 16 B state gather, 16 B scatter, 4 B last_T

    # SASGD mode of the same pass, measured after the timed region
    sas_ms = []
    for r in range(3):
        a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        base = st.T
        a.record()
        fa.sasgd_apply_updates(st, pool[:K], clients[base:base + K], ts[base:base + K])
        b_.record()
        torch.cuda.synchronize()
        sas_ms.append(a.elapsed_time(b_))
    sas_ms_avg = float(np.mean(sas_ms[1:]))
    sas_bytes = P * (8 + 4 * K)

    def batch_ms(fn, n):
        """Per-call ms of back-to-back calls (the median over groups of n
        calls between two events): the rate the kernels sustain, without
        per-call event and dispatch gaps."""
        return grouped_b2b(torch, fn, n)

    # the push selection back to back on the step's last inputs
    sel_b2b_ms, sel_b2b_range = batch_ms(lambda: fa.bfasgd_select_compact(st, pool[K], c, EPS_C, SEED, st.T,
                                                                          clients[st.T], idx, val, cnt, ws), 20)
    m_b2b = int(cnt.item())
    sel_b2b_bytes = P * 8 + m_b2b * 8
    # the dense pass at K = 1, 8, 32 (gradients fused per pass), back to back
    dense_k = {}
    for k in KS:
        def dense_pass(k=k):
            base = st.T
            fa.fasgd_apply_updates(st, pool[:k], clients[base:base + k], ts[base:base + k])
        kms, krange = batch_ms(dense_pass, 10)
        dense_k[str(k)] = {"ms": kms, "ms_range": krange, "GB/s": P * (32 + 4 * k) / (kms * 1e-3) / 1e9,
                           "frac": P * (32 + 4 * k) / (kms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                           "param_updates_per_s": P * k / (kms * 1e-3)}

    def timed(fn, reps=3):
        out = []
        for _ in range(reps):
            a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b_.record()
            torch.cuda.synchronize()
            out.append(a.elapsed_time(b_))
        return float(np.mean(out[1:]))

    # widened paths at the same shape, after the timed region
    #   cached push: the list of the last push written into one client's cache,
    #   then the whole cache applied (Sec. 2.3's re-apply of dropped values)
    #   (with the list's index: merged into the cache inside the one pass;
    #   without it: the list copy, then the pass)
    extra = torch.zeros_like(pool[0])
    fa.bfasgd_select_compact(st, pool[K], c, EPS_C, SEED, st.T, clients[st.T], idx, val, cnt, ws, seg_start=seg)
    cached_ms = timed(lambda: fa.bfasgd_apply_cached(st, idx, val, cnt, extra, clients[st.T], ts[st.T],
                                                     seg_start=seg))
    cached_two_ms = timed(lambda: fa.bfasgd_apply_cached(st, idx, val, cnt, extra, clients[st.T], ts[st.T]))
    m_last = int(cnt.item())
    #   fetch: selection over the server's theta, copied into a client's copy
    #   (with the list's index the copy rewrites whole segments; without it,
    #   one scattered write per entry)
    def fetch():
        fa.bfasgd_select_compact(st, theta, c, EPS_C, SEED ^ 0xFE7C, st.T, clients[st.T], idx, val, cnt, ws,
                                 seg_start=seg)
        fa.bfasgd_apply_fetch(extra, idx, val, cnt, seg_start=seg)

    def fetch_scatter():
        fa.bfasgd_select_compact(st, theta, c, EPS_C, SEED ^ 0xFE7C, st.T, clients[st.T], idx, val, cnt, ws)
        fa.bfasgd_apply_fetch(extra, idx, val, cnt)
    fetch_seg_ms = timed(fetch)
    fetch_scatter_ms = timed(fetch_scatter)
    m_fetch = int(cnt.item())
    fetch_by_segments = fetch_copy_by_segments(P, m_fetch)
    fetch_ms = fetch_seg_ms if fetch_by_segments else fetch_scatter_ms
    #   the paper's own decision: one per push from the mean of v, and one per
    #   segment for 64 equal segments; then the push applied on the sent ones
    seg1 = np.array([0, P], np.int64)
    seg64 = np.linspace(0, P, 65).astype(np.int64)
    dsel = torch.zeros(64, device=dev, dtype=torch.uint8)
    wseg = torch.empty(fa.bfasgd_segments_workspace_bytes(P, 64), device=dev, dtype=torch.uint8)
    dec1_ms = timed(lambda: fa.bfasgd_decide_segments(st, seg1, c, EPS_C, SEED, st.T, 0, dsel[:1], wseg))
    dec64_ms = timed(lambda: fa.bfasgd_decide_segments(st, seg64, c, EPS_C, SEED, st.T, 0, dsel, wseg))
    dsel.fill_(1)
    segapply_ms = timed(lambda: fa.bfasgd_apply_segments(st, pool[K], seg64, dsel, clients[st.T], ts[st.T]))
    #   synchronous SGD step with lambda = K clients (the Sec. 3 listing)
    sync_st = fa.fasgd_init_state(theta, None, None, None, last_T, lam=K, alpha=w.alpha_sasgd)
    sync_ms = timed(lambda: fa.sgd_sync_apply(sync_st, pool[:K], w.alpha_sasgd))
    del extra

    # plain copies of one gradient buffer (4P bytes read, 4P written): the
    # library's streaming copy (fasgd_copy_anchor), the bandwidth anchor the
    # pass is read against, and torch's copy, the known-size kernel that
    # calibrates the rocprofv3 FETCH_SIZE / WRITE_SIZE counters
    anchor = torch.empty_like(pool[0])
    cp_ms = []
    for r in range(3):
        a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        anchor.copy_(pool[r % K])
        b_.record()
        torch.cuda.synchronize()
        cp_ms.append(a.elapsed_time(b_))
    copy_gbs = 8 * P / (float(np.mean(cp_ms[1:])) * 1e-3) / 1e9
    anchor_ms, anchor_range = grouped_b2b(torch, lambda: fa.fasgd_copy_anchor(pool[0], anchor), 4)
    anchor_gbs = 8 * P / (anchor_ms * 1e-3) / 1e9
    del anchor
    small = small_configs(fa, workload, dev, mode)
    large = large_25m(fa, workload, dev, mode) if args.workload != "large" else None

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "param-updates/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warm,
        "ms_per_step": wall / steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {w.name}, P={P}, lambda={w.lam}, per step one call: a pass "
                               f"applying the previous B-FASGD push (~{int(f * 100)}% transmitted) and K={K} "
                               f"FASGD updates and taking the next push's transmit decisions, then that push's "
                               f"compaction; {args.math} math",
                   "P": P, "K": K, "lambda": w.lam, "math": args.math, "transmit_fraction": f, "c": c},
        "roofline": {"bound": "hbm", "kernel": "fasgd_dense_push_lane", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic, "algorithmic_bytes": pass_bytes},
        "kernels": {
            "fasgd_apply_with_push_and_select": {
                "pass_ms": pass_ms, "pass_GB/s": achieved,
                "pass_param_updates_per_s": (P * K + m_avg) / (pass_ms * 1e-3),
                "selection_after_the_pass_ms": sel_ms,
                "selection_after_the_pass_GB/s": sel_bytes / (sel_ms * 1e-3) / 1e9},
            "step_as_two_calls": {"ms": two_ms_avg,
                                  "calls": "fasgd_apply_with_push, bfasgd_select_compact"},
            "fasgd_apply_updates": {"ms": dense_k[str(K)]["ms"] if str(K) in dense_k else None,
                                    "GB/s": dense_k[str(K)]["GB/s"] if str(K) in dense_k else None,
                                    "back_to_back_by_K": dense_k},
            "step_as_separate_calls": {"ms": sep_ms_avg,
                                       "calls": "fasgd_apply_updates, bfasgd_select_compact, bfasgd_apply_sparse"},
            "bfasgd_select_compact": {"ms_back_to_back": sel_b2b_ms, "ms_back_to_back_range": sel_b2b_range,
                                      "GB/s_back_to_back": sel_b2b_bytes / (sel_b2b_ms * 1e-3) / 1e9,
                                      "frac_back_to_back": sel_b2b_bytes / (sel_b2b_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                                      "transmitted_fraction": m_avg / P},
            "bfasgd_apply_sparse": {"ms": sp_ms, "GB/s_algorithmic": sp_bytes / (sp_ms * 1e-3) / 1e9,
                                    "ms_by_segments": sp_seg_ms},
            "sasgd_apply_updates": {"ms": sas_ms_avg, "GB/s": sas_bytes / (sas_ms_avg * 1e-3) / 1e9},
            "sgd_sync_apply": {"ms": sync_ms, "lambda": K,
                               "GB/s": P * (8 + 4 * K) / (sync_ms * 1e-3) / 1e9},
            "bfasgd_apply_cached": {"ms": cached_ms, "transmitted": m_last,
                                    "GB/s_algorithmic": (36 * P + 12 * m_last) / (cached_ms * 1e-3) / 1e9,
                                    "ms_two_steps": cached_two_ms},
            "fetch_select_and_copy": {"ms": fetch_ms, "transmitted": m_fetch,
                                      "GB/s_algorithmic": (8 * P + 20 * m_fetch) / (fetch_ms * 1e-3) / 1e9,
                                      "copy": "by segments" if fetch_by_segments else "scattered",
                                      "ms_copy_by_segments": fetch_seg_ms, "ms_scattered_copy": fetch_scatter_ms},
            "bfasgd_decide_segments": {"ms_whole_vector": dec1_ms, "ms_64_segments": dec64_ms,
                                       "GB/s": 4 * P / (dec1_ms * 1e-3) / 1e9},
            "bfasgd_apply_segments": {"ms_all_sent": segapply_ms,
                                      "GB/s": 40 * P / (segapply_ms * 1e-3) / 1e9},
            "copy_anchor": {"kernel": "fasgd_copy_anchor", "GB/s": anchor_gbs, "frac": anchor_gbs / HBM_PEAK_GBS,
                            "ms": anchor_ms, "ms_range": anchor_range, "bytes": 8 * P,
                            "pass_vs_anchor": achieved / anchor_gbs, "torch_copy_GB/s": copy_gbs},
            "small_configs": small,
            "large_25m": large,
        },
    }
    if args.cpu_params:
        P_s = min(args.cpu_params, P)
        cb = cpu_baseline(pool, theta0_host, clients, ts, c, w, K, P_s)
        out["cpu_baseline"] = {"value": cb["value"], "unit": "param-updates/s", "cores": 1, "kind": "oracle",
                               "sample": f"first {P_s} parameters of the same workload, one step "
                                         f"({K} dense updates + 1 push, {cb['transmitted']} transmitted), "
                                         f"{cb['seconds']:.1f} s on one pinned CPU",
                               "pinned_core": cb["pinned_core"], "host_logical_cpus": cb["host_logical_cpus"],
                               "cpus_available": cb["cpus_available"], "cpu_model": cb["cpu_model"],
                               "all_cores": cb["all_cores"]}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
