"""Pins for the oracle's B-FASGD send/skip selection (Sec. 2.3) and its Philox.

 * Philox4x32-10 against rocRAND's implementation (a library routine, compiled
   for the host from its public header);
 * the fp32 decision against the transmit rule r < 1/(1 + c/(v + eps))
   evaluated in exact rational arithmetic on the same fp32 inputs;
 * the limits the paper states (v large: nearly always transmit; v near 0:
   nearly never) and c = 0 (always);
 * the transmit rate against the mean transmit probability (binomial z-test);
 * the compacted list (ascending, values bit-copied, count) and the sparse
   apply (c = 0 reproduces dense FASGD; unlisted parameters untouched).
"""
import os
import shutil
import subprocess
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workload

ROCRAND_HDR = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"

_ROCRAND_PROBE = r"""
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
int main() {
    unsigned c0, c1, c2, c3, k0, k1;
    while (std::scanf("%x %x %x %x %x %x", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
        unsigned long long seed = ((unsigned long long)k1 << 32) | k0;
        unsigned long long sub  = ((unsigned long long)c3 << 32) | c2;
        unsigned long long q    = ((unsigned long long)c1 << 32) | c0;   /* c1 < 2^30 */
        rocrand_device::philox4x32_10_engine e(seed, sub, 4ull * q);
        uint4 r = e.next4();
        std::printf("%08x %08x %08x %08x\n", r.x, r.y, r.z, r.w);
    }
    return 0;
}
"""


@pytest.mark.skipif(not os.path.exists(ROCRAND_HDR) or shutil.which("g++") is None,
                    reason="rocRAND header or g++ not available")
def test_philox_matches_rocrand(tmp_path):
    """rocRAND's engine seeded with (seed, subsequence, offset) evaluates
    Philox4x32-10 at counter (offset/4 low, offset/4 high, subsequence low,
    subsequence high) under key (seed low, seed high)."""
    src = tmp_path / "probe.cpp"
    src.write_text(_ROCRAND_PROBE)
    exe = tmp_path / "probe"
    subprocess.run(["g++", "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", str(src), "-o", str(exe)],
                   check=True)
    rng = np.random.default_rng(2024)
    cases = [(0, 0, 0, 0, 0, 0), (0x3FFFFFFF, 0x3FFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF)]
    for _ in range(300):
        c = rng.integers(0, 2 ** 32, size=6, dtype=np.uint64)
        c[1] &= 0x3FFFFFFF
        cases.append(tuple(int(x) for x in c))
    inp = "\n".join(" ".join("%x" % x for x in cs) for cs in cases) + "\n"
    out = subprocess.run([str(exe)], input=inp, capture_output=True, text=True, check=True).stdout.split("\n")
    for cs, line in zip(cases, out):
        want = [int(x, 16) for x in line.split()]
        got = oracle.philox4x32_10(cs[:4], cs[4:]).tolist()
        assert got == want, (cs, got, want)


def _philox_r(j, seed, T, client):
    q = j >> 2
    w = oracle.philox4x32_10([q & 0xFFFFFFFF, q >> 32, T & 0xFFFFFFFF, client & 0xFFFFFFFF],
                             [seed & 0xFFFFFFFF, seed >> 32])[j & 3]
    return Fraction(int(w) >> 8, 1 << 24)


def test_decision_matches_exact_rule():
    """Away from a relative margin of 2^-21 around the threshold (the two
    fp32 sums v + eps and (v + eps) + c each round by at most 2^-24), the
    decision equals r < 1/(1 + c/(v + eps)) evaluated exactly."""
    rng = np.random.default_rng(7)
    n = 4000
    js = rng.integers(0, 2 ** 31 - 1, size=n)
    v = np.exp(rng.uniform(np.log(1e-6), np.log(1e6), size=n)).astype(np.float32)
    cs = np.exp(rng.uniform(np.log(1e-6), np.log(1e6), size=n)).astype(np.float32)
    seed, T, client = 0x0123456789ABCDEF, 77, 5
    eps_c = np.float32(1e-8)
    near = 0
    for i in range(n):
        d = oracle.bfasgd_decide(js[i:i + 1], v[i:i + 1], cs[i], eps_c, seed, T, client)[0]
        r = _philox_r(int(js[i]), seed, T, client)
        t = Fraction(float(v[i])) + Fraction(float(eps_c))
        p = 1 / (1 + Fraction(float(cs[i])) / t)
        if abs(r - p) <= p * Fraction(1, 2 ** 21):
            near += 1
            continue
        assert d == (r < p), (i, float(v[i]), float(cs[i]), float(r), float(p))
    assert near < n // 100


def test_c_zero_transmits_everything_and_huge_c_only_r_zero():
    P = 10_000
    v = workload.synthetic_v(P, seed=1)
    g = np.arange(P, dtype=np.float32)
    idx, val, m = oracle.bfasgd_select(v, g, 0.0, 1e-8, seed=9, T=3, client=1)
    assert m == P and (idx == np.arange(P)).all() and (val == g).all()
    idx, val, m = oracle.bfasgd_select(v, g, 3e38, 1e-8, seed=9, T=3, client=1)
    r_zero = [j for j in range(P) if _philox_r(j, 9, 3, 1) == 0]
    assert idx.tolist() == r_zero and m == len(r_zero)


def test_limits_in_v():
    """Sec. 2.3: v very large -> the threshold is close to 1; v near 0 -> close to 0."""
    P = 20_000
    js = np.arange(P)
    big = oracle.bfasgd_decide(js, np.full(P, 1e30, np.float32), 1.0, 1e-8, 5, 0, 0)
    assert big.all()
    small = oracle.bfasgd_decide(js, np.zeros(P, np.float32), 1.0, 1e-30, 5, 0, 0)
    assert not small.any()


@pytest.mark.parametrize("target", [0.2, 0.1, 0.5])
def test_transmit_rate_matches_probability(target):
    P = 200_000
    v = workload.synthetic_v(P, seed=2)
    vd = v.astype(np.float64) + 1e-8
    lo, hi = 0.0, 1e6                       # bisection for mean p = target
    for _ in range(100):
        c = 0.5 * (lo + hi)
        if (vd / (vd + c)).mean() > target:
            lo = c
        else:
            hi = c
    c = np.float32(c)
    p = vd / (vd + float(c))
    _, _, m = oracle.bfasgd_select(v, np.ones(P, np.float32), c, 1e-8, seed=123, T=41, client=7)
    z = (m - p.sum()) / np.sqrt((p * (1 - p)).sum())
    assert abs(z) < 5, (m, p.sum(), z)


def test_stream_is_keyed_by_seed_T_client_index():
    P = 20_000
    v = np.full(P, 1.0, np.float32)          # p = 1/2
    base = oracle.bfasgd_decide(np.arange(P), v, 1.0, 0.0, 11, 5, 3)
    for other in [(12, 5, 3), (11, 6, 3), (11, 5, 4), (11 + (1 << 32), 5, 3)]:
        d = oracle.bfasgd_decide(np.arange(P), v, 1.0, 0.0, *other)
        agree = (d == base).mean()
        assert 0.45 < agree < 0.55, (other, agree)
    shifted = oracle.bfasgd_decide(np.arange(1, P + 1), v, 1.0, 0.0, 11, 5, 3)
    assert 0.45 < (shifted == base).mean() < 0.55


def test_list_invariants_and_capacity():
    P = 50_001
    v = workload.synthetic_v(P, seed=3)
    g = np.random.default_rng(1).standard_normal(P).astype(np.float32)
    idx, val, m = oracle.bfasgd_select(v, g, 40.0, 1e-8, seed=5, T=100, client=2)
    assert m == len(idx) and 0 < m < P
    assert (np.diff(idx) > 0).all()
    assert (val.view(np.uint32) == g[idx].view(np.uint32)).all()
    dec = oracle.bfasgd_decide(np.arange(P), v, 40.0, 1e-8, 5, 100, 2)
    assert dec.sum() == m and (np.flatnonzero(dec) == idx).all()
    idx2, val2, m2 = oracle.bfasgd_select(v, g, 40.0, 1e-8, seed=5, T=100, client=2, capacity=m // 3)
    assert m2 == m and (idx2 == idx[: m // 3]).all() and (val2 == val[: m // 3]).all()


def test_transmit_all_sparse_apply_is_dense_fasgd():
    w = workload.WORKLOADS["tiny"]
    theta0, mm, s = workload.host_params(w, 3001)
    clients, ts = workload.schedule(w, 12)
    dense = oracle.init_state(theta0, alpha=0.01)
    sparse = oracle.init_state(theta0, alpha=0.01)
    for t in range(12):
        g = workload.host_gradient(w, mm, s, t)
        oracle.fasgd_apply(dense, g, ts[t])
        idx, val, m = oracle.bfasgd_select(sparse.v.astype(np.float32), g, 0.0, 1e-8, 0, sparse.T, clients[t])
        assert m == 3001
        oracle.bfasgd_apply_sparse(sparse, idx, val, ts[t])
    for name in ("theta", "n", "b", "v", "last_T"):
        np.testing.assert_array_equal(getattr(dense, name), getattr(sparse, name))
    assert dense.T == sparse.T == 12


def test_sparse_apply_leaves_unlisted_parameters():
    w = workload.WORKLOADS["tiny"]
    theta0, mm, s = workload.host_params(w, 1000)
    st = oracle.init_state(theta0, alpha=0.01)
    oracle.fasgd_apply(st, workload.host_gradient(w, mm, s, 0), 0)
    before = st.copy()
    idx = np.array([3, 10, 11, 999], np.int32)
    val = np.array([0.5, -0.25, 1.0, 2.0], np.float32)
    oracle.bfasgd_apply_sparse(st, idx, val, grad_ts=0)
    rest = np.setdiff1d(np.arange(1000), idx)
    for name in ("theta", "n", "b", "v", "last_T"):
        np.testing.assert_array_equal(getattr(st, name)[rest], getattr(before, name)[rest])
    assert (st.last_T[idx] == 1).all() and st.T == 2
    assert (st.theta[idx] != before.theta[idx]).all()
    # an empty push is still one server update
    oracle.bfasgd_apply_sparse(st, np.zeros(0, np.int32), np.zeros(0, np.float32), grad_ts=1)
    assert st.T == 3


def test_slices_with_index_base_reproduce_the_whole_selection():
    """A vector cut into slices at global offsets (multiples of 4), each
    selected with its offset as index_base, lists exactly the whole vector's
    transmitted indices (slice index + offset) and values: decisions follow
    the global index, so they do not depend on how the vector is cut."""
    P = 50_003
    v = workload.synthetic_v(P, seed=21)
    g = np.random.default_rng(22).standard_normal(P).astype(np.float32)
    idx, val, m = oracle.bfasgd_select(v, g, 30.0, 1e-8, 0xABC, 12, 3)
    for cuts in ([0, P], [0, 4, 16_384, 30_000, P], [0, 25_000, P]):
        parts_i, parts_v, total = [], [], 0
        for a, b in zip(cuts[:-1], cuts[1:]):
            i_s, v_s, m_s = oracle.bfasgd_select(v[a:b], g[a:b], 30.0, 1e-8, 0xABC, 12, 3, index_base=a)
            parts_i.append(i_s.astype(np.int64) + a)
            parts_v.append(v_s)
            total += m_s
        assert total == m
        np.testing.assert_array_equal(np.concatenate(parts_i), idx)
        np.testing.assert_array_equal(np.concatenate(parts_v).view(np.uint32), val.view(np.uint32))
    # an offset that is not the slice's true position changes the decisions
    i_w, _, _ = oracle.bfasgd_select(v[4:], g[4:], 30.0, 1e-8, 0xABC, 12, 3, index_base=0)
    assert not np.array_equal(i_w + 4, idx[idx >= 4])
