"""Seeded synthetic inputs for the FASGD server path.

This module is the only code that both the CPU oracle side (tests, CPU
baseline) and the GPU side consume.  It generates *inputs* -- initial
parameters, per-parameter gradient means and noise scales, client gradients,
client arrival order and gradient timestamps -- and holds none of the update
rules themselves.

The paper (arXiv:1601.04033, Sec. 4) trains an MNIST MLP; no data or weights
are used here.  The workloads below stand in for it with synthetic gradients
of a fixed shape:

  theta0_j ~ N(0, 0.05^2)                  initial parameters
  m_j      ~ N(0, (1e-3)^2)                per-parameter gradient mean
  s_j      log-uniform in [lo, hi]         per-parameter (or per-layer /
                                           per-block) gradient noise scale
  grad_j(t) = m_j + s_j * z_j(t),  z ~ N(0, 1) drawn afresh for update t

Client arrival is round-robin (client = T mod lambda); the staleness of the
gradient applied at server timestamp T is a random delay tau <= T, and the
gradient's timestamp is T - tau (Sec. 2.1: tau = i - j >= 0).

CPU arrays come from numpy PCG64 streams keyed by (seed, workload id, purpose,
t).  Large device arrays come from torch's device generator (Philox-based on
ROCm) keyed the same way; tests that compare at full size read the sampled
device inputs back to the host, so both sides always see identical inputs.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np

# purposes (third word of every stream key)
_THETA, _MEAN, _SCALE, _GRAD, _SCHED, _LAYER = 1, 2, 3, 4, 5, 6

# 784-1000-1000-10 MLP: (name, entries, is_bias)
MLP_LAYOUT = (("W1", 784 * 1000, False), ("b1", 1000, True),
              ("W2", 1000 * 1000, False), ("b2", 1000, True),
              ("W3", 1000 * 10, False), ("b3", 10, True))
MLP_P = sum(n for _, n, _ in MLP_LAYOUT)  # 1,796,010


@dataclass(frozen=True)
class Workload:
    """One synthetic workload shaped like the paper's experiments."""
    wid: int                 # stream key word
    name: str
    P: int                   # parameters
    lam: int                 # lambda, number of clients
    updates: int             # server updates in the run
    K: Sequence[int]         # gradients fused per kernel pass
    alpha_fasgd: float
    alpha_sasgd: float
    delay: str               # staleness recipe: "u0_3", "poisson", "u0_2lam"
    scale: str               # noise-scale recipe: "per_param", "mlp", "blocks"
    scale_lo: float = 1e-4
    scale_hi: float = 1e-1
    block: int = 500_000
    transmit_fraction: Optional[float] = None   # B-FASGD target m/P
    seed: int = 0
    extra: dict = field(default_factory=dict)


# The paper's best master rates (Sec. 4.1): 0.005 for FASGD and 0.04 for SASGD.
WORKLOADS = {
    "tiny": Workload(1, "tiny FASGD trace", 100_000, 4, 256, (1,), 0.01, 0.01,
                     "u0_3", "per_param"),
    "mlp": Workload(2, "MLP-shaped FASGD (784-1000-1000-10)", MLP_P, 16, 2000, (16,),
                    0.005, 0.04, "poisson", "mlp"),
    "mlp_bfasgd": Workload(3, "B-FASGD select + sparse apply, MLP layout", MLP_P, 16, 2000, (1,),
                           0.005, 0.04, "poisson", "mlp", transmit_fraction=0.2),
    "large": Workload(4, "large dense FASGD, 50 blocks of 500k", 25_000_000, 64, 512, (1, 8, 32),
                      0.005, 0.04, "u0_2lam", "blocks", scale_lo=1e-5, scale_hi=1e-1),
    "memscale": Workload(5, "memory-scale FASGD + B-FASGD", 1_000_000_000, 256, 64, (32,),
                         0.005, 0.04, "u0_2lam", "per_param", transmit_fraction=0.1),
}


def _rng(w: Workload, purpose: int, t: int = 0, seed: Optional[int] = None) -> np.random.Generator:
    s = w.seed if seed is None else seed
    return np.random.Generator(np.random.PCG64([s, w.wid, purpose, t]))


def _log_uniform(rng: np.random.Generator, lo: float, hi: float, size) -> np.ndarray:
    return np.exp(rng.uniform(np.log(lo), np.log(hi), size=size)).astype(np.float32)


def noise_scale(w: Workload, P: Optional[int] = None, seed: Optional[int] = None) -> np.ndarray:
    """s_j for the first P parameters of workload w (fp32, host)."""
    P = w.P if P is None else P
    if w.scale == "per_param":
        return _log_uniform(_rng(w, _SCALE, seed=seed), w.scale_lo, w.scale_hi, P)
    if w.scale == "blocks":
        nb = -(-P // w.block)
        per_block = _log_uniform(_rng(w, _SCALE, seed=seed), w.scale_lo, w.scale_hi, nb)
        return np.repeat(per_block, w.block)[:P].copy()
    if w.scale == "mlp":
        rng = _rng(w, _LAYER, seed=seed)
        out = []
        S = None
        for name, n, is_bias in MLP_LAYOUT:
            if not is_bias:
                S = _log_uniform(rng, w.scale_lo, w.scale_hi, 1)[0]
            out.append(np.full(n, np.float32(S * (0.1 if is_bias else 1.0)), dtype=np.float32))
        s = np.concatenate(out)
        if P > s.shape[0]:
            raise ValueError("the MLP layout has only %d parameters" % s.shape[0])
        return s[:P].copy()
    raise ValueError(w.scale)


def host_params(w: Workload, P: Optional[int] = None, seed: Optional[int] = None):
    """(theta0, m, s) as fp32 numpy arrays of length P (default w.P)."""
    P = w.P if P is None else P
    theta0 = (_rng(w, _THETA, seed=seed).standard_normal(P, dtype=np.float32) * np.float32(0.05))
    m = (_rng(w, _MEAN, seed=seed).standard_normal(P, dtype=np.float32) * np.float32(1e-3))
    s = noise_scale(w, P, seed=seed)
    return theta0.astype(np.float32), m.astype(np.float32), s


def host_gradient(w: Workload, m: np.ndarray, s: np.ndarray, t: int, seed: Optional[int] = None) -> np.ndarray:
    """Gradient for server update t: m + s * z, z ~ N(0, 1) (fp32, host)."""
    z = _rng(w, _GRAD, t, seed=seed).standard_normal(m.shape[0], dtype=np.float32)
    return (m + s * z).astype(np.float32)


def schedule(w: Workload, updates: Optional[int] = None, T0: int = 0, seed: Optional[int] = None):
    """Arrival order for server timestamps T0 .. T0+updates-1.

    Returns (clients int32, grad_ts int64): the client of timestamp T is
    T mod lambda; its gradient was computed on parameters with timestamp
    T - tau, with the delay tau drawn per the workload's recipe and capped at T.
    """
    U = w.updates if updates is None else updates
    rng = _rng(w, _SCHED, T0, seed=seed)
    T = np.arange(T0, T0 + U, dtype=np.int64)
    if w.delay == "u0_3":
        d = rng.integers(0, 4, size=U)
    elif w.delay == "poisson":
        d = np.clip(rng.poisson(w.lam - 1, size=U), 0, 4 * w.lam)
    elif w.delay == "u0_2lam":
        d = rng.integers(0, 2 * w.lam + 1, size=U)
    else:
        raise ValueError(w.delay)
    tau = np.minimum(d.astype(np.int64), T)
    clients = (T % w.lam).astype(np.int32)
    return clients, (T - tau).astype(np.int64)


def synthetic_v(P: int, seed: int = 0, lo: float = 1.0, hi: float = 300.0) -> np.ndarray:
    """A stand-alone fp32 array shaped like FASGD's v (positive, spread over
    two and a half decades) for testing the send/skip selection on its own."""
    rng = np.random.Generator(np.random.PCG64([seed, 0, 7, 0]))
    return _log_uniform(rng, lo, hi, P)


# --------------------------------------------------------------------------
# Device-side generation for workloads too large to build on the host.
# --------------------------------------------------------------------------
def _torch_gen(device, w: Workload, purpose: int, t: int = 0, seed: Optional[int] = None):
    import torch
    s = w.seed if seed is None else seed
    g = torch.Generator(device=device)
    g.manual_seed(((s * 1_000_003 + w.wid) * 1_000_003 + purpose) * 1_000_003 + t)
    return g


def device_params(w: Workload, device, P: Optional[int] = None, seed: Optional[int] = None):
    """(theta0, m, s) as fp32 device tensors.  Only the per-parameter
    log-uniform and per-block recipes are supported on the device."""
    import torch
    P = w.P if P is None else P
    theta0 = torch.randn(P, device=device, generator=_torch_gen(device, w, _THETA, seed=seed)) * 0.05
    m = torch.randn(P, device=device, generator=_torch_gen(device, w, _MEAN, seed=seed)) * 1e-3
    if w.scale == "per_param":
        u = torch.rand(P, device=device, generator=_torch_gen(device, w, _SCALE, seed=seed))
        lo, hi = float(np.log(w.scale_lo)), float(np.log(w.scale_hi))
        s = torch.exp(u * (hi - lo) + lo)
    elif w.scale == "blocks":
        s = torch.from_numpy(noise_scale(w, P, seed=seed)).to(device)
    else:
        raise ValueError("device generation supports per_param and blocks noise scales")
    return theta0.float().contiguous(), m.float().contiguous(), s.float().contiguous()


def device_gradient(w: Workload, m, s, t: int, out=None, seed: Optional[int] = None):
    """Gradient for server update t, generated on m's device: m + s * z."""
    import torch
    gen = _torch_gen(m.device, w, _GRAD, t, seed=seed)
    if out is None:
        out = torch.empty_like(m)
    torch.randn(out.shape, device=m.device, generator=gen, out=out)
    out.mul_(s).add_(m)
    return out
