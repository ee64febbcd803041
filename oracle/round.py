"""Float64 oracle of one synchronisation round (test infrastructure only).

Everything is evaluated in float64 with numpy, straight from the definitions:

  pseudo-gradient    Delta_k = theta - theta_k
                     (Alg. "AutoLoCo outer interval", local inner loops;
                     App. D.1 eq. diloco-local-trajectory)
  mean               Delta_bar = (1/K) sum_k Delta_k
                     (Sec. "Adaptive Interval Selection"; eq. diloco-outer-update)
  diagnostics        D = (1/K) sum_k ||Delta_k||^2,  C = K ||Delta_bar||^2 / (D + eps)
                     (eq. adaptive-h-core-diagnostics)
  disagreement       (1/K) sum_k ||Delta_k - Delta_bar||^2
                     (App. C.1 eqs. dc_variance_expansion, dc_endpoint_disagreement)
  normalisation      Delta_tilde = Delta_bar / rho, or Delta_bar when off
                     (eq. normalized-pseudo-gradient)
  corrected Nesterov v' = mu v + Delta_tilde;  d = Delta_tilde + mu v';
                     theta' = theta - eta d   (eq. autoloco-corrected-nesterov)
  reset              theta_k <- theta'  (every worker starts the next interval
                     from the synchronised parameters; Alg. "AutoLoCo outer
                     interval", first line of the local loop)

The paper writes the worker count as N; here it is K and N is the number of
parameters.  Inputs are fp32 arrays or bf16 bit patterns (uint16); both widen
to float64 exactly.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Sequence

import numpy as np


# ---------------------------------------------------------------- precision --
def widen(x: np.ndarray) -> np.ndarray:
    """fp32 values, or bf16 bit patterns held as uint16, to float64 (exact)."""
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if x.dtype == np.float32 or x.dtype == np.float64:
        return x.astype(np.float64)
    raise TypeError(f"unsupported replica dtype {x.dtype}")


_BF16_MAX = float.fromhex("0x1.fep127")


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 (round to nearest, ties to even) and return
    the uint16 bit patterns.  NaN stays NaN with its sign, infinities stay, and
    magnitudes past the largest finite bf16 plus half an ulp become infinities."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.float64)
    fin = np.isfinite(x)
    xf = x[fin]
    _, e = np.frexp(xf)                       # xf = m * 2**e, 0.5 <= |m| < 1
    q = np.maximum(e - 8, -133)               # 8 significant bits; bf16 subnormal quantum 2**-133
    r = np.ldexp(np.rint(np.ldexp(xf, -q)), q)  # np.rint rounds half to even
    big = np.abs(r) > _BF16_MAX
    r[big] = np.copysign(np.inf, r[big])
    out[fin] = r
    out[~fin] = x[~fin]
    bits = (out.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        sign = (np.signbit(x[nan]).astype(np.uint16) << 15)
        bits[nan] = sign | np.uint16(0x7FC0)
    return bits


# ------------------------------------------------------------- definitions --
def pseudo_gradients(theta: np.ndarray, replicas: Sequence[np.ndarray]) -> List[np.ndarray]:
    """Delta_k = theta - theta_k, one float64 array per worker."""
    th = widen(theta)
    return [th - widen(r) for r in replicas]


def mean_pseudo_gradient(deltas: Sequence[np.ndarray]) -> np.ndarray:
    """Delta_bar = (1/K) sum_k Delta_k."""
    total = np.zeros_like(deltas[0])
    for d in deltas:
        total = total + d
    return total / len(deltas)


@dataclass
class Stats:
    """Sums over parameters of one round: ||Delta_k||^2, ||Delta_k - Delta_bar||^2
    and ||Delta_bar||^2, and the scalars derived from them."""

    sq_norm: List[float] = field(default_factory=list)
    sq_dev: List[float] = field(default_factory=list)
    sq_mean: float = 0.0
    D: float = 0.0
    C: float = 0.0
    disagreement: float = 0.0
    finite: bool = True


def partial_sums(theta: np.ndarray, replicas: Sequence[np.ndarray]):
    """(S_k, Q_k, M) for one contiguous range of parameters."""
    deltas = pseudo_gradients(theta, replicas)
    mean = mean_pseudo_gradient(deltas)
    s = [float(np.sum(d * d)) for d in deltas]
    q = [float(np.sum((d - mean) * (d - mean))) for d in deltas]
    m = float(np.sum(mean * mean))
    return s, q, m


def finish_stats(s: Sequence[float], q: Sequence[float], m: float, eps: float) -> Stats:
    k = len(s)
    d_energy = sum(s) / k
    coherence = k * m / (d_energy + eps)
    disagreement = sum(q) / k
    vals = list(s) + list(q) + [m, d_energy, coherence, disagreement]
    finite = all(np.isfinite(v) for v in vals)
    return Stats(list(s), list(q), m, d_energy, coherence, disagreement, finite)


def round_stats(theta: np.ndarray, replicas: Sequence[np.ndarray], eps: float = 1e-12,
                chunk: int = 1 << 22) -> Stats:
    """Diagnostics of one round, summed over chunks of ``chunk`` parameters."""
    k = len(replicas)
    n = theta.shape[0]
    s_tot = [0.0] * k
    q_tot = [0.0] * k
    m_tot = 0.0
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        s, q, m = partial_sums(theta[lo:hi], [r[lo:hi] for r in replicas])
        s_tot = [a + b for a, b in zip(s_tot, s)]
        q_tot = [a + b for a, b in zip(q_tot, q)]
        m_tot += m
    return finish_stats(s_tot, q_tot, m_tot, eps)


def outer_update(theta: np.ndarray, momentum: np.ndarray, mean: np.ndarray,
                 mu: float, eta: float, rho: float, normalize: bool):
    """Corrected Nesterov step on float64 arrays; returns (theta', v')."""
    th = widen(theta)
    v = widen(momentum)
    dt = mean / rho if normalize else mean
    v_new = mu * v + dt
    d = dt + mu * v_new
    th_new = th - eta * d
    return th_new, v_new


@dataclass
class RoundResult:
    theta: np.ndarray        # float64 [n]
    momentum: np.ndarray     # float64 [n]
    stats: Stats


def sync_round(theta: np.ndarray, momentum: np.ndarray, replicas: Sequence[np.ndarray],
               mu: float, eta: float, rho: float, normalize: bool, eps: float = 1e-12,
               chunk: int = 1 << 22) -> RoundResult:
    """One whole round: diagnostics of theta_t's pseudo-gradients and the
    corrected Nesterov step.  The reset copies theta' into every replica; see
    ``reset_replicas``."""
    n = theta.shape[0]
    k = len(replicas)
    th_out = np.empty(n, dtype=np.float64)
    v_out = np.empty(n, dtype=np.float64)
    s_tot = [0.0] * k
    q_tot = [0.0] * k
    m_tot = 0.0
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        reps = [r[lo:hi] for r in replicas]
        deltas = pseudo_gradients(theta[lo:hi], reps)
        mean = mean_pseudo_gradient(deltas)
        for i, d in enumerate(deltas):
            s_tot[i] += float(np.sum(d * d))
            q_tot[i] += float(np.sum((d - mean) * (d - mean)))
        m_tot += float(np.sum(mean * mean))
        th_out[lo:hi], v_out[lo:hi] = outer_update(theta[lo:hi], momentum[lo:hi], mean,
                                                   mu, eta, rho, normalize)
    return RoundResult(th_out, v_out, finish_stats(s_tot, q_tot, m_tot, eps))


def reset_replicas(theta_new: np.ndarray, k: int, replica_dtype: str) -> List[np.ndarray]:
    """Every worker restarts from theta': fp32 replicas take theta' rounded to
    fp32, bf16 replicas take it rounded to bf16 (bit patterns, uint16)."""
    if replica_dtype == "f32":
        r = np.asarray(theta_new, dtype=np.float64).astype(np.float32)
    elif replica_dtype == "bf16":
        r = to_bf16_bits(theta_new)
    else:
        raise ValueError(replica_dtype)
    return [r.copy() for _ in range(k)]


def model_average(replicas: Sequence[np.ndarray]) -> np.ndarray:
    """Arithmetic mean of the local endpoints, (1/K) sum_k theta_k
    (App. C.1 eq. dc_endpoint_mean: it equals theta - Delta_bar)."""
    total = np.zeros(replicas[0].shape, dtype=np.float64)
    for r in replicas:
        total = total + widen(r)
    return total / len(replicas)
