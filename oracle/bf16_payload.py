"""The round with BF16 pseudo-gradient payloads (test infrastructure only).

The paper's main runs communicate each worker's pseudo-gradient as a BF16
tensor (Table "Quality and communication cost": payload in full-model BF16
tensors per worker; the UltraChat tables: both methods communicate BF16
pseudo-gradients), while the master parameters, the outer reference and the
Nesterov momentum stay in FP32 (App. G.1).  One round:

  Delta_k  = theta - theta_k                          FP32 (theta_k widened exactly)
  b_k      = bf16(Delta_k)                            the payload of worker k
  mean     = fp32( (sum_k b_k) * (1/K) )              sum in float64, worker order
  agg      = bf16(mean)                               what every worker receives
  S_k = ||Delta_k||^2 (before rounding), Q_k = ||Delta_k - agg||^2, M = ||agg||^2
  corrected Nesterov step with agg, reset of the replicas

bf16(.) is round to nearest, ties to even.  Readings of what the text leaves
open, chosen alike to the INT8 configuration the paper spells out (App. G.1):
the payloads are averaged in FP32 (the float64 sum of at most 16 BF16 values in
worker order, times float64(1/K), rounded once to FP32), the mean is rounded to
BF16 once for distribution, D is measured before the payload rounding and C on
the aggregate every worker receives.
"""
from __future__ import annotations

import numpy as np

from . import round as orr


def payload(delta32: np.ndarray) -> np.ndarray:
    """BF16 bit patterns of FP32 pseudo-gradients."""
    return orr.to_bf16_bits(np.asarray(delta32, dtype=np.float32).astype(np.float64))


def aggregate(payloads) -> np.ndarray:
    """BF16 bits of the mean every worker receives."""
    total = np.zeros(payloads[0].shape, dtype=np.float64)
    for p in payloads:
        total = total + orr.widen(p)
    mean32 = (total * (1.0 / len(payloads))).astype(np.float32)
    return orr.to_bf16_bits(mean32.astype(np.float64))


class Bf16Round:
    def __init__(self, theta, momentum, stats, mean_bits):
        self.theta = theta
        self.momentum = momentum
        self.stats = stats
        self.mean_bits = mean_bits


def bf16_round(theta: np.ndarray, momentum: np.ndarray, replicas, mu: float, eta: float, rho: float,
               normalize: bool, eps: float = 1e-12) -> Bf16Round:
    th32 = np.asarray(theta, dtype=np.float32)
    deltas = [th32 - orr.widen(r).astype(np.float32) for r in replicas]
    bits = aggregate([payload(d) for d in deltas])
    agg = orr.widen(bits)
    d64 = [d.astype(np.float64) for d in deltas]
    s = [float(np.sum(d * d)) for d in d64]
    q = [float(np.sum((d - agg) * (d - agg))) for d in d64]
    m = float(np.sum(agg * agg))
    stats = orr.finish_stats(s, q, m, eps)
    th_new, v_new = orr.outer_update(theta, momentum, agg, mu, eta, rho, normalize)
    return Bf16Round(th_new, v_new, stats, bits)
