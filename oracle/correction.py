"""Inner learning-rate schedule, learning-rate masses and the Outer Optimizer
Correction, in plain Python doubles (test infrastructure only).

  learning-rate mass   Lambda = sum_{h=1..H} eta_{t,h},  eta_{t,h} = eta(s_t + h - 1)
                       (App. B.2 eq. app-outer-correction-lr-masses)
  interval ratio       rho = max(Lambda / (Lambda_base + eps), 1)
                       (eq. outer-correction-ratio; eq. app-outer-correction-ratios)
  momentum retention   mu_t = clip(mu_base ** rho, mu_min, mu_max)
  step scale           kappa_t = min(rho, kappa_max)  (eq. app-outer-step-scale)
  outer learning rate  eta_t = eta_base * kappa_t * (1 - mu_t) / (1 - mu_base)
                       (eq. adjusted-outer-learning-rate; App. C.3)

The schedule is the training recipe's cosine decay after a linear warm-up
(Table "Training settings": cosine, 1,000 warm-up steps, peak 4e-4 for C4).
The paper does not print the formula; the reading used is
  eta(s) = peak * (s + 1) / W                                  for s < W,
  eta(s) = min_lr + (peak - min_lr) * (1 + cos(pi * min(1, (s - W) / (T - W)))) / 2
with s the 0-based global inner step, W the warm-up length and T the budget.
"""
from __future__ import annotations

import math
from dataclasses import dataclass


@dataclass(frozen=True)
class Schedule:
    peak: float = 4e-4
    min_lr: float = 0.0
    warmup: int = 1000
    total: int = 50_000


def inner_lr(sched: Schedule, step: int) -> float:
    if step < sched.warmup:
        return sched.peak * (step + 1) / sched.warmup
    span = sched.total - sched.warmup
    frac = (step - sched.warmup) / span if span > 0 else 1.0
    if frac > 1.0:
        frac = 1.0
    return sched.min_lr + (sched.peak - sched.min_lr) * 0.5 * (1.0 + math.cos(math.pi * frac))


def lr_mass(sched: Schedule, start: int, steps: int) -> float:
    """Sum of the inner learning rates of ``steps`` steps starting at ``start``."""
    total = 0.0
    for h in range(1, steps + 1):
        total += inner_lr(sched, start + h - 1)
    return total


@dataclass(frozen=True)
class OuterConfig:
    eta_base: float = 0.7
    mu_base: float = 0.9
    mu_min: float = 0.45
    mu_max: float = 0.90
    kappa_max: float = 1.6
    eps: float = 1e-12
    normalize: bool = False


@dataclass(frozen=True)
class OuterCoeffs:
    rho: float
    mu: float
    kappa: float
    eta: float
    normalize: bool


def interval_ratio(lam: float, lam_base: float, eps: float) -> float:
    r = lam / (lam_base + eps)
    return r if r > 1.0 else 1.0


def outer_correction(cfg: OuterConfig, lam: float, lam_base: float) -> OuterCoeffs:
    rho = interval_ratio(lam, lam_base, cfg.eps)
    mu = cfg.mu_base ** rho
    if mu < cfg.mu_min:
        mu = cfg.mu_min
    if mu > cfg.mu_max:
        mu = cfg.mu_max
    kappa = rho if rho < cfg.kappa_max else cfg.kappa_max
    eta = cfg.eta_base * kappa * ((1.0 - mu) / (1.0 - cfg.mu_base))
    return OuterCoeffs(rho, mu, kappa, eta, cfg.normalize)
