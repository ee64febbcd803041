"""Inner AdamW step of every worker, in float64 (test infrastructure only).

Each worker runs H local AdamW steps between synchronisations (Alg. "AutoLoCo
outer interval", local inner loops; the paper follows DiLoCo in using AdamW as
the inner optimiser).  The training recipe fixes the settings (Table "Training
settings": AdamW coefficients (0.9, 0.95) for C4 and (0.9, 0.999) for SFT,
weight decay 0.1 / 0, gradient-norm clipping 1.0, the cosine schedule), and
App. G.1 keeps the master parameters and the AdamW states in FP32 while the
model computes in BF16.

One step of one worker, with gradient g of its parameters theta, first and
second moments m and v, step count t (1 for the first step), learning rate
eta (the schedule's value at this step) and weight decay lambda:

  norm     = || g ||_2 over all of the worker's parameters
  c        = max_norm / (norm + 1e-6), capped at 1   (no clipping: c = 1)
  g        = c g
  theta    = theta (1 - eta lambda)                   decoupled weight decay
  m        = beta1 m + (1 - beta1) g
  v        = beta2 v + (1 - beta2) g^2
  m_hat    = m / (1 - beta1^t),  v_hat = v / (1 - beta2^t)
  theta    = theta - eta m_hat / (sqrt(v_hat) + epsilon)

Readings of what the recipe leaves open:
  * AdamW is the decoupled form of Loshchilov and Hutter with the decay scaled
    by the learning rate and applied before the Adam step (the form of the
    common PyTorch optimiser); epsilon = 1e-8 sits outside the square root of
    the bias-corrected second moment;
  * "gradient-norm clipping 1.0" clips each worker's own global gradient norm
    (workers do not communicate inside the interval), with the usual 1e-6
    guard in the denominator; a non-finite norm is not an error: the step
    then produces non-finite values and the round's statistics report it;
  * the BF16 compute copy of a worker's parameters is the round-to-nearest-even
    BF16 value of its updated FP32 master parameters.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Sequence

import numpy as np

CLIP_GUARD = 1e-6


@dataclass(frozen=True)
class AdamWConfig:
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    weight_decay: float = 0.1
    max_grad_norm: float = 1.0        # 0 = no clipping


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def grad_norm(grad) -> float:
    """Euclidean norm of a worker's whole gradient (one flat array)."""
    g = _f64(grad)
    return math.sqrt(float(np.sum(g * g)))


def clip_coefficient(norm: float, max_norm: float) -> float:
    """Factor the gradient is multiplied by; NaN stays NaN (no clipping: 1)."""
    if max_norm == 0.0:
        return 1.0
    c = max_norm / (norm + CLIP_GUARD)
    return 1.0 if c > 1.0 else c


def adamw_step(param, exp_avg, exp_avg_sq, grad, lr: float, step: int, cfg: AdamWConfig, coef: float = 1.0):
    """One AdamW step of one worker on float64 copies; returns (theta', m', v')."""
    if step < 1:
        raise ValueError("the step count starts at 1")
    g = _f64(grad) * coef
    th = _f64(param) * (1.0 - lr * cfg.weight_decay)
    m = cfg.beta1 * _f64(exp_avg) + (1.0 - cfg.beta1) * g
    v = cfg.beta2 * _f64(exp_avg_sq) + (1.0 - cfg.beta2) * g * g
    m_hat = m / (1.0 - cfg.beta1 ** step)
    v_hat = v / (1.0 - cfg.beta2 ** step)
    th = th - lr * m_hat / (np.sqrt(v_hat) + cfg.eps)
    return th, m, v


@dataclass
class InnerStep:
    params: List[np.ndarray]         # float64 [n] per worker
    exp_avg: List[np.ndarray]
    exp_avg_sq: List[np.ndarray]
    grad_norm: List[float]
    clip_coef: List[float]


def inner_step(params: Sequence, exp_avg: Sequence, exp_avg_sq: Sequence, grads: Sequence,
               lr: float, step: int, cfg: AdamWConfig) -> InnerStep:
    """One inner step of every worker: its own clipping, then its AdamW step."""
    out = InnerStep([], [], [], [], [])
    for p, m, v, g in zip(params, exp_avg, exp_avg_sq, grads):
        norm = grad_norm(g)
        c = clip_coefficient(norm, cfg.max_grad_norm)
        th, m2, v2 = adamw_step(p, m, v, g, lr, step, cfg, c)
        out.params.append(th)
        out.exp_avg.append(m2)
        out.exp_avg_sq.append(v2)
        out.grad_norm.append(norm)
        out.clip_coef.append(c)
    return out
