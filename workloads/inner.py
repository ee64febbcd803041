"""Seeded synthetic state of the workers' inner AdamW step.

For each of K workers: FP32 master parameters, first and second moments and
one step's gradient.  The parameters are the round inputs' replicas (or
N(0, param_std) draws), m ~ N(0, m_std), v = z^2 with z ~ N(0, v_std), and the
gradient of worker k is N(0, 1) scaled so that its Euclidean norm is about
norms[k % len(norms)] (the defaults straddle the clipping threshold 1.0 of the
training recipe, so some workers are clipped and others are not).  Every draw
comes from torch's seeded generator per (seed, role, worker, chunk) on the
CPU or the GPU; none of the optimiser's arithmetic lives here.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

import torch

from .drift import CHUNK, _generator

ROLE_PARAM, ROLE_M, ROLE_V, ROLE_GRAD = 11, 12, 13, 14


@dataclass(frozen=True)
class InnerRecipe:
    param_std: float = 0.02
    m_std: float = 1e-4
    v_std: float = 1e-4
    norms: Sequence[float] = (0.5, 2.0, 0.9, 4.0)


@dataclass
class InnerState:
    params: List[torch.Tensor]
    exp_avg: List[torch.Tensor]
    exp_avg_sq: List[torch.Tensor]
    grads: List[torch.Tensor]

    @property
    def n(self) -> int:
        return self.params[0].numel()

    @property
    def k(self) -> int:
        return len(self.params)


def _fill(out: torch.Tensor, std: float, seed: int, role: int, k: int, square: bool = False) -> None:
    n = out.numel()
    for c, lo in enumerate(range(0, n, CHUNK)):
        hi = min(n, lo + CHUNK)
        torch.randn(hi - lo, generator=_generator(seed, role, k, c, out.device), device=out.device,
                    dtype=torch.float32, out=out[lo:hi])
        out[lo:hi].mul_(std)
        if square:
            out[lo:hi].mul_(out[lo:hi])


def empty_state(n: int, k: int, device="cpu", params: Optional[List[torch.Tensor]] = None) -> InnerState:
    def e():
        return torch.empty(n, dtype=torch.float32, device=device)
    return InnerState(params if params is not None else [e() for _ in range(k)],
                      [e() for _ in range(k)], [e() for _ in range(k)], [e() for _ in range(k)])


def fill_state(st: InnerState, seed: int, recipe: InnerRecipe = InnerRecipe(), fill_params: bool = True) -> None:
    for k in range(st.k):
        if fill_params:
            _fill(st.params[k], recipe.param_std, seed, ROLE_PARAM, k)
        _fill(st.exp_avg[k], recipe.m_std, seed, ROLE_M, k)
        _fill(st.exp_avg_sq[k], recipe.v_std, seed, ROLE_V, k, square=True)


def fill_grads(st: InnerState, seed: int, step: int, recipe: InnerRecipe = InnerRecipe()) -> None:
    """Gradient of every worker for one step (a fresh draw per step)."""
    n = st.n
    for k in range(st.k):
        std = recipe.norms[k % len(recipe.norms)] / math.sqrt(max(n, 1))
        _fill(st.grads[k], std, seed * 7919 + step, ROLE_GRAD, k)


def make_state(n: int, k: int, seed: int = 42, recipe: InnerRecipe = InnerRecipe(), device="cpu") -> InnerState:
    st = empty_state(n, k, device)
    fill_state(st, seed, recipe)
    fill_grads(st, seed, 0, recipe)
    return st
