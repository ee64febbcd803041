"""Seeded synthetic inputs for one synchronisation round.

These generators stand in for the inner loop of every worker (K local
trajectories of AdamW steps, which need a model and a dataset): they write the
synchronised parameters theta, the outer momentum v and K worker endpoints
theta_k = theta + a*s + b*e_k built from a drift s shared by all workers and an
independent drift e_k per worker.  Everything is a normal draw from torch's
seeded generator, on the CPU or on the GPU; no part of the round's arithmetic
lives here, and both the oracle and the GPU path read the exact bits written.

Each buffer draws from its own generator, seeded from (seed, role, worker,
chunk), so a buffer can be regenerated chunk by chunk without holding the
whole of it in temporary memory.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import torch

CHUNK = 1 << 26  # elements per generator substream

ROLE_THETA, ROLE_MOMENTUM, ROLE_SHARED, ROLE_INDEP = 1, 2, 3, 4


@dataclass(frozen=True)
class DriftRecipe:
    """theta ~ N(0, theta_std); v ~ N(0, momentum_std);
    theta_k = theta + shared_coef*s + indep_coef*e_k with s ~ N(0, shared_std),
    e_k ~ N(0, indep_std).  All *_std are standard deviations."""

    theta_std: float = 0.02
    momentum_std: float = 1e-4
    shared_std: float = 1e-3
    indep_std: float = 1e-3
    shared_coef: float = 0.7
    indep_coef: float = 0.3


# Tiny / 1.1B / 3B recipe: theta_k = theta + 0.7 s + 0.3 e_k, s, e_k ~ N(0, 1e-3).
MIXED = DriftRecipe()


def spread_recipe(sigma: float) -> DriftRecipe:
    """GPT-2-small recipe: theta_k = theta + s + e_k, s ~ N(0,1e-3), e_k ~ N(0,sigma)."""
    return DriftRecipe(shared_coef=1.0, indep_coef=1.0, indep_std=sigma)


def _generator(seed: int, role: int, k: int, chunk: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    key = (((seed * 1_000_003 + role) * 10_007 + k) * 1_000_033 + chunk) & 0x7FFF_FFFF_FFFF_FFFF
    g.manual_seed(key)
    return g


def _normal_into(out: torch.Tensor, std: float, seed: int, role: int, k: int) -> None:
    """Fill a flat fp32 tensor with N(0, std) draws, chunk by chunk."""
    n = out.numel()
    for c, lo in enumerate(range(0, n, CHUNK)):
        hi = min(n, lo + CHUNK)
        g = _generator(seed, role, k, c, out.device)
        torch.randn(hi - lo, generator=g, device=out.device, dtype=torch.float32, out=out[lo:hi])
        out[lo:hi].mul_(std)


@dataclass
class RoundInputs:
    theta: torch.Tensor             # [n] fp32
    momentum: torch.Tensor          # [n] fp32
    replicas: List[torch.Tensor]    # k x [n], fp32 or bf16

    @property
    def n(self) -> int:
        return self.theta.numel()

    @property
    def k(self) -> int:
        return len(self.replicas)


def empty_inputs(n: int, k: int, replica_dtype=torch.float32, device="cpu") -> RoundInputs:
    theta = torch.empty(n, dtype=torch.float32, device=device)
    mom = torch.empty(n, dtype=torch.float32, device=device)
    reps = [torch.empty(n, dtype=replica_dtype, device=device) for _ in range(k)]
    return RoundInputs(theta, mom, reps)


def fill_theta_momentum(inp: RoundInputs, seed: int, recipe: DriftRecipe = MIXED) -> None:
    _normal_into(inp.theta, recipe.theta_std, seed, ROLE_THETA, 0)
    _normal_into(inp.momentum, recipe.momentum_std, seed, ROLE_MOMENTUM, 0)


def fill_replicas(inp: RoundInputs, seed: int, recipe: DriftRecipe = MIXED,
                  scale: float = 1.0, indep_scale: Optional[List[float]] = None) -> None:
    """theta_k = theta + scale*(shared_coef*s + indep_coef*indep_scale[k]*e_k).

    ``scale`` and ``indep_scale`` let a multi-round workload grow or jitter the
    drift; the default is the plain recipe."""
    n = inp.n
    dev = inp.theta.device
    for lo in range(0, n, CHUNK):
        hi = min(n, lo + CHUNK)
        c = lo // CHUNK
        s = torch.randn(hi - lo, generator=_generator(seed, ROLE_SHARED, 0, c, dev),
                        device=dev, dtype=torch.float32)
        s.mul_(recipe.shared_std * recipe.shared_coef * scale)
        base = inp.theta[lo:hi] + s
        del s
        for k, rep in enumerate(inp.replicas):
            e = torch.randn(hi - lo, generator=_generator(seed, ROLE_INDEP, k, c, dev),
                            device=dev, dtype=torch.float32)
            f = recipe.indep_std * recipe.indep_coef * scale
            if indep_scale is not None:
                f *= indep_scale[k]
            e.mul_(f)
            e.add_(base)
            rep[lo:hi].copy_(e)  # cast to the replica dtype (bf16: round to nearest even)
            del e
        del base


def make_round_inputs(n: int, k: int, seed: int = 42, recipe: DriftRecipe = MIXED,
                      replica_dtype=torch.float32, device="cpu") -> RoundInputs:
    inp = empty_inputs(n, k, replica_dtype, device)
    fill_theta_momentum(inp, seed, recipe)
    fill_replicas(inp, seed, recipe)
    return inp
