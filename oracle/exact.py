"""Exact rational evaluation of one synchronisation round (test infrastructure).

For tiny inputs (a handful of parameters and workers) every quantity of the
round is computed in ``fractions.Fraction`` arithmetic, element by element and
term by term, with no library routine at all:

  Delta_k = theta - theta_k, Delta_bar = (1/K) sum_k Delta_k,
  D = (1/K) sum_k ||Delta_k||^2, C = K ||Delta_bar||^2 / (D + eps),
  disagreement = (1/K) sum_k ||Delta_k - Delta_bar||^2
      (eq. adaptive-h-core-diagnostics; App. C.1),
  v' = mu v + Delta_tilde, d = Delta_tilde + mu v', theta' = theta - eta d
      (eq. autoloco-corrected-nesterov; Delta_tilde = Delta_bar / rho when
      normalised, eq. normalized-pseudo-gradient).

Binary floating-point inputs convert to fractions exactly, so this pins the
float64 oracle to within its own rounding.
"""
from __future__ import annotations

from fractions import Fraction
from typing import Dict, List, Sequence


def frac(x) -> Fraction:
    return x if isinstance(x, Fraction) else Fraction(float(x))


def exact_round(theta: Sequence, momentum: Sequence, replicas: Sequence[Sequence],
                mu, eta, rho, normalize: bool, eps) -> Dict[str, object]:
    th = [frac(x) for x in theta]
    v = [frac(x) for x in momentum]
    reps = [[frac(x) for x in r] for r in replicas]
    mu, eta, rho, eps = frac(mu), frac(eta), frac(rho), frac(eps)
    n = len(th)
    k = len(reps)
    deltas: List[List[Fraction]] = []
    for r in reps:
        deltas.append([th[j] - r[j] for j in range(n)])
    mean = []
    for j in range(n):
        acc = Fraction(0)
        for i in range(k):
            acc += deltas[i][j]
        mean.append(acc / k)
    sq_norm = []
    sq_dev = []
    for i in range(k):
        s = Fraction(0)
        q = Fraction(0)
        for j in range(n):
            s += deltas[i][j] * deltas[i][j]
            q += (deltas[i][j] - mean[j]) * (deltas[i][j] - mean[j])
        sq_norm.append(s)
        sq_dev.append(q)
    sq_mean = Fraction(0)
    for j in range(n):
        sq_mean += mean[j] * mean[j]
    d_energy = sum(sq_norm, Fraction(0)) / k
    coherence = k * sq_mean / (d_energy + eps)
    disagreement = sum(sq_dev, Fraction(0)) / k
    th_new = []
    v_new = []
    for j in range(n):
        dt = mean[j] / rho if normalize else mean[j]
        vn = mu * v[j] + dt
        d = dt + mu * vn
        v_new.append(vn)
        th_new.append(th[j] - eta * d)
    return {
        "deltas": deltas, "mean": mean, "sq_norm": sq_norm, "sq_dev": sq_dev,
        "sq_mean": sq_mean, "D": d_energy, "C": coherence,
        "disagreement": disagreement, "theta": th_new, "momentum": v_new,
    }
