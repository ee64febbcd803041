"""Scripted observation sequences for the interval controller.

``drive`` runs a controller through a training budget.  By default every
completed interval reports diagnostics that sit exactly on the current
reference profile (D = D_ref * xi^2, C = C_ref, so both residuals are ~0 and the
interval is increase-supported); a script can instead inject a coherence loss
of a chosen size at chosen intervals, so that z_max lands in a chosen class of
Table "Interval assessments", or a non-finite statistic.  The reference values
are read from the oracle controller, which is what makes the sequence
self-consistent; the recorded observations can then be replayed verbatim into
any other implementation of the controller.
"""
import math
from dataclasses import dataclass
from typing import Callable, Dict, List, Optional

from oracle.controller import ControllerConfig, Observation, OracleController
from oracle.correction import lr_mass

TOKENS_PER_STEP = float(1 << 20)


@dataclass
class Event:
    # coherence-loss residual to inject (r_C ~ loss); None keeps the interval on-profile
    loss: Optional[float] = None
    nonfinite: bool = False


def drive(cfg: ControllerConfig = ControllerConfig(),
          script: Optional[Dict[int, Event]] = None,
          density: Optional[Callable[[int], float]] = None,
          max_intervals: int = 10_000):
    """Returns (decisions, observations); interval numbering starts at 1."""
    script = script or {}
    ctl = OracleController(cfg)
    dec = ctl.select_interval(None)
    decisions = [dec]
    observations: List[Observation] = []
    t = 1
    while not dec.done and t <= max_intervals:
        lam = lr_mass(cfg.sched, dec.start_step, dec.h_step)
        if ctl.d_ref > 0.0 and ctl.l_ref > 0.0:
            xi = lam / (ctl.l_ref + cfg.eps)
            d = ctl.d_ref * xi * xi
            c = ctl.c_ref
        else:
            d = (10.0 * lam) ** 2
            c = 5.0
        ev = script.get(t)
        finite = True
        if ev is not None:
            if ev.loss is not None:
                c = c * math.exp(-ev.loss)
            if ev.nonfinite:
                d = float("nan")
                finite = False
        n = TOKENS_PER_STEP if density is None else density(t)
        obs = Observation(d, c, lam, n * dec.h_step, dec.h_step, finite)
        observations.append(obs)
        dec = ctl.select_interval(obs)
        decisions.append(dec)
        t += 1
    return decisions, observations


def runs(decisions):
    """Collapse executed step horizons into (horizon, count) runs."""
    out = []
    for d in decisions:
        if d.done:
            break
        if out and out[-1][0] == d.h_step:
            out[-1][1] += 1
        else:
            out.append([d.h_step, 1])
    return [tuple(x) for x in out]
