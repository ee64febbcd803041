"""Adaptive interval controller and token mapper, in plain Python doubles
(test infrastructure only).

Follows Sec. "Adaptive Interval Selection" (eqs. adaptive-h-lr-mass,
adaptive-h-core-residuals, adaptive-h-core-deviation, adaptive-h-token-mapping)
and App. A (current-run reference, interval evaluation, horizon updates, Table
"Interval assessments"), with the constants of Table "AutoLoCo configuration".
Horizons H below are token-equivalent horizons (H^tok) unless named h_step or
h_ref.

Phases, in the order the paper describes them:
  WARMUP    recipe horizon H_base while the inner learning-rate warm-up runs;
            an interval whose last step completes the warm-up is the first
            reference interval.
  REF_BOOT  two finite intervals at H_base; the reference (D_ref, C_ref) is the
            geometric mean of their diagnostics, Lambda_ref the latest one.
  INIT      after an adoption, a return or a reduction: one interval at the new
            horizon sets the reference.
  VAR       three further intervals at the accepted horizon; their residuals
            fill the residual histories unconditionally.
  MONITOR   each interval is assessed by z_max (Table "Interval assessments"):
            increase-supported proposes a candidate, reference-consistent keeps
            the horizon, two consecutive moderate deviations reduce it by 1.20,
            a severe deviation reduces it by 1.50.  Only supported or
            consistent intervals at the accepted horizon update the histories,
            the log-space EMA of D_ref and C_ref, and Lambda_ref.
  CAND1/2   a supported first candidate interval is adopted at once, a
            consistent one earns one more interval at the candidate, and a
            moderate or severe one (in either) rejects the candidate, leaves a
            rejected-horizon bound and returns to the accepted horizon.
  DONE      the training budget is spent.

Readings of points the paper leaves open (each also listed in the oracle
package docstring as parity unpinned where no printed value fixes it):
  * robust scale s = max(1.4826 * MAD, 1e-3); an empty history contributes 0;
  * log-space EMA coefficient 0.9 for D_ref and C_ref, skipped for a
    non-positive value;
  * a reduction snaps to the admissible multiple of q_H nearest H/factor that
    is strictly below the accepted H (ties to the lower one); the geometric
    midpoint under a bound picks the admissible H strictly between the
    accepted and the rejected horizon nearest sqrt(H_acc * H_rej) (ties lower);
  * two consecutive severe-or-invalid intervals fall back to H_min;
  * a non-finite required statistic is "invalid": the reduction path with the
    severe divisor outside the candidate phases, a rejection inside them;
    warm-up intervals ignore the diagnostics;
  * the rejected-horizon bound stores the previewed learning-rate mass of the
    rejected interval and retires once a preview at the bound falls to at most
    0.90 of it;
  * the token-mapped step horizon rounds half up to a multiple of q_H and is
    at least q_H; before M_base is known, H^step = H^tok and H^ref = H_base;
  * the last interval is truncated to the remaining budget.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from enum import IntEnum
from typing import List, Optional, Tuple

from .correction import OuterCoeffs, OuterConfig, Schedule, lr_mass, outer_correction


class Phase(IntEnum):
    WARMUP = 0
    REF_BOOT = 1
    INIT = 2
    VAR = 3
    MONITOR = 4
    CAND1 = 5
    CAND2 = 6
    DONE = 7


class Assessment(IntEnum):
    NONE = -1
    SUPPORTED = 0
    CONSISTENT = 1
    MODERATE = 2
    SEVERE = 3
    INVALID = 4


@dataclass(frozen=True)
class ControllerConfig:
    h_base: int = 500
    h_min: int = 250
    h_max: int = 750
    q_h: int = 50
    budget_steps: int = 50_000
    beta_tok: float = 0.9
    eps: float = 1e-12
    thr_cand: float = 1.5
    thr_mod: float = 2.5
    thr_sev: float = 4.0
    cand_exposure: float = 1.15
    retire_frac: float = 0.90
    red_moderate: float = 1.20
    red_severe: float = 1.50
    ref_ema: float = 0.9
    mad_scale: float = 1.4826
    scale_floor: float = 1e-3
    n_mapper_boot: int = 3
    n_ref_boot: int = 2
    n_var: int = 3
    hist_max: int = 16
    moderate_confirm: int = 2
    fallback_count: int = 2
    sched: Schedule = field(default_factory=Schedule)
    outer: OuterConfig = field(default_factory=OuterConfig)


@dataclass(frozen=True)
class Observation:
    D: float
    C: float
    lambda_done: float
    tokens: float
    h_step_done: int
    finite: bool = True


@dataclass(frozen=True)
class Decision:
    start_step: int
    h_tok: int
    h_step: int
    h_ref: int
    lambda_sel: float
    lambda_base: float
    z_max: float
    assessment: int
    phase: int
    coeffs: OuterCoeffs
    done: bool


def _median(xs: List[float]) -> float:
    s = sorted(xs)
    n = len(s)
    if n % 2 == 1:
        return s[n // 2]
    return (s[n // 2 - 1] + s[n // 2]) / 2


class OracleController:
    def __init__(self, cfg: ControllerConfig = ControllerConfig()):
        self.cfg = cfg
        self.phase = Phase.WARMUP
        self.started = False
        self.start = 0          # first step of the interval in flight
        self.h_cur = cfg.h_base  # H^tok of the interval in flight
        self.h_step = 0
        self.lambda_sel = 0.0
        self.h_acc = cfg.h_base
        self.h_cand = 0
        self.boot: List[Tuple[float, float, float]] = []
        self.d_ref = 0.0
        self.c_ref = 0.0
        self.l_ref = 0.0
        self.hist_d: List[float] = []
        self.hist_c: List[float] = []
        self.var_count = 0
        self.mod_streak = 0
        self.bad_streak = 0
        self.bound: Optional[Tuple[int, float]] = None
        self.m_samples: List[float] = []
        self.m_base: Optional[float] = None
        self.n_hat: Optional[float] = None
        self.interval = 0

    # ------------------------------------------------------------ helpers --
    def admissible(self) -> List[int]:
        q = self.cfg.q_h
        lo = -(-self.cfg.h_min // q)
        hi = self.cfg.h_max // q
        return [m * q for m in range(lo, hi + 1)]

    def map_steps(self, h_tok: int) -> int:
        """Token-equivalent horizon -> executable steps (eq. adaptive-h-token-mapping)."""
        cfg = self.cfg
        if self.m_base is None or self.n_hat is None:
            return h_tok
        x = self.m_base * h_tok / (cfg.h_base * (self.n_hat + cfg.eps))
        h = cfg.q_h * math.floor(x / cfg.q_h + 0.5)
        return max(h, cfg.q_h)

    def ref_steps(self) -> int:
        if self.m_base is None or self.n_hat is None:
            return self.cfg.h_base
        return self.map_steps(self.cfg.h_base)

    def _residuals(self, obs: Observation) -> Tuple[float, float]:
        eps = self.cfg.eps
        xi = obs.lambda_done / (self.l_ref + eps)
        r_d = math.log(math.sqrt(obs.D) / (math.sqrt(self.d_ref) * xi + eps) + eps)
        r_c = -math.log(obs.C / (self.c_ref + eps) + eps)
        return r_d, r_c

    def _z(self, hist: List[float], r: float) -> float:
        if not hist:
            return 0.0
        c = _median(hist)
        mad = _median([abs(h - c) for h in hist])
        s = self.cfg.mad_scale * mad
        if s < self.cfg.scale_floor:
            s = self.cfg.scale_floor
        dev = r - c
        if dev < 0.0:
            dev = 0.0
        return dev / s

    def _classify(self, z: float) -> Assessment:
        cfg = self.cfg
        if math.isnan(z):
            return Assessment.INVALID
        if z < cfg.thr_cand:
            return Assessment.SUPPORTED
        if z < cfg.thr_mod:
            return Assessment.CONSISTENT
        if z < cfg.thr_sev:
            return Assessment.MODERATE
        return Assessment.SEVERE

    def _push(self, r_d: float, r_c: float) -> None:
        self.hist_d.append(r_d)
        self.hist_c.append(r_c)
        if len(self.hist_d) > self.cfg.hist_max:
            self.hist_d.pop(0)
            self.hist_c.pop(0)

    def _set_reference(self, d: float, c: float, lam: float) -> None:
        self.d_ref, self.c_ref, self.l_ref = d, c, lam
        self.hist_d = []
        self.hist_c = []
        self.var_count = 0
        self.phase = Phase.VAR

    def _ema(self, d: float, c: float, lam: float) -> None:
        a = self.cfg.ref_ema
        if d > 0.0 and self.d_ref > 0.0:
            self.d_ref = math.exp(a * math.log(self.d_ref) + (1.0 - a) * math.log(d))
        if c > 0.0 and self.c_ref > 0.0:
            self.c_ref = math.exp(a * math.log(self.c_ref) + (1.0 - a) * math.log(c))
        self.l_ref = lam

    def _snap_below(self, x: float, h_cur: int) -> int:
        best = None
        for h in self.admissible():
            if h >= h_cur:
                continue
            if best is None or abs(h - x) < abs(best - x):
                best = h
        return h_cur if best is None else best

    def _reduce(self, factor: float) -> None:
        if self.bad_streak >= self.cfg.fallback_count:
            h_new = self.cfg.h_min
        else:
            h_new = self._snap_below(self.h_acc / factor, self.h_acc)
        self.h_acc = h_new
        self.mod_streak = 0
        self.boot = []
        self.phase = Phase.INIT

    def _reject(self) -> None:
        self.bound = (self.h_cur, self.lambda_sel)
        self.phase = Phase.INIT

    def _candidate(self, start: int) -> Optional[int]:
        cfg = self.cfg
        if self.bound is not None:
            h_rej, l_rej = self.bound
            if lr_mass(cfg.sched, start, self.map_steps(h_rej)) <= cfg.retire_frac * l_rej:
                self.bound = None
        if self.bound is not None:
            h_rej = self.bound[0]
            g = math.sqrt(self.h_acc * h_rej)
            best = None
            for h in self.admissible():
                if self.h_acc < h < h_rej:
                    if best is None or abs(h - g) < abs(best - g):
                        best = h
            return best
        l_acc = lr_mass(cfg.sched, start, self.map_steps(self.h_acc))
        best = None
        for h in self.admissible():
            if h > self.h_acc:
                if lr_mass(cfg.sched, start, self.map_steps(h)) <= cfg.cand_exposure * l_acc:
                    best = h
        return best

    # ---------------------------------------------------------- the step --
    def _observe(self, obs: Observation) -> Tuple[Assessment, float]:
        cfg = self.cfg
        # token mapper: density EMA every interval, M_base from the first ones
        if obs.h_step_done > 0 and math.isfinite(obs.tokens):
            n_bar = obs.tokens / obs.h_step_done
            if self.n_hat is None:
                self.n_hat = n_bar
            else:
                self.n_hat = cfg.beta_tok * self.n_hat + (1.0 - cfg.beta_tok) * n_bar
            if len(self.m_samples) < cfg.n_mapper_boot:
                self.m_samples.append(obs.tokens)
                if len(self.m_samples) == cfg.n_mapper_boot:
                    self.m_base = _median(self.m_samples)

        end = self.start + self.h_step
        if self.phase == Phase.WARMUP:
            if end < cfg.sched.warmup:
                return Assessment.NONE, math.nan
            self.phase = Phase.REF_BOOT

        finite = (bool(obs.finite) and math.isfinite(obs.D) and math.isfinite(obs.C)
                  and math.isfinite(obs.lambda_done) and obs.D >= 0.0 and obs.C >= 0.0)
        if not finite:
            self.bad_streak += 1
            self.mod_streak = 0
            if self.phase in (Phase.CAND1, Phase.CAND2):
                self._reject()
            else:
                self._reduce(cfg.red_severe)
            return Assessment.INVALID, math.nan

        ph = self.phase
        if ph == Phase.REF_BOOT:
            self.bad_streak = 0
            self.boot.append((obs.D, obs.C, obs.lambda_done))
            if len(self.boot) >= cfg.n_ref_boot:
                pd = 1.0
                pc = 1.0
                for d, c, _ in self.boot:
                    pd *= d
                    pc *= c
                n = len(self.boot)
                if n == 2:
                    d_ref, c_ref = math.sqrt(pd), math.sqrt(pc)
                else:
                    d_ref, c_ref = pd ** (1.0 / n), pc ** (1.0 / n)
                self._set_reference(d_ref, c_ref, self.boot[-1][2])
                self.boot = []
            return Assessment.NONE, math.nan
        if ph == Phase.INIT:
            self.bad_streak = 0
            self._set_reference(obs.D, obs.C, obs.lambda_done)
            return Assessment.NONE, math.nan

        r_d, r_c = self._residuals(obs)
        if ph == Phase.VAR:
            self.bad_streak = 0
            self._push(r_d, r_c)
            self.var_count += 1
            if self.var_count >= cfg.n_var:
                self.phase = Phase.MONITOR
            return Assessment.NONE, math.nan

        z_d = self._z(self.hist_d, r_d)
        z_c = self._z(self.hist_c, r_c)
        z = z_d if z_d > z_c else z_c
        a = self._classify(z)
        if a == Assessment.INVALID:
            self.bad_streak += 1
            self.mod_streak = 0
            if ph in (Phase.CAND1, Phase.CAND2):
                self._reject()
            else:
                self._reduce(cfg.red_severe)
            return a, z

        if ph == Phase.MONITOR:
            if a in (Assessment.SUPPORTED, Assessment.CONSISTENT):
                self._push(r_d, r_c)
                self._ema(obs.D, obs.C, obs.lambda_done)
                self.mod_streak = 0
                self.bad_streak = 0
                if a == Assessment.SUPPORTED:
                    cand = self._candidate(end)
                    if cand is not None:
                        self.h_cand = cand
                        self.phase = Phase.CAND1
            elif a == Assessment.MODERATE:
                self.mod_streak += 1
                self.bad_streak = 0
                if self.mod_streak >= cfg.moderate_confirm:
                    self._reduce(cfg.red_moderate)
            else:
                self.bad_streak += 1
                self.mod_streak = 0
                self._reduce(cfg.red_severe)
            return a, z

        # candidate phases
        self.bad_streak = 0
        adopt = a == Assessment.SUPPORTED or (a == Assessment.CONSISTENT and ph == Phase.CAND2)
        if adopt:
            self.h_acc = self.h_cur
            self.mod_streak = 0
            self._set_reference(obs.D, obs.C, obs.lambda_done)
        elif a == Assessment.CONSISTENT:
            self.phase = Phase.CAND2
        else:
            self._reject()
        return a, z

    def _next_h_tok(self) -> int:
        if self.phase in (Phase.CAND1, Phase.CAND2):
            return self.h_cand
        return self.h_acc

    def select_interval(self, obs: Optional[Observation]) -> Decision:
        cfg = self.cfg
        if self.phase == Phase.DONE:
            raise RuntimeError("training budget already spent")
        if not self.started:
            if obs is not None:
                raise ValueError("the first call takes no observation")
            self.started = True
            a, z = Assessment.NONE, math.nan
            start = 0
        else:
            if obs is None:
                raise ValueError("an observation of the completed interval is required")
            a, z = self._observe(obs)
            start = self.start + self.h_step
        if start >= cfg.budget_steps:
            self.phase = Phase.DONE
            one = outer_correction(cfg.outer, 0.0, 0.0)
            return Decision(start, 0, 0, 0, 0.0, 0.0, z, int(a), int(Phase.DONE), one, True)
        h_tok = self._next_h_tok()
        h_step = self.map_steps(h_tok)
        h_ref = self.ref_steps()
        if start + h_step > cfg.budget_steps:
            h_step = cfg.budget_steps - start
        lam = lr_mass(cfg.sched, start, h_step)
        lam_b = lr_mass(cfg.sched, start, h_ref)
        coeffs = outer_correction(cfg.outer, lam, lam_b)
        self.start = start
        self.h_cur = h_tok
        self.h_step = h_step
        self.lambda_sel = lam
        self.interval += 1
        return Decision(start, h_tok, h_step, h_ref, lam, lam_b, z, int(a), int(self.phase),
                        coeffs, False)
