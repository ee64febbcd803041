"""Pins of the controller's log-space reference EMA (App. A.1), its
median / MAD deviation scale (eq. adaptive-h-core-deviation) and the H_min
fallback (App. A.3 "Reducing the horizon"), with hand-derived expected values
(tests/controller_pins.py), and checks that plausible mistakes planted in the
oracle fail them: a linear-space EMA, a swapped EMA coefficient, a mean- or
standard-deviation scale, the wrong middle of an even history, no consistency
factor, r_D without the square roots or without the learning-rate ratio xi,
and a fallback after one or three
intervals instead of two."""
import math

import pytest

from oracle import controller as oc
from tests import controller_pins as pins


@pytest.mark.parametrize("name", [n for n, _ in pins.SCENARIOS])
def test_hand_derived_pin(name):
    run = dict(pins.SCENARIOS)[name]
    _, checks = run()
    assert pins.failures(checks) == []


def _fails(run) -> bool:
    try:
        _, checks = run()
    except Exception:            # a mutant may also crash the scenario
        return True
    return bool(pins.failures(checks))


def test_linear_space_ema_fails(monkeypatch):
    def linear(self, d, c, lam):
        a = self.cfg.ref_ema
        self.d_ref = a * self.d_ref + (1 - a) * d
        self.c_ref = a * self.c_ref + (1 - a) * c
        self.l_ref = lam
    monkeypatch.setattr(oc.OracleController, "_ema", linear)
    assert _fails(pins.run_ema)


def test_swapped_ema_coefficient_fails(monkeypatch):
    monkeypatch.setattr(pins, "stable", lambda h: oc.ControllerConfig(h_base=h, h_min=250, h_max=h, ref_ema=0.1))
    assert _fails(pins.run_ema)


def test_ema_on_moderate_interval_fails(monkeypatch):
    orig = oc.OracleController._observe

    def observe(self, obs):
        a, z = orig(self, obs)
        if a == oc.Assessment.MODERATE:
            self._ema(obs.D, obs.C, obs.lambda_done)
        return a, z
    monkeypatch.setattr(oc.OracleController, "_observe", observe)
    assert _fails(pins.run_ema)


def _z_with_scale(scale_fn):
    def z(self, hist, r):
        if not hist:
            return 0.0
        c = oc._median(hist)
        s = max(scale_fn(hist, c), self.cfg.scale_floor)
        return max(r - c, 0.0) / s
    return z


def test_mean_absolute_deviation_scale_fails(monkeypatch):
    monkeypatch.setattr(oc.OracleController, "_z",
                        _z_with_scale(lambda h, c: 1.4826 * sum(abs(x - c) for x in h) / len(h)))
    assert _fails(pins.run_mad)


def test_standard_deviation_scale_fails(monkeypatch):
    def std(h, c):
        m = sum(h) / len(h)
        return math.sqrt(sum((x - m) ** 2 for x in h) / len(h))
    monkeypatch.setattr(oc.OracleController, "_z", _z_with_scale(std))
    assert _fails(pins.run_mad)


def test_missing_consistency_factor_fails(monkeypatch):
    monkeypatch.setattr(oc.OracleController, "_z",
                        _z_with_scale(lambda h, c: oc._median([abs(x - c) for x in h])))
    assert _fails(pins.run_mad)


def test_upper_middle_of_even_history_fails(monkeypatch):
    def upper(xs):
        s = sorted(xs)
        return s[len(s) // 2]
    monkeypatch.setattr(oc, "_median", upper)
    assert _fails(pins.run_mad)


def test_drift_residual_without_square_roots_fails(monkeypatch):
    def residuals(self, obs):
        eps = self.cfg.eps
        xi = obs.lambda_done / (self.l_ref + eps)
        r_d = math.log(obs.D / (self.d_ref * xi + eps) + eps)
        r_c = -math.log(obs.C / (self.c_ref + eps) + eps)
        return r_d, r_c
    monkeypatch.setattr(oc.OracleController, "_residuals", residuals)
    assert _fails(pins.run_ema)


def test_drift_residual_without_learning_rate_ratio_fails(monkeypatch):
    def residuals(self, obs):
        eps = self.cfg.eps
        r_d = math.log(math.sqrt(obs.D) / (math.sqrt(self.d_ref) + eps) + eps)
        r_c = -math.log(obs.C / (self.c_ref + eps) + eps)
        return r_d, r_c
    monkeypatch.setattr(oc.OracleController, "_residuals", residuals)
    assert _fails(pins.run_ema)


@pytest.mark.parametrize("count", [1, 3])
def test_other_fallback_counts_fail(monkeypatch, count):
    monkeypatch.setattr(pins, "stable",
                        lambda h: oc.ControllerConfig(h_base=h, h_min=250, h_max=h, fallback_count=count))
    failed = [name for name, run in pins.SCENARIOS if name.startswith("fallback") and _fails(run)]
    assert failed, f"a fallback after {count} interval(s) passes every fallback pin"
