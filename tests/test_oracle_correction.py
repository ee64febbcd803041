"""Pins of the oracle's schedule, learning-rate masses and Outer Optimizer
Correction against closed forms and the special cases the paper states."""
import math
from fractions import Fraction

import pytest

from oracle.correction import (OuterConfig, Schedule, inner_lr, interval_ratio, lr_mass,
                               outer_correction)

SCHED = Schedule()          # peak 4e-4, warm-up 1000, budget 50000, min 0
CFG9 = OuterConfig(mu_base=0.9)
CFG7 = OuterConfig(mu_base=0.7)


def test_warmup_mass_closed_form():
    # sum_{s=a}^{b-1} peak (s+1)/W = peak/W * (b(b+1)/2 - a(a+1)/2)
    for a, n in [(0, 500), (500, 500), (0, 1000), (123, 77)]:
        b = a + n
        exact = Fraction(SCHED.peak) / SCHED.warmup * Fraction(b * (b + 1) - a * (a + 1), 2)
        assert lr_mass(SCHED, a, n) == pytest.approx(float(exact), rel=1e-13)


def test_cosine_mass_closed_form():
    # sum_{j<n} cos(alpha + j beta) = sin(n beta/2)/sin(beta/2) cos(alpha + (n-1) beta/2)
    W, T, pk, mn = SCHED.warmup, SCHED.total, SCHED.peak, SCHED.min_lr
    beta = math.pi / (T - W)
    for a, n in [(1000, 500), (20000, 75), (20000, 50), (16000, 750), (49000, 1000)]:
        alpha = math.pi * (a - W) / (T - W)
        csum = math.sin(n * beta / 2) / math.sin(beta / 2) * math.cos(alpha + (n - 1) * beta / 2)
        closed = n * (mn + (pk - mn) / 2) + (pk - mn) / 2 * csum
        assert lr_mass(SCHED, a, n) == pytest.approx(closed, rel=1e-11)


def test_schedule_shape():
    assert inner_lr(SCHED, 999) == SCHED.peak
    assert inner_lr(SCHED, 1000) == SCHED.peak
    assert inner_lr(SCHED, 50_000) == pytest.approx(0.0, abs=1e-20)
    assert inner_lr(SCHED, 60_000) == inner_lr(SCHED, 50_000)   # held at min after the budget
    assert lr_mass(SCHED, 20_000, 0) == 0.0


def test_rho_one_recovers_base_exactly():
    # eq. fixed-horizon-correction: rho = 1 gives mu_base, kappa 1, eta_base exactly
    for cfg in (CFG9, CFG7):
        lam = lr_mass(SCHED, 20_000, 500)
        c = outer_correction(cfg, lam, lam)
        assert c.rho == 1.0 and c.mu == cfg.mu_base and c.kappa == 1.0 and c.eta == cfg.eta_base


def test_short_interval_floors_ratio_at_one():
    # eq. app-outer-correction-ratios: rho_unc < 1 uses rho = 1
    c = outer_correction(CFG9, lr_mass(SCHED, 20_000, 250), lr_mass(SCHED, 20_000, 500))
    assert c.rho == 1.0 and c.mu == 0.9 and c.eta == 0.7
    assert interval_ratio(0.0, 0.0, 1e-12) == 1.0


@pytest.mark.parametrize("cfg", [CFG9, CFG7])
@pytest.mark.parametrize("rho", [1.0, 1.2, 1.5, 2.0, 3.0, 5.0])
def test_scale_matching_and_bounds(cfg, rho):
    # eq. app-outer-step-ratio: eta/(1-mu) = kappa eta_base/(1-mu_base);
    # mu within [mu_min, mu_max]; kappa = min(rho, kappa_max)
    c = outer_correction(cfg, rho, 1.0 - cfg.eps)  # lam/(lam_base+eps) = rho
    assert c.rho == pytest.approx(rho, rel=1e-15)
    assert cfg.mu_min <= c.mu <= cfg.mu_max
    assert c.kappa == min(c.rho, cfg.kappa_max)
    assert c.eta / (1 - c.mu) == pytest.approx(c.kappa * cfg.eta_base / (1 - cfg.mu_base), rel=1e-14)


def test_integer_ratio_is_repeated_retention():
    # App. B.4: for integer rho, mu_base^rho is the retention of rho repeated base updates
    for rho, mb in [(2, 0.9), (3, 0.9), (2, 0.7)]:
        c = outer_correction(OuterConfig(mu_base=mb), float(rho), 1.0 - 1e-12)
        rep = 1.0
        for _ in range(rho):
            rep *= mb
        expect = min(max(rep, 0.45), 0.90)
        assert c.mu == pytest.approx(expect, rel=1e-14)


def test_printed_bounds_active():
    # Table "AutoLoCo configuration": mu in [0.45, 0.90], kappa_max 1.6
    c = outer_correction(CFG7, 3.0, 1.0 - 1e-12)      # 0.7^3 = 0.343 < 0.45
    assert c.mu == 0.45 and c.kappa == 1.6
    c = outer_correction(CFG9, 2.0, 1.0 - 1e-12)      # 0.81, kappa capped at 1.6
    assert c.mu == pytest.approx(0.81, rel=1e-15) and c.kappa == 1.6
    assert c.eta == pytest.approx(0.7 * 1.6 * 0.19 / 0.1, rel=1e-14)
