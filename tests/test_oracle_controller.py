"""Pins of the oracle's adaptive interval controller.

The executed horizon sequence of the C4 run (App. F.2) pins the bootstrap,
calibration, candidate and saturation timing; the remaining tests check the
rules of App. A as the text states them (reductions by 1.20 and 1.50 onto an
admissible multiple strictly below, candidate evaluation and rejection, the
rejected-horizon bound, the token mapper) and the DiLoCo special case
(App. D.2)."""
import math
import os

import pytest

from oracle.controller import Assessment, ControllerConfig, Phase
from oracle.correction import Schedule, lr_mass
from tests.controller_driver import TOKENS_PER_STEP, Event, drive, runs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_sequence():
    vals = {}
    with open(os.path.join(GOLDEN, "c4_executed_intervals.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                k, v = [p.strip() for p in line.split("=", 1)]
                vals[k] = v
    seq = [tuple(int(x) for x in tok.split("x")) for tok in vals["sequence"].split()]
    return seq, int(vals["intervals"]), int(vals["total_steps"])


def test_c4_executed_interval_sequence():
    seq, n_int, total = _golden_sequence()
    decs, _ = drive(ControllerConfig())
    assert runs(decs) == seq
    executed = [d for d in decs if not d.done]
    assert len(executed) == n_int
    assert sum(d.h_step for d in executed) == total
    assert decs[-1].done


def test_candidate_is_longest_within_exposure_multiplier():
    # App. A.2: the candidate is the longest admissible horizon whose previewed
    # LR exposure is at most 1.15x that of the accepted horizon, from the same step.
    cfg = ControllerConfig()
    decs, _ = drive(cfg)
    prev_acc = cfg.h_base
    seen = 0
    for d in decs:
        if d.done:
            break
        if d.phase == Phase.CAND1:
            seen += 1
            base = lr_mass(cfg.sched, d.start_step, prev_acc)
            assert lr_mass(cfg.sched, d.start_step, d.h_tok) <= 1.15 * base
            nxt = d.h_tok + cfg.q_h
            if nxt <= cfg.h_max:
                assert lr_mass(cfg.sched, d.start_step, nxt) > 1.15 * base
            prev_acc = d.h_tok
    assert seen == 5


def test_diloco_special_case_fixed_horizon():
    # App. D.2: a controller that always keeps H_base at the reference density gives
    # H^step = H^ref = H_base, rho = 1 and the base outer coefficients in every interval.
    cfg = ControllerConfig(h_min=500, h_max=500)
    decs, _ = drive(cfg)
    executed = [d for d in decs if not d.done]
    assert len(executed) == 100
    for d in executed:
        assert d.h_step == d.h_ref == 500
        assert d.lambda_sel == d.lambda_base
        assert d.coeffs.rho == 1.0 and d.coeffs.mu == 0.9 and d.coeffs.eta == 0.7


def _stable(h=500, **kw):
    # H_max = H_base: no admissible horizon above the accepted one, so monitoring never proposes a candidate
    return ControllerConfig(h_base=h, h_min=250, h_max=h, **kw)


def _after(decs, t):
    """Decision taken after observing interval t (interval numbering from 1)."""
    return decs[t]


def test_two_moderate_deviations_reduce_by_1_2():
    decs, _ = drive(_stable(), {10: Event(loss=3e-3), 11: Event(loss=3e-3)})
    assert _after(decs, 10).assessment == Assessment.MODERATE
    assert _after(decs, 10).h_tok == 500            # one moderate keeps the horizon
    d = _after(decs, 11)
    assert d.assessment == Assessment.MODERATE
    assert d.h_tok == 400                           # 500/1.2 = 416.7 -> 400
    assert d.phase == Phase.INIT
    # then 1 init + 3 variability + 1 monitoring interval before an increase
    assert [x.phase for x in decs[12:16]] == [Phase.VAR] * 3 + [Phase.MONITOR]


def test_moderate_streak_resets():
    decs, _ = drive(_stable(), {10: Event(loss=3e-3), 12: Event(loss=3e-3)})
    assert all(d.h_tok == 500 for d in decs[:30] if not d.done)


def test_consistent_keeps_horizon():
    decs, _ = drive(_stable(), {10: Event(loss=2e-3)})
    assert _after(decs, 10).assessment == Assessment.CONSISTENT
    assert _after(decs, 10).h_tok == 500 and _after(decs, 10).phase == Phase.MONITOR


def test_severe_reduces_by_1_5_at_once():
    decs, _ = drive(_stable(), {10: Event(loss=5e-3)})
    d = _after(decs, 10)
    assert d.assessment == Assessment.SEVERE
    assert d.h_tok == 350                           # 500/1.5 = 333.3 -> 350
    assert d.phase == Phase.INIT


def test_reduction_tie_goes_to_lower_multiple():
    decs, _ = drive(_stable(750), {10: Event(loss=3e-3), 11: Event(loss=3e-3)})
    assert _after(decs, 11).h_tok == 600            # 750/1.2 = 625: 600 and 650 tie


def test_nonfinite_takes_reduction_path_and_fallback():
    decs, _ = drive(_stable(), {10: Event(nonfinite=True), 11: Event(nonfinite=True)})
    assert _after(decs, 10).assessment == Assessment.INVALID
    assert _after(decs, 10).h_tok == 350
    assert _after(decs, 11).assessment == Assessment.INVALID
    assert _after(decs, 11).h_tok == 250            # repeated invalid: H_min fallback


def test_nonfinite_during_warmup_keeps_recipe_horizon():
    decs, _ = drive(ControllerConfig(), {1: Event(nonfinite=True)})
    assert _after(decs, 1).h_tok == 500 and _after(decs, 1).phase == Phase.WARMUP


def test_candidate_rejected_returns_and_leaves_bound():
    cfg = ControllerConfig()
    decs, _ = drive(cfg, {8: Event(loss=3e-3)})    # interval 8 is the first 550 candidate
    assert decs[7].phase == Phase.CAND1 and decs[7].h_tok == 550
    d = _after(decs, 8)
    assert d.assessment == Assessment.MODERATE
    assert d.h_tok == 500 and d.phase == Phase.INIT  # return, no extra reduction
    # with the bound at 550 and the accepted horizon 500 no admissible horizon lies
    # strictly between, so no candidate is proposed until the bound retires
    later = [x for x in decs[9:] if x.phase == Phase.CAND1]
    assert later, "bound never retired"
    first = later[0]
    # retirement: a preview at the bound has fallen to <= 0.90 of the stored mass
    stored = decs[7].lambda_sel
    assert lr_mass(cfg.sched, first.start_step, 550) <= 0.90 * stored
    # and the first monitoring intervals before retirement proposed nothing
    blocked = [x for x in decs[9:] if x.phase == Phase.MONITOR and x.start_step < first.start_step]
    assert blocked


def test_geometric_midpoint_under_bound():
    # exposure multiplier 1.5 lets the first candidate jump several quanta, so the
    # bound it leaves has admissible horizons strictly inside it.
    cfg = ControllerConfig(cand_exposure=1.5)
    decs, _ = drive(cfg, {8: Event(loss=5e-3)})
    h_rej = decs[7].h_tok
    assert decs[7].phase == Phase.CAND1 and h_rej >= 650
    nxt = [x for x in decs[9:] if x.phase == Phase.CAND1][0]
    g = math.sqrt(500 * h_rej)
    inside = [h for h in range(550, h_rej, 50)]
    best = min(inside, key=lambda h: (abs(h - g), h))
    assert nxt.h_tok == best


def test_consistent_candidate_gets_second_interval():
    decs, _ = drive(ControllerConfig(), {8: Event(loss=2e-3)})
    assert _after(decs, 8).assessment == Assessment.CONSISTENT
    assert _after(decs, 8).phase == Phase.CAND2 and _after(decs, 8).h_tok == 550
    assert _after(decs, 9).phase == Phase.VAR and _after(decs, 9).h_tok == 550   # adopted


def test_second_candidate_interval_can_reject():
    decs, _ = drive(ControllerConfig(), {8: Event(loss=2e-3), 9: Event(loss=3e-3)})
    assert _after(decs, 9).h_tok == 500 and _after(decs, 9).phase == Phase.INIT


def test_token_mapper_median_and_density_ema():
    # Eq. adaptive-h-token-mapping with App. A.3: M_base is the median token mass of
    # the first three intervals, n_hat an EMA (beta 0.9) started at the first interval.
    masses = {1: 1.0, 2: 1.25, 3: 0.5}              # tokens per step relative to 2^20
    dens = lambda t: TOKENS_PER_STEP * (masses.get(t, 0.5))
    cfg = ControllerConfig()
    decs, obs = drive(cfg, density=dens, max_intervals=6)
    m = sorted(o.tokens for o in obs[:3])[1]
    n_hat = obs[0].tokens / obs[0].h_step_done
    for o in obs[1:4]:
        n_hat = 0.9 * n_hat + 0.1 * (o.tokens / o.h_step_done)
    x = m * decs[4].h_tok / (cfg.h_base * (n_hat + cfg.eps))
    assert decs[4].h_step == 50 * math.floor(x / 50 + 0.5)
    # the first three intervals execute the token horizon unmapped
    assert [d.h_step for d in decs[:3]] == [500, 500, 500]
    # lower density -> more steps per token horizon
    assert decs[4].h_step > decs[4].h_tok


def test_budget_truncation_and_done():
    cfg = ControllerConfig(budget_steps=2_300, h_min=500, h_max=500,
                           sched=Schedule(total=2_300))
    decs, _ = drive(cfg)
    executed = [d for d in decs if not d.done]
    assert [d.h_step for d in executed] == [500, 500, 500, 500, 300]
    assert decs[-1].done
