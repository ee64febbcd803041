"""Whole-run simulation of the interval controller (host only).

For many random runs over the full training budget, a synthetic statistics
process drives the controller: the drift energy follows the learning-rate
mass of the executed interval (D ~ (c Lambda)^2) with multiplicative noise,
the coherence fluctuates, the token density per step varies (padding), and
random intervals carry a coherence loss or a non-finite statistic.  The
library's C++ controller must take exactly the oracle controller's decisions,
and every decision must respect the rules that hold at any point of a run
(App. A; Table "AutoLoCo configuration")."""
import math
import random
import warnings

import pytest

import paper_2609_36662_amd as al
from oracle import controller as oc
from oracle import correction as ocorr
from tests.test_lib_host import _ccfg

CONFIGS = {
    "c4": oc.ControllerConfig(),
    "c4_mu07_norm": oc.ControllerConfig(outer=ocorr.OuterConfig(mu_base=0.7, normalize=True)),
    "sft": oc.ControllerConfig(h_base=100, h_min=50, h_max=150, q_h=10, budget_steps=6490,
                               sched=ocorr.Schedule(peak=5e-6, warmup=195, total=6490),
                               outer=ocorr.OuterConfig(mu_base=0.7, normalize=True)),
}


def _simulate(cfg: oc.ControllerConfig, seed: int, noise: float, p_event: float):
    rng = random.Random(seed)
    ctl = oc.OracleController(cfg)
    dec = ctl.select_interval(None)
    decs, obs = [dec], []
    c_level = rng.uniform(2.0, 7.0)
    while not dec.done:
        lam = ocorr.lr_mass(cfg.sched, dec.start_step, dec.h_step)
        d = (30.0 * lam) ** 2 * math.exp(rng.gauss(0.0, noise))
        c = c_level * math.exp(rng.gauss(0.0, noise))
        finite = True
        u = rng.random()
        if u < p_event:
            c *= math.exp(-rng.uniform(0.002, 0.05))          # coherence loss of random size
        elif u < 1.5 * p_event:
            d, finite = float("nan"), False
        density = 1_048_576.0 * rng.uniform(0.85, 1.0)
        o = oc.Observation(d, c, lam, density * dec.h_step, dec.h_step, finite)
        obs.append(o)
        dec = ctl.select_interval(o)
        decs.append(dec)
    return decs, obs


def _check_rules(cfg, decs):
    executed = [d for d in decs if not d.done]
    assert sum(d.h_step for d in executed) == cfg.budget_steps
    assert decs[-1].done
    starts = [d.start_step for d in executed]
    assert starts == sorted(starts) and starts[0] == 0
    for d in executed[:-1]:
        assert d.h_step % cfg.q_h == 0 or d.h_step == d.h_tok, d
        assert d.h_step >= cfg.q_h
    for d in executed:
        assert cfg.h_min <= d.h_tok <= cfg.h_max
        c = d.coeffs
        assert c.rho >= 1.0 and cfg.outer.mu_min <= c.mu <= cfg.outer.mu_max and c.kappa <= cfg.outer.kappa_max
        assert c.eta / (1 - c.mu) == pytest.approx(c.kappa * cfg.outer.eta_base / (1 - cfg.outer.mu_base), rel=1e-12)
        assert c.rho == max(d.lambda_sel / (d.lambda_base + cfg.outer.eps), 1.0)


@pytest.mark.parametrize("name", sorted(CONFIGS))
@pytest.mark.parametrize("seed", range(8))
def test_full_run_library_equals_oracle(name, seed):
    cfg = CONFIGS[name]
    noise = [0.002, 0.01, 0.05][seed % 3]
    p_event = [0.0, 0.03, 0.1][(seed // 3) % 3]
    decs, obs = _simulate(cfg, 1000 * seed + len(name), noise, p_event)
    _check_rules(cfg, decs)
    ties = [(i, d.z_max) for i, d in enumerate(decs) if not math.isnan(d.z_max)
            and any(abs(d.z_max - t) < 1e-6 for t in (cfg.thr_cand, cfg.thr_mod, cfg.thr_sev))]
    if ties:
        warnings.warn(f"near-tie z values in {name}/{seed}: {ties}")
    ctl = al.autoloco_controller_create(_ccfg(cfg))
    got = al.autoloco_select_interval(ctl, None)
    for i, o in enumerate(obs):
        r = decs[i]
        assert (got.start_step, got.h_tok, got.h_step, got.h_ref, got.phase) == \
            (r.start_step, r.h_tok, r.h_step, r.h_ref, r.phase), i
        assert (got.coeffs.mu, got.coeffs.eta_out, got.coeffs.rho) == (r.coeffs.mu, r.coeffs.eta, r.coeffs.rho), i
        got = al.autoloco_select_interval(ctl, al.make_observation(o.D, o.C, o.lambda_done, o.tokens,
                                                                   o.h_step_done, o.finite))
        assert got.assessment == decs[i + 1].assessment, i
        z_o = decs[i + 1].z_max
        assert (math.isnan(got.z_max) and math.isnan(z_o)) or got.z_max == z_o, i
    assert got.done
