"""The whole method on one GPU, interval after interval (Alg. "AutoLoCo outer
interval"): every worker takes H^step inner AdamW steps on its own replica
(synthetic gradients: a part shared by all workers and a part of its own,
drawn per step), then the fused round computes the statistics, applies the
corrected Nesterov step with the controller's coefficients and resets the
replicas; the statistics drive the library's controller, whose next decision
fixes the next interval's length and coefficients.  The optimiser states stay
with their workers across rounds.

The oracle runs the same loop in float64 (its AdamW, round and controller) on
the same gradient draws, starting every interval from the GPU's state (so the
fp32 rounding of the GPU's stored state does not accumulate across intervals).
Every decision must be identical.  Within an interval each inner step stores
the replicas in fp32, a relative rounding of at most 2^-24 per step, so after H
steps a pseudo-gradient may differ from the float64 one by H 2^-23 |theta_k|;
the element bounds are the round's (1e-5 (|o| + rms(o))) plus that term carried
through the step (v' = mu v + Delta/rho, theta' = theta - eta (Delta/rho + mu v'))."""
import math

import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al
from oracle import adamw as oa
from oracle import controller as oc
from oracle import correction as ocorr
from oracle import round as orr
from tests.gpu_common import assert_close_elementwise
from tests.test_lib_host import _ccfg

pytestmark = pytest.mark.gpu
EPS = 1e-12
TOKENS_PER_STEP = float(1 << 18)
SCHED = ocorr.Schedule(peak=4e-4, warmup=40, total=360)
CFG = oc.ControllerConfig(h_base=20, h_min=10, h_max=30, q_h=5, budget_steps=360, sched=SCHED)
ADAMW = oa.AdamWConfig()


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()


def _grads(n, k, step):
    """Worker gradients of one inner step: 0.6 shared + 0.8 own, unit-variance normals scaled to a norm ~1."""
    g = torch.Generator().manual_seed(50_000 + step)
    shared = torch.randn(n, generator=g)
    out = []
    for kk in range(k):
        gk = torch.Generator().manual_seed(60_000 + 31 * step + kk)
        own = torch.randn(n, generator=gk)
        out.append(((0.6 * shared + 0.8 * own) * (1.2 / math.sqrt(n))).to(torch.float32))
    return out


def test_intervals_of_inner_steps_rounds_and_controller(ctx):
    n, k = 65_539, 4
    gen = torch.Generator().manual_seed(42)
    theta0 = (torch.randn(n, generator=gen) * 0.02).to(torch.float32)
    # GPU state
    th_g = theta0.cuda()
    v_g = torch.zeros(n, device="cuda")
    reps_g = [th_g.clone() for _ in range(k)]
    m_g = [torch.zeros(n, device="cuda") for _ in range(k)]
    s_g = [torch.zeros(n, device="cuda") for _ in range(k)]
    g_g = [torch.empty(n, device="cuda") for _ in range(k)]
    ctl_g = al.autoloco_controller_create(_ccfg(CFG))
    dec_g = al.autoloco_select_interval(ctl_g, None)
    # oracle controller (its state is re-read from the GPU at every interval)
    ctl_o = oc.OracleController(CFG)
    dec_o = ctl_o.select_interval(None)

    intervals, steps = 0, 0
    phases = set()
    while not dec_o.done:
        assert not dec_g.done
        assert (dec_g.start_step, dec_g.h_tok, dec_g.h_step, dec_g.h_ref, dec_g.phase) == \
            (dec_o.start_step, dec_o.h_tok, dec_o.h_step, dec_o.h_ref, dec_o.phase), intervals
        assert (dec_g.coeffs.mu, dec_g.coeffs.eta_out, dec_g.coeffs.rho) == \
            (dec_o.coeffs.mu, dec_o.coeffs.eta, dec_o.coeffs.rho), intervals
        phases.add(dec_o.phase)
        # the oracle starts the interval from the GPU's state
        th_o, v_o = th_g.cpu().numpy().astype(np.float64), v_g.cpu().numpy().astype(np.float64)
        reps_o = [x.cpu().numpy().astype(np.float64) for x in reps_g]
        m_o = [x.cpu().numpy().astype(np.float64) for x in m_g]
        s_o = [x.cpu().numpy().astype(np.float64) for x in s_g]
        # the local inner loops
        H = dec_o.h_step
        for h in range(H):
            s = dec_o.start_step + h
            lr = ocorr.inner_lr(SCHED, s)
            grads = _grads(n, k, s)
            for kk in range(k):
                g_g[kk].copy_(grads[kk])
            co = al.make_adamw_coeffs(lr, s + 1, ADAMW.beta1, ADAMW.beta2, ADAMW.eps, ADAMW.weight_decay,
                                      ADAMW.max_grad_norm)
            st_in = al.autoloco_inner_adamw(ctx, reps_g, m_g, s_g, g_g, co)
            ref_in = oa.inner_step(reps_o, m_o, s_o, [x.numpy().astype(np.float64) for x in grads], lr, s + 1,
                                   ADAMW)
            reps_o, m_o, s_o = ref_in.params, ref_in.exp_avg, ref_in.exp_avg_sq
            for kk in range(k):
                assert st_in.grad_norm[kk] == pytest.approx(ref_in.grad_norm[kk], rel=1e-6)
                assert st_in.clip_coef[kk] == pytest.approx(ref_in.clip_coef[kk], rel=1e-6)
            steps += 1
        state_err = H * 2.0 ** -23 * np.max(np.abs(np.stack(reps_o)), axis=0)
        for kk in range(k):
            o = reps_o[kk]
            err = np.abs(reps_g[kk].cpu().numpy() - o)
            assert np.all(err <= 1e-5 * (np.abs(o) + np.sqrt(np.mean(o * o))) + state_err), (kk, intervals)
            assert_close_elementwise(m_g[kk].cpu().numpy(), m_o[kk], tol=1e-5, what=f"m[{kk}] {intervals}")
            assert_close_elementwise(s_g[kk].cpu().numpy(), s_o[kk], tol=1e-5, what=f"v_adam[{kk}] {intervals}")
        # the synchronisation round
        st = al.autoloco_outer_step(ctx, th_g, v_g, reps_g, dec_g.coeffs, al.FUSE_STATS | al.FUSE_RESET, EPS)
        c = dec_o.coeffs
        ref = orr.sync_round(th_o, v_o, reps_o, c.mu, c.eta, c.rho, c.normalize, EPS)
        for name in ("D", "C", "disagreement", "sq_mean"):
            assert getattr(st, name) == pytest.approx(getattr(ref.stats, name), rel=2e-4), (name, intervals)
        for got, o, extra, what in ((v_g, ref.momentum, state_err, "v'"),
                                    (th_g, ref.theta, c.eta * (1 + c.mu) * state_err, "theta'")):
            err = np.abs(got.cpu().numpy() - o)
            bound = 1e-5 * (np.abs(o) + np.sqrt(np.mean(o * o))) + extra
            bad = np.nonzero(~(err <= bound))[0]
            assert bad.size == 0, f"{what} interval {intervals}: {bad.size} elements, first {bad[:3]}"
        assert all(torch.equal(x, th_g) for x in reps_g)
        # the controller
        lam = dec_o.lambda_sel
        tokens = TOKENS_PER_STEP * dec_o.h_step
        dec_o = ctl_o.select_interval(oc.Observation(ref.stats.D, ref.stats.C, lam, tokens, dec_o.h_step,
                                                     ref.stats.finite))
        dec_g = al.autoloco_select_interval(ctl_g, al.make_observation(st.D, st.C, lam, tokens, dec_g.h_step,
                                                                       st.finite))
        assert dec_g.assessment == dec_o.assessment, intervals
        if not math.isnan(dec_o.z_max):
            for thr in (CFG.thr_cand, CFG.thr_mod, CFG.thr_sev):
                assert abs(dec_o.z_max - thr) > 1e-6, f"near-tie z at interval {intervals}: {dec_o.z_max}"
        intervals += 1
    assert dec_g.done
    assert steps == CFG.budget_steps and intervals >= 10
    assert {oc.Phase.WARMUP, oc.Phase.VAR, oc.Phase.MONITOR} <= phases
    assert {oc.Phase.CAND1} <= phases                      # a candidate was tried (and adopted)
