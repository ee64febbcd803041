"""Pins of the inner AdamW oracle (CPU).

The oracle is checked against what fixes it independently of its own code:
the AdamW optimiser and gradient-norm clipping of PyTorch run in float64 on
the CPU (a library routine for the same definition), closed forms of the
first step and of a constant gradient, the scale invariance of the Adam
direction, and the clipping coefficient's cases.  Planted mistakes (a dropped
bias correction, epsilon under the square root, decay after the step,
swapped coefficients, the square instead of the root of v) must each fail the
library pin."""
import math

import numpy as np
import pytest
import torch

from oracle import adamw as oa
from oracle import correction as ocorr

C4 = oa.AdamWConfig()                                                   # (0.9, 0.95), decay 0.1, clip 1.0
SFT = oa.AdamWConfig(beta2=0.999, weight_decay=0.0)


def _grads(rng, n, k, step):
    # magnitudes spread over six decades, so epsilon matters for some elements;
    # overall scale chosen so some workers clip and others do not
    out = []
    for i in range(k):
        mag = 10.0 ** rng.uniform(-9, -3, n)
        scale = [1.0, 30.0, 300.0][(i + step) % 3]
        out.append(rng.standard_normal(n) * mag * scale)
    return out


def _torch_run(p0, m0, v0, grads_by_step, lrs, cfg):
    """Each worker's parameters through torch.optim.AdamW and clip_grad_norm_ (float64)."""
    res = []
    for i in range(len(p0)):
        p = torch.nn.Parameter(torch.tensor(p0[i], dtype=torch.float64))
        opt = torch.optim.AdamW([p], lr=lrs[0], betas=(cfg.beta1, cfg.beta2), eps=cfg.eps,
                                weight_decay=cfg.weight_decay, foreach=False)
        st = opt.state[p]
        st["step"] = torch.tensor(0.0, dtype=torch.float64)
        st["exp_avg"] = torch.tensor(m0[i], dtype=torch.float64)
        st["exp_avg_sq"] = torch.tensor(v0[i], dtype=torch.float64)
        norms = []
        for s, lr in enumerate(lrs):
            p.grad = torch.tensor(grads_by_step[s][i], dtype=torch.float64)
            if cfg.max_grad_norm > 0:
                norms.append(float(torch.nn.utils.clip_grad_norm_([p], cfg.max_grad_norm)))
            opt.param_groups[0]["lr"] = lr
            opt.step()
        res.append((p.detach().numpy().copy(), st["exp_avg"].numpy().copy(), st["exp_avg_sq"].numpy().copy(),
                    norms))
    return res


def _oracle_run(p0, m0, v0, grads_by_step, lrs, cfg, step_fn=None):
    p, m, v = [np.array(x) for x in p0], [np.array(x) for x in m0], [np.array(x) for x in v0]
    norms = [[] for _ in p0]
    for s, lr in enumerate(lrs):
        if step_fn is None:
            r = oa.inner_step(p, m, v, grads_by_step[s], lr, s + 1, cfg)
            p, m, v = r.params, r.exp_avg, r.exp_avg_sq
            for i, nm in enumerate(r.grad_norm):
                norms[i].append(nm)
        else:
            out = [step_fn(p[i], m[i], v[i], grads_by_step[s][i], lr, s + 1, cfg) for i in range(len(p))]
            p, m, v = [o[0] for o in out], [o[1] for o in out], [o[2] for o in out]
    return p, m, v, norms


def _close(a, b, rel):
    a, b = np.asarray(a), np.asarray(b)
    return bool(np.all(np.abs(a - b) <= rel * (np.abs(b) + 1e-300)))


def _setup(seed, n=2000, k=3, steps=6, start=20_000):
    rng = np.random.default_rng(seed)
    p0 = [rng.standard_normal(n) * 0.02 for _ in range(k)]
    m0 = [rng.standard_normal(n) * 1e-5 for _ in range(k)]
    v0 = [(rng.standard_normal(n) * 1e-5) ** 2 for _ in range(k)]
    grads = [_grads(rng, n, k, s) for s in range(steps)]
    sched = ocorr.Schedule()
    lrs = [ocorr.inner_lr(sched, start + s) for s in range(steps)]
    return p0, m0, v0, grads, lrs


@pytest.mark.parametrize("cfg", [C4, SFT, oa.AdamWConfig(max_grad_norm=0.0)], ids=["c4", "sft", "noclip"])
def test_matches_torch_adamw(cfg):
    p0, m0, v0, grads, lrs = _setup(1)
    ref = _torch_run(p0, m0, v0, grads, lrs, cfg)
    p, m, v, norms = _oracle_run(p0, m0, v0, grads, lrs, cfg)
    clipped = 0
    for i in range(len(p0)):
        assert _close(p[i], ref[i][0], 1e-13)
        assert _close(m[i], ref[i][1], 1e-12)
        assert _close(v[i], ref[i][2], 1e-12)
        if cfg.max_grad_norm > 0:
            assert norms[i] == pytest.approx(ref[i][3], rel=1e-13)
            clipped += sum(nm > cfg.max_grad_norm for nm in norms[i])
    if cfg.max_grad_norm > 0:
        assert 0 < clipped < len(p0) * len(lrs)          # both branches of the clip were taken


def test_warmup_schedule_steps():
    # the first steps of training: warm-up learning rates from zero state
    rng = np.random.default_rng(5)
    n, k = 500, 2
    p0 = [rng.standard_normal(n) * 0.02 for _ in range(k)]
    z = [np.zeros(n) for _ in range(k)]
    grads = [_grads(rng, n, k, s) for s in range(4)]
    lrs = [ocorr.inner_lr(ocorr.Schedule(), s) for s in range(4)]
    ref = _torch_run(p0, z, z, grads, lrs, C4)
    p, m, v, _ = _oracle_run(p0, z, z, grads, lrs, C4)
    for i in range(k):
        assert _close(p[i], ref[i][0], 1e-13) and _close(v[i], ref[i][2], 1e-12)


def test_first_step_closed_form():
    # from zero moments, m_hat = g and v_hat = g^2: theta' = theta (1 - eta lambda) - eta g / (|g| + eps)
    rng = np.random.default_rng(2)
    n = 1000
    th = rng.standard_normal(n) * 0.02
    g = rng.standard_normal(n) * 10.0 ** rng.uniform(-10, -2, n)
    cfg = oa.AdamWConfig(max_grad_norm=0.0)
    lr = 3e-4
    t1, m1, v1 = oa.adamw_step(th, np.zeros(n), np.zeros(n), g, lr, 1, cfg)
    assert _close(t1, th * (1 - lr * 0.1) - lr * g / (np.abs(g) + 1e-8), 1e-14)
    assert _close(m1, 0.1 * g, 4e-15) and _close(v1, 0.05 * g * g, 4e-15)


def test_constant_gradient_closed_form():
    # a constant gradient makes the bias-corrected moments exactly g and g^2:
    # without decay, theta_n = theta_0 - (sum of the step sizes) g / (|g| + eps)
    rng = np.random.default_rng(3)
    n = 300
    th0 = rng.standard_normal(n) * 0.02
    g = rng.standard_normal(n) * 1e-3
    cfg = oa.AdamWConfig(weight_decay=0.0, max_grad_norm=0.0)
    lrs = [1e-4 * (1 + 0.1 * s) for s in range(12)]
    th, m, v = th0, np.zeros(n), np.zeros(n)
    for s, lr in enumerate(lrs):
        th, m, v = oa.adamw_step(th, m, v, g, lr, s + 1, cfg)
    assert _close(th, th0 - sum(lrs) * g / (np.abs(g) + 1e-8), 1e-12)
    assert _close(m, g * (1 - 0.9 ** 12), 1e-13)
    assert _close(v, g * g * (1 - 0.95 ** 12), 1e-13)


def test_scale_invariance_without_epsilon():
    # with epsilon 0 and no decay, the Adam direction does not depend on the gradient's scale
    rng = np.random.default_rng(4)
    n = 400
    th = rng.standard_normal(n)
    m = rng.standard_normal(n) * 1e-3
    v = (rng.standard_normal(n) * 1e-3) ** 2
    g = rng.standard_normal(n) * 1e-3
    cfg = oa.AdamWConfig(eps=0.0, weight_decay=0.0, max_grad_norm=0.0)
    a = oa.adamw_step(th, m, v, g, 1e-3, 7, cfg)[0]
    b = oa.adamw_step(th, m * 1024, v * 1024 ** 2, g * 1024, 1e-3, 7, cfg)[0]
    assert _close(a, b, 1e-13)


def test_decay_only():
    th = np.array([1.0, -2.0, 0.5])
    z = np.zeros(3)
    t1, m1, v1 = oa.adamw_step(th, z, z, z, 1e-2, 3, C4)
    assert np.array_equal(t1, th * (1 - 1e-2 * 0.1)) and not m1.any() and not v1.any()


def test_clip_coefficient_cases():
    assert oa.clip_coefficient(3.0, 1.0) == 1.0 / (3.0 + 1e-6)
    assert oa.clip_coefficient(0.25, 1.0) == 1.0
    assert oa.clip_coefficient(0.0, 1.0) == 1.0
    assert oa.clip_coefficient(5.0, 0.0) == 1.0
    assert oa.clip_coefficient(math.inf, 1.0) == 0.0
    assert math.isnan(oa.clip_coefficient(math.nan, 1.0))
    g = np.zeros(100)
    g[7], g[50] = 3.0, 4.0
    assert oa.grad_norm(g) == 5.0
    r = oa.inner_step([np.zeros(100)], [np.zeros(100)], [np.zeros(100)], [g], 1e-3, 1, C4)
    assert r.clip_coef[0] == 1.0 / 5.000001 and r.grad_norm[0] == 5.0


def test_non_finite_gradient_propagates():
    g = np.ones(8)
    g[3] = np.nan
    r = oa.inner_step([np.zeros(8)], [np.zeros(8)], [np.zeros(8)], [g], 1e-3, 1, C4)
    assert math.isnan(r.grad_norm[0]) and np.isnan(r.params[0]).all()


def test_step_count_starts_at_one():
    with pytest.raises(ValueError):
        oa.adamw_step(np.zeros(2), np.zeros(2), np.zeros(2), np.zeros(2), 1e-3, 0, C4)


# ---------------------------------------------------------- planted mistakes --
def _no_bias_correction(p, m, v, g, lr, t, cfg):
    th = p * (1 - lr * cfg.weight_decay)
    m = cfg.beta1 * m + (1 - cfg.beta1) * g
    v = cfg.beta2 * v + (1 - cfg.beta2) * g * g
    return th - lr * m / (np.sqrt(v) + cfg.eps), m, v


def _eps_inside_sqrt(p, m, v, g, lr, t, cfg):
    th = p * (1 - lr * cfg.weight_decay)
    m = cfg.beta1 * m + (1 - cfg.beta1) * g
    v = cfg.beta2 * v + (1 - cfg.beta2) * g * g
    return th - lr * (m / (1 - cfg.beta1 ** t)) / np.sqrt(v / (1 - cfg.beta2 ** t) + cfg.eps), m, v


def _decay_after_step(p, m, v, g, lr, t, cfg):
    m = cfg.beta1 * m + (1 - cfg.beta1) * g
    v = cfg.beta2 * v + (1 - cfg.beta2) * g * g
    th = p - lr * (m / (1 - cfg.beta1 ** t)) / (np.sqrt(v / (1 - cfg.beta2 ** t)) + cfg.eps)
    return th * (1 - lr * cfg.weight_decay), m, v


def _swapped_betas(p, m, v, g, lr, t, cfg):
    th = p * (1 - lr * cfg.weight_decay)
    m = cfg.beta2 * m + (1 - cfg.beta2) * g
    v = cfg.beta1 * v + (1 - cfg.beta1) * g * g
    return th - lr * (m / (1 - cfg.beta2 ** t)) / (np.sqrt(v / (1 - cfg.beta1 ** t)) + cfg.eps), m, v


def _unclipped(p, m, v, g, lr, t, cfg):
    return oa.adamw_step(p, m, v, g, lr, t, cfg, 1.0)


@pytest.mark.parametrize("mutant", [_no_bias_correction, _eps_inside_sqrt, _decay_after_step, _swapped_betas,
                                    _unclipped])
def test_library_pin_catches_planted_mistakes(mutant):
    p0, m0, v0, grads, lrs = _setup(7, n=400)
    ref = _torch_run(p0, m0, v0, grads, lrs, C4)
    p, _, _, _ = _oracle_run(p0, m0, v0, grads, lrs, C4, step_fn=mutant)
    assert not all(_close(p[i], ref[i][0], 1e-9) for i in range(len(p0)))
