"""Pins of the BF16-payload round oracle.

The payload rounding is checked against torch's own FP32 -> BF16 conversion
(round to nearest even), hand-computed cases fix the rounding of a
pseudo-gradient, its ties and the second rounding of the mean, inputs whose
payloads and mean are exactly representable reduce to the plain round (and to
the worked example's values), and the aggregate stays within the rounding
bound of the exact mean.  Planted mistakes in the order of the steps must
fail these pins."""
import numpy as np
import pytest
import torch

from oracle import bf16_payload as bp
from oracle import round as orr

EPS = 1e-12


def _f32(*v):
    return np.array(v, dtype=np.float32)


def test_payload_is_torch_bf16_conversion():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(200_000) * 10.0 ** rng.uniform(-30, 30, 200_000)).astype(np.float32)
    ties = (np.arange(1, 2000, dtype=np.uint32) << 16 | np.uint32(0x8000)).view(np.float32)   # exact halfway values
    x = np.concatenate([x, ties, -ties, _f32(0.0, -0.0, np.inf, -np.inf, 3.0e38, -3.0e38, 1e-40)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bp.payload(x), ref)


def _k1(delta: float):
    theta = _f32(2.0)
    rep = theta - _f32(delta)
    assert float(theta[0] - rep[0]) == delta          # the FP32 difference is the intended value
    return bp.bf16_round(theta, _f32(0.0), [rep], 0.9, 0.7, 1.0, False, EPS)


def test_pseudo_gradient_rounding_cases():
    r = _k1(1.0 + 2.0 ** -9)                      # below half a step: rounds down to 1
    assert orr.widen(r.mean_bits)[0] == 1.0
    assert r.stats.sq_norm[0] == (1.0 + 2.0 ** -9) ** 2 and r.stats.sq_dev[0] == 2.0 ** -18
    assert r.stats.sq_mean == 1.0
    assert r.stats.C == 1.0 / ((1.0 + 2.0 ** -9) ** 2 + EPS)
    assert orr.widen(_k1(1.0 + 2.0 ** -8).mean_bits)[0] == 1.0                  # tie, even below
    assert orr.widen(_k1(1.0 + 3 * 2.0 ** -8).mean_bits)[0] == 1.0 + 2.0 ** -6  # tie, even above
    assert orr.widen(_k1(-(1.0 + 3 * 2.0 ** -8)).mean_bits)[0] == -(1.0 + 2.0 ** -6)


def test_mean_is_rounded_again():
    # payloads 1 and 1 + 2^-7 are exact; their mean 1 + 2^-8 is a BF16 tie and goes to 1
    theta = _f32(4.0, 4.0)
    reps = [theta - _f32(1.0, 1.0), theta - _f32(1.0 + 2.0 ** -7, 1.0 + 2.0 ** -7)]
    r = bp.bf16_round(theta, _f32(0.0, 0.0), reps, 0.9, 0.7, 1.0, False, EPS)
    assert orr.widen(r.mean_bits).tolist() == [1.0, 1.0]
    assert r.stats.sq_mean == 2.0
    assert r.stats.sq_dev == [0.0, 2 * 2.0 ** -14]
    # the update uses the received mean: v' = 1, theta' = 4 - 0.7 (1 + 0.9) = 2.67
    assert r.momentum.tolist() == [1.0, 1.0]
    assert r.theta.tolist() == pytest.approx([4.0 - 0.7 * 1.9] * 2, rel=1e-15)


def test_exact_payloads_reduce_to_the_plain_round():
    # the worked example (K = 2, N = 2): every payload and the mean are exact in BF16
    theta = _f32(1.0, 2.0)
    reps = [_f32(0.0, 2.0), _f32(1.0, 1.0)]
    for mu, eta, rho, norm in ((0.9, 0.7, 1.0, False), (0.81, 2.128, 2.0, True)):
        b = bp.bf16_round(theta, _f32(0, 0), reps, mu, eta, rho, norm, EPS)
        p = orr.sync_round(theta, _f32(0, 0), reps, mu, eta, rho, norm, EPS)
        assert np.array_equal(b.theta, p.theta) and np.array_equal(b.momentum, p.momentum)
        assert b.stats == p.stats
    b = bp.bf16_round(theta, _f32(0, 0), reps, 0.9, 0.7, 1.0, False, EPS)
    assert b.theta.tolist() == pytest.approx([0.335, 1.335], rel=1e-15)
    # dyadic random inputs with few significant bits behave the same
    rng = np.random.default_rng(1)
    th = (rng.integers(-64, 64, 500) / 64.0).astype(np.float32)
    reps = [(th - rng.integers(-8, 8, 500) / 32.0).astype(np.float32) for _ in range(4)]
    b = bp.bf16_round(th, th * 0, reps, 0.9, 0.7, 1.0, False, EPS)
    p = orr.sync_round(th, th * 0, reps, 0.9, 0.7, 1.0, False, EPS)
    assert np.array_equal(b.theta, p.theta) and b.stats == p.stats


def test_identical_replicas():
    rng = np.random.default_rng(2)
    th = rng.standard_normal(1000).astype(np.float32)
    v = (rng.standard_normal(1000) * 1e-3).astype(np.float32)
    b = bp.bf16_round(th, v, [th.copy() for _ in range(3)], 0.9, 0.7, 1.0, False, EPS)
    assert not orr.widen(b.mean_bits).any() and b.stats.D == 0.0 and b.stats.C == 0.0
    assert np.array_equal(b.momentum, 0.9 * v.astype(np.float64))


def test_aggregate_within_rounding_bound_of_exact_mean():
    rng = np.random.default_rng(3)
    n, k = 20_000, 8
    th = (rng.standard_normal(n) * 0.02).astype(np.float32)
    s = rng.standard_normal(n) * 1e-3
    reps = [(th - 0.7 * s - 0.3 * rng.standard_normal(n) * 1e-3).astype(np.float32) for _ in range(k)]
    b = bp.bf16_round(th, th * 0, reps, 0.9, 0.7, 1.0, False, EPS)
    deltas = [th.astype(np.float64) - r.astype(np.float64) for r in reps]
    exact = sum(deltas) / k
    agg = orr.widen(b.mean_bits)
    bound = 2.0 ** -8 * (sum(np.abs(d) for d in deltas) / k + np.abs(agg)) + 1e-7 * np.abs(exact) + 1e-30
    assert np.all(np.abs(agg - exact) <= bound)
    assert np.abs(agg - exact).max() > 0          # the rounding is visible at this scale
    p = orr.round_stats(th, reps, EPS)
    assert b.stats.D == pytest.approx(p.D, rel=1e-6)       # D is taken before the payload rounding


# ---------------------------------------------------------- planted mistakes --
def _mutant_no_second_rounding(theta, momentum, replicas, mu, eta, rho, normalize, eps=EPS):
    th32 = np.asarray(theta, dtype=np.float32)
    deltas = [th32 - orr.widen(r).astype(np.float32) for r in replicas]
    total = sum(orr.widen(bp.payload(d)) for d in deltas)
    agg = (total * (1.0 / len(replicas))).astype(np.float32).astype(np.float64)
    d64 = [d.astype(np.float64) for d in deltas]
    st = orr.finish_stats([float(np.sum(d * d)) for d in d64], [float(np.sum((d - agg) ** 2)) for d in d64],
                          float(np.sum(agg * agg)), eps)
    return st, agg


def _mutant_truncating_payload(theta, momentum, replicas, mu, eta, rho, normalize, eps=EPS):
    th32 = np.asarray(theta, dtype=np.float32)
    deltas = [th32 - orr.widen(r).astype(np.float32) for r in replicas]
    cut = [(d.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32) for d in deltas]
    total = sum(c.astype(np.float64) for c in cut)
    bits = orr.to_bf16_bits((total / len(replicas)).astype(np.float32).astype(np.float64))
    agg = orr.widen(bits)
    d64 = [d.astype(np.float64) for d in deltas]
    st = orr.finish_stats([float(np.sum(d * d)) for d in d64], [float(np.sum((d - agg) ** 2)) for d in d64],
                          float(np.sum(agg * agg)), eps)
    return st, agg


@pytest.mark.parametrize("mutant", [_mutant_no_second_rounding, _mutant_truncating_payload])
def test_planted_mistakes_fail_the_hand_cases(mutant):
    theta = _f32(4.0, 2.0)
    reps = [theta - _f32(1.0, 1.0 + 3 * 2.0 ** -8), theta - _f32(1.0 + 2.0 ** -7, 1.0 + 3 * 2.0 ** -8)]
    good = bp.bf16_round(theta, _f32(0, 0), reps, 0.9, 0.7, 1.0, False, EPS)
    _, agg = mutant(theta, _f32(0, 0), reps, 0.9, 0.7, 1.0, False)
    assert not np.array_equal(agg, orr.widen(good.mean_bits))
