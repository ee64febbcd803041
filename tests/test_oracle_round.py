"""Pins of the float64 round oracle against values fixed by the paper and by
mathematics: a hand-derived worked example, exact rational brute force,
the identities and bounds of App. C.1, the DiLoCo special case (App. D.2) run
through torch's own Nesterov SGD, the fixed-input momentum closed form
(App. C.3) and plain model averaging."""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import exact
from oracle import round as orr

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
EPS = 1e-12


def _golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, val = [p.strip() for p in line.split("=", 1)]
            vals[key] = val
    return vals


def _vec(s):
    return np.array([float(x) for x in s.split()])


# ------------------------------------------------------------ worked example
def test_worked_example_stats():
    g = _golden("worked_example_k2n2.txt")
    theta = _vec(g["theta"]).astype(np.float32)
    reps = [_vec(g["replica_1"]).astype(np.float32), _vec(g["replica_2"]).astype(np.float32)]
    st = orr.round_stats(theta, reps, eps=float(g["eps"]))
    assert st.sq_norm == list(_vec(g["sq_norm"]))
    assert st.sq_dev == list(_vec(g["sq_dev"]))
    assert st.sq_mean == float(g["sq_mean"])
    assert st.D == float(g["D"])
    assert st.C * (1 + EPS) == pytest.approx(float(g["C_times_1_plus_eps"]), rel=1e-15)
    assert st.disagreement == float(g["disagreement"])
    assert st.finite


@pytest.mark.parametrize("case,rho,normalize", [("rho1", 1.0, False), ("rho2_norm", 2.0, True),
                                                 ("rho2_raw", 2.0, False)])
def test_worked_example_update(case, rho, normalize):
    g = _golden("worked_example_k2n2.txt")
    theta = _vec(g["theta"]).astype(np.float32)
    reps = [_vec(g["replica_1"]).astype(np.float32), _vec(g["replica_2"]).astype(np.float32)]
    mom = _vec(g["momentum"]).astype(np.float32)
    key = "rho1" if rho == 1.0 else "rho2"
    mu, eta = float(g[key + ".mu"]), float(g[key + ".eta"])
    res = orr.sync_round(theta, mom, reps, mu, eta, rho, normalize, eps=EPS)
    np.testing.assert_allclose(res.momentum, _vec(g[case + ".momentum"]), rtol=1e-15, atol=1e-15)
    np.testing.assert_allclose(res.theta, _vec(g[case + ".theta"]), rtol=1e-14, atol=1e-15)


# ------------------------------------------------------- exact brute force
def _dyadic(rng, shape):
    # multiples of 2**-12 in (-1, 1): exact in fp32, so every input is exact
    return (rng.integers(-4095, 4096, size=shape) / 4096.0).astype(np.float32)


@pytest.mark.parametrize("seed", range(12))
def test_brute_force_fraction(seed):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(1, 17))
    k = int(rng.integers(1, 5))
    theta = _dyadic(rng, n)
    mom = _dyadic(rng, n)
    reps = [_dyadic(rng, n) for _ in range(k)]
    rho = [1, 2][seed % 2]
    mu = Fraction(9, 10) ** rho          # mu_base^rho, exact for integer rho
    eta = Fraction(7, 10) * Fraction(min(rho, Fraction(8, 5))) * (1 - mu) / Fraction(1, 10)
    normalize = seed % 3 == 0
    ex = exact.exact_round(theta, mom, reps, mu, eta, rho, normalize, Fraction(EPS))
    res = orr.sync_round(theta, mom, reps, float(mu), float(eta), float(rho), normalize, eps=EPS)

    def close(a, b, rel=4e-16, floor=0.0):
        b = float(b)
        assert abs(a - b) <= rel * abs(b) + floor, (a, b)

    for i in range(k):
        close(res.stats.sq_norm[i], ex["sq_norm"][i], rel=1e-15)
        close(res.stats.sq_dev[i], ex["sq_dev"][i], rel=1e-15, floor=1e-18)
    close(res.stats.sq_mean, ex["sq_mean"], rel=1e-15)
    close(res.stats.D, ex["D"], rel=1e-15)
    close(res.stats.C, ex["C"], rel=1e-14)
    close(res.stats.disagreement, ex["disagreement"], rel=1e-15, floor=1e-18)
    scale = max(1e-300, max(abs(float(x)) for x in ex["theta"]))
    for j in range(n):
        close(res.momentum[j], ex["momentum"][j], rel=1e-15, floor=1e-16)
        close(res.theta[j], ex["theta"][j], rel=1e-15, floor=1e-15 * scale)


# ------------------------------------------------- identities and bounds
def _rand_round(rng, n, k, dtype=np.float32, spread=1e-3):
    theta = rng.normal(0, 0.02, n).astype(dtype)
    s = rng.normal(0, 1e-3, n)
    reps = [(theta + 0.7 * s + 0.3 * rng.normal(0, spread, n)).astype(dtype) for _ in range(k)]
    return theta, reps


@pytest.mark.parametrize("k", [1, 2, 3, 5, 8, 16])
def test_disagreement_identity_and_bounds(k):
    rng = np.random.default_rng(k)
    theta, reps = _rand_round(rng, 4099, k)
    st = orr.round_stats(theta, reps, eps=EPS, chunk=1000)
    # App. C.1 eq. dc_variance_expansion: disagreement = D - ||Delta_bar||^2
    assert st.disagreement == pytest.approx(st.D - st.sq_mean, rel=1e-9, abs=1e-12 * st.D)
    # eq. dc_endpoint_disagreement: disagreement = D - C (D + eps) / K
    assert st.disagreement == pytest.approx(st.D - st.C * (st.D + EPS) / k, rel=1e-9,
                                            abs=1e-12 * st.D)
    # eq. dc_ranges: 0 <= C <= K D / (D + eps) < K ; 0 <= disagreement <= D
    assert 0.0 <= st.C <= k * st.D / (st.D + EPS) * (1 + 1e-12) < k
    assert 0.0 <= st.disagreement <= st.D


def test_chunking_does_not_change_sums():
    rng = np.random.default_rng(7)
    theta, reps = _rand_round(rng, 10_001, 4)
    a = orr.round_stats(theta, reps, eps=EPS, chunk=10_001)
    b = orr.round_stats(theta, reps, eps=EPS, chunk=97)
    assert a.D == pytest.approx(b.D, rel=1e-13)
    assert a.C == pytest.approx(b.C, rel=1e-13)


def test_single_worker_full_coherence():
    # K=1: Delta_bar = Delta_1, so disagreement is 0 and C = D/(D+eps), the bound of
    # eq. dc_identical_updates with N=1.
    rng = np.random.default_rng(3)
    theta, reps = _rand_round(rng, 777, 1)
    st = orr.round_stats(theta, reps, eps=EPS)
    assert st.sq_dev == [0.0]
    assert st.C == st.D / (st.D + EPS) or st.C == pytest.approx(st.D / (st.D + EPS), rel=1e-15)


@pytest.mark.parametrize("k", [2, 4, 7])
def test_identical_replicas(k):
    # identical pseudo-gradients: zero disagreement and C = K D/(D+eps)  (eq. dc_identical_updates)
    rng = np.random.default_rng(k)
    theta, reps = _rand_round(rng, 1000, 1)
    reps = [reps[0].copy() for _ in range(k)]
    st = orr.round_stats(theta, reps, eps=EPS)
    assert max(st.sq_dev) <= 1e-30 * st.D
    assert st.C == pytest.approx(k * st.D / (st.D + EPS), rel=1e-14)
    # replicas equal to theta: D = 0 implies C = 0 (App. C.1, the D_t = 0 case)
    st0 = orr.round_stats(theta, [theta.copy() for _ in range(k)], eps=EPS)
    assert st0.D == 0.0 and st0.C == 0.0 and st0.disagreement == 0.0


def test_zero_drift_update_is_pure_momentum():
    # theta_k = theta: v' = mu v and theta' = theta - eta mu^2 v
    rng = np.random.default_rng(11)
    theta = rng.normal(0, 0.02, 513).astype(np.float32)
    mom = rng.normal(0, 1e-4, 513).astype(np.float32)
    res = orr.sync_round(theta, mom, [theta.copy(), theta.copy()], 0.8, 0.7, 1.0, False, EPS)
    np.testing.assert_allclose(res.momentum, 0.8 * mom.astype(np.float64), rtol=1e-15)
    np.testing.assert_allclose(res.theta, theta - 0.7 * 0.64 * mom.astype(np.float64), rtol=1e-14)


def test_nan_marks_not_finite():
    rng = np.random.default_rng(5)
    theta, reps = _rand_round(rng, 100, 3)
    with np.errstate(invalid="ignore"):   # inf - inf and nan arithmetic are the point here
        reps[1][17] = np.nan
        assert not orr.round_stats(theta, reps, eps=EPS).finite
        reps[1][17] = np.inf
        assert not orr.round_stats(theta, reps, eps=EPS).finite


# -------------------------------------------- DiLoCo special case (App. D.2)
@pytest.mark.parametrize("mu,eta", [(0.9, 0.7), (0.7, 0.7)])
def test_rho_one_is_torch_nesterov_sgd(mu, eta):
    # At rho = 1 the corrected step is DiLoCo's Nesterov outer step: SGD with
    # Nesterov momentum applied to the gradient Delta_bar with the momentum buffer
    # holding v (eq. fixed-horizon-nesterov).  torch.optim.SGD is the textbook routine.
    rng = np.random.default_rng(21)
    n, k = 300, 4
    theta, reps = _rand_round(rng, n, k)
    mom = rng.normal(0, 1e-4, n).astype(np.float32)
    res = orr.sync_round(theta, mom, reps, mu, eta, 1.0, True, EPS)

    p = torch.nn.Parameter(torch.from_numpy(theta.astype(np.float64)))
    opt = torch.optim.SGD([p], lr=eta, momentum=mu, nesterov=True, dampening=0.0)
    opt.state[p]["momentum_buffer"] = torch.from_numpy(mom.astype(np.float64)).clone()
    grad = torch.from_numpy(theta.astype(np.float64)) - torch.stack(
        [torch.from_numpy(r.astype(np.float64)) for r in reps]).mean(0)
    p.grad = grad
    opt.step()
    np.testing.assert_allclose(res.theta, p.detach().numpy(), rtol=1e-13, atol=1e-17)
    np.testing.assert_allclose(res.momentum, opt.state[p]["momentum_buffer"].numpy(),
                               rtol=1e-13, atol=1e-19)


# ------------------------------------------- fixed-input response (App. C.3)
@pytest.mark.parametrize("normalize", [False, True])
def test_fixed_input_momentum_closed_form(normalize):
    # Holding Delta_k fixed and repeating the step: v_n - Dt/(1-mu) = mu^n (v_0 - Dt/(1-mu))
    # (eq. oc_momentum_fixed_point), so v_n = mu^n v_0 + Dt (1-mu^n)/(1-mu), and the
    # direction tends to Dt/(1-mu) (eq. oc_steady_response).
    rng = np.random.default_rng(9)
    n, k, mu, eta, rho = 64, 3, 0.81, 2.128, 2.0
    theta0, reps0 = _rand_round(rng, n, k, dtype=np.float64)
    deltas = [theta0 - r for r in reps0]
    dbar = sum(deltas) / k
    dt = dbar / rho if normalize else dbar
    v0 = rng.normal(0, 1e-4, n)
    theta, v = theta0.copy(), v0.copy()
    rounds = 60
    for _ in range(rounds):
        reps = [theta - d for d in deltas]
        res = orr.sync_round(theta, v, reps, mu, eta, rho, normalize, EPS)
        prev_theta = theta
        theta, v = res.theta, res.momentum
    expect_v = mu ** rounds * v0 + dt * (1 - mu ** rounds) / (1 - mu)
    np.testing.assert_allclose(v, expect_v, rtol=1e-11, atol=1e-18)
    d_last = (prev_theta - theta) / eta
    np.testing.assert_allclose(d_last, dt / (1 - mu), rtol=1e-4)


# --------------------------------------------------- model averaging (P-I8)
def test_plain_averaging_special_case():
    # mu = 0, eta = 1, v = 0, no normalisation: theta' = theta - Delta_bar, the
    # arithmetic mean of the local endpoints (App. C.1 eq. dc_endpoint_mean).
    rng = np.random.default_rng(31)
    theta, reps = _rand_round(rng, 1001, 5)
    res = orr.sync_round(theta, np.zeros(1001, np.float32), reps, 0.0, 1.0, 1.0, False, EPS)
    mean = np.mean(np.stack([r.astype(np.float64) for r in reps]), axis=0)
    np.testing.assert_allclose(res.theta, mean, rtol=1e-13, atol=1e-18)


# ------------------------------------------------------ bf16 reset rounding
def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.normal(0, 1, 20000), rng.normal(0, 1e-3, 2000),
                        np.ldexp(rng.uniform(1, 2, 500), -130),     # bf16 subnormals
                        [0.0, -0.0, 1.0, 3.0e38, -3.3e38, 1e-45]]).astype(np.float32)
    ours = orr.to_bf16_bits(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)


def test_bf16_ties_and_specials():
    one = 1.0
    ulp = 2.0 ** -7
    # exactly halfway between 1 and 1+ulp: ties to even (1.0); 1+ulp+half: up to 1+2ulp
    bits = orr.to_bf16_bits(np.array([one + ulp / 2, one + 1.5 * ulp, np.inf, -np.inf, np.nan, -np.nan]))
    assert bits[0] == 0x3F80
    assert bits[1] == 0x3F82
    assert bits[2] == 0x7F80 and bits[3] == 0xFF80
    assert bits[4] == 0x7FC0 and bits[5] == 0xFFC0
    # fp64 input just above a tie rounds up even when fp32 would have made it a tie
    just_above = one + ulp / 2 + 2.0 ** -40
    assert orr.to_bf16_bits(np.array([just_above]))[0] == 0x3F81
    # overflow past max + half ulp becomes infinity
    assert orr.to_bf16_bits(np.array([3.4e38]))[0] == 0x7F80


def test_widen_bf16_is_exact():
    bits = np.array([0x3F80, 0xBF81, 0x0001, 0x7F7F], dtype=np.uint16)
    w = orr.widen(bits)
    assert w[0] == 1.0 and w[1] == -(1 + 2 ** -7) and w[2] == 2.0 ** -133
    assert w[3] == float.fromhex("0x1.fep127")
