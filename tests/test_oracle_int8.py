"""Pins of the oracle's INT8 blockwise codec (App. G.1) against what the text
fixes: zero blocks use scale 1, the largest element of a block encodes to
+-127, round-to-nearest-even on exact ties, codes stay in [-127, 127], the
decode error is at most half a scale step, blocks are independent, D is taken
before quantisation and C on the decoded aggregate, and on dyadic inputs
(where every FP32 step is exact) the whole codec round equals an exact
rational evaluation."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import int8_codec as ic
from oracle import round as orr


def test_zero_block_uses_scale_one():
    codes, scales = ic.encode(np.zeros(5000, dtype=np.float32))
    assert scales.tolist() == [1.0, 1.0] and not codes.any()


def test_block_maximum_maps_to_127():
    rng = np.random.default_rng(0)
    for _ in range(20):
        x = rng.normal(0, rng.uniform(1e-6, 1e2), 4096).astype(np.float32)
        codes, scales = ic.encode(x)
        j = int(np.argmax(np.abs(x)))
        assert codes[j] == (127 if x[j] > 0 else -127)
        assert np.abs(codes.astype(np.int32)).max() <= 127 and codes.min() >= -127


def test_ties_round_to_even():
    s = 1.0 / 128.0                       # block maximum 127/128 gives the exact scale 1/128
    x = np.array([127, 2.5, 3.5, -2.5, 0.5, 1.5, -3.5, -0.5], dtype=np.float32) * np.float32(s)
    codes, scales = ic.encode(x)
    assert scales[0] == np.float32(s)
    assert codes.tolist() == [127, 2, 4, -2, 0, 2, -4, 0]


def test_decode_error_at_most_half_a_step():
    rng = np.random.default_rng(1)
    x = (rng.normal(0, 1e-3, 3 * 4096 + 17) * rng.uniform(0.1, 10, 3 * 4096 + 17)).astype(np.float32)
    codes, scales = ic.encode(x)
    dec = ic.decode(codes, scales)
    per = np.repeat(scales, 4096)[: x.size].astype(np.float64)
    err = np.abs(dec.astype(np.float64) - x.astype(np.float64))
    # half a step plus the FP32 roundings of the division and the decode product
    assert np.all(err <= per * (0.5 + 1e-5) + np.abs(x) * 2e-7)


def test_blocks_are_independent_and_last_block_is_short():
    x = np.concatenate([np.full(4096, 1.0), np.full(5, 1e-3)]).astype(np.float32)
    codes, scales = ic.encode(x)
    assert scales.size == 2
    assert scales[0] == np.float32(1.0) / np.float32(127.0)
    assert scales[1] == np.float32(1e-3) / np.float32(127.0)
    assert (codes == 127).all()


def test_scale_bound_for_tiny_blocks():
    x = np.array([1e-40, -1e-41, 0.0], dtype=np.float32)   # subnormal maximum
    codes, scales = ic.encode(x)
    assert scales[0] == np.float32(2.0 ** -126)
    assert not codes.any()


def test_d_before_quantisation_c_on_decoded_aggregate():
    # worker 1 has one large entry, so its small entries quantise to zero; the
    # decoded aggregate therefore differs from the exact mean
    n = 64
    theta = np.zeros(n, dtype=np.float32)
    d1 = np.full(n, 1e-3, dtype=np.float32)
    d1[0] = 1.0
    d2 = np.full(n, 1e-3, dtype=np.float32)
    reps = [theta - d1, theta - d2]
    r = ic.int8_round(theta, np.zeros(n, np.float32), reps, 0.9, 0.7, 1.0, False, 1e-12)
    exact = orr.round_stats(theta, reps, 1e-12)
    assert r.stats.D == pytest.approx(exact.D, rel=1e-12)          # D: pre-quantisation
    agg = r.mean_decoded.astype(np.float64)
    assert agg[1] != pytest.approx(1e-3, rel=1e-3)                 # the small entries moved
    assert r.stats.C == pytest.approx(2 * float(np.sum(agg * agg)) / (r.stats.D + 1e-12), rel=1e-14)
    assert abs(r.stats.C - exact.C) > 1e-6


def _round_half_even(f: Fraction) -> int:
    lo = f.numerator // f.denominator
    rem = f - lo
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1):
        return lo + 1
    return lo


@pytest.mark.parametrize("seed", range(6))
def test_dyadic_round_equals_exact_rational(seed):
    # Every worker's block b holds entries m * 2^-(e_b+1), |m| <= 254, with the
    # block maximum 127 * 2^-e_b at the block's first element: each scale is the
    # power of two 2^-e_b, the worker mean keeps that maximum (so its scale is
    # exact too), and every quotient is a multiple of 1/8: all FP32 steps are exact.
    rng = np.random.default_rng(seed)
    k, blk, nb = 4, 16, 3
    n = blk * nb - 5
    deltas = []
    exps = rng.integers(3, 9, nb)
    for w in range(k):
        d = np.empty(n, dtype=np.float64)
        for b in range(nb):
            lo, hi = b * blk, min(n, (b + 1) * blk)
            m = rng.integers(-254, 255, hi - lo)
            m[0] = 254                                            # the block maximum
            d[lo:hi] = m * 2.0 ** -(int(exps[b]) + 1)
        deltas.append(d.astype(np.float32))
    theta = np.zeros(n, dtype=np.float32)
    reps = [theta - d for d in deltas]
    r = ic.int8_round(theta, np.zeros(n, np.float32), reps, 0.9, 0.7, 1.0, False, 0.0, block=blk)

    # exact: codes, decode, mean over workers, encode the mean, decode
    dec = []
    for w in range(k):
        out = []
        for b in range(nb):
            seg = [Fraction(float(x)) for x in deltas[w][b * blk:(b + 1) * blk]]
            s = max(abs(v) for v in seg) / 127
            out += [max(-127, min(127, _round_half_even(v / s))) * s for v in seg]
        dec.append(out)
    mean = [sum(dec[w][j] for w in range(k)) / k for j in range(n)]
    agg = []
    for b in range(nb):
        seg = mean[b * blk:(b + 1) * blk]
        mx = max(abs(v) for v in seg)
        s = Fraction(1) if mx == 0 else mx / 127
        assert float(s) == float(np.float32(float(s)))         # still exact in FP32
        agg += [max(-127, min(127, _round_half_even(v / s))) * s for v in seg]
    assert [float(a) for a in agg] == r.mean_decoded.astype(np.float64).tolist()


def test_near_half_cases_need_the_exact_quotient():
    # The GPU parity cases of tests/int8_cases.py are only a test of the codec's
    # exact path if the product with the rounded reciprocal gives a different
    # code than the paper's division for some of them: count those.
    from tests.int8_cases import block_scale, near_half_block
    rng = np.random.default_rng(11)
    differ = ties = 0
    for amax in (1.0, 3.7, 0.3, 2.0 ** -100 * 5.0):
        x = near_half_block(amax, 4096, rng)
        s = block_scale(amax)
        codes, scales = ic.encode(x)
        assert scales[0] == s and np.max(np.abs(x)) == np.float32(amax)
        fast = np.clip(np.rint(x * (np.float32(1.0) / s)), -127, 127).astype(np.int8)
        differ += int(np.sum(fast != codes))
        qf = x / s                                 # the FP32 quotient the codes are defined on
        ties += int(np.sum(qf - np.floor(qf) == np.float32(0.5)))
    assert differ > 0, "no case where the product and the quotient round apart"
    assert ties > 0, "no FP32 quotient on a tie, where rounding to even decides"
