"""INT8 blockwise pseudo-gradient codec and the round that communicates
through it (test infrastructure only).

App. G.1 ("Low-precision communication configuration"):
  * a tensor part is cut into contiguous blocks of up to 4,096 elements;
  * a nonzero block's FP32 scale is its largest absolute value divided by 127;
    a zero block uses scale 1;
  * elements are divided by the scale, rounded to the nearest integer with
    ties to even and clipped to [-127, 127];
  * decoding multiplies the signed INT8 values by the block scale in FP32;
  * no error feedback; worker contributions are decoded and averaged in FP32,
    and the mean is encoded once more for distribution (every worker,
    including the one that reduced the part, receives the same decoded mean);
  * D is measured on the local pseudo-gradients before quantisation and C on
    the decoded aggregate.

The codes are integers decided by FP32 arithmetic, so this module computes
every step of the codec in the paper's precision (numpy float32, whose
division and rounding are IEEE round-to-nearest-even), as the GPU does.
Readings of what the text leaves open:
  * the tensor part is the whole flat buffer: blocks are [4096 j, 4096 j + 4096)
    and the last block is shorter;
  * the "scale bound" keeps the scale a normal FP32 number:
    scale = max(maxabs / 127, 2^-126), so the division never meets a zero or
    subnormal scale;
  * "averaged in FP32" is the FP32 rounding of the mean: the decoded
    contributions are summed in float64 in worker order, multiplied by the
    float64 value of 1/K and rounded once to FP32;
  * the decoded aggregate that C is computed on, and that the outer step
    uses, is the mean after its own encoding and decoding (what every worker
    receives);
  * the per-worker deviation sums are taken against that same decoded mean.
"""
from __future__ import annotations

import numpy as np

from . import round as orr

BLOCK = 4096
_F127 = np.float32(127.0)
_SCALE_MIN = np.float32(2.0 ** -126)


def encode(x: np.ndarray, block: int = BLOCK):
    """FP32 values -> (int8 codes, FP32 block scales)."""
    x = np.asarray(x, dtype=np.float32)
    n = x.shape[0]
    nb = (n + block - 1) // block
    codes = np.empty(n, dtype=np.int8)
    scales = np.empty(nb, dtype=np.float32)
    for b in range(nb):
        seg = x[b * block:(b + 1) * block]
        m = np.max(np.abs(seg)) if seg.size else np.float32(0)
        if m == 0:
            s = np.float32(1.0)
        else:
            s = np.float32(m) / _F127
            if s < _SCALE_MIN:
                s = _SCALE_MIN
        q = np.rint(seg / s)
        q = np.clip(q, -127, 127)
        codes[b * block:(b + 1) * block] = q.astype(np.int8)
        scales[b] = s
    return codes, scales


def decode(codes: np.ndarray, scales: np.ndarray, block: int = BLOCK) -> np.ndarray:
    """Codes times their block scale, in FP32."""
    n = codes.shape[0]
    per = np.repeat(scales, block)[:n]
    return codes.astype(np.float32) * per


def roundtrip(x: np.ndarray, block: int = BLOCK) -> np.ndarray:
    c, s = encode(x, block)
    return decode(c, s, block)


def fp32_mean(parts) -> np.ndarray:
    """FP32 rounding of the mean of FP32 arrays (float64 sum in order, times 1/K)."""
    total = np.zeros(parts[0].shape, dtype=np.float64)
    for p in parts:
        total = total + p.astype(np.float64)
    return (total * (1.0 / len(parts))).astype(np.float32)


class Int8Round:
    """Result of one INT8-communicating round."""

    def __init__(self, theta, momentum, stats, mean_codes, mean_scales, mean_decoded):
        self.theta = theta
        self.momentum = momentum
        self.stats = stats
        self.mean_codes = mean_codes
        self.mean_scales = mean_scales
        self.mean_decoded = mean_decoded


def int8_round(theta: np.ndarray, momentum: np.ndarray, replicas, mu: float, eta: float, rho: float,
               normalize: bool, eps: float = 1e-12, block: int = BLOCK) -> Int8Round:
    """One round whose pseudo-gradient average travels through the INT8 codec."""
    th32 = np.asarray(theta, dtype=np.float32)
    # FP32 pseudo-gradients (master parameters and the outer reference are FP32)
    deltas = [th32 - orr.widen(r).astype(np.float32) for r in replicas]
    decoded = [roundtrip(d, block) for d in deltas]
    mean_dec = fp32_mean(decoded)
    mcodes, mscales = encode(mean_dec, block)
    agg = decode(mcodes, mscales, block)
    k = len(replicas)
    d64 = [d.astype(np.float64) for d in deltas]
    a64 = agg.astype(np.float64)
    s = [float(np.sum(d * d)) for d in d64]
    q = [float(np.sum((d - a64) * (d - a64))) for d in d64]
    m = float(np.sum(a64 * a64))
    stats = orr.finish_stats(s, q, m, eps)
    th_new, v_new = orr.outer_update(theta, momentum, a64, mu, eta, rho, normalize)
    return Int8Round(th_new, v_new, stats, mcodes, mscales, agg)
