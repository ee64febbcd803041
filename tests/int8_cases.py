"""Codec blocks crowded at the rounding boundaries of their own scale: the tie
points (j + 1/2) s for every code step j, each rounded to FP32, with its
neighbours up to three FP32 ulps away on either side.  For a scale that is not
a power of two, x * fp32(1/s) and the IEEE quotient x / s then round to
different integers for some of these values, so only a codec that takes the
exact quotient where it matters reproduces the oracle's codes."""
import numpy as np

from oracle import int8_codec as ic


def block_scale(amax: float) -> np.float32:
    """The oracle's scale of a block whose largest magnitude is amax."""
    return ic.encode(np.array([amax], dtype=np.float32))[1][0]


def near_half_block(amax: float, m: int, rng: np.random.Generator) -> np.ndarray:
    """m FP32 values with largest magnitude amax, most of them at or next to a
    tie point of the block's scale, the rest uniform in [-amax, amax]."""
    s = np.float64(block_scale(amax))
    vals = [np.float32(amax)]
    for j in range(-127, 127):
        c = np.float32((j + 0.5) * s)
        vals.append(c)
        up = dn = c
        for _ in range(3):
            up = np.nextafter(up, np.float32(np.inf))
            dn = np.nextafter(dn, np.float32(-np.inf))
            vals += [up, dn]
    x = np.array(vals, dtype=np.float32)
    x = x[np.abs(x) <= np.float32(amax)][:m]
    fill = rng.uniform(-amax, amax, m - x.size).astype(np.float32)
    out = np.concatenate([x, fill])
    rng.shuffle(out)
    return out
