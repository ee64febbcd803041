"""Helpers shared by the GPU tests: seeded inputs on the CPU and device copies,
bit views of bf16 tensors, and the tolerance checks (element-wise
|g - o| <= 1e-5 (|o| + rms(o)) for the updated fp32 buffers, relative 1e-4 for
the statistics)."""
import numpy as np
import torch

from workloads import drift

THETA_TOL = 1e-5
STATS_TOL = 1e-4


def bits16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def host_array(t: torch.Tensor) -> np.ndarray:
    """fp32 tensor -> fp32 numpy; bf16 tensor -> uint16 bit patterns."""
    if t.dtype == torch.bfloat16:
        return bits16(t)
    return t.detach().cpu().numpy().copy()


def cpu_inputs(n, k, seed=42, recipe=drift.MIXED, replica_dtype=torch.float32):
    return drift.make_round_inputs(n, k, seed=seed, recipe=recipe, replica_dtype=replica_dtype, device="cpu")


def to_device(inp, device="cuda"):
    return drift.RoundInputs(inp.theta.to(device).contiguous(), inp.momentum.to(device).contiguous(),
                             [r.to(device).contiguous() for r in inp.replicas])


def assert_close_elementwise(got: np.ndarray, ref: np.ndarray, tol=THETA_TOL, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    err = np.abs(got - ref)
    bound = tol * (np.abs(ref) + rms)
    bad = np.nonzero(~(err <= bound))[0]
    assert bad.size == 0, (f"{what}: {bad.size} of {ref.size} elements out of tolerance; first at {bad[:5]}: "
                           f"got {got[bad[:5]]}, oracle {ref[bad[:5]]}")


def assert_stats_close(st, ref, tol=STATS_TOL, floor=0.0):
    """GPU autoloco_stats against oracle Stats; ``floor`` is an absolute slack
    for sums that are zero or near zero in exact arithmetic."""
    k = st.k
    assert k == len(ref.sq_norm)
    pairs = [("sq_mean", st.sq_mean, ref.sq_mean), ("D", st.D, ref.D), ("C", st.C, ref.C),
             ("disagreement", st.disagreement, ref.disagreement)]
    pairs += [(f"sq_norm[{i}]", st.sq_norm[i], ref.sq_norm[i]) for i in range(k)]
    pairs += [(f"sq_dev[{i}]", st.sq_dev[i], ref.sq_dev[i]) for i in range(k)]
    for name, g, o in pairs:
        assert abs(g - o) <= tol * abs(o) + floor, f"{name}: gpu {g!r} oracle {o!r}"
    assert bool(st.finite) == bool(ref.finite)


def assert_bf16_reset_close(bits: np.ndarray, ref: np.ndarray, tol=THETA_TOL, what="bf16 reset"):
    """bf16 replicas written by the reset against the oracle's float64 theta'.

    The reset is round-to-nearest of the GPU's fp32 theta' g, so
    |bf16(g) - o| <= |bf16(g) - g| + |g - o| <= 2^-8 |bf16(g)| (1 + 2^-7) + tol (|o| + rms(o)):
    half a bf16 ulp (8 significant bits) plus the fp32 tolerance of theta' itself.  (Near a zero
    crossing of theta' the fp32 error alone can exceed one bf16 ulp, so an ulp
    count against the oracle's own rounding is not a valid bar there.)"""
    w = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    bound = 2.0 ** -8 * np.abs(w) * (1 + 2.0 ** -7) + tol * (np.abs(ref) + rms)
    bad = np.nonzero(~(np.abs(w - ref) <= bound))[0]
    assert bad.size == 0, f"{what}: {bad.size} elements out of bound; first at {bad[:5]}: {w[bad[:5]]} vs {ref[bad[:5]]}"
