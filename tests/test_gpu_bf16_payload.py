"""GPU parity of the round with BF16 pseudo-gradient payloads against the oracle.

The received mean is a BF16 value decided by FP32/float64 arithmetic the
reading fixes, so its bits must equal the oracle's; theta', v' and the
statistics match within the round's tolerances.  Covered: ragged sizes, every
worker count with fp32 and bf16 replicas, the flag combinations, identical
replicas, determinism, argument errors, and sampled parameters of the full
1.1B model (the received mean of a parameter depends on that parameter only,
so the oracle computes sampled ones one by one)."""
import ctypes as C

import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al
from oracle import bf16_payload as bp
from oracle import round as orr
from tests.gpu_common import (assert_bf16_reset_close, assert_close_elementwise, assert_stats_close, bits16,
                              cpu_inputs, host_array, to_device)
from workloads import drift, shapes

pytestmark = pytest.mark.gpu
EPS = 1e-12
MU, ETA, RHO = 0.8545853971914775, 1.5181396589623761, 1.4914395799922477


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()


def _check(ctx, n, k, dtype=torch.float32, normalize=False, seed=1, flags=al.FUSE_STATS | al.FUSE_RESET,
           recipe=drift.MIXED, payload=True):
    inp = cpu_inputs(n, k, seed=seed, recipe=recipe, replica_dtype=dtype)
    dev = to_device(inp)
    c = al.make_coeffs(MU, ETA, RHO, normalize)
    ref = bp.bf16_round(inp.theta.numpy(), inp.momentum.numpy(), [host_array(r) for r in inp.replicas],
                        c.mu, c.eta_out, c.rho, normalize, EPS)
    mean = torch.empty(max(n, 1), dtype=torch.bfloat16, device="cuda") if payload else None
    st = al.autoloco_outer_step_bf16(ctx, dev.theta, dev.momentum, dev.replicas, c, flags, EPS, mean_bf16=mean)
    torch.cuda.synchronize()
    if payload:
        assert np.array_equal(bits16(mean)[:n], ref.mean_bits), "received mean differs"
    if flags & al.FUSE_STATS:
        assert_stats_close(st, ref.stats, floor=1e-9 * max(ref.stats.D, 1e-30))
    th = dev.theta.cpu().numpy()
    assert_close_elementwise(th, ref.theta, what="theta'")
    assert_close_elementwise(dev.momentum.cpu().numpy(), ref.momentum, what="v'")
    for r, r0 in zip(dev.replicas, inp.replicas):
        if not flags & al.FUSE_RESET:
            assert torch.equal(r.cpu(), r0)
        elif dtype == torch.float32:
            assert np.array_equal(r.cpu().numpy().view(np.uint32), th.view(np.uint32))
        else:
            assert np.array_equal(bits16(r), bits16(dev.theta.to(torch.bfloat16)))
            assert_bf16_reset_close(bits16(r), ref.theta)
    return st, ref


@pytest.mark.parametrize("n", [1, 5, 7, 8, 9, 4096 + 3, (1 << 20) + 5])
def test_sizes(ctx, n):
    _check(ctx, n, 4, seed=n % 89)


@pytest.mark.parametrize("k", [1, 2, 3, 5, 8, 9, 12, 16])
def test_worker_counts_fp32(ctx, k):
    _check(ctx, 50_003, k, seed=40 + k, normalize=k % 2 == 1)


@pytest.mark.parametrize("k", [1, 4, 8, 16])
def test_worker_counts_bf16(ctx, k):
    _check(ctx, 70_001, k, dtype=torch.bfloat16, seed=60 + k, normalize=True)


@pytest.mark.parametrize("flags", [0, al.FUSE_STATS, al.FUSE_RESET])
def test_flag_combinations(ctx, flags):
    _check(ctx, 30_011, 3, seed=7, flags=flags)


def test_without_payload_output(ctx):
    _check(ctx, 30_011, 5, seed=8, payload=False)


def test_spread_recipe(ctx):
    st, _ = _check(ctx, 200_003, 8, seed=3, recipe=drift.spread_recipe(1e-2))
    assert 0.5 < st.C < 1.5


def test_identical_replicas(ctx):
    n, k = 20_000, 4
    inp = cpu_inputs(n, 1, seed=4)
    th = inp.theta.cuda()
    reps = [th.clone() for _ in range(k)]
    mom = inp.momentum.cuda()
    mean = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    st = al.autoloco_outer_step_bf16(ctx, th, mom, reps, al.make_coeffs(0.9, 0.7), al.FUSE_STATS, EPS,
                                     mean_bf16=mean)
    assert st.D == 0.0 and st.C == 0.0 and not bits16(mean).any()


def test_deterministic(ctx):
    inp = cpu_inputs(1_000_003, 8, seed=8)
    outs = []
    for _ in range(2):
        dev = to_device(inp)
        mean = torch.empty(inp.theta.numel(), dtype=torch.bfloat16, device="cuda")
        st = al.autoloco_outer_step_bf16(ctx, dev.theta, dev.momentum, dev.replicas, al.make_coeffs(MU, ETA, RHO, True),
                                         al.FUSE_STATS | al.FUSE_RESET, EPS, mean_bf16=mean)
        outs.append((bytes(st), bits16(mean).tobytes(), dev.theta.cpu().numpy().tobytes()))
    assert outs[0] == outs[1]


def test_payload_argument_checks(ctx):
    n = 8192
    dev = to_device(cpu_inputs(n, 2, seed=9))
    mean = torch.empty(n + 8, dtype=torch.bfloat16, device="cuda")
    b = al.make_buffers(dev.theta, dev.replicas, dev.momentum)
    cf = al.make_coeffs(0.9, 0.7)
    st = al._lib.Stats()
    f = al.lib().autoloco_outer_step_bf16
    assert f(ctx.handle, C.byref(b), C.byref(cf), 1, EPS, C.byref(st), C.c_void_p(mean.data_ptr() + 2)) == -2
    assert f(ctx.handle, C.byref(b), C.byref(cf), 1, EPS, C.byref(st), C.c_void_p(dev.momentum.data_ptr())) == -3
    assert f(ctx.handle, C.byref(b), C.byref(cf), 4, EPS, C.byref(st), None) == -1       # unknown flag
    assert f(ctx.handle, C.byref(b), C.byref(cf), 1, EPS, C.byref(st), C.c_void_p(mean.data_ptr())) == 0


def test_llama_1b1_sampled(ctx):
    n, k = shapes.llama_1b1().n_params, 8
    ts, _ = al.spread_tensors(ctx, n, [torch.float32] * (k + 2))
    inp = drift.RoundInputs(ts[0], ts[1], ts[2:])
    drift.fill_theta_momentum(inp, seed=42)
    drift.fill_replicas(inp, seed=42)
    rng = np.random.default_rng(5)
    idx = np.unique(np.concatenate([rng.integers(0, n, 20_000), [0, 1, n - 2, n - 1]]))
    it = torch.as_tensor(idx, device="cuda")
    th0, v0 = inp.theta[it].cpu().numpy(), inp.momentum[it].cpu().numpy()
    reps0 = [r[it].cpu().numpy() for r in inp.replicas]
    plain = al.autoloco_round_stats(ctx, inp.theta, inp.replicas, EPS)
    mean = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    c = al.make_coeffs(MU, ETA, RHO, False)
    st = al.autoloco_outer_step_bf16(ctx, inp.theta, inp.momentum, inp.replicas, c, al.FUSE_STATS | al.FUSE_RESET,
                                     EPS, mean_bf16=mean)
    torch.cuda.synchronize()
    ref = bp.bf16_round(th0, v0, reps0, c.mu, c.eta_out, c.rho, False, EPS)
    assert np.array_equal(bits16(mean[it]), ref.mean_bits)
    assert_close_elementwise(inp.theta[it].cpu().numpy(), ref.theta, what="1.1B theta'")
    assert_close_elementwise(inp.momentum[it].cpu().numpy(), ref.momentum, what="1.1B v'")
    # D is taken before the payload rounding: the plain statistics pass agrees
    for i in range(k):
        assert st.sq_norm[i] == pytest.approx(plain.sq_norm[i], rel=1e-6)
    assert st.D == pytest.approx(plain.D, rel=1e-6) and st.finite
    # the received mean differs from the exact one by BF16 rounding only
    assert st.sq_mean == pytest.approx(plain.sq_mean, rel=1e-2)
    del inp, ts
    torch.cuda.empty_cache()
