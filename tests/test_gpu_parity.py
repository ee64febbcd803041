"""GPU parity of the round kernels against the float64 oracle, through the C ABI.

Sizes span several workgroups and grid-stride passes with ragged tails; every
worker count 1..16 and both replica types are exercised, as are the flag
combinations, the standalone statistics and reset calls, the degenerate cases
of App. C.1 and the argument checks."""
import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al
from oracle import correction as ocorr
from oracle import round as orr
from tests.gpu_common import (assert_bf16_reset_close, assert_close_elementwise, assert_stats_close, bits16,
                              cpu_inputs, host_array, to_device)
from workloads import drift

pytestmark = pytest.mark.gpu
EPS = 1e-12


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()


def _tiny_coeffs(normalize):
    # H^step = 75 against H^ref = 50 from step 20,000 of the C4 schedule
    sched = ocorr.Schedule()
    lam, lam_b = ocorr.lr_mass(sched, 20_000, 75), ocorr.lr_mass(sched, 20_000, 50)
    c = al.autoloco_outer_correction(al.make_outer_cfg(normalize=normalize), lam, lam_b)
    return c


def _oracle_round(inp_cpu, c):
    th = inp_cpu.theta.numpy()
    mom = inp_cpu.momentum.numpy()
    reps = [host_array(r) for r in inp_cpu.replicas]
    return orr.sync_round(th, mom, reps, c.mu, c.eta_out, c.rho, bool(c.normalize), EPS)


def _check_full_round(ctx, n, k, replica_dtype=torch.float32, normalize=False, seed=42,
                      recipe=drift.MIXED, coeffs=None):
    inp = cpu_inputs(n, k, seed=seed, recipe=recipe, replica_dtype=replica_dtype)
    dev = to_device(inp)
    c = coeffs if coeffs is not None else _tiny_coeffs(normalize)
    ref = _oracle_round(inp, c)
    st = al.autoloco_outer_step(ctx, dev.theta, dev.momentum, dev.replicas, c,
                                al.FUSE_STATS | al.FUSE_RESET, EPS)
    torch.cuda.synchronize()
    assert_stats_close(st, ref.stats, floor=1e-9 * max(ref.stats.D, 1e-30))
    th = dev.theta.cpu().numpy()
    assert_close_elementwise(th, ref.theta, what="theta'")
    assert_close_elementwise(dev.momentum.cpu().numpy(), ref.momentum, what="v'")
    if replica_dtype == torch.float32:
        for r in dev.replicas:
            assert np.array_equal(r.cpu().numpy().view(np.uint32), th.view(np.uint32))
    else:
        mine = bits16(dev.theta.to(torch.bfloat16))      # torch's own rounding of the GPU theta'
        for r in dev.replicas:
            rb = bits16(r)
            assert np.array_equal(rb, mine)
            assert_bf16_reset_close(rb, ref.theta)
    return st, ref


@pytest.mark.parametrize("normalize", [False, True])
def test_tiny_config(ctx, normalize):
    # N = 1,048,576 fp32, K = 4, theta_k = theta + 0.7 s + 0.3 e_k
    st, ref = _check_full_round(ctx, 1 << 20, 4, normalize=normalize)
    assert 0.55 < st.D < 0.67 and 3.3 < st.C < 3.7


@pytest.mark.parametrize("k", list(range(1, 17)))
def test_every_worker_count_fp32(ctx, k):
    _check_full_round(ctx, 65_537, k, seed=100 + k, normalize=k % 2 == 0)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5, 7, 8, 12, 16])
def test_every_worker_count_bf16(ctx, k):
    _check_full_round(ctx, 65_539, k, replica_dtype=torch.bfloat16, seed=200 + k, normalize=k % 2 == 1)


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 7, 8, 9, 255, 1023, 1025, 5000, 7579, 262_147, 2_097_155])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_ragged_sizes(ctx, n, dtype):
    _check_full_round(ctx, n, 3, replica_dtype=dtype, seed=n % 97)


def test_many_grid_stride_passes(ctx):
    # more vectors than threads in the grid: several passes per thread, ragged tail
    al.autoloco_set_grid_limit(ctx, 7)
    try:
        _check_full_round(ctx, 7 * 256 * 4 * 5 + 3, 5, seed=5)
    finally:
        al.autoloco_set_grid_limit(ctx, 0)


def test_spread_recipe_coherence_range(ctx):
    # theta_k = theta + s + e_k with e_k ~ N(0, sigma): C falls as sigma grows
    cs = []
    for sigma in (1e-4, 1e-3, 1e-2):
        st, _ = _check_full_round(ctx, 300_001, 8, recipe=drift.spread_recipe(sigma), seed=7)
        cs.append(st.C)
    assert cs[0] > 7.5 and 4.0 < cs[1] < 5.0 and cs[2] < 1.3


@pytest.mark.parametrize("flags", [0, al.FUSE_STATS, al.FUSE_RESET])
def test_flag_subsets(ctx, flags):
    n, k = 100_003, 6
    inp = cpu_inputs(n, k, seed=3)
    dev = to_device(inp)
    c = _tiny_coeffs(True)
    before = [r.clone() for r in dev.replicas]
    ref = _oracle_round(inp, c)
    st = al.autoloco_outer_step(ctx, dev.theta, dev.momentum, dev.replicas, c, flags, EPS)
    torch.cuda.synchronize()
    assert_close_elementwise(dev.theta.cpu().numpy(), ref.theta, what="theta'")
    assert_close_elementwise(dev.momentum.cpu().numpy(), ref.momentum, what="v'")
    if flags & al.FUSE_STATS:
        assert_stats_close(st, ref.stats)
    else:
        assert st is None
    for r, b in zip(dev.replicas, before):
        if flags & al.FUSE_RESET:
            assert torch.equal(r, dev.theta)
        else:
            assert torch.equal(r, b)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("k", [3, 5, 6, 8])
def test_standalone_stats_match_fused_bitwise(ctx, dtype, k):
    # every K on both sides of the grid thresholds (one workgroup per compute
    # unit from K = 5 with fp32 replicas and from K = 6 with bf16)
    n = 1_000_003
    inp = cpu_inputs(n, k, seed=11, replica_dtype=dtype)
    dev = to_device(inp)
    ref = _oracle_round(inp, _tiny_coeffs(False))
    s1 = al.autoloco_round_stats(ctx, dev.theta, dev.replicas, EPS)
    s2 = al.autoloco_round_stats(ctx, dev.theta, dev.replicas, EPS)
    assert_stats_close(s1, ref.stats)
    assert bytes(s1) == bytes(s2)
    fused = al.autoloco_outer_step(ctx, dev.theta, dev.momentum, dev.replicas, _tiny_coeffs(False),
                                   al.FUSE_STATS, EPS)
    assert bytes(fused) == bytes(s1)


def test_statistics_bit_stable_across_runs(ctx):
    n, k = 3_000_001, 8
    inp = cpu_inputs(n, k, seed=13)
    dev = to_device(inp)
    c = _tiny_coeffs(False)
    outs = []
    for _ in range(6):
        th, mom = dev.theta.clone(), dev.momentum.clone()
        reps = [r.clone() for r in dev.replicas]
        st = al.autoloco_outer_step(ctx, th, mom, reps, c, al.FUSE_STATS | al.FUSE_RESET, EPS)
        outs.append((bytes(st), th.cpu().numpy().tobytes(), mom.cpu().numpy().tobytes()))
    assert all(o == outs[0] for o in outs[1:])


_CHILD = """
import sys
sys.path.insert(0, {root!r})
import hashlib, torch
import paper_2609_36662_amd as al
from tests.gpu_common import cpu_inputs, to_device
dev = to_device(cpu_inputs({n}, {k}, seed=23))
ctx = al.autoloco_create(0)
st = al.autoloco_round_stats(ctx, dev.theta, dev.replicas, 1e-12)
c = al.autoloco_outer_correction(al.make_outer_cfg(normalize=True), 2.0e-2, 1.25e-2)
st2 = al.autoloco_outer_step(ctx, dev.theta, dev.momentum, dev.replicas, c, al.FUSE_STATS | al.FUSE_RESET, 1e-12)
h = hashlib.sha256(dev.theta.cpu().numpy().tobytes() + dev.momentum.cpu().numpy().tobytes()).hexdigest()
print(bytes(st).hex(), bytes(st2).hex(), h)
ctx.close()
"""


def test_statistics_bit_stable_across_processes(ctx):
    # the same round in a fresh process gives the same bits (statistics, theta', v')
    import hashlib
    import os
    import subprocess
    import sys
    n, k = 2_500_001, 8
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    dev = to_device(cpu_inputs(n, k, seed=23))
    st = al.autoloco_round_stats(ctx, dev.theta, dev.replicas, EPS)
    c = al.autoloco_outer_correction(al.make_outer_cfg(normalize=True), 2.0e-2, 1.25e-2)
    st2 = al.autoloco_outer_step(ctx, dev.theta, dev.momentum, dev.replicas, c, al.FUSE_STATS | al.FUSE_RESET, EPS)
    h = hashlib.sha256(dev.theta.cpu().numpy().tobytes() + dev.momentum.cpu().numpy().tobytes()).hexdigest()
    print(f"child process: n={n} k={k}", flush=True)
    p = subprocess.run([sys.executable, "-c", _CHILD.format(root=root, n=n, k=k)], capture_output=True, text=True,
                       timeout=100)
    assert p.returncode == 0, p.stderr[-2000:]
    assert p.stdout.split() == [bytes(st).hex(), bytes(st2).hex(), h]


def test_grid_size_changes_only_rounding(ctx):
    n, k = 2_000_003, 4
    inp = cpu_inputs(n, k, seed=17)
    dev = to_device(inp)
    ref = _oracle_round(inp, _tiny_coeffs(False))
    try:
        for g in (1, 3, 64, 1000, 4096):
            al.autoloco_set_grid_limit(ctx, g)
            st = al.autoloco_round_stats(ctx, dev.theta, dev.replicas, EPS)
            assert_stats_close(st, ref.stats)
    finally:
        al.autoloco_set_grid_limit(ctx, 0)


@pytest.mark.parametrize("n,k", [(17_000_003, 9), (67_200_003, 2)])
def test_largest_grid(ctx, n, k):
    # 16,384 workgroups (the scratch capacity): every partial slot in use, and the
    # finishing kernel's strided loop runs 64 times per thread
    inp = cpu_inputs(n, k, seed=19)
    dev = to_device(inp)
    c = _tiny_coeffs(True)
    ref = _oracle_round(inp, c)
    try:
        al.autoloco_set_grid_limit(ctx, 16384)
        assert al.autoloco_launch_shape(ctx, n, k)[0] == 16384
        st = al.autoloco_outer_step(ctx, dev.theta, dev.momentum, dev.replicas, c, al.FUSE_STATS | al.FUSE_RESET, EPS)
        torch.cuda.synchronize()
    finally:
        al.autoloco_set_grid_limit(ctx, 0)
    assert_stats_close(st, ref.stats)
    assert_close_elementwise(dev.theta.cpu().numpy(), ref.theta, what="theta'")
    assert_close_elementwise(dev.momentum.cpu().numpy(), ref.momentum, what="v'")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("k", [1, 2, 3, 8, 16])
@pytest.mark.parametrize("n,grid", [(1, 0), (3, 0), (4 * 256 + 3, 0), (8 * 512 * 3 + 5, 3), (300_001, 0),
                                    (300_001, 5), (8 * 1024 * 5 + 2 * 1024 + 7, 3), (8 * 1024 * 7 + 1, 2)])
def test_broadcast_reset_shapes(ctx, dtype, k, n, grid):
    # the reset's window loop over ragged sizes, the last window shorter than one
    # run per lane, a last span of fewer windows than a full one (8 windows of
    # 1,024 elements from three fp32 replicas on), and a capped grid that takes
    # several grid-stride passes
    inp = cpu_inputs(n, k, seed=23 + k, replica_dtype=dtype)
    dev = to_device(inp)
    al.autoloco_set_grid_limit(ctx, grid)
    try:
        al.autoloco_broadcast_reset(ctx, dev.theta, dev.replicas)
        torch.cuda.synchronize()
    finally:
        al.autoloco_set_grid_limit(ctx, 0)
    exp_bits = orr.reset_replicas(inp.theta.numpy(), 1, "f32" if dtype == torch.float32 else "bf16")[0]
    for r in dev.replicas:
        assert np.array_equal(host_array(r).view(np.uint8), exp_bits.view(np.uint8))
    assert torch.equal(dev.theta.cpu(), inp.theta)


def test_broadcast_reset(ctx):
    for dtype in (torch.float32, torch.bfloat16):
        n, k = 777_777, 5
        inp = cpu_inputs(n, k, seed=19, replica_dtype=dtype)
        dev = to_device(inp)
        al.autoloco_broadcast_reset(ctx, dev.theta, dev.replicas)
        torch.cuda.synchronize()
        want = dev.theta if dtype == torch.float32 else dev.theta.to(torch.bfloat16)
        exp_bits = orr.reset_replicas(inp.theta.numpy(), 1, "f32" if dtype == torch.float32 else "bf16")[0]
        for r in dev.replicas:
            assert torch.equal(r, want)
            assert np.array_equal(host_array(r).view(np.uint8), exp_bits.view(np.uint8))


# ---------------------------------------------------------- degenerate cases
def test_empty_input(ctx):
    z = torch.empty(0, device="cuda")
    st = al.autoloco_outer_step(ctx, z, torch.empty(0, device="cuda"), [torch.empty(0, device="cuda")] * 3,
                                _tiny_coeffs(False), al.FUSE_STATS | al.FUSE_RESET, EPS)
    assert st.D == 0.0 and st.C == 0.0 and st.disagreement == 0.0 and st.finite
    st = al.autoloco_round_stats(ctx, z, [torch.empty(0, device="cuda")], EPS)
    assert st.D == 0.0 and st.k == 1


@pytest.mark.parametrize("k", [1, 2, 4, 8, 16])
def test_identical_replicas_zero_disagreement(ctx, k):
    # identical pseudo-gradients: sq_dev = 0 exactly (pairwise sum of K equal terms,
    # K a power of two) and C = K D/(D+eps) (App. C.1 eq. dc_identical_updates)
    n = 500_001
    inp = cpu_inputs(n, 1, seed=23)
    dev = to_device(inp)
    reps = [dev.replicas[0].clone() for _ in range(k)]
    st = al.autoloco_round_stats(ctx, dev.theta, reps, EPS)
    assert all(st.sq_dev[i] == 0.0 for i in range(k))
    assert st.C == pytest.approx(k * st.D / (st.D + EPS), rel=1e-12)
    # replicas equal to theta: D = 0, C = 0
    st0 = al.autoloco_round_stats(ctx, dev.theta, [dev.theta.clone() for _ in range(k)], EPS)
    assert st0.D == 0.0 and st0.C == 0.0 and st0.finite


def test_plain_averaging_special_case(ctx):
    # mu = 0, eta = 1, v = 0, no normalisation: theta' is the mean of the replicas
    n, k = 123_457, 8
    inp = cpu_inputs(n, k, seed=29)
    dev = to_device(inp)
    dev.momentum.zero_()
    al.autoloco_outer_step(ctx, dev.theta, dev.momentum, dev.replicas, al.make_coeffs(0.0, 1.0, 1.0, False), 0)
    mean = np.mean(np.stack([r.numpy().astype(np.float64) for r in inp.replicas]), axis=0)
    assert_close_elementwise(dev.theta.cpu().numpy(), mean, what="model average")


def test_rho_one_matches_torch_nesterov(ctx):
    # DiLoCo special case (App. D.2): torch's Nesterov SGD in float64 on the CPU
    n, k, mu, eta = 200_003, 4, 0.9, 0.7
    inp = cpu_inputs(n, k, seed=31)
    dev = to_device(inp)
    al.autoloco_outer_step(ctx, dev.theta, dev.momentum, dev.replicas, al.make_coeffs(mu, eta, 1.0, True), 0)
    p = torch.nn.Parameter(inp.theta.double())
    opt = torch.optim.SGD([p], lr=eta, momentum=mu, nesterov=True, dampening=0.0)
    opt.state[p]["momentum_buffer"] = inp.momentum.double().clone()
    p.grad = inp.theta.double() - torch.stack([r.double() for r in inp.replicas]).mean(0)
    opt.step()
    assert_close_elementwise(dev.theta.cpu().numpy(), p.detach().numpy(), what="theta'")
    assert_close_elementwise(dev.momentum.cpu().numpy(), opt.state[p]["momentum_buffer"].numpy(), what="v'")


def test_nonfinite_is_reported_not_fatal(ctx):
    n, k = 10_007, 3
    inp = cpu_inputs(n, k, seed=37)
    inp.replicas[1][4321] = float("nan")
    dev = to_device(inp)
    st = al.autoloco_outer_step(ctx, dev.theta, dev.momentum, dev.replicas, _tiny_coeffs(False),
                                al.FUSE_STATS, EPS)
    assert not st.finite
    th = dev.theta.cpu().numpy()
    assert np.isnan(th[4321]) and np.isfinite(np.delete(th, 4321)).all()


# ------------------------------------------------------------ argument checks
def _raw(ctx, theta, mom, reps, n, k, dtype=al.F32, flags=al.FUSE_STATS | al.FUSE_RESET, eps=EPS):
    import ctypes as C
    b = al._lib.Buffers()
    b.n, b.k, b.replica_dtype = n, k, dtype
    b.theta, b.momentum = theta, mom
    for i, r in enumerate(reps):
        b.replicas[i] = r
    st = al._lib.Stats()
    c = _tiny_coeffs(False)
    return al.lib().autoloco_outer_step(ctx.handle, C.byref(b), C.byref(c), flags, eps, C.byref(st))


def test_rejects_bad_arguments_without_touching_buffers(ctx):
    n = 4096
    inp = cpu_inputs(n + 8, 2, seed=41)
    dev = to_device(inp)
    snap = [t.clone() for t in [dev.theta, dev.momentum] + dev.replicas]
    th, mo = dev.theta.data_ptr(), dev.momentum.data_ptr()
    r0, r1 = dev.replicas[0].data_ptr(), dev.replicas[1].data_ptr()
    assert _raw(ctx, th + 4, mo, [r0, r1], n, 2) == -2            # misaligned theta
    assert _raw(ctx, th, mo, [r0, r1 + 8], n, 2) == -2            # misaligned replica
    assert _raw(ctx, th, mo, [r0, th], n, 2) == -3                # replica aliases theta
    assert _raw(ctx, th, th + 16, [r0, r1], n, 2) == -3           # momentum overlaps theta
    assert _raw(ctx, th, mo, [r0, r1], n, 0) == -1                # k = 0
    assert _raw(ctx, th, mo, [r0, r1], n, 17) == -1               # k = 17
    assert _raw(ctx, th, None, [r0, r1], n, 2) == -1              # no momentum
    assert _raw(ctx, th, mo, [r0, r1], n, 2, dtype=7) == -1       # unknown dtype
    assert _raw(ctx, th, mo, [r0, r1], n, 2, flags=4) == -1       # unknown flag
    assert _raw(ctx, th, mo, [r0, r1], -1, 2) == -1               # negative n
    assert _raw(ctx, th, mo, [r0, r1], 2**56 + 1, 2) == -1        # n beyond 2^56
    assert "2^56" in al.autoloco_last_error(ctx)
    for bad_eps in (0.0, -1e-12, float("nan"), float("inf")):    # eps > 0 (eq. adaptive-h-core-diagnostics)
        assert _raw(ctx, th, mo, [r0, r1], n, 2, eps=bad_eps) == -1
    assert al.autoloco_last_error(ctx)                            # a message was left
    torch.cuda.synchronize()
    for t, s in zip([dev.theta, dev.momentum] + dev.replicas, snap):
        assert torch.equal(t, s)
    with pytest.raises(al.AutolocoError):
        al.autoloco_round_stats(ctx, dev.theta, [dev.theta], EPS)
    with pytest.raises(al.AutolocoError):
        al.autoloco_round_stats(ctx, dev.theta, dev.replicas, 0.0)


def test_rejects_host_memory(ctx):
    # pinned host memory (reachable by the GPU, so a missed check could not fault) in
    # place of a replica is refused before any launch, with a message
    n = 4096
    dev = to_device(cpu_inputs(n, 2, seed=44))
    host = torch.empty(n, dtype=torch.float32, pin_memory=True)
    host.fill_(7.0)
    snap = dev.theta.clone()
    th, mo = dev.theta.data_ptr(), dev.momentum.data_ptr()
    assert _raw(ctx, th, mo, [dev.replicas[0].data_ptr(), host.data_ptr()], n, 2) == -1
    assert "not device memory" in al.autoloco_last_error(ctx)
    torch.cuda.synchronize()
    assert torch.equal(dev.theta, snap) and bool((host == 7.0).all())


def test_timing_events(ctx):
    E_STATE = -6   # AUTOLOCO_E_STATE
    inp = to_device(cpu_inputs(1 << 20, 4, seed=43))
    al.autoloco_set_timing(ctx, True)
    try:
        with pytest.raises(al.AutolocoError) as ei:   # nothing timed yet
            al.autoloco_last_kernel_ms(ctx)
        assert ei.value.status == E_STATE
        al.autoloco_outer_step(ctx, inp.theta, inp.momentum, inp.replicas, _tiny_coeffs(False),
                               al.FUSE_STATS | al.FUSE_RESET, EPS)
        ms = al.autoloco_last_kernel_ms(ctx)
        assert 0.0 < ms < 100.0
        # a call refused before launching anything leaves the last timing in place
        with pytest.raises(al.AutolocoError):
            al.autoloco_outer_step(ctx, inp.theta, inp.momentum, inp.replicas, _tiny_coeffs(False), 8, EPS)
        assert al.autoloco_last_kernel_ms(ctx) == ms
        with pytest.raises(al.AutolocoError) as ei:   # the last timed call was no AdamW step
            al.autoloco_last_adamw_ms(ctx)
        assert ei.value.status == E_STATE
        al.autoloco_broadcast_reset(ctx, inp.theta, inp.replicas)
        assert 0.0 < al.autoloco_last_kernel_ms(ctx) < 100.0
    finally:
        al.autoloco_set_timing(ctx, False)
    with pytest.raises(al.AutolocoError) as ei:   # switching timing off drops it
        al.autoloco_last_kernel_ms(ctx)
    assert ei.value.status == E_STATE
