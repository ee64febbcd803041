"""GPU parity of the INT8-codec round (App. G.1) against the oracle.

The codes and block scales of the encoded mean are integers and FP32 values
decided by FP32 arithmetic the paper fixes, so they must match the oracle bit
for bit; θ', v' and the statistics match within the round's tolerances.  At
the full 1.1B (fp32 replicas) and 3B (bf16 replicas) sizes the codec is
checked block by block on sampled codec blocks (the codec is local to a
block), and D against the plain statistics pass."""
import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al
from oracle import int8_codec as ic
from tests.gpu_common import (assert_bf16_reset_close, assert_close_elementwise, assert_stats_close, bits16,
                              cpu_inputs, host_array, to_device)
from workloads import drift, shapes

pytestmark = pytest.mark.gpu
EPS = 1e-12
COEFFS = dict(mu=0.8545853971914775, eta_out=1.5181396589623761, rho=1.4914395799922477)


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()


def _payload(n):
    nb = (n + 4095) // 4096
    return (torch.empty(max(n, 1), dtype=torch.int8, device="cuda"),
            torch.empty(max(nb, 1), dtype=torch.float32, device="cuda"))


def _check(ctx, n, k, dtype=torch.float32, normalize=False, seed=1, recipe=drift.MIXED):
    inp = cpu_inputs(n, k, seed=seed, recipe=recipe, replica_dtype=dtype)
    dev = to_device(inp)
    c = al.make_coeffs(COEFFS["mu"], COEFFS["eta_out"], COEFFS["rho"], normalize)
    ref = ic.int8_round(inp.theta.numpy(), inp.momentum.numpy(), [host_array(r) for r in inp.replicas],
                        c.mu, c.eta_out, c.rho, normalize, EPS)
    codes, scales = _payload(n)
    st = al.autoloco_outer_step_int8(ctx, dev.theta, dev.momentum, dev.replicas, c, al.FUSE_STATS | al.FUSE_RESET,
                                     EPS, mean_codes=codes, mean_scales=scales)
    torch.cuda.synchronize()
    nb = (n + 4095) // 4096
    assert np.array_equal(codes[:n].cpu().numpy(), ref.mean_codes), "mean codes differ"
    assert np.array_equal(scales[:nb].cpu().numpy().view(np.uint32), ref.mean_scales.view(np.uint32)), "scales differ"
    assert_stats_close(st, ref.stats, floor=1e-9 * max(ref.stats.D, 1e-30))
    th = dev.theta.cpu().numpy()
    assert_close_elementwise(th, ref.theta, what="theta'")
    assert_close_elementwise(dev.momentum.cpu().numpy(), ref.momentum, what="v'")
    for r in dev.replicas:
        if dtype == torch.float32:
            assert np.array_equal(r.cpu().numpy().view(np.uint32), th.view(np.uint32))
        else:
            assert np.array_equal(bits16(r), bits16(dev.theta.to(torch.bfloat16)))
            assert_bf16_reset_close(bits16(r), ref.theta)
    return st, ref


@pytest.mark.parametrize("n", [1, 5, 4095, 4096, 4097, 3 * 4096 + 13, (1 << 20) + 3])
def test_sizes_fp32(ctx, n):
    _check(ctx, n, 4, seed=n % 101)


@pytest.mark.parametrize("k", [1, 2, 3, 5, 8, 9, 12, 16])
def test_worker_counts_fp32(ctx, k):
    _check(ctx, 3 * 4096 + 777, k, seed=10 + k, normalize=k % 2 == 0)


@pytest.mark.parametrize("k", [1, 4, 8, 16])
def test_worker_counts_bf16(ctx, k):
    _check(ctx, 5 * 4096 + 321, k, dtype=torch.bfloat16, seed=30 + k, normalize=True)


def test_spread_recipe_and_codec_effect(ctx):
    # with sigma = 1e-2 the per-worker noise dominates the shared drift; the decoded
    # aggregate still matches the oracle bit for bit
    st, ref = _check(ctx, 200_003, 8, seed=3, recipe=drift.spread_recipe(1e-2))
    assert 0.5 < st.C < 1.5


def test_zero_blocks_and_identical_replicas(ctx):
    n, k = 3 * 4096, 4
    inp = cpu_inputs(n, 1, seed=4)
    th = inp.theta.cuda()
    reps = [th.clone() for _ in range(k)]                  # zero pseudo-gradients: zero blocks, scale 1
    mom = inp.momentum.cuda()
    codes, scales = _payload(n)
    st = al.autoloco_outer_step_int8(ctx, th, mom, reps, al.make_coeffs(0.9, 0.7, 1.0, False),
                                     al.FUSE_STATS, EPS, mean_codes=codes, mean_scales=scales)
    assert st.D == 0.0 and st.C == 0.0
    assert not codes.any().item() and torch.all(scales[:3] == 1.0).item()


def test_deterministic(ctx):
    n, k = 1_000_003, 8
    inp = cpu_inputs(n, k, seed=8)
    outs = []
    for _ in range(3):
        dev = to_device(inp)
        codes, scales = _payload(n)
        st = al.autoloco_outer_step_int8(ctx, dev.theta, dev.momentum, dev.replicas,
                                         al.make_coeffs(0.85, 1.5, 1.49, True), al.FUSE_STATS | al.FUSE_RESET,
                                         EPS, mean_codes=codes, mean_scales=scales)
        outs.append((bytes(st), codes.cpu().numpy().tobytes(), dev.theta.cpu().numpy().tobytes()))
    assert outs[0] == outs[1] == outs[2]


def test_payload_argument_checks(ctx):
    import ctypes as C
    n = 8192
    dev = to_device(cpu_inputs(n, 2, seed=9))
    codes, scales = _payload(n)
    with pytest.raises(ValueError):
        al.autoloco_outer_step_int8(ctx, dev.theta, dev.momentum, dev.replicas, al.make_coeffs(0.9, 0.7),
                                    al.FUSE_STATS, EPS, mean_codes=codes)
    b = al.make_buffers(dev.theta, dev.replicas, dev.momentum)
    cf = al.make_coeffs(0.9, 0.7)
    st = al._lib.Stats()
    f = al.lib().autoloco_outer_step_int8
    assert f(ctx.handle, C.byref(b), C.byref(cf), 1, EPS, C.byref(st), C.c_void_p(codes.data_ptr() + 4),
             C.c_void_p(scales.data_ptr())) == -2                        # misaligned codes
    assert f(ctx.handle, C.byref(b), C.byref(cf), 1, EPS, C.byref(st), C.c_void_p(dev.theta.data_ptr()),
             C.c_void_p(scales.data_ptr())) == -3                        # codes alias theta
    assert f(ctx.handle, C.byref(b), C.byref(cf), 1, EPS, C.byref(st), C.c_void_p(codes.data_ptr()),
             None) == -1                                                  # only one payload buffer


def _sampled_codec_blocks(ctx, shape, k, dtype, normalize, seed):
    n = shapes.SHAPES[shape]().n_params
    ts, _ = al.spread_tensors(ctx, n, [torch.float32] * 2 + [dtype] * k)
    inp = drift.RoundInputs(ts[0], ts[1], ts[2:])
    drift.fill_theta_momentum(inp, seed=42)
    drift.fill_replicas(inp, seed=42)
    nb = (n + 4095) // 4096
    rng = np.random.default_rng(seed)
    blocks = sorted(set(rng.integers(0, nb, 48).tolist()) | {0, nb - 1})
    saved = {}
    for b in blocks:
        lo, hi = b * 4096, min(n, (b + 1) * 4096)
        saved[b] = (inp.theta[lo:hi].cpu().numpy(), inp.momentum[lo:hi].cpu().numpy(),
                    [host_array(r[lo:hi]) for r in inp.replicas])
    plain = al.autoloco_round_stats(ctx, inp.theta, inp.replicas, EPS)
    codes = torch.empty(n, dtype=torch.int8, device="cuda")
    scales = torch.empty(nb, dtype=torch.float32, device="cuda")
    c = al.make_coeffs(COEFFS["mu"], COEFFS["eta_out"], COEFFS["rho"], normalize)
    print(f"{shape}: n={n:,} K={k} {dtype}, {len(blocks)} sampled codec blocks", flush=True)
    st = al.autoloco_outer_step_int8(ctx, inp.theta, inp.momentum, inp.replicas, c, al.FUSE_STATS | al.FUSE_RESET,
                                     EPS, mean_codes=codes, mean_scales=scales)
    torch.cuda.synchronize()
    # D is taken on the pre-quantisation pseudo-gradients: the plain statistics pass agrees
    for i in range(k):
        assert st.sq_norm[i] == pytest.approx(plain.sq_norm[i], rel=1e-6)
    assert st.D == pytest.approx(plain.D, rel=1e-6) and st.finite
    for b in blocks:
        lo, hi = b * 4096, min(n, (b + 1) * 4096)
        th, mo, reps = saved[b]
        ref = ic.int8_round(th, mo, reps, c.mu, c.eta_out, c.rho, normalize, EPS)
        assert np.array_equal(codes[lo:hi].cpu().numpy(), ref.mean_codes), b
        assert scales[b].cpu().numpy().view(np.uint32) == ref.mean_scales.view(np.uint32)[0], b
        got_th = inp.theta[lo:hi].cpu().numpy()
        assert_close_elementwise(got_th, ref.theta, what=f"theta' block {b}")
        assert_close_elementwise(inp.momentum[lo:hi].cpu().numpy(), ref.momentum, what=f"v' block {b}")
        for r in inp.replicas:
            if dtype == torch.float32:
                assert np.array_equal(r[lo:hi].cpu().numpy().view(np.uint32), got_th.view(np.uint32)), b
            else:
                assert np.array_equal(bits16(r[lo:hi]), bits16(inp.theta[lo:hi].to(torch.bfloat16))), b
    del inp, ts
    torch.cuda.empty_cache()


def test_llama_1b1_sampled_codec_blocks(ctx):
    _sampled_codec_blocks(ctx, "llama-1.1b", 8, torch.float32, False, seed=3)


def test_llama_3b_bf16_sampled_codec_blocks(ctx):
    _sampled_codec_blocks(ctx, "llama-3b", 8, torch.bfloat16, True, seed=5)


@pytest.mark.parametrize("dtype,k", [(torch.float32, 1), (torch.float32, 3), (torch.bfloat16, 2)])
def test_codes_at_rounding_boundaries(ctx, dtype, k):
    # theta holds blocks crowded at the tie points of their own scale (and next
    # to them), the replicas are zero, so every worker's pseudo-gradient is
    # exactly theta and its codes are decided at those boundaries; the last block
    # is ragged.  Codes and scales of the encoded mean must equal the oracle's.
    from tests.int8_cases import near_half_block
    rng = np.random.default_rng(17)
    amaxes = (1.0, 3.7, 0.3)
    n = 3 * 4096 - 1000
    theta = np.concatenate([near_half_block(a, min(4096, n - 4096 * i), rng) for i, a in enumerate(amaxes)])
    momentum = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    inp = drift.RoundInputs(torch.from_numpy(theta), torch.from_numpy(momentum),
                            [torch.zeros(n, dtype=dtype) for _ in range(k)])
    dev = to_device(inp)
    c = al.make_coeffs(COEFFS["mu"], COEFFS["eta_out"], COEFFS["rho"], True)
    ref = ic.int8_round(theta, momentum, [host_array(r) for r in inp.replicas], c.mu, c.eta_out, c.rho, True, EPS)
    codes, scales = _payload(n)
    st = al.autoloco_outer_step_int8(ctx, dev.theta, dev.momentum, dev.replicas, c, al.FUSE_STATS | al.FUSE_RESET,
                                     EPS, mean_codes=codes, mean_scales=scales)
    torch.cuda.synchronize()
    assert np.array_equal(codes[:n].cpu().numpy(), ref.mean_codes), "mean codes differ"
    assert np.array_equal(scales[:3].cpu().numpy().view(np.uint32), ref.mean_scales.view(np.uint32)), "scales differ"
    assert_stats_close(st, ref.stats, floor=1e-9 * max(ref.stats.D, 1e-30))
    assert_close_elementwise(dev.theta.cpu().numpy(), ref.theta, what="theta'")
    assert_close_elementwise(dev.momentum.cpu().numpy(), ref.momentum, what="v'")


@pytest.mark.parametrize("grid", [1, 2, 3])
@pytest.mark.parametrize("dtype,k", [(torch.bfloat16, 8), (torch.bfloat16, 16), (torch.float32, 8)])
def test_many_blocks_per_workgroup(ctx, grid, dtype, k):
    # a capped grid gives every workgroup several codec blocks, even and odd
    # counts, so the prefetching loops go round (bf16 up to K = 8: blocks in pairs
    # with the two register sets swapping roles; fp32 up to K = 8: the LDS
    # prefetch) and the ragged last block follows them
    al.autoloco_set_grid_limit(ctx, grid)
    try:
        _check(ctx, 7 * 4096 + 100, k, dtype=dtype, seed=50 + grid + k, normalize=grid % 2 == 1)
    finally:
        al.autoloco_set_grid_limit(ctx, 0)


@pytest.mark.parametrize("k,dtype", [(4, torch.float32), (8, torch.bfloat16)])
def test_non_finite_blocks_stay_local(ctx, k, dtype):
    # a NaN in one block and an infinity in another: the round reports non-finite
    # statistics, the planted elements come out non-finite, and every other codec
    # block is exactly what the oracle gives (the codec and the step are local to
    # a block; inside the planted blocks the paper fixes no NaN arithmetic)
    n = 6 * 4096 + 1000
    inp = cpu_inputs(n, k, seed=77, replica_dtype=dtype)
    nan_at, inf_at = 1 * 4096 + 17, 3 * 4096 + 100
    inp.replicas[1][nan_at] = float("nan")
    inp.replicas[k - 1][inf_at] = float("inf")
    dev = to_device(inp)
    c = al.make_coeffs(COEFFS["mu"], COEFFS["eta_out"], COEFFS["rho"], True)
    with np.errstate(all="ignore"):
        ref = ic.int8_round(inp.theta.numpy(), inp.momentum.numpy(), [host_array(r) for r in inp.replicas],
                            c.mu, c.eta_out, c.rho, True, EPS)
    codes, scales = _payload(n)
    st = al.autoloco_outer_step_int8(ctx, dev.theta, dev.momentum, dev.replicas, c, al.FUSE_STATS | al.FUSE_RESET,
                                     EPS, mean_codes=codes, mean_scales=scales)
    torch.cuda.synchronize()
    assert not st.finite
    th, v = dev.theta.cpu().numpy(), dev.momentum.cpu().numpy()
    assert not np.isfinite(th[nan_at]) and not np.isfinite(th[inf_at])
    keep = [b for b in range((n + 4095) // 4096) if b not in (1, 3)]
    got_codes, got_scales = codes[:n].cpu().numpy(), scales.cpu().numpy()
    for b in keep:
        lo, hi = 4096 * b, min(n, 4096 * (b + 1))
        assert np.array_equal(got_codes[lo:hi], ref.mean_codes[lo:hi]), b
        assert got_scales[b].view(np.uint32) == ref.mean_scales[b].view(np.uint32), b
        assert_close_elementwise(th[lo:hi], ref.theta[lo:hi], what=f"theta' block {b}")
        assert_close_elementwise(v[lo:hi], ref.momentum[lo:hi], what=f"v' block {b}")
