"""One GPU's share of a round with one worker replica per GPU.

On one GPU the collectives are stand-ins (the payload shards are views of
each worker's payload; theta is shared, so the all-gather is a no-op), and
the decomposition - every worker's payload, then every shard's step, then the
reset - must give exactly the bits of the fused BF16-payload round, and the
oracle's values.  At the full 1.1B size the per-GPU shapes are checked on
sampled parameters against the oracle."""
import ctypes as C

import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al
from oracle import bf16_payload as bp
from oracle import round as orr
from tests.gpu_common import assert_close_elementwise, assert_stats_close, bits16, cpu_inputs, host_array, to_device
from workloads import drift, shapes

pytestmark = pytest.mark.gpu
EPS = 1e-12
MU, ETA, RHO = 0.8545853971914775, 1.5181396589623761, 1.4914395799922477


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()


def _shards(n, g):
    step = -(-n // g)
    step = -(-step // 8) * 8                     # shard boundaries on 16-byte payload vectors
    return [(lo, min(n, lo + step)) for lo in range(0, n, step)]


def _decomposed(ctx, dev, k, coeffs, n, g):
    payloads = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(k)]
    sq = [al.autoloco_rank_payload(ctx, dev.theta, dev.replicas[r], payloads[r]) for r in range(k)]
    mean = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    m = 0.0
    for lo, hi in _shards(n, g):
        m += al.autoloco_shard_step(ctx, dev.theta[lo:hi], dev.momentum[lo:hi], [p[lo:hi] for p in payloads],
                                    coeffs, mean_bf16=mean[lo:hi])
    al.autoloco_broadcast_reset(ctx, dev.theta, dev.replicas)
    torch.cuda.synchronize()
    d = sum(sq) / k
    return sq, m, d, mean, payloads


@pytest.mark.parametrize("n,k,dtype,g", [(1_000_003, 8, torch.float32, 8), (4096 + 5, 4, torch.float32, 4),
                                         (300_001, 1, torch.float32, 1), (250_007, 8, torch.bfloat16, 8),
                                         (77, 3, torch.float32, 3), (131_072, 16, torch.float32, 5)])
def test_decomposition_equals_fused_round(ctx, n, k, dtype, g):
    inp = cpu_inputs(n, k, seed=n % 1000, replica_dtype=dtype)
    a, b = to_device(inp), to_device(inp)
    c = al.make_coeffs(MU, ETA, RHO, k % 2 == 0)
    mean_a = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    st = al.autoloco_outer_step_bf16(ctx, a.theta, a.momentum, a.replicas, c, al.FUSE_STATS | al.FUSE_RESET, EPS,
                                     mean_bf16=mean_a)
    sq, m, d, mean_b, _ = _decomposed(ctx, b, k, c, n, g)
    assert torch.equal(a.theta, b.theta) and torch.equal(a.momentum, b.momentum)
    assert np.array_equal(bits16(mean_a), bits16(mean_b))
    for ra, rb in zip(a.replicas, b.replicas):
        assert torch.equal(ra.view(torch.int16) if dtype == torch.bfloat16 else ra,
                           rb.view(torch.int16) if dtype == torch.bfloat16 else rb)
    # the same float64 sums, with fp32 partials over 8 instead of 4 or 8 parameters
    for r in range(k):
        assert sq[r] == pytest.approx(st.sq_norm[r], rel=1e-6)
    assert d == pytest.approx(st.D, rel=1e-6)
    assert m == pytest.approx(st.sq_mean, rel=1e-6)
    # and the oracle's values
    ref = bp.bf16_round(inp.theta.numpy(), inp.momentum.numpy(), [host_array(r) for r in inp.replicas],
                        c.mu, c.eta_out, c.rho, bool(c.normalize), EPS)
    assert np.array_equal(bits16(mean_b), ref.mean_bits)
    assert_close_elementwise(b.theta.cpu().numpy(), ref.theta, what="theta'")
    assert_close_elementwise(b.momentum.cpu().numpy(), ref.momentum, what="v'")
    assert d == pytest.approx(ref.stats.D, rel=1e-4)
    assert k * m / (d + EPS) == pytest.approx(ref.stats.C, rel=1e-4)


def test_payload_matches_oracle(ctx):
    n = 100_003
    inp = cpu_inputs(n, 2, seed=5, replica_dtype=torch.bfloat16)
    dev = to_device(inp)
    p = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    s = al.autoloco_rank_payload(ctx, dev.theta, dev.replicas[1], p)
    delta = inp.theta.numpy() - orr.widen(host_array(inp.replicas[1])).astype(np.float32)
    assert np.array_equal(bits16(p), bp.payload(delta))
    assert s == pytest.approx(float(np.sum(delta.astype(np.float64) ** 2)), rel=1e-6)
    assert al.autoloco_rank_payload(ctx, dev.theta, dev.replicas[0], p, sq_norm=False) is None


def test_argument_errors(ctx):
    n = 4096
    dev = to_device(cpu_inputs(n, 2, seed=6))
    p = torch.empty(n + 16, dtype=torch.bfloat16, device="cuda")
    L = al.lib()
    out = C.c_double()
    th, rep = C.c_void_p(dev.theta.data_ptr()), C.c_void_p(dev.replicas[0].data_ptr())
    assert L.autoloco_rank_payload(ctx.handle, n, th, rep, 0, C.c_void_p(p.data_ptr() + 2), C.byref(out)) == -2
    assert L.autoloco_rank_payload(ctx.handle, n, th, rep, 0, C.c_void_p(dev.replicas[0].data_ptr() + 16),
                                   C.byref(out)) == -3
    assert L.autoloco_rank_payload(ctx.handle, n, th, rep, 7, C.c_void_p(p.data_ptr()), C.byref(out)) == -1
    assert L.autoloco_rank_payload(ctx.handle, n, th, None, 0, C.c_void_p(p.data_ptr()), C.byref(out)) == -1
    b = al._lib.ShardBuffers()
    b.n, b.k = n, 2
    b.theta, b.momentum = dev.theta.data_ptr(), dev.momentum.data_ptr()
    b.payloads[0], b.payloads[1] = p.data_ptr(), dev.replicas[1].data_ptr()
    cf = al.make_coeffs(0.9, 0.7)
    assert L.autoloco_shard_step(ctx.handle, C.byref(b), C.byref(cf), None, C.byref(out)) == 0
    b.payloads[1] = dev.theta.data_ptr() + 32
    assert L.autoloco_shard_step(ctx.handle, C.byref(b), C.byref(cf), None, C.byref(out)) == -3
    b.payloads[1] = None
    assert L.autoloco_shard_step(ctx.handle, C.byref(b), C.byref(cf), None, C.byref(out)) == -1
    b.k = 0
    assert L.autoloco_shard_step(ctx.handle, C.byref(b), C.byref(cf), None, C.byref(out)) == -1
    b.k, b.n = 2, 0
    assert L.autoloco_shard_step(ctx.handle, C.byref(b), C.byref(cf), None, C.byref(out)) == 0 and out.value == 0.0


def test_llama_1b1_per_gpu_shapes(ctx):
    # worker 3 of 8 computes its payload over the whole model; GPU 3 steps its eighth of the parameters
    n, k, g, r = shapes.llama_1b1().n_params, 8, 8, 3
    ts, _ = al.spread_tensors(ctx, n, [torch.float32] * 3)
    theta, mom, rep = ts
    inp = drift.RoundInputs(theta, mom, [rep])
    drift.fill_theta_momentum(inp, seed=42)
    drift.fill_replicas(inp, seed=42)
    payload = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    s = al.autoloco_rank_payload(ctx, theta, rep, payload)
    rng = np.random.default_rng(9)
    idx = np.unique(np.concatenate([rng.integers(0, n, 20_000), [0, n - 1]]))
    it = torch.as_tensor(idx, device="cuda")
    delta = theta[it].cpu().numpy() - rep[it].cpu().numpy()
    assert np.array_equal(bits16(payload[it]), bp.payload(delta))
    assert s > 0 and np.isfinite(s)
    lo, hi = _shards(n, g)[r]
    ns = hi - lo
    # the K payload shards GPU 3 would receive: this worker's, and seeded stand-ins for the others
    shards = [payload[lo:hi].clone()]
    for w in range(1, k):
        x = torch.empty(ns, dtype=torch.float32, device="cuda")
        drift._normal_into(x, 1e-3, 100 + w, 4, w)
        shards.append(x.to(torch.bfloat16))
    th_s, v_s = theta[lo:hi].clone(), mom[lo:hi].clone()
    sidx = np.unique(np.concatenate([rng.integers(0, ns, 20_000), [0, ns - 1]]))
    sit = torch.as_tensor(sidx, device="cuda")
    th0, v0 = th_s[sit].cpu().numpy(), v_s[sit].cpu().numpy()
    b0 = [bits16(x[sit]) for x in shards]
    c = al.make_coeffs(MU, ETA, RHO, False)
    mean = torch.empty(ns, dtype=torch.bfloat16, device="cuda")
    m = al.autoloco_shard_step(ctx, th_s, v_s, shards, c, mean_bf16=mean)
    torch.cuda.synchronize()
    bits = bp.aggregate(b0)
    assert np.array_equal(bits16(mean[sit]), bits)
    agg = orr.widen(bits)
    th_ref, v_ref = orr.outer_update(th0, v0, agg, c.mu, c.eta_out, c.rho, False)
    assert_close_elementwise(th_s[sit].cpu().numpy(), th_ref, what="shard theta'")
    assert_close_elementwise(v_s[sit].cpu().numpy(), v_ref, what="shard v'")
    full = orr.widen(bits16(mean))
    assert m == pytest.approx(float(np.sum(full * full)), rel=1e-6)
    del inp, ts, theta, mom, rep, shards
    torch.cuda.empty_cache()
