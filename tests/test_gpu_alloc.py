"""GPU tests of the placement-aware allocator: buffers are distinct, aligned
and usable by the round (parity with the oracle on them), they free cleanly,
and bad arguments are refused."""
import ctypes as C

import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al
from oracle import round as orr
from tests.gpu_common import assert_close_elementwise, assert_stats_close
from workloads import drift

pytestmark = pytest.mark.gpu
EPS = 1e-12


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()


def test_spread_buffers_are_distinct_and_aligned(ctx):
    nbytes = 64 << 20
    ptrs, spread = al.autoloco_alloc_spread(ctx, 10, nbytes)
    try:
        assert len(set(ptrs)) == 10 and all(p % 256 == 0 for p in ptrs)
        srt = sorted(ptrs)
        assert all(b - a >= nbytes for a, b in zip(srt, srt[1:]))
    finally:
        for p in ptrs:
            al.autoloco_free(ctx, p)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_round_on_spread_buffers_matches_oracle(ctx, dtype):
    n, k = 1_000_003, 8
    ts, _ = al.spread_tensors(ctx, n, [torch.float32, torch.float32] + [dtype] * k)
    inp = drift.RoundInputs(ts[0], ts[1], ts[2:])
    drift.fill_theta_momentum(inp, seed=5)
    drift.fill_replicas(inp, seed=5)
    th = inp.theta.cpu().numpy()
    mo = inp.momentum.cpu().numpy()
    reps = [r.cpu().view(torch.int16).numpy().view(np.uint16) if dtype == torch.bfloat16 else r.cpu().numpy()
            for r in inp.replicas]
    c = al.make_coeffs(0.85, 1.5, 1.49, True)
    ref = orr.sync_round(th, mo, reps, c.mu, c.eta_out, c.rho, True, EPS)
    st = al.autoloco_outer_step(ctx, inp.theta, inp.momentum, inp.replicas, c, al.FUSE_STATS | al.FUSE_RESET, EPS)
    assert_stats_close(st, ref.stats)
    assert_close_elementwise(inp.theta.cpu().numpy(), ref.theta, what="theta'")
    assert_close_elementwise(inp.momentum.cpu().numpy(), ref.momentum, what="v'")
    del inp, ts
    torch.cuda.synchronize()


def test_alloc_spread_rejects_bad_arguments(ctx):
    out = (C.c_void_p * 2)()
    assert al.lib().autoloco_alloc_spread(ctx.handle, 0, 1024, out, None) == -1
    assert al.lib().autoloco_alloc_spread(ctx.handle, 65, 1024, out, None) == -1
    assert al.lib().autoloco_alloc_spread(ctx.handle, 2, 0, out, None) == -1
    assert al.lib().autoloco_alloc_spread(ctx.handle, 2, 1024, None, None) == -1
    assert al.lib().autoloco_free(ctx.handle, None) == 0


def test_buffers_outliving_their_context_are_freed():
    # closing the context while its spread buffers are still alive detaches it
    # from the API at once; the buffers keep their memory until they are
    # collected and then return it (the native context goes with the last one)
    import gc
    gc.collect()
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info(0)
    c = al.autoloco_create(0)
    n = 256 << 20   # 1 GiB per fp32 buffer
    ts, _ = al.spread_tensors(c, n, [torch.float32] * 2)
    ts[0].fill_(1.5)
    ts[1].copy_(ts[0])
    c.close()
    assert c.handle is None
    with pytest.raises(Exception):
        al.autoloco_launch_shape(c, 1024, 2)
    # still this process's memory after the close
    assert [float(ts[1][i]) for i in (0, n // 2, n - 1)] == [1.5] * 3
    held, _ = torch.cuda.mem_get_info(0)
    assert free0 - held >= 2 * (n * 4)
    del ts
    gc.collect()
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info(0)
    assert c._held is None and c._live == 0
    assert free1 >= free0 - (64 << 20), (free0, free1)
