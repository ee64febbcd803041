"""GPU tests that no kernel writes past the n elements a call is given.

Every buffer is allocated with a guard band of GUARD elements after the n the
call receives, filled with random bits, and the band is compared bit for bit
afterwards.  The sizes leave the last window, span or codec block of each
kernel short of full and add a ragged tail of n mod 4 elements: 5 (tail only),
two windows of two runs plus 7, three eight-window spans of the reset plus
five windows plus 3, and three codec blocks plus 1,001."""
import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al

pytestmark = pytest.mark.gpu

GUARD = 8200      # more than the longest span any kernel takes (8 windows of 1,024: the reset)
SIZES = [5, 4 * 256 * 2 + 7, 8 * 1024 * 3 + 5 * 1024 + 3, 4096 * 3 + 1001]
EPS = 1e-12


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()


def _buf(n, dtype, seed, positive=False):
    g = torch.Generator().manual_seed(seed)
    if dtype == torch.int8:
        t = torch.randint(-128, 128, (n + GUARD,), generator=g, dtype=torch.int8)
    else:
        t = torch.randn(n + GUARD, generator=g)
        t = (t.abs() if positive else t).to(dtype)
    return t.cuda()


def _band(t, n):
    x = t[n:].detach().cpu()
    return x.view(torch.int16 if x.element_size() == 2 else torch.int8 if x.element_size() == 1 else torch.int32).numpy().copy()


class Guarded:
    """Buffers whose bands past n are recorded at construction and checked later."""

    def __init__(self, n):
        self.n = n
        self.items = []

    def add(self, t, n=None):
        self.items.append((t, self.n if n is None else n, _band(t, self.n if n is None else n)))
        return t

    def check(self, what):
        torch.cuda.synchronize()
        for i, (t, n, band) in enumerate(self.items):
            assert np.array_equal(_band(t, n), band), f"{what}: buffer {i} written past n = {n}"


def _round_bufs(n, k, dtype, seed):
    g = Guarded(n)
    th = g.add(_buf(n, torch.float32, seed))
    v = g.add(_buf(n, torch.float32, seed + 1))
    reps = [g.add((th + 0.01 * _buf(n, torch.float32, seed + 2 + j)).to(dtype)) for j in range(k)]
    return g, th, v, reps


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("k", [3, 8])
@pytest.mark.parametrize("flags", [al.FUSE_STATS | al.FUSE_RESET, 0])
def test_fused_round(ctx, n, dtype, k, flags):
    g, th, v, reps = _round_bufs(n, k, dtype, seed=n + k)
    al.autoloco_outer_step(ctx, th, v, reps, al.make_coeffs(0.9, 0.7), flags, EPS, n=n)
    g.check("outer step")


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("dtype,k", [(torch.float32, 1), (torch.float32, 2), (torch.float32, 3),
                                     (torch.float32, 8), (torch.bfloat16, 1), (torch.bfloat16, 8)])
def test_reset(ctx, n, dtype, k):
    g, th, _, reps = _round_bufs(n, k, dtype, seed=2 * n + k)
    al.autoloco_broadcast_reset(ctx, th, reps, n=n)
    g.check("reset")


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_int8_round(ctx, n, dtype):
    g, th, v, reps = _round_bufs(n, 4, dtype, seed=3 * n)
    blocks = (n + 4095) // 4096
    codes = g.add(_buf(n, torch.int8, 7))
    scales = g.add(_buf(blocks, torch.float32, 8), n=blocks)
    al.autoloco_outer_step_int8(ctx, th, v, reps, al.make_coeffs(0.9, 0.7), al.FUSE_STATS | al.FUSE_RESET, EPS,
                                n=n, mean_codes=codes, mean_scales=scales)
    g.check("INT8 round")


@pytest.mark.parametrize("n", SIZES)
def test_bf16_payload_round(ctx, n):
    g, th, v, reps = _round_bufs(n, 4, torch.float32, seed=4 * n)
    mean = g.add(_buf(n, torch.bfloat16, 9))
    al.autoloco_outer_step_bf16(ctx, th, v, reps, al.make_coeffs(0.9, 0.7), al.FUSE_STATS | al.FUSE_RESET, EPS,
                                mean_bf16=mean, n=n)
    g.check("BF16-payload round")


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_share_kernels(ctx, n, dtype):
    g = Guarded(n)
    th = g.add(_buf(n, torch.float32, 10))
    rep = g.add(_buf(n, dtype, 11))
    payload = g.add(_buf(n, torch.bfloat16, 12))
    al.autoloco_rank_payload(ctx, th, rep, payload, n=n)
    g.check("worker payload")
    v = g.add(_buf(n, torch.float32, 13))
    shards = [g.add(_buf(n, torch.bfloat16, 14 + j)) for j in range(8)]
    mean = g.add(_buf(n, torch.bfloat16, 30))
    al.autoloco_shard_step(ctx, th, v, shards, al.make_coeffs(0.9, 0.7), mean_bf16=mean, n=n)
    g.check("shard step")


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("copy", [False, True])
def test_inner_adamw(ctx, n, copy):
    g = Guarded(n)
    k = 2
    params = [g.add(_buf(n, torch.float32, 40 + j)) for j in range(k)]
    m = [g.add(_buf(n, torch.float32, 50 + j)) for j in range(k)]
    v2 = [g.add(_buf(n, torch.float32, 60 + j, positive=True)) for j in range(k)]
    grads = [g.add(_buf(n, torch.float32, 70 + j)) for j in range(k)]
    model = [g.add(_buf(n, torch.bfloat16, 80 + j)) for j in range(k)] if copy else None
    al.autoloco_inner_adamw(ctx, params, m, v2, grads, al.make_adamw_coeffs(1e-3, 3), model_bf16=model, n=n)
    g.check("inner AdamW")
