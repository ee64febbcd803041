"""GPU tests of the traffic reference (the fused round's loads and stores
without its arithmetic): every buffer holds its old bits afterwards, across
worker counts, both replica types, ragged sizes and a grid cap that forces
several grid-stride passes, and bad arguments launch nothing."""
import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al
from tests.gpu_common import cpu_inputs, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()


def _bits(t):
    t = t.detach().cpu()
    return t.view(torch.int16).numpy().copy() if t.dtype == torch.bfloat16 else t.view(torch.int32).numpy().copy()


@pytest.mark.parametrize("rdt", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("k", [1, 3, 8, 16])
@pytest.mark.parametrize("n", [1, 5, 4 * 256 + 3, 8 * 256 * 7 + 9, 300_001])
def test_buffers_unchanged(ctx, rdt, k, n):
    dev = to_device(cpu_inputs(n, k, seed=7 + k, replica_dtype=rdt))
    before = [_bits(dev.theta), _bits(dev.momentum)] + [_bits(r) for r in dev.replicas]
    al.autoloco_set_grid_limit(ctx, 3)   # several grid-stride passes at these sizes
    try:
        al.autoloco_traffic_reference(ctx, dev.theta, dev.momentum, dev.replicas)
        torch.cuda.synchronize()
    finally:
        al.autoloco_set_grid_limit(ctx, 0)
    after = [_bits(dev.theta), _bits(dev.momentum)] + [_bits(r) for r in dev.replicas]
    for i, (b, a) in enumerate(zip(before, after)):
        assert np.array_equal(b, a), f"buffer {i} changed"


def test_timed_and_default_grid(ctx):
    n, k = 1 << 22, 8
    dev = to_device(cpu_inputs(n, k, seed=3))
    before = _bits(dev.replicas[5])
    al.autoloco_set_timing(ctx, True)
    try:
        al.autoloco_traffic_reference(ctx, dev.theta, dev.momentum, dev.replicas)
        ms = al.autoloco_last_kernel_ms(ctx)
    finally:
        al.autoloco_set_timing(ctx, False)
    assert ms > 0.0
    assert np.array_equal(before, _bits(dev.replicas[5]))


def test_rejects_aliasing_and_host_memory(ctx):
    n, k = 4096, 2
    dev = to_device(cpu_inputs(n, k, seed=1))
    th0 = _bits(dev.theta)
    with pytest.raises(al.AutolocoError):
        al.autoloco_traffic_reference(ctx, dev.theta, dev.theta, dev.replicas)
    host = torch.empty(n, dtype=torch.float32, pin_memory=True)
    host.fill_(7.0)
    b = al.make_buffers(dev.theta, dev.replicas, dev.momentum)
    b.momentum = host.data_ptr()
    assert al.lib().autoloco_traffic_reference(ctx.handle, b) == -1
    assert "not device memory" in al.autoloco_last_error(ctx)
    torch.cuda.synchronize()
    assert np.array_equal(th0, _bits(dev.theta)) and bool((host == 7.0).all())
