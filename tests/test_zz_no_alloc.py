"""GPU test of autoloco_outer_step_static, the outer step for callers that
cannot allocate: called through the C ABI, it gives theta', v', the replicas
and the statistics of autoloco_outer_step (with a context) bit for bit, on
two calls in a row (the second on a smaller input that reuses the static
scratch with fewer workgroups' partials), for every flag subset and both
replica types; a bad device or a missing stats output launches nothing; and
repeated calls leave the device's free memory unchanged."""
import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al
from oracle import correction as ocorr
from tests.gpu_common import cpu_inputs, to_device

pytestmark = pytest.mark.gpu

EPS = 1e-12


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()


def _coeffs():
    sched = ocorr.Schedule()
    return al.autoloco_outer_correction(al.make_outer_cfg(normalize=True), ocorr.lr_mass(sched, 20_000, 750),
                                        ocorr.lr_mass(sched, 20_000, 500))


def _bits(t):
    t = t.detach().cpu()
    return t.view(torch.int16).numpy() if t.dtype == torch.bfloat16 else t.view(torch.int32).numpy()


def _same_stats(a, b, k):
    fields = [a.sq_mean, a.D, a.C, a.disagreement] + list(a.sq_norm[:k]) + list(a.sq_dev[:k])
    other = [b.sq_mean, b.D, b.C, b.disagreement] + list(b.sq_norm[:k]) + list(b.sq_dev[:k])
    return np.array_equal(np.array(fields, dtype=np.float64).view(np.int64),
                          np.array(other, dtype=np.float64).view(np.int64)) and a.finite == b.finite and a.k == b.k


# two calls in a row per case: a large input, then a smaller one
CASES = [((3 << 20) + 5, 8, torch.float32), (100_003, 3, torch.bfloat16)]


@pytest.mark.parametrize("flags", [al.FUSE_STATS | al.FUSE_RESET, al.FUSE_STATS, al.FUSE_RESET, 0])
def test_static_step_equals_context_step(ctx, flags):
    coeffs = _coeffs()
    for i, (n, k, dtype) in enumerate(CASES):
        inp = cpu_inputs(n, k, seed=61 + i, replica_dtype=dtype)
        a, b = to_device(inp), to_device(inp)
        st_ctx = al.autoloco_outer_step(ctx, a.theta, a.momentum, a.replicas, coeffs, flags, EPS)
        st_static = al.autoloco_outer_step_static(b.theta, b.momentum, b.replicas, coeffs, flags, EPS)
        torch.cuda.synchronize()
        if flags & al.FUSE_STATS:
            assert _same_stats(st_ctx, st_static, k), (n, k)
        else:
            assert st_static is None
        for x, y in zip([a.theta, a.momentum] + a.replicas, [b.theta, b.momentum] + b.replicas):
            assert np.array_equal(_bits(x), _bits(y)), (n, k, flags)


def test_bad_arguments_launch_nothing():
    n, k = 4096, 2
    inp = cpu_inputs(n, k, seed=67)
    dev = to_device(inp)
    snap = [t.clone() for t in [dev.theta, dev.momentum] + dev.replicas]
    with pytest.raises(al.AutolocoError) as e:
        al.autoloco_outer_step_static(dev.theta, dev.momentum, dev.replicas, _coeffs(), device=99)
    assert e.value.status == -1
    import ctypes as C
    bufs = al.make_buffers(dev.theta, dev.replicas, dev.momentum)
    stream = torch.cuda.current_stream().cuda_stream
    status = al.lib().autoloco_outer_step_static(0, C.c_void_p(stream), C.byref(bufs), C.byref(_coeffs()),
                                                 al.FUSE_STATS, EPS, None)
    assert status == -1                                      # FUSE_STATS needs an output
    status = al.lib().autoloco_outer_step_static(0, C.c_void_p(stream), C.byref(bufs), C.byref(_coeffs()),
                                                 al.FUSE_STATS, 0.0, C.byref(al._lib.Stats()))
    assert status == -1                                      # eps > 0
    torch.cuda.synchronize()
    for t, s in zip([dev.theta, dev.momentum] + dev.replicas, snap):
        assert torch.equal(t, s)


def test_repeated_calls_allocate_nothing():
    n, k = 1 << 20, 4
    dev = to_device(cpu_inputs(n, k, seed=71))
    coeffs = _coeffs()
    al.autoloco_outer_step_static(dev.theta, dev.momentum, dev.replicas, coeffs)   # set-up on first use
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    for _ in range(5):
        al.autoloco_outer_step_static(dev.theta, dev.momentum, dev.replicas, coeffs)
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert free1 == free0
