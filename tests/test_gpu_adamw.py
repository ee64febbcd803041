"""GPU parity of the workers' inner AdamW step against the oracle.

Every worker's parameters, moments and gradient norm are compared with the
float64 oracle (element-wise |g - o| <= 1e-5 (|o| + rms(o)); norms and
clipping factors to relative 1e-6), over ragged sizes, every worker count,
both recipes' settings, several consecutive steps of an interval on the
cosine schedule, the BF16 compute copy, the no-clipping and asynchronous
paths, a non-finite gradient and argument errors.  At the full 1.1B size the
update is checked on sampled elements, with the clipping factor taken from
an independent float64 norm of the same gradients."""
import ctypes as C
import math

import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al
from oracle import adamw as oa
from oracle import correction as ocorr
from tests.gpu_common import assert_bf16_reset_close, assert_close_elementwise, bits16
from workloads import inner, shapes

pytestmark = pytest.mark.gpu
C4 = oa.AdamWConfig()
SFT = oa.AdamWConfig(beta2=0.999, weight_decay=0.0)


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()


def _coeffs(cfg, lr, step):
    return al.make_adamw_coeffs(lr, step, cfg.beta1, cfg.beta2, cfg.eps, cfg.weight_decay, cfg.max_grad_norm)


def _dev(st):
    return inner.InnerState(*[[t.cuda() for t in group] for group in
                              (st.params, st.exp_avg, st.exp_avg_sq, st.grads)])


def _np(ts):
    return [t.detach().cpu().numpy().astype(np.float64) for t in ts]


def _check_state(dev, ref, what=""):
    for i in range(dev.k):
        assert_close_elementwise(dev.params[i].cpu().numpy(), ref.params[i], what=f"{what} params[{i}]")
        assert_close_elementwise(dev.exp_avg[i].cpu().numpy(), ref.exp_avg[i], what=f"{what} m[{i}]")
        assert_close_elementwise(dev.exp_avg_sq[i].cpu().numpy(), ref.exp_avg_sq[i], what=f"{what} v[{i}]")


def _check_stats(st, ref, k):
    assert st.k == k
    for i in range(k):
        assert st.grad_norm[i] == pytest.approx(ref.grad_norm[i], rel=1e-6, abs=1e-30)
        assert st.clip_coef[i] == pytest.approx(ref.clip_coef[i], rel=1e-6)
    assert bool(st.finite) == all(math.isfinite(x) for x in ref.grad_norm)


def _one_step(ctx, n, k, cfg=C4, step=1, lr=3e-4, seed=1, copy=False):
    host = inner.make_state(n, k, seed=seed)
    dev = _dev(host)
    ref = oa.inner_step(_np(host.params), _np(host.exp_avg), _np(host.exp_avg_sq), _np(host.grads), lr, step, cfg)
    cp = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(k)] if copy else None
    st = al.autoloco_inner_adamw(ctx, dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads, _coeffs(cfg, lr, step),
                                 model_bf16=cp)
    torch.cuda.synchronize()
    _check_state(dev, ref, f"n={n} k={k}")
    _check_stats(st, ref, k)
    return dev, ref, st, cp


@pytest.mark.parametrize("n", [1, 3, 4, 5, 1023, 4096 + 3, (1 << 20) + 7])
def test_sizes(ctx, n):
    _one_step(ctx, n, 3, step=1 + n % 5, seed=n % 97)


@pytest.mark.parametrize("k", [1, 2, 5, 8, 13, 16])
def test_worker_counts(ctx, k):
    _, ref, st, _ = _one_step(ctx, 100_003, k, cfg=SFT if k % 2 else C4, step=k, seed=20 + k)
    if k >= 4:
        assert any(c < 1.0 for c in ref.clip_coef) and any(c == 1.0 for c in ref.clip_coef)


@pytest.mark.parametrize("cfg", [C4, SFT], ids=["c4", "sft"])
def test_interval_of_steps(ctx, cfg):
    # eight consecutive steps on the cosine schedule from step 20,000, a fresh gradient each step;
    # the oracle carries its state in float64 throughout
    n, k, seed = 300_007, 4, 5
    host = inner.make_state(n, k, seed=seed)
    dev = _dev(host)
    p, m, v = _np(host.params), _np(host.exp_avg), _np(host.exp_avg_sq)
    sched = ocorr.Schedule()
    for h in range(8):
        if h:
            inner.fill_grads(host, seed, h)
            for i in range(k):
                dev.grads[i].copy_(host.grads[i])
        lr = ocorr.inner_lr(sched, 20_000 + h)
        ref = oa.inner_step(p, m, v, _np(host.grads), lr, 100 + h, cfg)
        p, m, v = ref.params, ref.exp_avg, ref.exp_avg_sq
        st = al.autoloco_inner_adamw(ctx, dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads,
                                     _coeffs(cfg, lr, 100 + h))
        _check_stats(st, ref, k)
    torch.cuda.synchronize()
    _check_state(dev, ref, "after 8 steps")


def test_warmup_first_steps(ctx):
    # the very first steps of training: zero moments, warm-up learning rates
    n, k = 65_537, 2
    host = inner.make_state(n, k, seed=9)
    for t in host.exp_avg + host.exp_avg_sq:
        t.zero_()
    dev = _dev(host)
    p, m, v = _np(host.params), _np(host.exp_avg), _np(host.exp_avg_sq)
    for s in range(3):
        lr = ocorr.inner_lr(ocorr.Schedule(), s)
        ref = oa.inner_step(p, m, v, _np(host.grads), lr, s + 1, C4)
        p, m, v = ref.params, ref.exp_avg, ref.exp_avg_sq
        al.autoloco_inner_adamw(ctx, dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads, _coeffs(C4, lr, s + 1))
    torch.cuda.synchronize()
    _check_state(dev, ref, "warm-up")


def test_bf16_copy(ctx):
    dev, ref, _, cp = _one_step(ctx, 200_003, 3, copy=True, seed=11)
    for i in range(3):
        assert np.array_equal(bits16(cp[i]), bits16(dev.params[i].to(torch.bfloat16)))
        assert_bf16_reset_close(bits16(cp[i]), ref.params[i], what=f"bf16 copy {i}")


@pytest.mark.parametrize("copy", [False, True])
def test_traffic_reference_keeps_the_state(ctx, copy):
    # the update pass's traffic reference (a measurement) leaves every buffer as
    # the last step left it: state bits unchanged, the BF16 copies rewritten with
    # the same bits, gradients untouched; bad buffers launch nothing
    n, k = 3 * 4096 * 64 + 5, 3
    dev, _, _, cp = _one_step(ctx, n, k, copy=copy, seed=21)
    torch.cuda.synchronize()
    before = [t.clone() for t in dev.params + dev.exp_avg + dev.exp_avg_sq + dev.grads + (cp or [])]
    al.autoloco_adamw_traffic_reference(ctx, dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads, model_bf16=cp)
    torch.cuda.synchronize()
    after = dev.params + dev.exp_avg + dev.exp_avg_sq + dev.grads + (cp or [])
    for x, y in zip(before, after):
        assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x.view(torch.int32),
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32))
    f = al.lib().autoloco_adamw_traffic_reference
    b = al.make_adamw_buffers(dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads)
    b.params[1] = dev.params[1].data_ptr() + 4
    assert f(ctx.handle, C.byref(b)) == -2
    b.params[1] = dev.exp_avg[0].data_ptr()
    assert f(ctx.handle, C.byref(b)) == -3
    torch.cuda.synchronize()
    assert torch.equal(dev.exp_avg[0].view(torch.int32), before[k].view(torch.int32))


def test_no_clipping_asynchronous(ctx):
    cfg = oa.AdamWConfig(max_grad_norm=0.0)
    n, k = 123_457, 4
    host = inner.make_state(n, k, seed=12)
    dev = _dev(host)
    ref = oa.inner_step(_np(host.params), _np(host.exp_avg), _np(host.exp_avg_sq), _np(host.grads), 2e-4, 3, cfg)
    assert al.autoloco_inner_adamw(ctx, dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads,
                                   _coeffs(cfg, 2e-4, 3), stats=False) is None
    torch.cuda.synchronize()
    _check_state(dev, ref, "no clipping")
    # the same settings with stats: norms reported, factors 1
    host2 = inner.make_state(n, k, seed=12)
    dev2 = _dev(host2)
    st = al.autoloco_inner_adamw(ctx, dev2.params, dev2.exp_avg, dev2.exp_avg_sq, dev2.grads,
                                 _coeffs(cfg, 2e-4, 3))
    _check_stats(st, ref, k)
    assert all(st.clip_coef[i] == 1.0 for i in range(k))
    for i in range(k):
        assert torch.equal(dev.params[i], dev2.params[i])


def test_non_finite_gradient(ctx):
    n, k = 40_000, 3
    host = inner.make_state(n, k, seed=13)
    host.grads[1][777] = float("nan")
    dev = _dev(host)
    ref = oa.inner_step(_np(host.params), _np(host.exp_avg), _np(host.exp_avg_sq), _np(host.grads), 1e-4, 5, C4)
    st = al.autoloco_inner_adamw(ctx, dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads, _coeffs(C4, 1e-4, 5))
    assert not st.finite and math.isnan(st.grad_norm[1])
    assert torch.isnan(dev.params[1]).all().item()
    for i in (0, 2):
        assert_close_elementwise(dev.params[i].cpu().numpy(), ref.params[i], what=f"params[{i}]")


def test_deterministic(ctx):
    outs = []
    for _ in range(2):
        host = inner.make_state(500_001, 5, seed=14)
        dev = _dev(host)
        st = al.autoloco_inner_adamw(ctx, dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads, _coeffs(C4, 3e-4, 9))
        outs.append((bytes(st), b"".join(t.cpu().numpy().tobytes() for t in dev.params + dev.exp_avg_sq)))
    assert outs[0] == outs[1]


def test_argument_errors(ctx):
    n, k = 4096, 2
    dev = _dev(inner.make_state(n, k, seed=15))
    f = al.lib().autoloco_inner_adamw
    good = _coeffs(C4, 1e-4, 1)
    st = al._lib.AdamWStats()

    def call(b, co=good):
        return f(ctx.handle, C.byref(b), C.byref(co), C.byref(st))

    b = al.make_adamw_buffers(dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads)
    assert call(b) == 0
    b.params[1] = dev.params[1].data_ptr() + 4
    assert call(b) == -2                                       # misaligned
    b.params[1] = dev.exp_avg[0].data_ptr()
    assert call(b) == -3                                       # params[1] aliases exp_avg[0]
    b = al.make_adamw_buffers(dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads)
    cp = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    b.model_bf16[0] = cp.data_ptr()
    assert call(b) == -1                                       # copy for one worker only
    b.model_bf16[0] = None
    b.grads[0] = None
    assert call(b) == -1                                       # null gradient
    b = al.make_adamw_buffers(dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads)
    for bad in (al.make_adamw_coeffs(1e-4, 0), al.make_adamw_coeffs(-1e-4, 1), al.make_adamw_coeffs(1e-4, 1, beta2=1.0),
                al.make_adamw_coeffs(1e-4, 1, max_grad_norm=float("nan")), al.make_adamw_coeffs(1e-4, 1, eps=-1.0)):
        assert call(b, bad) == -1
    b.k = 17
    assert call(b) == -1
    b.k = 2
    host = torch.zeros(n, dtype=torch.float32, pin_memory=True)
    b.grads[1] = host.data_ptr()                                # pinned host memory, not device memory
    assert call(b) == -1 and "not device memory" in al.autoloco_last_error(ctx)
    b = al.make_adamw_buffers(dev.params, dev.exp_avg, dev.exp_avg_sq, dev.grads)
    b.k = 2
    b.n = 0
    assert call(b) == 0 and st.k == 2 and st.clip_coef[0] == 1.0 and st.grad_norm[1] == 0.0


def test_llama_1b1_sampled(ctx):
    n, k = shapes.llama_1b1().n_params, 8
    ts, _ = al.spread_tensors(ctx, n, [torch.float32] * (4 * k))
    st_dev = inner.InnerState(ts[0:k], ts[k:2 * k], ts[2 * k:3 * k], ts[3 * k:4 * k])
    inner.fill_state(st_dev, seed=42)
    inner.fill_grads(st_dev, seed=42, step=0)
    rng = np.random.default_rng(6)
    idx = np.unique(np.concatenate([rng.integers(0, n, 4000), [0, 1, n - 2, n - 1]]))
    it = torch.as_tensor(idx, device="cuda")
    before = [[g[i][it].cpu().numpy().astype(np.float64) for i in range(k)]
              for g in (st_dev.params, st_dev.exp_avg, st_dev.exp_avg_sq, st_dev.grads)]
    norms = [float(torch.linalg.vector_norm(g.double()).item()) for g in st_dev.grads]   # independent of the library
    lr = ocorr.inner_lr(ocorr.Schedule(), 20_000)
    st = al.autoloco_inner_adamw(ctx, st_dev.params, st_dev.exp_avg, st_dev.exp_avg_sq, st_dev.grads,
                                 _coeffs(C4, lr, 2000))
    torch.cuda.synchronize()
    assert st.finite
    for i in range(k):
        assert st.grad_norm[i] == pytest.approx(norms[i], rel=1e-6)
        c = oa.clip_coefficient(norms[i], C4.max_grad_norm)
        assert st.clip_coef[i] == pytest.approx(c, rel=1e-6)
        p, m, v = oa.adamw_step(before[0][i], before[1][i], before[2][i], before[3][i], lr, 2000, C4, c)
        assert_close_elementwise(st_dev.params[i][it].cpu().numpy(), p, what=f"1.1B params[{i}]")
        assert_close_elementwise(st_dev.exp_avg[i][it].cpu().numpy(), m, what=f"1.1B m[{i}]")
        assert_close_elementwise(st_dev.exp_avg_sq[i][it].cpu().numpy(), v, what=f"1.1B v[{i}]")
    assert any(oa.clip_coefficient(x, 1.0) < 1.0 for x in norms) and any(oa.clip_coefficient(x, 1.0) == 1.0
                                                                         for x in norms)
    del st_dev, ts
    torch.cuda.empty_cache()
