"""GPU parity at the full model sizes, in the launch configuration the
benchmark times (library default grid).

GPT-2 small (124,439,808 parameters, K = 8 fp32): the oracle streams every
parameter back to the host and sums the statistics in float64; θ', v' and the
reset replicas are compared on sampled parameters.

Llama-style 1.1B (K = 8 fp32) and 3B (K = 8 bf16 replicas): too large for the
oracle to read whole in a test, so
  * θ', v' and the reset replicas are compared with the oracle on 2^20 sampled
    parameters (plus the first and last ones), computed one by one;
  * the full-size statistics must equal the sum of the statistics of disjoint
    sub-ranges (each its own launch) to fp64 rounding, and two of those
    sub-ranges (one of them the last) are compared with the oracle in full;
  * the App. C.1 identity disagreement = D - ||Delta_bar||^2 holds at any size."""
import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al
from oracle import correction as ocorr
from oracle import round as orr
from tests.gpu_common import (assert_bf16_reset_close, assert_close_elementwise, assert_stats_close,
                              host_array)
from workloads import drift, shapes

pytestmark = pytest.mark.gpu
EPS = 1e-12


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()
    torch.cuda.empty_cache()


def _coeffs(h_sel=750, h_ref=500, normalize=False):
    s = ocorr.Schedule()
    return al.autoloco_outer_correction(al.make_outer_cfg(normalize=normalize), ocorr.lr_mass(s, 20_000, h_sel),
                                        ocorr.lr_mass(s, 20_000, h_ref))


def _sample_index(n, m=1 << 20, seed=0):
    rng = np.random.default_rng(seed)
    edge = np.array([0, 1, 2, 3, 4, 7, 8, n // 2, n - 9, n - 8, n - 5, n - 4, n - 3, n - 2, n - 1])
    idx = np.unique(np.concatenate([rng.integers(0, n, m), edge[(edge >= 0) & (edge < n)]]))
    return torch.from_numpy(idx).cuda()


def _gather(inp, idx):
    th = inp.theta.index_select(0, idx).cpu().numpy()
    mo = inp.momentum.index_select(0, idx).cpu().numpy()
    reps = [host_array(r.index_select(0, idx)) for r in inp.replicas]
    return th, mo, reps


def _oracle_chunked_stats(inp, lo, hi, chunk=1 << 22):
    """Oracle statistics of parameters [lo, hi), streamed to the host in chunks."""
    k = inp.k
    s_tot, q_tot, m_tot = [0.0] * k, [0.0] * k, 0.0
    for a in range(lo, hi, chunk):
        b = min(hi, a + chunk)
        th = inp.theta[a:b].cpu().numpy()
        reps = [host_array(r[a:b]) for r in inp.replicas]
        s, q, m = orr.partial_sums(th, reps)
        s_tot = [x + y for x, y in zip(s_tot, s)]
        q_tot = [x + y for x, y in zip(q_tot, q)]
        m_tot += m
    return orr.finish_stats(s_tot, q_tot, m_tot, EPS)


def _check_sampled_outputs(inp, idx, sample_in, coeffs, replica_dtype):
    th, mo, reps = sample_in
    ref = orr.sync_round(th, mo, reps, coeffs.mu, coeffs.eta_out, coeffs.rho, bool(coeffs.normalize), EPS)
    got_th = inp.theta.index_select(0, idx).cpu().numpy()
    assert_close_elementwise(got_th, ref.theta, what="theta' (sampled)")
    assert_close_elementwise(inp.momentum.index_select(0, idx).cpu().numpy(), ref.momentum, what="v' (sampled)")
    for r in inp.replicas:
        g = host_array(r.index_select(0, idx))
        if replica_dtype == torch.float32:
            assert np.array_equal(g.view(np.uint32), got_th.view(np.uint32))
        else:
            assert_bf16_reset_close(g, ref.theta)


@pytest.mark.parametrize("sigma", [1e-4, 1e-3, 1e-2])
def test_gpt2_small_full(ctx, sigma):
    n = shapes.gpt2_small().n_params
    assert n == 124_439_808
    inp = drift.make_round_inputs(n, 8, seed=42, recipe=drift.spread_recipe(sigma), device="cuda")
    ref_stats = _oracle_chunked_stats(inp, 0, n)
    idx = _sample_index(n, seed=1)
    sample_in = _gather(inp, idx)
    c = _coeffs()
    st = al.autoloco_outer_step(ctx, inp.theta, inp.momentum, inp.replicas, c, al.FUSE_STATS | al.FUSE_RESET, EPS)
    torch.cuda.synchronize()
    assert_stats_close(st, ref_stats)
    _check_sampled_outputs(inp, idx, sample_in, c, torch.float32)
    expect_c = {1e-4: 7.93, 1e-3: 4.50, 1e-2: 1.07}[sigma]
    assert st.C == pytest.approx(expect_c, rel=0.01)
    del inp
    torch.cuda.empty_cache()


def _large(ctx, shape, k, replica_dtype, parts, oracle_parts, normalize):
    n = shapes.SHAPES[shape]().n_params
    inp = drift.make_round_inputs(n, k, seed=42, replica_dtype=replica_dtype, device="cuda")
    idx = _sample_index(n, seed=2)
    sample_in = _gather(inp, idx)

    full = al.autoloco_round_stats(ctx, inp.theta, inp.replicas, EPS)
    # disjoint sub-ranges, boundaries on multiples of 16 parameters (pointers stay 16-byte aligned)
    bounds = [0] + [((n * p) // parts) // 16 * 16 for p in range(1, parts)] + [n]
    s_tot, q_tot, m_tot = [0.0] * k, [0.0] * k, 0.0
    sub = []
    for p in range(parts):
        lo, hi = bounds[p], bounds[p + 1]
        st = al.autoloco_round_stats(ctx, inp.theta[lo:], [r[lo:] for r in inp.replicas], EPS, n=hi - lo)
        sub.append(st)
        s_tot = [a + st.sq_norm[i] for i, a in enumerate(s_tot)]
        q_tot = [a + st.sq_dev[i] for i, a in enumerate(q_tot)]
        m_tot += st.sq_mean
    for i in range(k):
        assert full.sq_norm[i] == pytest.approx(s_tot[i], rel=1e-11)
        assert full.sq_dev[i] == pytest.approx(q_tot[i], rel=1e-11)
    assert full.sq_mean == pytest.approx(m_tot, rel=1e-11)
    assert full.disagreement == pytest.approx(full.D - full.sq_mean, rel=1e-4)
    for p in oracle_parts:
        lo, hi = bounds[p], bounds[p + 1]
        assert_stats_close(sub[p], _oracle_chunked_stats(inp, lo, hi))

    c = _coeffs(normalize=normalize)
    st = al.autoloco_outer_step(ctx, inp.theta, inp.momentum, inp.replicas, c, al.FUSE_STATS | al.FUSE_RESET, EPS)
    torch.cuda.synchronize()
    assert bytes(st) == bytes(full)          # same partition, same bits
    _check_sampled_outputs(inp, idx, sample_in, c, replica_dtype)
    del inp
    torch.cuda.empty_cache()


def test_llama_1b1_full(ctx):
    _large(ctx, "llama-1.1b", 8, torch.float32, parts=16, oracle_parts=[5, 15], normalize=False)


def test_llama_3b_bf16_full(ctx):
    _large(ctx, "llama-3b", 8, torch.bfloat16, parts=64, oracle_parts=[17, 63], normalize=True)


def test_llama_1b1_interval_ratios(ctx):
    # the 1.1B configuration's selected/base interval ratios 0.5, 1, 1.5, 2 (H^ref = 500
    # from step 20,000): rho = 1, 1, 1.4914, 1.9771, each round on freshly drawn replicas,
    # with and without normalisation
    n, k = shapes.llama_1b1().n_params, 8
    ts, _ = al.spread_tensors(ctx, n, [torch.float32] * (k + 2))
    inp = drift.RoundInputs(ts[0], ts[1], ts[2:])
    drift.fill_theta_momentum(inp, seed=42)
    idx = _sample_index(n, m=1 << 18, seed=4)
    rhos = []
    for i, (h_sel, normalize) in enumerate([(250, False), (500, True), (750, True), (1000, False)]):
        drift.fill_replicas(inp, seed=60 + i)
        c = _coeffs(h_sel=h_sel, normalize=normalize)
        rhos.append(c.rho)
        sample_in = _gather(inp, idx)
        print(f"1.1B ratio {h_sel / 500}: rho {c.rho:.6f} normalise {normalize}", flush=True)
        st = al.autoloco_outer_step(ctx, inp.theta, inp.momentum, inp.replicas, c, al.FUSE_STATS | al.FUSE_RESET,
                                    EPS)
        torch.cuda.synchronize()
        assert st.finite and st.disagreement == pytest.approx(st.D - st.sq_mean, rel=1e-4)
        _check_sampled_outputs(inp, idx, sample_in, c, torch.float32)
    assert rhos[0] == 1.0 and rhos[1] == 1.0
    assert rhos[2] == pytest.approx(1.491439580, rel=1e-9) and rhos[3] == pytest.approx(1.977132131, rel=1e-9)
    del inp, ts
    torch.cuda.empty_cache()
