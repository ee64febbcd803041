"""The synthetic workloads (CPU): model shapes against the closed-form
parameter counts of their architectures, the 16-byte alignment of every
tensor view, and the seeded generators' determinism and scales."""
import math

import pytest
import torch

from workloads import drift, inner, shapes


def _llama_count(layers, d, ffn, vocab, kv):
    per_layer = 2 * d * d + 2 * kv * d + 3 * d * ffn + 2 * d   # q, o; k, v; gate, up, down; two norms
    return 2 * vocab * d + layers * per_layer + d               # embedding, untied head, final norm


@pytest.mark.parametrize("name,count,tensors", [
    ("gpt2-small", 50257 * 768 + 1024 * 768 + 12 * (12 * 768 * 768 + 13 * 768) + 2 * 768, 148),
    ("llama-1.1b", _llama_count(22, 2048, 5632, 32000, 256), 201),
    ("llama-3b", _llama_count(26, 3072, 8192, 32000, 3072), 237),
    ("llama-7b", _llama_count(32, 4096, 11008, 32000, 4096), 291),
])
def test_shape_counts(name, count, tensors):
    s = shapes.SHAPES[name]()
    assert s.n_params == count and s.n_tensors == tensors
    assert all(off % 4 == 0 and size % 4 == 0 for _, off, size in s.offsets())


def test_published_totals():
    # GPT-2 small with tied head, TinyLlama-style 1.1B, Llama-2-style 7B
    assert shapes.SHAPES["gpt2-small"]().n_params == 124_439_808
    assert shapes.SHAPES["llama-1.1b"]().n_params == 1_100_048_384
    assert shapes.SHAPES["llama-7b"]().n_params == 6_738_415_616
    assert shapes.SHAPES["llama-3b"]().n_params == 3_141_172_224


def test_drift_inputs_are_seeded_and_scaled():
    a = drift.make_round_inputs(50_000, 3, seed=5)
    b = drift.make_round_inputs(50_000, 3, seed=5)
    c = drift.make_round_inputs(50_000, 3, seed=6)
    assert torch.equal(a.theta, b.theta) and all(torch.equal(x, y) for x, y in zip(a.replicas, b.replicas))
    assert not torch.equal(a.theta, c.theta)
    assert float(a.theta.std()) == pytest.approx(0.02, rel=0.03)
    assert float(a.momentum.std()) == pytest.approx(1e-4, rel=0.03)
    # theta_k - theta = 0.7 s + 0.3 e_k with s, e_k of std 1e-3
    d = [(r - a.theta).double() for r in a.replicas]
    assert float(d[0].std()) == pytest.approx(1e-3 * math.hypot(0.7, 0.3), rel=0.05)
    shared = float(((d[0] - d[0].mean()) * (d[1] - d[1].mean())).mean())
    assert shared == pytest.approx((0.7e-3) ** 2, rel=0.1)


def test_inner_state_norms_straddle_the_clip():
    st = inner.make_state(200_000, 4, seed=3)
    norms = [float(torch.linalg.vector_norm(g.double())) for g in st.grads]
    for got, want in zip(norms, inner.InnerRecipe().norms):
        assert got == pytest.approx(want, rel=0.02)
    assert min(norms) < 1.0 < max(norms)
    assert all(float(v.min()) >= 0.0 for v in st.exp_avg_sq)
    st2 = inner.make_state(200_000, 4, seed=3)
    assert all(torch.equal(x, y) for x, y in zip(st.grads, st2.grads))
    inner.fill_grads(st2, seed=3, step=1)
    assert not torch.equal(st.grads[0], st2.grads[0])
