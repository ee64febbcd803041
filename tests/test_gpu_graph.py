"""The asynchronous entry points under HIP graph capture.

The workers' AdamW step (with gradient clipping, so its norm pass and the
reduction kernel run on the device), the corrected outer step with the reset
and the reset alone, captured once on the context's stream and replayed
several times, with the program's own eager work and synchronisations between
the replays, give bit for bit what the same calls give eagerly on a second set
of buffers.  (The calls that return statistics wait for them on the host and
are not captured; one of them runs between the replays.)"""
import pytest
import torch

import paper_2609_36662_amd as al
from tests.gpu_common import cpu_inputs, to_device

pytestmark = pytest.mark.gpu
EPS = 1e-12


def _same(a, b):
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_captured_steps_replay_like_eager():
    n, k = 100_003, 3
    s = torch.cuda.Stream()
    ctx = al.autoloco_create(0, s)
    try:
        inp = cpu_inputs(n, k, seed=61)
        eag, gra = to_device(inp), to_device(inp)
        gen = torch.Generator().manual_seed(7)
        grads_src = [[torch.randn(n, generator=gen) * 1e-2 for _ in range(k)] for _ in range(4)]

        def adamw_state():
            return ([torch.zeros(n, device="cuda") for _ in range(k)], [torch.zeros(n, device="cuda") for _ in range(k)],
                    [torch.empty(n, device="cuda") for _ in range(k)])

        m_e, v_e, g_e = adamw_state()
        m_g, v_g, g_g = adamw_state()
        co = al.make_adamw_coeffs(3e-4, step=5, max_grad_norm=1.0)
        c = al.make_coeffs(0.85, 0.7, 1.3, True)

        def step(bufs, m, v, g):
            al.autoloco_inner_adamw(ctx, bufs.replicas, m, v, g, co, stats=False)
            al.autoloco_outer_step(ctx, bufs.theta, bufs.momentum, bufs.replicas, c, al.FUSE_RESET, EPS)
            al.autoloco_broadcast_reset(ctx, bufs.theta, bufs.replicas)

        for t, src in zip(g_g, grads_src[0]):
            t.copy_(src)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=s, capture_error_mode="thread_local"):
            step(gra, m_g, v_g, g_g)
        torch.cuda.synchronize()
        # capture recorded the work without running it
        assert _same(gra.theta, eag.theta) and all(_same(a, b) for a, b in zip(gra.replicas, eag.replicas))

        for r in range(4):
            for a, b, src in zip(g_e, g_g, grads_src[r]):
                a.copy_(src)
                b.copy_(src)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            step(eag, m_e, v_e, g_e)
            torch.cuda.synchronize()
            for name, x, y in [("theta", gra.theta, eag.theta), ("momentum", gra.momentum, eag.momentum)] + \
                    [(f"replica {i}", x, y) for i, (x, y) in enumerate(zip(gra.replicas, eag.replicas))] + \
                    [(f"exp_avg {i}", x, y) for i, (x, y) in enumerate(zip(m_g, m_e))] + \
                    [(f"exp_avg_sq {i}", x, y) for i, (x, y) in enumerate(zip(v_g, v_e))]:
                assert _same(x, y), f"replay {r}: {name} differs from the eager run"
            # eager work between the replays: a statistics call that waits on the host
            st_g = al.autoloco_round_stats(ctx, gra.theta, gra.replicas, EPS)
            st_e = al.autoloco_round_stats(ctx, eag.theta, eag.replicas, EPS)
            assert st_g.finite and st_g.D == st_e.D == 0.0   # the reset left every replica at theta
        assert not torch.equal(gra.theta.cpu(), inp.theta)      # the replays did change the state
    finally:
        torch.cuda.synchronize()
        ctx.close()
