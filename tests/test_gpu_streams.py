"""Contexts bound to their own HIP streams: asynchronous rounds on two
streams at once (each context owns its reduction scratch) give the oracle's
results, and a context's launches are ordered on its stream."""
import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al
from oracle import round as orr
from tests.gpu_common import assert_close_elementwise, assert_stats_close, cpu_inputs, host_array, to_device

pytestmark = pytest.mark.gpu
EPS = 1e-12


def test_two_streams_two_contexts():
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    c1, c2 = al.autoloco_create(0, s1), al.autoloco_create(0, s2)
    try:
        a = cpu_inputs(1_000_003, 4, seed=61)
        b = cpu_inputs(700_001, 8, seed=62)
        da, db = to_device(a), to_device(b)
        torch.cuda.synchronize()
        co = al.make_coeffs(0.85, 1.5, 1.49, True)
        for _ in range(3):   # three asynchronous rounds (update + reset) on each stream, interleaved
            al.autoloco_outer_step(c1, da.theta, da.momentum, da.replicas, co, al.FUSE_RESET, EPS)
            al.autoloco_outer_step(c2, db.theta, db.momentum, db.replicas, co, al.FUSE_RESET, EPS)
        st1 = al.autoloco_round_stats(c1, da.theta, da.replicas, EPS)   # ordered after the rounds on s1
        st2 = al.autoloco_round_stats(c2, db.theta, db.replicas, EPS)
        torch.cuda.synchronize()
        for inp, dev, st in ((a, da, st1), (b, db, st2)):
            th, v = inp.theta.numpy().astype(np.float64), inp.momentum.numpy().astype(np.float64)
            reps = [host_array(r) for r in inp.replicas]
            for _ in range(3):
                ref = orr.sync_round(th, v, reps, co.mu, co.eta_out, co.rho, True, EPS)
                th, v = ref.theta, ref.momentum
                reps = orr.reset_replicas(th, len(reps), "f32")
            assert_close_elementwise(dev.theta.cpu().numpy(), th, tol=3e-5, what="theta after 3 rounds")
            assert_close_elementwise(dev.momentum.cpu().numpy(), v, tol=3e-5, what="v after 3 rounds")
            assert st.D == 0.0 and st.C == 0.0   # after the reset every replica equals theta
            assert_stats_close(st, orr.round_stats(dev.theta.cpu().numpy(), [x.cpu().numpy() for x in dev.replicas]))
    finally:
        c1.close()
        c2.close()
