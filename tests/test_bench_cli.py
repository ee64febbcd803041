"""bench.py's command line on the CPU: more than one GPU is refused with a
message and exit status 2, before anything touches a device."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    for n in (2, 8):
        p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                           capture_output=True, text=True, timeout=120)
        assert p.returncode == 2
        assert "one GPU" in p.stderr and p.stdout == ""


def test_help_lists_the_modes():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--help"], capture_output=True, text=True,
                       timeout=120)
    assert p.returncode == 0
    for word in ("--codec", "--step", "--workload", "--steps", "--warmup", "closed-loop", "inner", "share"):
        assert word in p.stdout


def test_metric_names_the_workload_it_measured():
    import types
    sys.path.insert(0, ROOT)
    import bench
    a = types.SimpleNamespace(workload="llama-1.1b", steps=20)
    assert bench.metric_name(bench.METRIC, a, 8) == bench.METRIC
    assert bench.metric_name(bench.METRIC, a, 4).endswith(", 1.1B params K=4")
    a = types.SimpleNamespace(workload="tiny", steps=5)
    assert bench.metric_name(bench.METRIC, a, 4).endswith("(% of peak), 1M params K=4")
    assert bench.metric_name(bench.CLOSED_LOOP_METRIC, a, 4, True).endswith("(% of peak), 1M params K=4, 5 rounds")
    a = types.SimpleNamespace(workload="llama-7b", steps=20)
    assert bench.metric_name(bench.CLOSED_LOOP_METRIC, a, 4, True) == bench.CLOSED_LOOP_METRIC


def test_streamed_cpu_baseline_equals_one_oracle_pass():
    # the CPU baseline's chunked, multi-process oracle pass over a workload gives
    # the statistics of one oracle pass over all of it (float64, chunk order)
    import numpy as np
    import torch
    sys.path.insert(0, ROOT)
    import bench
    import paper_2609_36662_amd as al
    from oracle import round as orr
    from workloads import drift
    old = bench.CPU_CHUNK
    bench.CPU_CHUNK = 1 << 14
    try:
        for rdt, dt in (("f32", torch.float32), ("bf16", torch.bfloat16)):
            n, k = 3 * (1 << 14) + 13, 4
            pool = bench.make_cpu_pool(n, k, rdt, 2)
            try:
                inp = drift.make_round_inputs(n, k, seed=5, device="cpu", replica_dtype=dt)
                coeffs = al.make_coeffs(0.85, 1.5, 1.49, True)
                par, one, st = bench.cpu_baseline_stream(inp, coeffs, rdt, "check", pool, 2)
                par2, none, st2 = bench.cpu_baseline_stream(inp, coeffs, rdt, "check", pool, 2, one_core=False)
            finally:
                bench.close_cpu_pool(pool)
            reps = [r.numpy() if rdt == "f32" else r.view(torch.int16).numpy().view(np.uint16) for r in inp.replicas]
            ref = orr.sync_round(inp.theta.numpy(), inp.momentum.numpy(), reps, 0.85, 1.5, 1.49, True, 1e-12)
            for a, b in ((st.D, ref.stats.D), (st.C, ref.stats.C), (st.disagreement, ref.stats.disagreement)):
                assert abs(a - b) <= 1e-12 * abs(b)
            assert par["cores"] == 2 and one["cores"] == 1 and "4 chunks" in par["sample"]
            assert none is None and par2["cores"] == 2 and (st2.D, st2.C) == (st.D, st.C)
    finally:
        bench.CPU_CHUNK = old


def test_streamed_inner_cpu_baseline_gives_the_oracle_norms():
    # the inner step's chunked, multi-process oracle pass computes each worker's
    # gradient norm over the whole gradient (float64, chunk order)
    import math
    sys.path.insert(0, ROOT)
    import bench
    from oracle import adamw as oa
    from workloads import inner
    old = bench.CPU_CHUNK
    bench.CPU_CHUNK = 1 << 14
    try:
        n, k = 2 * (1 << 14) + 21, 3
        st = inner.make_state(n, k, seed=9)
        pool = bench.make_inner_pool(n, 2)
        try:
            leg, norms = bench.inner_cpu_baseline_stream(st, 3e-4, 5, "check", pool, 2)
        finally:
            bench.close_cpu_pool(pool)
        for w in range(k):
            ref = oa.grad_norm(st.grads[w].numpy())
            assert math.isclose(norms[w], ref, rel_tol=1e-12)
        assert leg["cores"] == 2 and "3 chunks" in leg["sample"] and leg["value"] > 0
    finally:
        bench.CPU_CHUNK = old
