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
