"""bench.py's output contract on a small workload: one JSON line with the
metric, value, timing, configuration, roofline and CPU-baseline fields, for the
round step and the closed loop."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args):
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                       timeout=200)
    assert p.returncode == 0, p.stderr[-3000:]
    lines = [l for l in p.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, p.stdout
    return json.loads(lines[0])


def _common(d, steps, warmup):
    for key, typ in (("metric", str), ("value", float), ("unit", str), ("n_gpus", int), ("steps", int),
                     ("warmup", int), ("ms_per_step", float), ("higher_is_better", bool), ("scaling", str),
                     ("dtype", str), ("data", str), ("config", dict), ("roofline", dict)):
        assert isinstance(d[key], typ), key
    assert d["n_gpus"] == 1 and d["steps"] == steps and d["warmup"] == warmup
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["higher_is_better"] is True
    assert d["vs_baseline"] is None and d["data"] == "synthetic" and d["scaling"] == "weak"
    assert isinstance(d["config"]["workload"], str)
    r = d["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert r["achieved"] > 0 and r["frac"] == pytest.approx(r["achieved"] / r["peak"])
    assert r["traffic"] is None or r["traffic"] > 0


def test_round_line():
    d = _run(["--workload", "tiny", "--steps", "3", "--warmup", "1", "--perturbed", "2", "--cpu-seconds", "0.5",
              "--cpu-sample", str(1 << 16)])
    _common(d, 3, 1)
    assert d["unit"] == "params/s" and d["config"]["n_params"] == 1 << 20
    assert d["metric"].endswith(", 1M params K=4")
    assert d["value"] == pytest.approx(d["config"]["n_params"] / (d["ms_per_step"] * 1e-3), rel=1e-9)
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0 and cb["unit"] == "params/s"
    assert isinstance(cb["sample"], str) and d["cpu_baseline_one_thread"]["cores"] == 1
    ref = d["traffic_reference"]
    assert ref["gbs"] > 0 and ref["bytes"] == d["config"]["bytes_per_round"]
    assert d["first_round_stats"]["finite"] is True


def test_closed_loop_line():
    d = _run(["--step", "closed-loop", "--workload", "tiny", "--steps", "4", "--warmup", "1", "--no-cpu-baseline"])
    _common(d, 4, 1)
    assert len(d["rounds"]) == 5 and all(r["h_step"] > 0 for r in d["rounds"])
    assert d["metric"].endswith(", 1M params K=4, 4 rounds")
