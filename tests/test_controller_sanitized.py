"""The host controller built with AddressSanitizer and UndefinedBehaviorSanitizer
(g++/gcc, host code only) and driven through the C ABI by a plain-C program
(`tests/c_abi/controller_from_c.c`) over every scripted scenario of the
controller tests, with a checkpoint save / load every seventh interval: no
sanitizer report, and every decision equal, field by field and bit for bit, to
the library's (built without sanitizers).  Crafted checkpoints with counts or
horizons out of range are refused under the same checks."""
import ctypes as C
import math
import os
import shutil
import subprocess

import pytest

import paper_2609_36662_amd as al
from paper_2609_36662_amd import _lib
from tests.controller_driver import drive
from tests.test_lib_host import CORRUPT_STATES, SCENARIOS, StateHead, _ccfg, saved_in_reference_bootstrap

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_36662_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
DRIVER = os.path.join(ROOT, "tests", "c_abi", "controller_from_c.c")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert p.returncode == 0, f"{' '.join(map(str, cmd))}\n{p.stdout}"


@pytest.fixture(scope="module")
def exe(tmp_path_factory):
    gxx, gcc = shutil.which("g++"), shutil.which("gcc")
    if gxx is None or gcc is None:
        pytest.skip("g++/gcc not available")
    tmp = tmp_path_factory.mktemp("sanitized_controller")
    objs = []
    for src in ("controller.cpp", "scalar.cpp"):
        obj = str(tmp / (src + ".o"))
        # the library's own floating-point flags, so the decisions can be compared bit for bit
        _run([gxx, "-std=c++17", "-ffp-contract=off", "-fno-fast-math", *SAN, "-I", INCLUDE, "-c",
              os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    drv = str(tmp / "driver.o")
    _run([gcc, "-std=c11", "-Wall", "-Wextra", "-Werror", *SAN, "-I", INCLUDE, "-c", DRIVER, "-o", drv])
    out = str(tmp / "controller_from_c")
    _run([gxx, *SAN, drv, *objs, "-o", out, "-lm"])
    return out


def _fields(d):
    return (d.start_step, d.h_tok, d.h_step, d.h_ref, d.lambda_sel, d.lambda_base, d.z_max, d.assessment,
            d.phase, d.done, d.coeffs.mu, d.coeffs.eta_out, d.coeffs.rho, d.coeffs.normalize)


def _same(a, b):
    return all((isinstance(x, float) and math.isnan(x) and math.isnan(y)) or x == y for x, y in zip(a, b))


@pytest.mark.parametrize("name", sorted(SCENARIOS))
def test_sanitized_controller_matches_library(exe, name):
    cfg, script = SCENARIOS[name]
    dens = (lambda t: float(1 << 20) * (1.0 if t < 25 else 0.8)) if name == "mixed" else None
    _, obs = drive(cfg, script, density=dens)
    ccfg = _ccfg(cfg)
    cobs = [al.make_observation(o.D, o.C, o.lambda_done, o.tokens, o.h_step_done, o.finite) for o in obs]
    ctl = al.autoloco_controller_create(ccfg)
    ref = [_fields(al.autoloco_select_interval(ctl, None))]
    ref += [_fields(al.autoloco_select_interval(ctl, o)) for o in cobs]

    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    p = subprocess.run([exe], input=bytes(ccfg) + b"".join(bytes(o) for o in cobs), capture_output=True,
                       env=env, timeout=120)
    err = p.stderr.decode(errors="replace")
    assert p.returncode == 0, err[-3000:]
    assert "runtime error" not in err and "Sanitizer" not in err, err[-3000:]
    size = C.sizeof(_lib.Decision)
    assert len(p.stdout) == size * len(ref)
    got = [_fields(_lib.Decision.from_buffer_copy(p.stdout[i:i + size])) for i in range(0, len(p.stdout), size)]
    bad = [i for i, (g, r) in enumerate(zip(got, ref)) if not _same(g, r)]
    assert not bad, f"decisions differ from interval {bad[0]}: {got[bad[0]]} vs {ref[bad[0]]}"


@pytest.mark.parametrize("name", sorted(CORRUPT_STATES) + ["good"])
def test_sanitized_checkpoint_load(exe, name):
    # crafted checkpoints are refused before any field indexes an array; the
    # good one loads and takes its next decision, with no sanitizer report
    blob = saved_in_reference_bootstrap()
    if name != "good":
        field, value = CORRUPT_STATES[name]
        setattr(StateHead.from_buffer(blob), field, value)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    p = subprocess.run([exe, "load"], input=bytes(blob), capture_output=True, env=env, timeout=120)
    err = p.stderr.decode(errors="replace")
    assert p.returncode == 0, err[-3000:]
    assert "runtime error" not in err and "Sanitizer" not in err, err[-3000:]
    status = int.from_bytes(p.stdout[:4], "little", signed=True)
    if name == "good":
        assert status == 0 and int.from_bytes(p.stdout[4:8], "little", signed=True) == 0
        d = _lib.Decision.from_buffer_copy(p.stdout[8:8 + C.sizeof(_lib.Decision)])
        assert d.phase == 3
    else:
        assert status == -1 and len(p.stdout) == 4
