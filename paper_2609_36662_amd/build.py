"""Build the AutoLoCo round library (libautoloco.so) in-tree for gfx950.

The round kernels are compiled as ten slices (replica type x mode) in
parallel; the host-side scalar code (schedule, correction, controller) is
plain C++ built with g++ without floating-point contraction; hipcc links the
shared library next to this file.
"""
from __future__ import annotations

import hashlib
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libautoloco.so")
ARCH = "gfx950"

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    # no packed-fp32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{CSRC}",
]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-ffp-contract=off", "-fno-fast-math", f"-I{INCLUDE}"]


def source_files(root: str = ROOT):
    """The files the library is built from: the C++/HIP sources, the header and
    this build script (its flags shape the code)."""
    csrc = os.path.join(root, "paper_2609_36662_amd", "csrc")
    inc = os.path.join(root, "include")
    files = [os.path.join(csrc, f) for f in sorted(os.listdir(csrc)) if f.endswith((".hip", ".hpp", ".cpp"))]
    files += [os.path.join(inc, f) for f in sorted(os.listdir(inc)) if f.endswith(".h")]
    files.append(os.path.join(root, "paper_2609_36662_amd", "build.py"))
    return files


def source_hash(root: str = ROOT) -> str:
    """SHA-256 (first 16 hex digits) over the names and contents of source_files()."""
    h = hashlib.sha256()
    for path in source_files(root):
        h.update(os.path.relpath(path, root).replace(os.sep, "/").encode())
        h.update(b"\0")
        with open(path, "rb") as f:
            h.update(f.read())
        h.update(b"\0")
    return h.hexdigest()[:16]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the ROCm toolchain is required to build libautoloco.so")


def _run(cmd):
    proc = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in proc.stdout.splitlines() if "packed-fp32-ops" not in l
                    and "target feature" not in l)
    if proc.returncode != 0:
        raise RuntimeError(f"build step failed ({proc.returncode}): {' '.join(cmd)}\n{out}")
    return out


def jobs():
    hipcc = _hipcc()
    cmds = []
    for rt, rtname in ((0, "f32"), (1, "bf16")):
        for mode in range(9):
            obj = os.path.join(BUILD, f"round_{rtname}_m{mode}.o")
            cmds.append([hipcc, *HIP_FLAGS, f"-DAL_RT={rt}", f"-DAL_RTNAME={rtname}", f"-DAL_MODE={mode}",
                         "-c", os.path.join(CSRC, "round_inst.hip"), "-o", obj])
    for rt, rtname in ((0, "f32"), (1, "bf16")):
        for st in (0, 1):
            for rs in (0, 1):
                obj = os.path.join(BUILD, f"int8_{rtname}_s{st}r{rs}.o")
                cmds.append([hipcc, *HIP_FLAGS, f"-DAL_RT={rt}", f"-DAL_RTNAME={rtname}", f"-DAL_STATS={st}",
                             f"-DAL_RESET={rs}", "-c", os.path.join(CSRC, "int8_inst.hip"), "-o", obj])
    cmds.append([hipcc, *HIP_FLAGS, "-c", os.path.join(CSRC, "adamw_inst.hip"), "-o", os.path.join(BUILD, "adamw.o")])
    cmds.append([hipcc, *HIP_FLAGS, "-c", os.path.join(CSRC, "shard_inst.hip"), "-o", os.path.join(BUILD, "shard.o")])
    cmds.append([hipcc, *HIP_FLAGS, "-c", os.path.join(CSRC, "reduce_inst.hip"), "-o", os.path.join(BUILD, "reduce.o")])
    cmds.append([hipcc, *HIP_FLAGS, "-c", os.path.join(CSRC, "probe_inst.hip"), "-o", os.path.join(BUILD, "probe.o")])
    cmds.append([hipcc, *HIP_FLAGS, f'-DAUTOLOCO_BUILD_ID="{source_hash()}"', "-c", os.path.join(CSRC, "api.hip"),
                 "-o", os.path.join(BUILD, "api.o")])
    for src in ("scalar.cpp", "controller.cpp"):
        cmds.append(["g++", *CXX_FLAGS, "-c", os.path.join(CSRC, src),
                     "-o", os.path.join(BUILD, src.replace(".cpp", ".o"))])
    return hipcc, cmds


def build(verbose: bool = False) -> str:
    """Compile every source and link libautoloco.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    hipcc, cmds = jobs()
    workers = max(1, min(len(cmds), os.cpu_count() or 1, 16))
    with ThreadPoolExecutor(workers) as pool:
        for out in pool.map(_run, cmds):
            if verbose and out.strip():
                print(out)
    objs = [c[c.index("-o") + 1] for c in cmds]
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    _build_c_abi_check()
    return LIB


C_ABI_SRC = os.path.join(os.path.dirname(PKG), "tests", "c_abi", "round_from_c.c")
C_ABI_BIN = os.path.join(os.path.dirname(PKG), "tests", "c_abi", "round_from_c")


def _build_c_abi_check() -> None:
    """The plain-C program the tests use to drive a round through the C ABI
    (gcc, C11, the HIP runtime for device memory; linked against the library)."""
    if not os.path.exists(C_ABI_SRC):
        return
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    _run(["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
          f"-I{rocm}/include", f"-I{INCLUDE}", C_ABI_SRC, "-o", C_ABI_BIN, f"-L{PKG}", "-lautoloco",
          f"-L{rocm}/lib", "-lamdhip64", "-Wl,-rpath,$ORIGIN/../../paper_2609_36662_amd",
          f"-Wl,-rpath,{rocm}/lib"])


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
