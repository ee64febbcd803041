"""CPU check of the window loops of the standalone reset and of the per-GPU
share kernels in the gfx950 assembly.

These kernels split each grid-stride loop into whole windows, which take no
per-lane bounds test, and the last, shorter window.  The point of the split
is that the loads of a window are issued without first waiting for the
previous window's stores: when the loaded values were instead kept live
across iterations under per-lane tests, the compiler put an
`s_waitcnt vmcnt(0)` in front of every load, which serialised the store and
load latencies (13 % at one replica).  This test compiles the instances the
library launches and checks, in the block that holds a whole window's loads,
that every load of the window is there and that no vector-memory wait comes
before the first of them."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_36662_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")

# (symbol, loads of one whole window): the spans the reset launcher picks
# (one window for one fp32 replica, eight from three on, two for bf16), the
# payload kernel (theta and an fp32 replica, two runs) and the shard step
# (theta and v in place plus 8 bf16 payload shards, two runs).
KERNELS = [
    ("_ZN8autoloco12reset_kernelILi1ELi0ELi1EEEvNS_9RoundArgsE", 1),
    ("_ZN8autoloco12reset_kernelILi3ELi0ELi8EEEvNS_9RoundArgsE", 8),
    ("_ZN8autoloco12reset_kernelILi8ELi0ELi8EEEvNS_9RoundArgsE", 8),
    ("_ZN8autoloco12reset_kernelILi8ELi1ELi2EEEvNS_9RoundArgsE", 2),
    ("_ZN8autoloco19rank_payload_kernelILi0EEEvNS_15RankPayloadArgsE", 4),
    ("_ZN8autoloco17shard_step_kernelILi8EEEvNS_9ShardArgsE", 2 * (2 + 8)),
]

SOURCE = """
#include "reset_kernels.hpp"
#include "shard_kernels.hpp"
namespace autoloco {
template __global__ void reset_kernel<1, RT_F32, 1>(RoundArgs);
template __global__ void reset_kernel<3, RT_F32, 8>(RoundArgs);
template __global__ void reset_kernel<8, RT_F32, 8>(RoundArgs);
template __global__ void reset_kernel<8, RT_BF16, 2>(RoundArgs);
template __global__ void rank_payload_kernel<RT_F32>(RankPayloadArgs);
template __global__ void shard_step_kernel<8>(ShardArgs);
}
"""


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    return None


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    hipcc = _hipcc()
    if hipcc is None:
        pytest.skip("hipcc not available")
    tmp = tmp_path_factory.mktemp("isa_windows")
    src = tmp / "windows.hip"
    src.write_text(SOURCE)
    out = tmp / "windows.s"
    cmd = [hipcc, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", f"-I{INCLUDE}", f"-I{CSRC}", "--cuda-device-only", "-S", str(src), "-o", str(out)]
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert p.returncode == 0, p.stdout[-3000:]
    return out.read_text()


def _blocks(text, symbol):
    start = text.index(symbol + ":")
    body = text[start:text.index("s_endpgm", start)].split("\n")
    blocks, cur = [], []
    for line in body:
        if line.startswith(".LBB") and cur:
            blocks.append(cur)
            cur = []
        cur.append(line.strip())
    blocks.append(cur)
    return blocks


@pytest.mark.parametrize("symbol,loads", KERNELS)
def test_whole_window_loads_wait_for_no_store(asm, symbol, loads):
    is_load = re.compile(r"^global_load_dword")
    blocks = _blocks(asm, symbol)
    # the whole-window path: the block with the most loads
    block = max(blocks, key=lambda b: sum(bool(is_load.match(l)) for l in b))
    n = sum(bool(is_load.match(l)) for l in block)
    assert n == loads, (symbol, n)
    first = next(i for i, l in enumerate(block) if is_load.match(l))
    waits = [l for l in block[:first] if l.startswith("s_waitcnt") and "vmcnt" in l]
    assert not waits, (symbol, waits)
