"""CPU check of the INT8 round's LDS prefetch in the gfx950 assembly.

With fp32 replicas and up to 8 workers, the next codec block's theta and
replica vectors stream into LDS through direct global-to-LDS loads, and the
loop waits for them with an explicit `s_waitcnt vmcnt(N)` at the start of the
next iteration, N being the number of stores the kernel issues after those
loads.  That wait is only sufficient if at least N vector memory instructions
really lie between the last direct load and the wait on the path round the
loop, and if it comes before the LDS reads.  The compiler's wait insertion
does not order these loads against later LDS reads by itself, so this test
compiles every (statistics, reset) variant for gfx950 and checks the loop the
compiler actually emitted, for every worker count that uses the prefetch."""
import os
import re
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_36662_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
VARIANTS = [(st, rs) for st in (0, 1) for rs in (0, 1)]


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
    tmp = tmp_path_factory.mktemp("isa")

    def one(v):
        st, rs = v
        out = str(tmp / f"int8_s{st}r{rs}.s")
        cmd = [hipcc, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
               "-packed-fp32-ops", f"-I{INCLUDE}", f"-I{CSRC}", "-DAL_RT=0", "-DAL_RTNAME=f32", f"-DAL_STATS={st}",
               f"-DAL_RESET={rs}", "--cuda-device-only", "-S", os.path.join(CSRC, "int8_inst.hip"), "-o", out]
        p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
        assert p.returncode == 0, p.stdout[-3000:]
        with open(out) as f:
            return v, f.read()

    with ThreadPoolExecutor(len(VARIANTS)) as pool:
        return dict(pool.map(one, VARIANTS))


def _loop(text, k, st, rs):
    name = f"_ZN8autoloco17int8_round_kernelILi{k}ELi0ELb{st}ELb{rs}EEEvNS_8Int8ArgsE"
    start = text.index(name + ":")
    return text[start:text.index("s_endpgm", start)].split("\n")


@pytest.mark.parametrize("st,rs", VARIANTS)
def test_prefetch_wait_covers_the_direct_loads(asm, st, rs):
    text = asm[(st, rs)]
    for k in range(1, 9):
        body = _loop(text, k, st, rs)
        heads = [i for i, l in enumerate(body) if l.startswith(".LBB") and "Inner Loop Header" in l]
        assert len(heads) == 1, (k, "expected one loop")
        h = heads[0]
        # in the loop, the wait for the prefetch comes before any LDS read or direct load
        first_wait = next(i for i in range(h, len(body)) if "s_waitcnt vmcnt(" in body[i])
        first_lds = next(i for i in range(h, len(body)) if "ds_read" in body[i] or "global_load_lds" in body[i])
        assert first_wait < first_lds, (k, "LDS used before the wait")
        n = int(re.search(r"vmcnt\((\d+)\)", body[first_wait]).group(1))
        assert n == 2 * (2 + (k if rs else 0)), (k, n)
        # the direct loads of the next block are issued inside the loop, after the LDS reads
        dma = [i for i in range(h, len(body)) if "global_load_lds" in body[i]]
        assert len([i for i in dma if i < h + 1000]) >= 2 * (k + 1), (k, "direct loads missing")
        head = body[h].split(":")[0]
        to_head = [i for i, l in enumerate(body) if re.search(r"\bs_(c)?branch\w*\s+" + re.escape(head) + r"\s*$", l)]
        latch = [i for i in to_head if i > h]
        last_dma = max(i for i in dma if i < h + 1000)
        if latch:
            # the loop is laid out in order: one branch back to the header ends the
            # iteration, and the block that ends with it (from the last label before
            # it, which every path of the iteration reaches) holds at least n stores
            # after the last direct load
            assert len(latch) == 1, (k, "several back edges")
            tail = max(i for i in range(latch[0]) if re.match(r"^\.LBB\d+_\d+:", body[i]))
            assert tail > last_dma, (k, "direct loads after the last join of the iteration")
            stores = sum(1 for l in body[tail:latch[0]] if re.search(r"\bglobal_store", l))
            assert stores >= n, (k, stores, n)
            close = latch[0]
        else:
            # the loop is rotated: the block that falls into the header ends the
            # iteration; every branch back into the loop goes there, and it holds at
            # least n stores
            tail = max(i for i in range(h) if re.match(r"^\.LBB\d+_\d+:", body[i]))
            label = body[tail].split(":")[0]
            back = [i for i, l in enumerate(body) if re.search(r"\bs_(c)?branch\w*\s+" + re.escape(label) + r"\s*$", l)]
            assert back and all(i > h for i in back), (k, "unexpected loop shape")
            stores = sum(1 for l in body[tail:h] if re.search(r"\bglobal_store", l))
            assert stores >= n, (k, stores, n)
            # nothing on the back-edge path between the last direct load and the header may
            # skip the tail: the header is entered from the tail (fall through) or from before
            # the loop
            assert all(i < tail for i in to_head), (k, "header reached around the tail")
            close = max(back)
        # before the loop: the first block's direct loads are followed by a full wait
        start = h if latch else tail
        pro = [i for i in range(start) if "global_load_lds" in body[i]]
        assert pro, (k, "no prologue prefetch")
        assert any("s_waitcnt vmcnt(0)" in body[i] for i in range(pro[-1], start)), (k, "prologue not drained")
        # after the loop (the code after its last branch back into it): a full wait
        # comes before any LDS instruction and before the end of the program
        rest = body[close + 1:]
        w = next((i for i, l in enumerate(rest) if "s_waitcnt vmcnt(0)" in l), None)
        assert w is not None, (k, "no full wait after the loop")
        assert not any(re.search(r"\bds_|s_endpgm", l) for l in rest[:w]), (k, "LDS used before the final wait")
