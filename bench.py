#!/usr/bin/env python3
"""Benchmark of one fused AutoLoCo synchronisation round on one MI355X.

A step is one whole round through the C ABI: autoloco_outer_step with fused
statistics and replica reset (pseudo-gradients, their mean, D/C diagnostics,
corrected Nesterov step, reset of every replica), including the copy of the
2K+1 sums to the host.  The default workload is the 1.1B-parameter
Llama-style model (22 layers, d=2048, FFN 5632, vocab 32000, 4 KV heads) with
K=8 fp32 replicas, inputs resident in HBM.  Prints one JSON line.

    python bench.py [--steps 20] [--warmup 3] [--workload llama-1.1b]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "sync-round params/s and achieved HBM GB/s (% of peak), 1.1B params K=8"
PEAK_HBM_GBS = 8000.0
PROFILE_DIR = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2609_36662_amd", "csrc")
KERNEL_SOURCES = [os.path.join(CSRC, f) for f in ("round_kernels.hpp", "reduce.hpp", "round_inst.hip")]
INT8_SOURCES = KERNEL_SOURCES + [os.path.join(CSRC, f) for f in ("int8_kernels.hpp", "int8_inst.hip")]
ADAMW_SOURCES = [os.path.join(CSRC, f) for f in ("adamw_kernels.hpp", "adamw_inst.hip", "round_kernels.hpp",
                                                  "reduce.hpp")]
INNER_METRIC = "inner AdamW step worker-params/s and achieved HBM GB/s (% of peak), 1.1B params K=8"

# name -> (shape, K, replica dtype, recipe, selected horizon, base horizon)
WORKLOADS = {
    "llama-1.1b": ("llama-1.1b", 8, "f32", "mixed", 750, 500),
    "gpt2-small": ("gpt2-small", 8, "f32", "spread1e-3", 750, 500),
    "llama-3b-bf16": ("llama-3b", 8, "bf16", "mixed", 750, 500),
    "llama-7b": ("llama-7b", 4, "f32", "mixed", 750, 500),
    "tiny": (None, 4, "f32", "mixed", 75, 50),
}


_LABEL = {"llama-1.1b": "1.1B params", "gpt2-small": "124M params (GPT-2 small)", "llama-3b-bf16": "3B params",
          "llama-7b": "7B params", "tiny": "1M params"}


def metric_name(base: str, args, k: int, steps_tail: bool = False) -> str:
    """The metric string: `base` names its headline workload after the last
    comma; another workload or K replaces that part with its own."""
    head, _, tail = base.rpartition(", ")
    own = f"{_LABEL[args.workload]} K={k}" + (f", {args.steps} rounds" if steps_tail else "")
    if steps_tail:
        head, _, mid = head.rpartition(", ")
        tail = f"{mid}, {tail}"
    return base if tail == own else f"{head}, {own}"


def alloc_label(alloc: str, spread: bool) -> str:
    """How the streamed buffers were placed."""
    if alloc != "spread":
        return "torch"
    return "spread" if spread else "spread requested, plain (too little free memory)"


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash(sources=None) -> str:
    h = hashlib.sha256()
    for p in sources or KERNEL_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def committed_traffic(tag: str, sources=None):
    """HBM bytes per launch from the committed rocprofv3 counter summary of this
    kernel, if it was taken on the current kernel source; else None."""
    path = os.path.join(PROFILE_DIR, f"{tag}_traffic.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_source_sha256_16") != kernel_source_hash(sources):
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


CPU_CHUNK = 1 << 24          # parameters per device-to-host chunk of the CPU baseline

# A worker process's view of the shared chunk buffers: (theta, v, replicas, rdt).
_SHARED = None


def _attach(names, n, k, rdt):
    """Worker initialiser: map the shared chunk buffers (numpy views)."""
    import numpy as np
    from multiprocessing import shared_memory
    global _SHARED
    shms = [shared_memory.SharedMemory(name=x) for x in names]
    rt = np.float32 if rdt == "f32" else np.uint16
    arr = [np.ndarray((n,), dtype=np.float32, buffer=shms[0].buf), np.ndarray((n,), dtype=np.float32, buffer=shms[1].buf)]
    arr += [np.ndarray((n,), dtype=rt, buffer=m.buf) for m in shms[2:2 + k]]
    _SHARED = (arr[0], arr[1], arr[2:], rdt, shms)


def _oracle_part(job):
    """The oracle's round (statistics, corrected step, reset) on [lo, hi) of the
    shared chunk; returns the chunk part's sums."""
    from oracle import round as orr
    lo, hi, mu, eta, rho, normalize = job
    th, mom, reps, rdt, _ = _SHARED
    res = orr.sync_round(th[lo:hi], mom[lo:hi], [r[lo:hi] for r in reps], mu, eta, rho, normalize, 1e-12)
    orr.reset_replicas(res.theta, len(reps), rdt)
    return list(res.stats.sq_norm), list(res.stats.sq_dev), res.stats.sq_mean


def cpu_procs(requested: int = 0) -> int:
    """Worker processes of the CPU baseline: the cores this process may use
    (sched_getaffinity), at most 16, the host share of one GPU on the
    machines this runs on; `requested` > 0 overrides it."""
    try:
        p = len(os.sched_getaffinity(0))
    except AttributeError:
        p = os.cpu_count() or 1
    return max(1, requested if requested > 0 else min(16, p))


def make_cpu_pool(n, k, rdt, procs):
    """Shared chunk buffers and a pool of worker processes started fresh
    (spawn), before this process touches the GPU; returns (pool, buffers)."""
    import multiprocessing as mp
    from multiprocessing import shared_memory
    c = min(n, CPU_CHUNK)
    rb = 4 if rdt == "f32" else 2
    shms = [shared_memory.SharedMemory(create=True, size=c * 4) for _ in range(2)]
    shms += [shared_memory.SharedMemory(create=True, size=c * rb) for _ in range(k)]
    names = [m.name for m in shms]
    pool = mp.get_context("spawn").Pool(procs, initializer=_attach, initargs=(names, c, k, rdt)) if procs > 1 else None
    _attach(names, c, k, rdt)                   # this process's own view (the one-core leg)
    return pool, shms


def close_cpu_pool(pool_shms) -> None:
    """Stop the worker processes and release the shared chunk buffers."""
    if pool_shms is None:
        return
    pool, shms = pool_shms
    if pool is not None:
        pool.close()
        pool.join()
    for shm in shms:
        shm.close()
        shm.unlink()


def cpu_baseline_stream(inp, coeffs, rdt, desc, pool_shms, procs, one_core=True):
    """The float64 oracle, as it stands, over the whole workload.  The inputs
    move device-to-host in chunks of 2^24 parameters into shared memory (not
    timed); on each chunk the oracle runs once in this process (one core, when
    `one_core` is set or there is no pool) and once split over `procs` worker
    processes, and only that compute is timed.  The chunk sums are added in
    chunk order.  Returns the two legs (the one-core leg None when skipped) and
    the oracle's statistics of the whole workload."""
    import numpy as np
    import torch
    from oracle import round as orr
    pool, _ = pool_shms
    th_s, mom_s, reps_s, _, _ = _SHARED
    n, k = inp.theta.numel(), len(inp.replicas)
    mu, eta, rho, nz = coeffs.mu, coeffs.eta_out, coeffs.rho, bool(coeffs.normalize)
    s_tot, q_tot, m_tot = [0.0] * k, [0.0] * k, 0.0
    t_one = t_par = 0.0
    for c0 in range(0, n, CPU_CHUNK):
        c1 = min(n, c0 + CPU_CHUNK)
        m = c1 - c0
        th_s[:m] = inp.theta[c0:c1].cpu().numpy()
        mom_s[:m] = inp.momentum[c0:c1].cpu().numpy()
        for dst, src in zip(reps_s, inp.replicas):
            x = src[c0:c1].cpu()
            dst[:m] = x.numpy() if rdt == "f32" else x.view(torch.int16).numpy().view(np.uint16)
        if one_core or pool is None:
            t0 = time.perf_counter()
            one = _oracle_part((0, m, mu, eta, rho, nz))
            t_one += time.perf_counter() - t0
        step = -(-m // procs)
        jobs = [(lo, min(m, lo + step), mu, eta, rho, nz) for lo in range(0, m, step)]
        t0 = time.perf_counter()
        parts = pool.map(_oracle_part, jobs) if pool is not None else [one]
        t_par += time.perf_counter() - t0
        for sn, sd, sm in parts:                # worker order within the chunk
            s_tot = [a + b for a, b in zip(s_tot, sn)]
            q_tot = [a + b for a, b in zip(q_tot, sd)]
            m_tot += sm
        if (c0 // CPU_CHUNK) % 64 == 63:
            log(f"oracle: {c1:,} of {n:,} parameters, {t_par:.1f} s of oracle time so far")
    stats = orr.finish_stats(s_tot, q_tot, m_tot, 1e-12)
    nchunks = -(-n // CPU_CHUNK)
    what = (f"{desc}: the whole workload, {n:,} parameters of every buffer, streamed device-to-host in "
            f"{nchunks} chunks of up to {CPU_CHUNK:,} (transfer not timed); numpy float64 oracle")
    par = {"value": n / t_par, "unit": "params/s", "cores": procs, "kind": "oracle",
           "sample": what + (f", each chunk split over {procs} worker processes" if procs > 1 else ", one process"),
           "seconds": t_par}
    one_leg = {"value": n / t_one, "unit": "params/s", "cores": 1, "kind": "oracle",
               "sample": what + ", one process on one core", "seconds": t_one} \
        if one_core or pool is None else None
    return par, one_leg, stats


def cpu_model() -> str:
    """Model name of the host CPU with its family, model and stepping numbers
    (Linux /proc/cpuinfo, first processor), or "unknown"."""
    fields = {}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if not line.strip():
                    break                      # first processor only
                key, _, val = line.partition(":")
                fields[key.strip()] = val.strip()
    except OSError:
        return "unknown"
    name = fields.get("model name", "unknown")
    ids = [f"{k} {fields[k]}" for k in ("cpu family", "model", "stepping") if k in fields]
    return f"{name} ({', '.join(ids)})" if ids else name


def host_threads() -> int:
    """Host cores this process may use, capped at a one-GPU share of 16."""
    try:
        p = len(os.sched_getaffinity(0))
    except AttributeError:
        p = os.cpu_count() or 1
    return max(1, min(16, p))


def copy_ceiling(torch, dev) -> float:
    """GB/s of a 4 GiB device-to-device copy (median of five after one warm-up);
    also the calibration kernel of the HBM byte counters."""
    nbytes = 4 << 30
    src = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    times = []
    for _ in range(6):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        e1.synchronize()
        times.append(e0.elapsed_time(e1))
    del src, dst
    gbs = 2 * nbytes / (statistics.median(times[1:]) * 1e-3) / 1e9
    log(f"device-to-device copy of 4 GiB: {gbs:.0f} GB/s")
    return gbs


def inner_cpu_baseline(sample, lr, step, seconds: float, desc: str, threads: int = 1):
    """The float64 oracle's inner step on a bounded sample: every worker's first
    parameters, one worker per task (on a pool of threads when threads > 1)."""
    from concurrent.futures import ThreadPoolExecutor
    from oracle import adamw as oa
    params, m, v, g = sample
    n, k = params[0].shape[0], len(params)
    cfg = oa.AdamWConfig()

    def worker(i):
        return oa.inner_step([params[i]], [m[i]], [v[i]], [g[i]], lr, step, cfg)

    pool = ThreadPoolExecutor(threads) if threads > 1 else None
    try:
        done = 0
        t0 = time.perf_counter()
        while True:
            if pool is not None:
                list(pool.map(worker, range(k)))
            else:
                for i in range(k):
                    worker(i)
            done += n * k
            if time.perf_counter() - t0 >= seconds:
                break
        dt = time.perf_counter() - t0
    finally:
        if pool is not None:
            pool.shutdown()
    how = "one thread" if threads == 1 else f"one worker per task on {threads} threads"
    return {"value": done / dt, "unit": "worker-params/s", "cores": threads, "kind": "oracle",
            "sample": f"{desc}: first {n:,} parameters of each of {k} workers (clipping on the sample's own "
                      f"norm), step repeated {done // (n * k)}x over {dt:.1f} s (numpy float64, {how})"}


# A worker process's view of the inner step's shared chunk buffers: (theta, m, v, g).
_INNER = None


def _attach_inner(names, c):
    """Worker initialiser: map the inner step's shared chunk buffers (numpy views)."""
    import numpy as np
    from multiprocessing import shared_memory
    global _INNER
    shms = [shared_memory.SharedMemory(name=x) for x in names]
    _INNER = [np.ndarray((c,), dtype=np.float32, buffer=m.buf) for m in shms] + [shms]


def _inner_norm_part(job):
    """The oracle's gradient norm of [lo, hi) of the shared chunk, squared."""
    from oracle import adamw as oa
    lo, hi = job
    return oa.grad_norm(_INNER[3][lo:hi]) ** 2


def _inner_update_part(job):
    """The oracle's AdamW step on [lo, hi) of the shared chunk (results dropped)."""
    from oracle import adamw as oa
    lo, hi, lr, step, coef = job
    th, m, v, g = _INNER[:4]
    oa.adamw_step(th[lo:hi], m[lo:hi], v[lo:hi], g[lo:hi], lr, step, oa.AdamWConfig(), coef)
    return None


def make_inner_pool(n, procs):
    """Shared chunk buffers (theta, m, v, g) and a pool of worker processes started
    fresh (spawn), before this process touches the GPU; returns (pool, buffers)."""
    import multiprocessing as mp
    from multiprocessing import shared_memory
    c = min(n, CPU_CHUNK)
    shms = [shared_memory.SharedMemory(create=True, size=c * 4) for _ in range(4)]
    names = [m.name for m in shms]
    pool = mp.get_context("spawn").Pool(procs, initializer=_attach_inner, initargs=(names, c))
    _attach_inner(names, c)
    return pool, shms


def inner_cpu_baseline_stream(st, lr, step, desc, pool_shms, procs):
    """The float64 oracle's inner step, as it stands, over the whole workload:
    for each worker, its gradient's norm (chunk by chunk, the parts' squares
    added in chunk order) and clipping factor, then its AdamW step.  The buffers
    move device-to-host in chunks of 2^24 parameters into shared memory (not
    timed); each chunk's oracle work is split over `procs` worker processes, and
    only that compute is timed.  Returns the leg and the oracle's norms."""
    import math
    from oracle import adamw as oa
    pool, _ = pool_shms
    th_s, m_s, v_s, g_s = _INNER[:4]
    n, k = st.params[0].numel(), len(st.params)
    cfg = oa.AdamWConfig()
    t_par, norms, done = 0.0, [], 0

    def jobs(m):
        step_ = -(-m // procs)
        return [(lo, min(m, lo + step_)) for lo in range(0, m, step_)]

    for w in range(k):
        sq = 0.0
        for c0 in range(0, n, CPU_CHUNK):
            c1 = min(n, c0 + CPU_CHUNK)
            g_s[:c1 - c0] = st.grads[w][c0:c1].cpu().numpy()
            t0 = time.perf_counter()
            parts = pool.map(_inner_norm_part, jobs(c1 - c0))
            t_par += time.perf_counter() - t0
            for x in parts:
                sq += x
        norm = math.sqrt(sq)
        coef = oa.clip_coefficient(norm, cfg.max_grad_norm)
        norms.append(norm)
        for c0 in range(0, n, CPU_CHUNK):
            c1 = min(n, c0 + CPU_CHUNK)
            for dst, src in ((th_s, st.params[w]), (m_s, st.exp_avg[w]), (v_s, st.exp_avg_sq[w]), (g_s, st.grads[w])):
                dst[:c1 - c0] = src[c0:c1].cpu().numpy()
            t0 = time.perf_counter()
            pool.map(_inner_update_part, [(lo, hi, lr, step, coef) for lo, hi in jobs(c1 - c0)])
            t_par += time.perf_counter() - t0
        done += n
        log(f"oracle: worker {w + 1} of {k} done, {t_par:.1f} s of oracle time so far")
    nchunks = -(-n // CPU_CHUNK)
    leg = {"value": n * k / t_par, "unit": "worker-params/s", "cores": procs, "kind": "oracle",
           "sample": f"{desc}: the whole workload, {n:,} parameters of each of {k} workers, streamed "
                     f"device-to-host in {nchunks} chunks of up to {CPU_CHUNK:,} per buffer (transfer not timed); "
                     f"numpy float64 oracle (gradient norm, clipping, AdamW step), each chunk split over "
                     f"{procs} worker processes", "seconds": t_par}
    return leg, norms


def bench_inner(args) -> int:
    """One AdamW step of every worker (gradient-norm pass + update pass) per timed step."""
    import torch
    import paper_2609_36662_amd as al
    from workloads import inner, shapes

    shape_name, k = WORKLOADS[args.workload][0], WORKLOADS[args.workload][1]
    if args.k:
        k = args.k
    n = (1 << 20) if shape_name is None else shapes.SHAPES[shape_name]().n_params
    update_bytes = n * k * (28 + (2 if args.copy else 0))
    norm_bytes = n * k * 4
    # the CPU baseline's worker processes start before this process touches the GPU
    pool = procs = None
    if not args.no_cpu_baseline:
        procs = cpu_procs(args.cpu_procs)
        pool = make_inner_pool(n, procs)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sched = al.make_schedule()
    s0 = 20_000
    log(f"inner step {args.workload}: n={n:,} K={k} update bytes={update_bytes / 1e9:.3f} GB "
        f"norm bytes={norm_bytes / 1e9:.3f} GB")
    ctx = al.autoloco_create(0)
    t = time.perf_counter()
    dtypes = [torch.float32] * (4 * k) + ([torch.bfloat16] * k if args.copy else [])
    spread = False
    if args.alloc == "spread":
        ts, spread = al.spread_tensors(ctx, n, dtypes)
    else:
        ts = [torch.empty(n, dtype=d, device=dev) for d in dtypes]
    st = inner.InnerState(ts[0:k], ts[k:2 * k], ts[2 * k:3 * k], ts[3 * k:4 * k])
    copies = ts[4 * k:5 * k] if args.copy else None
    inner.fill_state(st, seed=42)
    inner.fill_grads(st, seed=42, step=0)
    torch.cuda.synchronize()
    log(f"buffers ({args.alloc}{', spread' if spread else ''}) allocated and filled in "
        f"{time.perf_counter() - t:.1f} s")

    sample = None
    if not args.no_cpu_baseline:
        s = min(n, args.cpu_sample // 4)
        sample = tuple([t_[:s].cpu().numpy().astype("float64") for t_ in grp]
                       for grp in (st.params, st.exp_avg, st.exp_avg_sq, st.grads))

    if args.grid:
        al.autoloco_set_grid_limit(ctx, args.grid)
    al.autoloco_set_timing(ctx, True)
    step_no = [1000]

    def one_step():
        lr = al.autoloco_inner_lr(sched, s0 + step_no[0])
        co = al.make_adamw_coeffs(lr, step_no[0])
        out = al.autoloco_inner_adamw(ctx, st.params, st.exp_avg, st.exp_avg_sq, st.grads, co, model_bf16=copies)
        step_no[0] += 1
        return out, al.autoloco_last_adamw_ms(ctx)

    first = None
    for i in range(args.warmup):
        out, _ = one_step()
        if i == 0:
            first = out
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")
    norm_ms, upd_ms = [], []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        _, (a, b) = one_step()
        norm_ms.append(a)
        upd_ms.append(b)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall / args.steps * 1e3
    upd_mean, norm_mean = statistics.mean(upd_ms), statistics.mean(norm_ms)
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step wall; update pass {upd_mean:.3f} ms "
        f"({update_bytes / upd_mean / 1e6:.0f} GB/s), norm pass {norm_mean:.3f} ms "
        f"({norm_bytes / norm_mean / 1e6:.0f} GB/s)")
    ceiling = None if args.no_ceiling else copy_ceiling(torch, dev)
    achieved = update_bytes / (upd_mean * 1e-3) / 1e9

    # The update pass's loads and stores without its arithmetic, on the same
    # buffers and grid; and the norm pass's pattern (K streams read) from the
    # streaming probe at one, two and three workgroups per compute unit.
    reference = None
    if not args.no_ceiling:
        ref_ms = []
        for _ in range(10):
            al.autoloco_adamw_traffic_reference(ctx, st.params, st.exp_avg, st.exp_avg_sq, st.grads,
                                                model_bf16=copies)
            ref_ms.append(al.autoloco_last_kernel_ms(ctx))
        ref_med = statistics.median(ref_ms)
        reference = {"kernel": "adamw_kernel traffic reference (the update pass's loads and stores, no arithmetic)",
                     "kernel_ms_median": ref_med, "gbs": update_bytes / (ref_med * 1e-3) / 1e9,
                     "update_frac_of_reference": ref_med / upd_mean}
        log(f"update pass traffic reference: {ref_med:.3f} ms ({update_bytes / ref_med / 1e6:.0f} GB/s); the "
            f"update runs at {100 * ref_med / upd_mean:.1f} % of it")
        if k in (1, 2, 4, 8, 10):
            cus = torch.cuda.get_device_properties(0).multi_processor_count
            best = None
            for per in (1, 2, 3):
                pm = []
                for _ in range(5):
                    al.autoloco_traffic_probe(ctx, [(g, al.PROBE_READ) for g in st.grads], al.PROBE_RUN1, cus * per)
                    pm.append(al.autoloco_last_kernel_ms(ctx))
                m = statistics.median(pm)
                best = m if best is None else min(best, m)
            reference["norm_probe_ms"] = best
            reference["norm_probe_gbs"] = norm_bytes / (best * 1e-3) / 1e9
            reference["norm_frac_of_probe"] = best / norm_mean
            log(f"norm pass: probe of {k} streams read {best:.3f} ms ({norm_bytes / best / 1e6:.0f} GB/s); the norm "
                f"pass runs at {100 * best / norm_mean:.1f} % of it")
    tag = f"adamw_f32_k{k}_{args.workload}" + ("_copy" if args.copy else "")
    traffic = committed_traffic(tag, ADAMW_SOURCES)

    cpu = cpu1 = None
    if sample is not None:
        desc = f"{args.workload} K={k} inner AdamW"
        lr = al.autoloco_inner_lr(sched, s0)
        log("timing the oracle on the CPU sample on one thread")
        cpu1 = inner_cpu_baseline(sample, lr, 1000, args.cpu_seconds, desc)
        log(f"timing the oracle over the whole workload on {procs} processes")
        cpu, onorms = inner_cpu_baseline_stream(st, lr, 1000, desc, pool, procs)
        gnorms = list(first.grad_norm[:k]) if first is not None else []
        match = len(gnorms) == k and all(abs(a - b) <= 1e-6 * abs(b) for a, b in zip(gnorms, onorms))
        log(f"oracle gradient norms over the whole workload {'within' if match else 'OUTSIDE'} 1e-6 of the GPU's")
        cpu["grad_norms_match_gpu_within_1e-6"] = match
        for leg in (cpu, cpu1):
            leg["cpu_model"] = cpu_model()
            leg["gpu_speedup"] = (n * k / (ms_per_step * 1e-3)) / leg["value"]

    out = {
        "metric": metric_name(INNER_METRIC, args, k),
        "value": n * k / (ms_per_step * 1e-3),
        "unit": "worker-params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{args.workload} inner AdamW step: {n:,} parameters x K={k} workers, fp32 master "
                        f"parameters, moments and gradients, per-worker gradient-norm clipping 1.0, "
                        f"betas (0.9, 0.95), weight decay 0.1" + (", BF16 compute copy" if args.copy else ""),
            "n_params": n, "k": k, "update_bytes": update_bytes, "norm_bytes": norm_bytes,
            "alloc": alloc_label(args.alloc, spread),
        },
        "roofline": {
            "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS, "traffic": traffic, "kernel": "adamw_kernel (update pass)",
        },
        "update_ms_mean": upd_mean,
        "norm_ms_mean": norm_mean,
        "norm_pass_gbs": norm_bytes / (norm_mean * 1e-3) / 1e9,
        "traffic_reference": reference,
        "copy_ceiling_gbs": ceiling,
        "first_step_grad_norms": list(first.grad_norm[:k]) if first is not None else None,
        "cpu_baseline": cpu,
        "cpu_baseline_one_thread": cpu1,
        "kernel_source_sha256_16": kernel_source_hash(ADAMW_SOURCES),
    }
    print(json.dumps(out), flush=True)
    close_cpu_pool(pool)
    del st, copies, ts
    ctx.close()
    return 0


SHARE_METRIC = "per-GPU share of a one-replica-per-GPU round (BF16 payloads) params/s, 1.1B params K=8 GPUs"
SHARE_SOURCES = [os.path.join(CSRC, f) for f in ("shard_kernels.hpp", "shard_inst.hip", "round_kernels.hpp",
                                                  "reduce.hpp", "reset_kernels.hpp")]


def bench_share(args) -> int:
    """GPU 0 of K: its worker's payload over the whole model, the step of its
    1/K shard from K received payload shards, and its replica's reset.  The
    all-to-all and all-gather between them are not run (one GPU)."""
    import torch
    import paper_2609_36662_amd as al
    from workloads import drift, shapes

    shape_name, k, rdt = WORKLOADS[args.workload][0], WORKLOADS[args.workload][1], WORKLOADS[args.workload][2]
    if args.k:
        k = args.k
    n = (1 << 20) if shape_name is None else shapes.SHAPES[shape_name]().n_params
    tdtype = torch.float32 if rdt == "f32" else torch.bfloat16
    s_r = 4 if rdt == "f32" else 2
    step8 = -(-(-(-n // k)) // 8) * 8
    ns = min(n, step8)                                    # shard of GPU 0
    b_payload, b_shard, b_reset = n * (4 + s_r + 2), ns * (16 + 2 * k), n * (4 + s_r)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sched = al.make_schedule()
    coeffs = al.autoloco_outer_correction(al.make_outer_cfg(), al.autoloco_lr_mass(sched, 20_000, 750),
                                          al.autoloco_lr_mass(sched, 20_000, 500))
    log(f"per-GPU share {args.workload}: n={n:,} K={k} GPUs, shard {ns:,}; bytes payload "
        f"{b_payload / 1e9:.2f} GB, shard step {b_shard / 1e9:.2f} GB, reset {b_reset / 1e9:.2f} GB")
    ctx = al.autoloco_create(0)
    # every buffer from the placement-aware allocator (shard buffers as views of full-size ones)
    ts, spread = al.spread_tensors(ctx, n, [torch.float32, tdtype, torch.bfloat16, torch.float32]
                                   + [torch.bfloat16] * (k + 1))
    theta, rep, payload = ts[0], ts[1], ts[2]
    v_shard = ts[3][:ns]
    recv = [t[:ns] for t in ts[4:4 + k]]
    mean = ts[4 + k][:ns]
    inp = drift.RoundInputs(theta, torch.empty(0, device=dev), [rep])
    drift._normal_into(theta, 0.02, 42, drift.ROLE_THETA, 0)
    drift.fill_replicas(inp, seed=42)
    drift._normal_into(v_shard, 1e-4, 42, drift.ROLE_MOMENTUM, 0)
    for w in range(k):                                  # stand-ins for the workers' payload shards
        x = torch.empty(ns, dtype=torch.float32, device=dev)
        drift._normal_into(x, 1e-3, 100 + w, drift.ROLE_INDEP, w)
        recv[w].copy_(x)
        del x
    torch.cuda.synchronize()
    if args.grid:
        al.autoloco_set_grid_limit(ctx, args.grid)
    al.autoloco_set_timing(ctx, True)

    def one_step():
        al.autoloco_rank_payload(ctx, theta, rep, payload)
        t_p = al.autoloco_last_kernel_ms(ctx)
        al.autoloco_shard_step(ctx, theta[:ns], v_shard, recv, coeffs, mean_bf16=mean)
        t_s = al.autoloco_last_kernel_ms(ctx)
        al.autoloco_broadcast_reset(ctx, theta, [rep])
        t_r = al.autoloco_last_kernel_ms(ctx)
        return t_p, t_s, t_r

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    times = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        times.append(one_step())
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall / args.steps * 1e3
    tp, tsh, tr = (statistics.mean(t[i] for t in times) for i in range(3))
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step wall; payload {tp:.3f} ms "
        f"({b_payload / tp / 1e6:.0f} GB/s), shard step {tsh:.3f} ms ({b_shard / tsh / 1e6:.0f} GB/s), "
        f"reset {tr:.3f} ms ({b_reset / tr / 1e6:.0f} GB/s)")
    # each kernel's traffic reference: the probe of its own loads and stores
    # (same shape and grid, no arithmetic)
    num_cus = torch.cuda.get_device_properties(dev).multi_processor_count
    R, W, RW = al.PROBE_READ, al.PROBE_WRITE, al.PROBE_READ | al.PROBE_WRITE
    refs = {
        "payload": ([(theta, R), (rep, R), (payload, W)], al.PROBE_RUN2, args.grid or 2 * num_cus),
        "shard_step": ([(theta[:ns], RW), (v_shard, RW)] + [(r, R) for r in recv] + [(mean, W)], al.PROBE_RUN2,
                       args.grid or 3 * num_cus),
        # the reset alone runs three workgroups per compute unit
        "reset": ([(theta, R), (rep, W)], al.PROBE_RUN1 if rdt == "f32" else al.PROBE_RUN2,
                  args.grid or 3 * num_cus),
    }
    ref_ms = {}
    for name, (streams, shape, blocks) in refs.items():
        ms = []
        for rep_i in range(args.warmup + args.steps):
            al.autoloco_traffic_probe(ctx, streams, shape, blocks)
            if rep_i >= args.warmup:
                ms.append(al.autoloco_last_kernel_ms(ctx))
        ref_ms[name] = statistics.median(ms)
    log("traffic references: " + ", ".join(f"{k_} {v:.3f} ms" for k_, v in ref_ms.items()))
    achieved = b_payload / (tp * 1e-3) / 1e9
    ceiling = None if args.no_ceiling else copy_ceiling(torch, dev)
    traffic = committed_traffic(f"share_{rdt}_k{k}_{args.workload}_payload", SHARE_SOURCES)
    out = {
        "metric": SHARE_METRIC,
        "value": n / (ms_per_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if rdt == "f32" else "f32 (bf16 replicas)",
        "data": "synthetic",
        "config": {
            "workload": f"{args.workload}: GPU 0 of K={k} (one worker replica per GPU), {n:,} parameters, "
                        f"{rdt} replica, BF16 payloads; shard of {ns:,} parameters; collectives not run",
            "n_params": n, "k": k, "shard": ns, "bytes": {"payload": b_payload, "shard_step": b_shard,
                                                          "reset": b_reset},
            "alloc": alloc_label("spread", spread),
        },
        "roofline": {
            "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS, "traffic": traffic, "kernel": "rank_payload_kernel",
        },
        "copy_ceiling_gbs": ceiling,
        "kernel_ms": {"payload": tp, "shard_step": tsh, "reset": tr},
        "traffic_reference_ms": ref_ms,
        "ratio_to_reference": {"payload": tp / ref_ms["payload"], "shard_step": tsh / ref_ms["shard_step"],
                               "reset": tr / ref_ms["reset"]},
        "kernel_gbs": {"payload": b_payload / tp / 1e6, "shard_step": b_shard / tsh / 1e6,
                       "reset": b_reset / tr / 1e6},
        "cpu_baseline": None,
        "kernel_source_sha256_16": kernel_source_hash(SHARE_SOURCES),
    }
    print(json.dumps(out), flush=True)
    del ts, theta, rep, inp, recv, payload, v_shard, mean
    ctx.close()
    return 0


RESET_METRIC = "standalone replica reset params/s and achieved HBM GB/s (% of peak), 1.1B params K=8"
RESET_SOURCES = [os.path.join(CSRC, f) for f in ("reset_kernels.hpp", "round_kernels.hpp")]


def reset_probe_shape(al, rdt: str, k: int) -> int:
    """The probe shape with the standalone reset's loads and stores: the runs
    per lane its launcher picks (eight from three fp32 replicas on, one below,
    two for bf16 replicas)."""
    if rdt != "f32":
        return al.PROBE_RUN2
    return al.PROBE_RUN8 if k >= 3 else al.PROBE_RUN1


def bench_reset(args) -> int:
    """The standalone reset (theta_k <- theta for every replica; Alg. "AutoLoCo
    outer interval") at the library's default grid, beside the probe of its own
    loads and stores (theta read, K replicas written) at the same grid."""
    import torch
    import paper_2609_36662_amd as al
    from workloads import drift, shapes

    shape_name, k, rdt = WORKLOADS[args.workload][0], WORKLOADS[args.workload][1], WORKLOADS[args.workload][2]
    if args.k:
        k = args.k
    n = (1 << 20) if shape_name is None else shapes.SHAPES[shape_name]().n_params
    tdtype = torch.float32 if rdt == "f32" else torch.bfloat16
    s_r = 4 if rdt == "f32" else 2
    nbytes = n * (4 + k * s_r)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    ctx = al.autoloco_create(0)
    ts, spread = al.spread_tensors(ctx, n, [torch.float32] + [tdtype] * k)
    theta, reps = ts[0], ts[1:]
    drift._normal_into(theta, 0.02, 42, drift.ROLE_THETA, 0)
    torch.cuda.synchronize()
    num_cus = torch.cuda.get_device_properties(dev).multi_processor_count
    if args.grid:
        al.autoloco_set_grid_limit(ctx, args.grid)
    al.autoloco_set_timing(ctx, True)
    log(f"reset {args.workload}: n={n:,} K={k} {rdt} replicas, {nbytes / 1e9:.2f} GB per reset "
        f"({'spread' if spread else 'plain'} buffers)")

    def median_ms(call):
        ms = []
        for i in range(args.warmup + args.steps):
            call()
            if i >= args.warmup:
                ms.append(al.autoloco_last_kernel_ms(ctx))
        return statistics.median(ms)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        al.autoloco_broadcast_reset(ctx, theta, reps)
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) / args.steps * 1e3
    ms = median_ms(lambda: al.autoloco_broadcast_reset(ctx, theta, reps))
    # the reset's own pattern at its grid (three workgroups per compute unit)
    blocks = args.grid or 3 * num_cus
    shape = reset_probe_shape(al, rdt, k)
    try:
        ref_ms = median_ms(lambda: al.autoloco_traffic_probe(ctx, [(theta, al.PROBE_READ)] +
                                                             [(r, al.PROBE_WRITE) for r in reps], shape, blocks))
    except al.AutolocoError as e:      # the probe instantiates the reset's pattern for some K only
        log(f"no traffic reference: {e}")
        ref_ms = None
    achieved = nbytes / (ms * 1e-3) / 1e9
    log(f"reset {ms:.3f} ms ({achieved:.0f} GB/s, {100 * achieved / PEAK_HBM_GBS:.1f} %)" +
        (f", its pattern {ref_ms:.3f} ms: {ms / ref_ms:.4f} x" if ref_ms else ""))
    ceiling = None if args.no_ceiling else copy_ceiling(torch, dev)
    out = {
        "metric": metric_name(RESET_METRIC, args, k), "value": n / (ms_per_step * 1e-3), "unit": "params/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32" if rdt == "f32" else "f32 (bf16 replicas)", "data": "synthetic",
        "config": {"workload": f"{args.workload}: theta ({n:,} fp32) into K={k} {rdt} replicas",
                   "n_params": n, "k": k, "bytes": nbytes, "alloc": alloc_label("spread", spread)},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "kernel": "reset_kernel",
                     "traffic": committed_traffic(f"reset_{rdt}_k{k}_{args.workload}", RESET_SOURCES)},
        "kernel_ms_median": ms, "traffic_reference_ms_median": ref_ms,
        "ratio_to_reference": ms / ref_ms if ref_ms else None,
        "copy_ceiling_gbs": ceiling, "cpu_baseline": None,
        "kernel_source_sha256_16": kernel_source_hash(RESET_SOURCES),
    }
    print(json.dumps(out), flush=True)
    del ts, theta, reps
    ctx.close()
    return 0


PROBE_METRIC = ("streaming-pattern probes: HBM GB/s (% of peak) of access patterns on the buffers of the 1.1B "
                "params K=8 round, and the standalone reset against its pattern")


def bench_probe(args) -> int:
    """What the device sustains for streaming access patterns on the round's own
    buffers (theta, v and 8 fp32 replicas of the 1.1B model, 4.4 GB each): the
    round's ten streams in place, the same streams read only or written only,
    fewer streams, out of place, LDS-staged tiles; then the fused round and its
    traffic reference, and the standalone reset at K = 8 and K = 1 beside the
    probe of its own pattern (one stream read, K written), over grids."""
    import torch
    import paper_2609_36662_amd as al
    from workloads import drift, shapes

    n = shapes.SHAPES["llama-1.1b"]().n_params
    k = 8
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    ctx = al.autoloco_create(0)
    spread = False
    if args.alloc == "spread":
        ts, spread = al.spread_tensors(ctx, n, [torch.float32] * (k + 2))
    else:
        ts = [torch.empty(n, dtype=torch.float32, device=dev) for _ in range(k + 2)]
    inp = drift.RoundInputs(ts[0], ts[1], ts[2:])
    drift.fill_theta_momentum(inp, seed=42, recipe=drift.MIXED)
    drift.fill_replicas(inp, seed=42, recipe=drift.MIXED)
    torch.cuda.synchronize()
    num_cus = torch.cuda.get_device_properties(dev).multi_processor_count
    al.autoloco_set_timing(ctx, True)
    R, W, RW = al.PROBE_READ, al.PROBE_WRITE, al.PROBE_READ | al.PROBE_WRITE
    log(f"probe buffers: {k + 2} x {n * 4 / 1e9:.2f} GB ({'spread' if spread else 'plain'}); {num_cus} CUs")

    def timed(call):
        times = []
        moved = 0.0
        for rep in range(args.warmup + args.steps):
            moved = call()
            ms = al.autoloco_last_kernel_ms(ctx)
            if rep >= args.warmup:
                times.append(ms)
        return moved, statistics.median(times), min(times)

    def probe(name, shape, spec, blocks=0):
        streams = [(ts[i], acc) for i, acc in spec]
        moved, med, best = timed(lambda: al.autoloco_traffic_probe(ctx, streams, shape, blocks))
        row = {"pattern": name, "shape": ["run1", "run2", "serial", "tile", "phased", "run8"][shape],
               "blocks": blocks or num_cus, "bytes": moved, "ms_median": med, "ms_min": best,
               "gbs": moved / med / 1e6, "frac_of_peak": moved / med / 1e6 / PEAK_HBM_GBS}
        log(f"  {name:52s} {row['shape']:6s} {row['blocks']:5d} wg  {med:8.3f} ms  {row['gbs']:7.0f} GB/s "
            f"({100 * row['frac_of_peak']:.1f} %)")
        return row

    # every pattern over grids from one workgroup per compute unit to eight:
    # patterns with few streams need more waves to keep enough bytes in flight
    grids = [num_cus * m for m in (1, 2, 3, 4, 8)]
    ten = list(range(k + 2))
    patterns = [
        ("10 streams in place (the round's pattern)", al.PROBE_RUN1, [(i, RW) for i in ten]),
        ("10 streams read", al.PROBE_RUN1, [(i, R) for i in ten]),
        ("10 streams written", al.PROBE_RUN1, [(i, W) for i in ten]),
        ("1 stream read", al.PROBE_RUN1, [(0, R)]),
        ("2 streams read", al.PROBE_RUN1, [(i, R) for i in range(2)]),
        ("4 streams read", al.PROBE_RUN1, [(i, R) for i in range(4)]),
        ("1 stream written", al.PROBE_RUN1, [(0, W)]),
        ("1 stream in place", al.PROBE_RUN1, [(0, RW)]),
        ("2 streams in place", al.PROBE_RUN1, [(i, RW) for i in range(2)]),
        ("4 streams in place", al.PROBE_RUN1, [(i, RW) for i in range(4)]),
        ("6 streams in place", al.PROBE_RUN1, [(i, RW) for i in range(6)]),
        ("5 streams read, 5 others written", al.PROBE_RUN1, [(i, R) for i in range(5)] + [(i, W) for i in range(5, 10)]),
        ("10 streams in place, two runs per lane", al.PROBE_RUN2, [(i, RW) for i in ten]),
        ("10 streams in place, eight runs per lane (32 KB per stream and workgroup)", al.PROBE_RUN8,
         [(i, RW) for i in ten]),
        ("10 streams read, eight runs per lane", al.PROBE_RUN8, [(i, R) for i in ten]),
        ("10 streams written, eight runs per lane", al.PROBE_RUN8, [(i, W) for i in ten]),
    ]
    rows = []
    for name, shape, spec in patterns:
        sweep = [probe(name, shape, spec, g) for g in grids]
        best = max(sweep, key=lambda r: r["gbs"])
        rows.append({**best, "at_one_per_cu_gbs": sweep[0]["gbs"], "grids": {r["blocks"]: r["gbs"] for r in sweep}})
    # LDS tiles hold 160 KB of one workgroup: one per compute unit
    for name, shape, spec in (
            ("10 streams in place, LDS tiles stream by stream", al.PROBE_SERIAL, [(i, RW) for i in ten]),
            ("10 streams in place, LDS tiles all streams at once", al.PROBE_TILE, [(i, RW) for i in ten]),
            ("10 streams read, LDS tiles stream by stream", al.PROBE_SERIAL, [(i, R) for i in ten]),
            ("10 streams read, LDS tiles all streams at once", al.PROBE_TILE, [(i, R) for i in ten]),
            ("10 streams written, LDS tiles", al.PROBE_TILE, [(i, W) for i in ten]),
            ("10 streams in place, grid-wide read and write phases", al.PROBE_PHASED, [(i, RW) for i in ten])):
        rows.append(probe(name, shape, spec, num_cus))

    # the fused round and its traffic reference on the same buffers
    coeffs = al.autoloco_outer_correction(al.make_outer_cfg(), al.autoloco_lr_mass(al.make_schedule(), 20_000, 750),
                                          al.autoloco_lr_mass(al.make_schedule(), 20_000, 500))
    flags = al.FUSE_STATS | al.FUSE_RESET
    b_round = n * (2 * k * 4 + 16)

    def round_call():
        al.autoloco_outer_step(ctx, inp.theta, inp.momentum, inp.replicas, coeffs, flags, 1e-12)
        return b_round

    def ref_call():
        al.autoloco_traffic_reference(ctx, inp.theta, inp.momentum, inp.replicas)
        return b_round

    kernels = []
    for name, call in (("fused round (round_kernel)", round_call), ("traffic reference (traffic_kernel)", ref_call)):
        moved, med, best = timed(call)
        kernels.append({"kernel": name, "bytes": moved, "ms_median": med, "gbs": moved / med / 1e6})
        log(f"  {name:48s} {med:8.3f} ms  {moved / med / 1e6:7.0f} GB/s")

    # standalone reset (theta read, K replicas written) against the probe of that pattern
    resets = []
    for kk in (8, 1):
        b_reset = n * (4 + 4 * kk)
        for blocks in (256, 512, 768, 1024):
            al.autoloco_set_grid_limit(ctx, blocks)
            _, med, _ = timed(lambda: (al.autoloco_broadcast_reset(ctx, inp.theta, inp.replicas[:kk]), b_reset)[1])
            al.autoloco_set_grid_limit(ctx, 0)
            ref = probe(f"reset pattern K={kk}: 1 stream read, {kk} written", reset_probe_shape(al, "f32", kk),
                        [(0, R)] + [(2 + j, W) for j in range(kk)], blocks)
            # the reset wrote theta into the replicas; the probe writes them the same words
            resets.append({"k": kk, "blocks": blocks, "bytes": b_reset, "reset_ms_median": med,
                           "reset_gbs": b_reset / med / 1e6, "reference_ms_median": ref["ms_median"],
                           "ratio_to_reference": med / ref["ms_median"]})
            log(f"  reset K={kk} at {blocks:5d} wg: {med:.3f} ms ({b_reset / med / 1e6:.0f} GB/s), "
                f"{med / ref['ms_median']:.3f} x its pattern")
        _, med, _ = timed(lambda: (al.autoloco_broadcast_reset(ctx, inp.theta, inp.replicas[:kk]), b_reset)[1])
        resets.append({"k": kk, "blocks": "default", "bytes": b_reset, "reset_ms_median": med,
                       "reset_gbs": b_reset / med / 1e6})
        log(f"  reset K={kk} at the default grid: {med:.3f} ms ({b_reset / med / 1e6:.0f} GB/s)")

    best = max(r["gbs"] for r in rows if r["pattern"].startswith("10 streams in place"))
    log("best of each pattern: " + "; ".join(f"{r['pattern']} {r['gbs']:.0f} GB/s at {r['blocks']}" for r in rows))
    out = {
        "metric": PROBE_METRIC, "value": best, "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "higher_is_better": True, "data": "synthetic",
        "config": {"workload": f"llama-1.1b buffers: {k + 2} x {n:,} fp32 elements",
                   "alloc": alloc_label(args.alloc, spread), "cus": num_cus},
        "probes": rows, "kernels": kernels, "reset": resets,
        "kernel_source_sha256_16": kernel_source_hash(KERNEL_SOURCES + [os.path.join(CSRC, "probe_kernels.hpp")]),
    }
    print(json.dumps(out), flush=True)
    del ts, inp
    ctx.close()
    return 0


CLOSED_LOOP_METRIC = ("closed-loop sync-round params/s (round + interval controller) and achieved HBM GB/s "
                      "(% of peak), 7B params K=4, 20 rounds")


def bench_closed_loop(args) -> int:
    """Consecutive rounds with the interval controller in the loop: each round's
    fused outer step runs with the coefficients of the controller's decision,
    and its statistics are the controller's next observation.  Between rounds
    (untimed), every worker endpoint is drawn around the new synchronised
    parameters, the drift growing with the learning-rate mass of the selected
    interval, with a per-round jitter of the per-worker part and, in the first
    assessed interval from round 12 on, a fault (per-worker part x10) that the
    controller must answer with a shorter horizon.  A timed step runs from the
    synchronisation before the round to the decision for the next interval."""
    import math
    from workloads import shapes

    shape_name, k, rdt = WORKLOADS[args.workload][0], WORKLOADS[args.workload][1], WORKLOADS[args.workload][2]
    if args.k:
        k = args.k
    n = (1 << 20) if shape_name is None else shapes.SHAPES[shape_name]().n_params
    # the CPU baseline's worker processes start before this process touches the GPU
    pool = procs = None
    if not args.no_cpu_baseline:
        procs = cpu_procs(args.cpu_procs)
        pool = make_cpu_pool(n, k, rdt, procs)

    import torch
    import paper_2609_36662_amd as al
    from workloads import drift
    tdtype = torch.float32 if rdt == "f32" else torch.bfloat16
    s_r = 4 if rdt == "f32" else 2
    bytes_per_round = n * (2 * k * s_r + 16)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"closed loop {args.workload}: n={n:,} K={k} replicas={rdt}, {args.warmup} + {args.steps} rounds, "
        f"bytes/round={bytes_per_round / 1e9:.3f} GB")
    ctx = al.autoloco_create(0)
    ts, spread = al.spread_tensors(ctx, n, [torch.float32, torch.float32] + [tdtype] * k)
    inp = drift.RoundInputs(ts[0], ts[1], ts[2:])
    drift.fill_theta_momentum(inp, seed=42)
    if args.grid:
        al.autoloco_set_grid_limit(ctx, args.grid)
    al.autoloco_set_timing(ctx, True)
    ctl = al.autoloco_controller_create()
    dec = al.autoloco_select_interval(ctl, None)
    lam1 = dec.lambda_sel
    tokens_per_step = float(1 << 20)
    assessed = (4, 5, 6)   # autoloco_phase: monitoring and the two candidate phases
    fault_done = False
    walls, kms, trace = [], [], []
    cpu = ost = None
    for r in range(args.warmup + args.steps):
        lam = dec.lambda_sel
        fault = not fault_done and r >= 12 and dec.phase in assessed
        jit = math.exp(0.05 * math.sin(1.7 * r + 0.3)) * (10.0 if fault else 1.0)
        drift.fill_replicas(inp, seed=100 + r, scale=lam / lam1, indep_scale=[jit] * k)
        if r == args.warmup and pool is not None:
            # untimed: the oracle over this round's whole state, with the decision's coefficients
            torch.cuda.synchronize()
            log(f"timing the oracle over the whole state of round {r} on {procs} processes")
            cpu, _, ost = cpu_baseline_stream(inp, dec.coeffs, rdt, f"{args.workload} K={k} {rdt} closed loop, "
                                              f"round {r}", pool, procs, one_core=False)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st = al.autoloco_outer_step(ctx, inp.theta, inp.momentum, inp.replicas, dec.coeffs,
                                    al.FUSE_STATS | al.FUSE_RESET, 1e-12)
        prev = dec
        dec = al.autoloco_select_interval(ctl, al.make_observation(st.D, st.C, lam, tokens_per_step * prev.h_step,
                                                                   prev.h_step, st.finite))
        wall = (time.perf_counter() - t0) * 1e3
        if fault:
            fault_done = True
        if r == args.warmup and cpu is not None:
            match = all(abs(a - b) <= 1e-4 * abs(b) for a, b in ((st.D, ost.D), (st.C, ost.C),
                                                                 (st.disagreement, ost.disagreement)))
            log(f"oracle on round {r}: D {ost.D:.9g} C {ost.C:.9g} (GPU D {st.D:.9g} C {st.C:.9g}, "
                f"{'within' if match else 'OUTSIDE'} 1e-4)")
            cpu["statistics_match_gpu_within_1e-4"] = match
        if r >= args.warmup:
            walls.append(wall)
            kms.append(al.autoloco_last_kernel_ms(ctx))
        trace.append({"round": r, "h_step": prev.h_step, "rho": prev.coeffs.rho, "D": st.D, "C": st.C,
                      "assessment_after": dec.assessment, "next_h_step": dec.h_step, "fault": fault})
        log(f"round {r}: H^step {prev.h_step} rho {prev.coeffs.rho:.4f} D {st.D:.4g} C {st.C:.4g} -> "
            f"assessment {dec.assessment}, next H^step {dec.h_step}; {wall:.3f} ms" + (" (fault)" if fault else ""))
    ms_per_step = statistics.mean(walls)
    mean_ms = statistics.mean(kms)
    achieved = bytes_per_round / (mean_ms * 1e-3) / 1e9
    if cpu is not None:
        cpu["cpu_model"] = cpu_model()
        cpu["gpu_speedup"] = (n / (ms_per_step * 1e-3)) / cpu["value"]
    tag = f"round_{rdt}_k{k}_{args.workload}"
    out = {
        "metric": metric_name(CLOSED_LOOP_METRIC, args, k, steps_tail=True),
        "value": n / (ms_per_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if rdt == "f32" else "f32 (bf16 replicas)",
        "data": "synthetic",
        "config": {
            "workload": f"{args.workload} closed loop: {n:,} parameters, K={k} {rdt} replicas, fused stats + "
                        f"Nesterov + reset with the coefficients the interval controller chose, the controller "
                        f"fed each round's statistics (C4 settings, budget 50,000 steps)",
            "n_params": n, "k": k, "replica_dtype": rdt, "bytes_per_round": bytes_per_round,
            "alloc": alloc_label("spread", spread), "fault_round": next((t["round"] for t in trace if t["fault"]), None),
        },
        "roofline": {
            "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS, "traffic": committed_traffic(tag),
        },
        "kernel_ms_mean": mean_ms,
        "round_ms_max": max(walls),
        "rounds": trace,
        "cpu_baseline": cpu,
        "kernel_source_sha256_16": kernel_source_hash(),
    }
    print(json.dumps(out), flush=True)
    close_cpu_pool(pool)
    del inp, ts
    ctx.close()
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama-1.1b", choices=sorted(WORKLOADS))
    ap.add_argument("--grid", type=int, default=0, help="cap on workgroups (0 = library default)")
    ap.add_argument("--k", type=int, default=0, help="override the workload's replica count")
    ap.add_argument("--codec", choices=("fp32", "int8", "bf16"), default="fp32",
                    help="int8: the worker average travels through the INT8 blockwise codec; "
                         "bf16: as BF16 pseudo-gradient payloads")
    ap.add_argument("--payload", action="store_true",
                    help="int8 / bf16: also write the mean every worker receives (codes + scales, or BF16)")
    ap.add_argument("--alloc", choices=("spread", "torch"), default="spread",
                    help="spread: the library's placement-aware allocator; torch: torch.empty")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--cpu-sample", type=int, default=1 << 22)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ceiling", action="store_true")
    ap.add_argument("--back-to-back", type=int, default=20,
                    help="round: also time this many rounds back to back on replicas already equal to theta'")
    ap.add_argument("--no-plain", action="store_true", help="round: skip the plain-allocation comparison")
    ap.add_argument("--cpu-procs", type=int, default=0,
                    help="worker processes of the CPU baseline (0: the cores this process may use, at most 16)")
    ap.add_argument("--perturbed", type=int, default=0,
                    help="ignored (every timed round runs on freshly drawn replicas); kept so older commands run")
    ap.add_argument("--step", choices=("round", "inner", "share", "closed-loop", "probe", "reset"), default="round",
                    help="round: the synchronisation round; inner: one AdamW step of every worker; share: one "
                         "GPU's share of a round with one worker replica per GPU (K GPUs, no collectives); "
                         "closed-loop: consecutive rounds with the interval controller choosing each one's "
                         "coefficients from the previous round's statistics (use --workload llama-7b); probe: "
                         "streaming-pattern probes on the round's buffers (the device's ceiling for each pattern); "
                         "reset: the standalone replica reset beside the probe of its own loads and stores")
    ap.add_argument("--copy", action="store_true", help="inner: also write each worker's BF16 compute copy")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the round keeps all K replicas on one device and has no "
              f"multi-GPU path (asked for --gpus {args.gpus})", file=sys.stderr)
        return 2

    if args.step == "inner":
        return bench_inner(args)
    if args.step == "share":
        return bench_share(args)
    if args.step == "probe":
        return bench_probe(args)
    if args.step == "reset":
        return bench_reset(args)
    if args.step == "closed-loop":
        return bench_closed_loop(args)

    from workloads import shapes
    shape_name, k, rdt, recipe_name, h_sel, h_base = WORKLOADS[args.workload]
    if args.k:
        k = args.k
    n = (1 << 20) if shape_name is None else shapes.SHAPES[shape_name]().n_params
    # the CPU baseline's worker processes start before this process touches the GPU
    pool = procs = None
    if not args.no_cpu_baseline:
        procs = cpu_procs(args.cpu_procs)
        pool = make_cpu_pool(n, k, rdt, procs)

    import torch
    import paper_2609_36662_amd as al
    from workloads import drift
    recipe = drift.MIXED if recipe_name == "mixed" else drift.spread_recipe(1e-3)
    tdtype = torch.float32 if rdt == "f32" else torch.bfloat16
    s_r = 4 if rdt == "f32" else 2
    bytes_per_round = n * (2 * k * s_r + 16)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    # Outer coefficients from the library's own schedule preview and correction.
    sched = al.make_schedule()
    lam = al.autoloco_lr_mass(sched, 20_000, h_sel)
    lam_b = al.autoloco_lr_mass(sched, 20_000, h_base)
    coeffs = al.autoloco_outer_correction(al.make_outer_cfg(), lam, lam_b)

    log(f"workload {args.workload}: n={n:,} K={k} replicas={rdt} bytes/round={bytes_per_round/1e9:.3f} GB")
    ctx = al.autoloco_create(0)
    t = time.perf_counter()
    spread = False
    if args.alloc == "spread":
        ts, spread = al.spread_tensors(ctx, n, [torch.float32, torch.float32] + [tdtype] * k)
        inp = drift.RoundInputs(ts[0], ts[1], ts[2:])
    else:
        inp = drift.empty_inputs(n, k, replica_dtype=tdtype, device=dev)
    drift.fill_theta_momentum(inp, seed=42, recipe=recipe)
    drift.fill_replicas(inp, seed=42, recipe=recipe)
    torch.cuda.synchronize()
    log(f"buffers ({args.alloc}{', spread' if spread else ''}) allocated and inputs generated in "
        f"{time.perf_counter() - t:.1f} s")


    if args.grid:
        al.autoloco_set_grid_limit(ctx, args.grid)
    blocks, threads = al.autoloco_launch_shape(ctx, n, k, al.F32 if rdt == "f32" else al.BF16)
    al.autoloco_set_timing(ctx, True)
    flags = al.FUSE_STATS | al.FUSE_RESET

    codes = scales = None
    if args.codec == "int8" and args.payload:
        codes = torch.empty(n, dtype=torch.int8, device=dev)
        scales = torch.empty((n + 4095) // 4096, dtype=torch.float32, device=dev)
        bytes_per_round += n + 4 * ((n + 4095) // 4096)
    if args.codec == "bf16" and args.payload:
        codes = torch.empty(n, dtype=torch.bfloat16, device=dev)
        bytes_per_round += 2 * n

    def one_round():
        if args.codec == "int8":
            st = al.autoloco_outer_step_int8(ctx, inp.theta, inp.momentum, inp.replicas, coeffs, flags, 1e-12,
                                             mean_codes=codes, mean_scales=scales)
        elif args.codec == "bf16":
            st = al.autoloco_outer_step_bf16(ctx, inp.theta, inp.momentum, inp.replicas, coeffs, flags, 1e-12,
                                             mean_bf16=codes)
        else:
            st = al.autoloco_outer_step(ctx, inp.theta, inp.momentum, inp.replicas, coeffs, flags, 1e-12)
        return st

    first_stats = None
    for i in range(args.warmup):
        st = one_round()
        if i == 0:
            first_stats = st.as_dict()
        drift.fill_replicas(inp, seed=43 + i, recipe=recipe)
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} rounds); grid {blocks} x {threads}")

    # Exactly `steps` timed rounds, each on freshly drawn replicas (drawn
    # untimed before it) and bracketed by device synchronisations; the call
    # itself returns once the sums are on the host.
    kernel_ms, round_ms = [], []
    for i in range(args.steps):
        drift.fill_replicas(inp, seed=1000 + i, recipe=recipe)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        one_round()
        torch.cuda.synchronize()
        round_ms.append((time.perf_counter() - t1) * 1e3)
        kernel_ms.append(al.autoloco_last_kernel_ms(ctx))      # read after the timed bracket
    ms_per_step = statistics.mean(round_ms)
    log(f"timed {args.steps} rounds on freshly drawn replicas: {ms_per_step:.3f} ms/round wall (mean), kernel mean "
        f"{statistics.mean(kernel_ms):.3f} ms")

    # the same rounds back to back, every replica already equal to theta' (the
    # kernel has no data-dependent control flow: the same time)
    b2b_ms = None
    if args.back_to_back:
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(args.back_to_back):
            one_round()
        torch.cuda.synchronize()
        b2b_ms = (time.perf_counter() - t1) / args.back_to_back * 1e3
        log(f"{args.back_to_back} rounds back to back: {b2b_ms:.3f} ms/round")

    ceiling = None if args.no_ceiling else copy_ceiling(torch, dev)

    mean_ms = statistics.mean(kernel_ms)
    achieved = bytes_per_round / (mean_ms * 1e-3) / 1e9

    # The round's loads and stores without its arithmetic, on the same buffers
    # with the plain round's launch shape: what the device sustains for this
    # access pattern (the buffers are left unchanged).
    reference = None
    if not args.no_ceiling:
        ref_ms = []
        for _ in range(10):
            al.autoloco_traffic_reference(ctx, inp.theta, inp.momentum, inp.replicas)
            ref_ms.append(al.autoloco_last_kernel_ms(ctx))
        ref_bytes = n * (2 * k * s_r + 16)
        ref_gbs = ref_bytes / (statistics.median(ref_ms) * 1e-3) / 1e9
        reference = {"kernel": "traffic_kernel (the round's loads and stores, no arithmetic)",
                     "kernel_ms_median": statistics.median(ref_ms), "bytes": ref_bytes, "gbs": ref_gbs,
                     "frac_of_peak": ref_gbs / PEAK_HBM_GBS, "round_frac_of_reference": achieved / ref_gbs}
        log(f"traffic reference (same loads and stores, no arithmetic): {statistics.median(ref_ms):.3f} ms, "
            f"{ref_gbs:.0f} GB/s; the round runs at {100 * achieved / ref_gbs:.1f} % of it")
    tag = f"round_{rdt}_k{k}_{args.workload}" + ("" if args.codec == "fp32" else f"_{args.codec}")
    traffic = committed_traffic(tag, INT8_SOURCES if args.codec == "int8" else None)

    # The same round on plain torch allocations (consecutive buffers, adjacent in
    # physical memory), for comparison with the spread placement above.
    plain = None
    need = n * (8 + k * s_r)
    free_b = torch.cuda.mem_get_info(dev)[0]
    if args.alloc == "spread" and not args.no_plain and args.codec == "fp32" and need > free_b - (2 << 30):
        log(f"plain allocations: skipped ({need / 1e9:.1f} GB more needed, {free_b / 1e9:.1f} GB free)")
        plain = {"skipped": f"{need / 1e9:.1f} GB needed beside the spread buffers, {free_b / 1e9:.1f} GB free"}
    elif args.alloc == "spread" and not args.no_plain and args.codec == "fp32":
        alt = drift.empty_inputs(n, k, replica_dtype=tdtype, device=dev)
        drift.fill_theta_momentum(alt, seed=42, recipe=recipe)
        pk, pw = [], []
        for i in range(6):
            drift.fill_replicas(alt, seed=2000 + i, recipe=recipe)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            al.autoloco_outer_step(ctx, alt.theta, alt.momentum, alt.replicas, coeffs, flags, 1e-12)
            torch.cuda.synchronize()
            if i:
                pw.append((time.perf_counter() - t1) * 1e3)
                pk.append(al.autoloco_last_kernel_ms(ctx))
        del alt
        torch.cuda.empty_cache()
        plain = {"ms_per_round_mean": statistics.mean(pw), "kernel_ms_mean": statistics.mean(pk),
                 "achieved_gbs": bytes_per_round / (statistics.mean(pk) * 1e-3) / 1e9, "rounds": len(pw),
                 "alloc": "torch (consecutive allocations made after the spread allocation returned its free slots; on a fresh device consecutive allocations run about 20 % slower, see --alloc torch)"}
        log(f"plain allocations: {plain['ms_per_round_mean']:.3f} ms/round, kernel {plain['kernel_ms_mean']:.3f} ms "
            f"({plain['achieved_gbs']:.0f} GB/s)")

    cpu = cpu1 = None
    if pool is not None:
        # fresh inputs for the oracle (the timed rounds left every replica at theta')
        drift.fill_replicas(inp, seed=3000, recipe=recipe)
        torch.cuda.synchronize()
        gst = al.autoloco_round_stats(ctx, inp.theta, inp.replicas, 1e-12)
        desc = f"{args.workload} K={k} {rdt}"
        log(f"timing the oracle over the whole workload: one core, then {procs} processes")
        cpu, cpu1, ost = cpu_baseline_stream(inp, coeffs, rdt, desc, pool, procs)
        match = all(abs(a - b) <= 1e-4 * abs(b) for a, b in ((gst.D, ost.D), (gst.C, ost.C),
                                                             (gst.disagreement, ost.disagreement)))
        log(f"oracle over the whole workload: D {ost.D:.9g} C {ost.C:.9g} (GPU D {gst.D:.9g} C {gst.C:.9g}, "
            f"{'within' if match else 'OUTSIDE'} 1e-4)")
        for leg in (cpu, cpu1):
            leg["cpu_model"] = cpu_model()
            leg["gpu_speedup"] = (n / (ms_per_step * 1e-3)) / leg["value"]
            leg["statistics_match_gpu_within_1e-4"] = match

    out = {
        "metric": metric_name(METRIC, args, k),
        "value": n / (ms_per_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if rdt == "f32" else "f32 (bf16 replicas)",
        "data": "synthetic",
        "config": {
            "workload": f"{args.workload}: {n:,} parameters as one flat arena per buffer, K={k} "
                        f"{rdt} replicas, fp32 theta and momentum, fused stats + Nesterov + reset"
                        + {"fp32": "", "int8": ", worker average through the INT8 blockwise codec",
                           "bf16": ", worker average as BF16 pseudo-gradient payloads"}[args.codec],
            "n_params": n, "k": k, "replica_dtype": rdt, "bytes_per_round": bytes_per_round,
            "grid": [blocks, threads] if args.codec == "fp32" else None, "alloc": alloc_label(args.alloc, spread),
            "codec": args.codec + (" + payload" if codes is not None else ""),
            "h_selected": h_sel, "h_base": h_base,
            "rho": coeffs.rho, "mu": coeffs.mu, "eta_out": coeffs.eta_out,
        },
        "roofline": {
            "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS, "traffic": traffic,
        },
        "timing": "mean of the timed rounds, each on freshly drawn replicas and bracketed by device "
                  "synchronisations (the call returns once the statistics are on the host)",
        "kernel_ms_mean": mean_ms,
        "kernel_ms_min": min(kernel_ms),
        "kernel_ms_median": statistics.median(kernel_ms),
        "round_ms_median": statistics.median(round_ms),
        "round_ms_back_to_back": b2b_ms,
        "plain_alloc": plain,
        "copy_ceiling_gbs": ceiling,
        "traffic_reference": reference,
        "first_round_stats": {k2: first_stats[k2] for k2 in ("D", "C", "disagreement", "finite")}
        if first_stats else None,
        "cpu_baseline": cpu,
        "cpu_baseline_one_thread": cpu1,
        "kernel_source_sha256_16": kernel_source_hash(INT8_SOURCES if args.codec == "int8" else None),
    }
    print(json.dumps(out), flush=True)
    close_cpu_pool(pool)
    del inp
    if args.alloc == "spread":
        del ts
    ctx.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
