"""ctypes binding of libautoloco.so (the C ABI declared in include/autoloco.h).

Argument marshalling only: torch tensors become raw device pointers and the
context is bound to a HIP stream; every step of a round runs in the library.
Loading fails loudly when the library is missing and cannot be built — there
is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import math
import os
import threading
from dataclasses import dataclass
from typing import List, Optional, Sequence

MAX_K = 16
F32, BF16 = 0, 1
FUSE_STATS, FUSE_RESET = 1, 2

STATUS = {0: "ok", -1: "invalid argument", -2: "misaligned", -3: "aliasing buffers",
          -4: "HIP runtime error", -5: "out of memory", -6: "call out of order"}

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libautoloco.so")


class AutolocoError(RuntimeError):
    def __init__(self, status: int, what: str, detail: str = ""):
        self.status = status
        msg = f"{what} failed: {STATUS.get(status, status)}"
        if detail:
            msg += f" ({detail})"
        super().__init__(msg)


# ------------------------------------------------------------------ structs --
class Buffers(C.Structure):
    _fields_ = [("n", C.c_int64), ("k", C.c_int32), ("replica_dtype", C.c_int32),
                ("theta", C.c_void_p), ("momentum", C.c_void_p), ("replicas", C.c_void_p * MAX_K)]


class Stats(C.Structure):
    _fields_ = [("sq_norm", C.c_double * MAX_K), ("sq_dev", C.c_double * MAX_K),
                ("sq_mean", C.c_double), ("D", C.c_double), ("C", C.c_double),
                ("disagreement", C.c_double), ("finite", C.c_int32), ("k", C.c_int32)]

    def as_dict(self):
        k = self.k
        return {"sq_norm": list(self.sq_norm[:k]), "sq_dev": list(self.sq_dev[:k]),
                "sq_mean": self.sq_mean, "D": self.D, "C": self.C,
                "disagreement": self.disagreement, "finite": bool(self.finite)}


class OuterCoeffs(C.Structure):
    _fields_ = [("mu", C.c_double), ("eta_out", C.c_double), ("rho", C.c_double),
                ("kappa", C.c_double), ("normalize", C.c_int32)]


class Schedule(C.Structure):
    _fields_ = [("peak", C.c_double), ("min_lr", C.c_double), ("warmup", C.c_int64),
                ("total", C.c_int64)]


class OuterCfg(C.Structure):
    _fields_ = [("eta_base", C.c_double), ("mu_base", C.c_double), ("mu_min", C.c_double),
                ("mu_max", C.c_double), ("kappa_max", C.c_double), ("eps", C.c_double),
                ("normalize", C.c_int32)]


class ControllerCfg(C.Structure):
    _fields_ = [("h_base", C.c_int64), ("h_min", C.c_int64), ("h_max", C.c_int64),
                ("q_h", C.c_int64), ("budget_steps", C.c_int64),
                ("beta_tok", C.c_double), ("eps", C.c_double), ("thr_cand", C.c_double),
                ("thr_mod", C.c_double), ("thr_sev", C.c_double), ("cand_exposure", C.c_double),
                ("retire_frac", C.c_double), ("red_moderate", C.c_double),
                ("red_severe", C.c_double), ("ref_ema", C.c_double), ("mad_scale", C.c_double),
                ("scale_floor", C.c_double),
                ("n_mapper_boot", C.c_int32), ("n_ref_boot", C.c_int32), ("n_var", C.c_int32),
                ("hist_max", C.c_int32), ("moderate_confirm", C.c_int32),
                ("fallback_count", C.c_int32),
                ("sched", Schedule), ("outer", OuterCfg)]


class Observation(C.Structure):
    _fields_ = [("D", C.c_double), ("C", C.c_double), ("lambda_done", C.c_double),
                ("tokens", C.c_double), ("h_step_done", C.c_int64), ("finite", C.c_int32)]


class Decision(C.Structure):
    _fields_ = [("start_step", C.c_int64), ("h_tok", C.c_int64), ("h_step", C.c_int64),
                ("h_ref", C.c_int64), ("lambda_sel", C.c_double), ("lambda_base", C.c_double),
                ("z_max", C.c_double), ("assessment", C.c_int32), ("phase", C.c_int32),
                ("done", C.c_int32), ("reserved", C.c_int32), ("coeffs", OuterCoeffs)]


class ShardBuffers(C.Structure):
    _fields_ = [("n", C.c_int64), ("k", C.c_int32), ("theta", C.c_void_p), ("momentum", C.c_void_p),
                ("payloads", C.c_void_p * MAX_K)]


class ProbeStream(C.Structure):
    _fields_ = [("ptr", C.c_void_p), ("elem_bytes", C.c_int32), ("access", C.c_int32)]


class AdamWBuffers(C.Structure):
    _fields_ = [("n", C.c_int64), ("k", C.c_int32), ("params", C.c_void_p * MAX_K),
                ("exp_avg", C.c_void_p * MAX_K), ("exp_avg_sq", C.c_void_p * MAX_K),
                ("grads", C.c_void_p * MAX_K), ("model_bf16", C.c_void_p * MAX_K)]


class AdamWCoeffs(C.Structure):
    _fields_ = [("lr", C.c_double), ("beta1", C.c_double), ("beta2", C.c_double), ("eps", C.c_double),
                ("weight_decay", C.c_double), ("max_grad_norm", C.c_double), ("step", C.c_int64)]


class AdamWStats(C.Structure):
    _fields_ = [("grad_norm", C.c_double * MAX_K), ("clip_coef", C.c_double * MAX_K),
                ("k", C.c_int32), ("finite", C.c_int32)]


# ---------------------------------------------------------------- loading --
_lib = None
_lock = threading.Lock()

# (name, restype, argtypes) of every symbol the header declares
SYMBOLS = [
    ("autoloco_status_string", C.c_char_p, [C.c_int]),
    ("autoloco_create", C.c_int, [C.c_int, C.c_void_p, C.POINTER(C.c_void_p)]),
    ("autoloco_destroy", None, [C.c_void_p]),
    ("autoloco_last_error", C.c_char_p, [C.c_void_p]),
    ("autoloco_set_timing", C.c_int, [C.c_void_p, C.c_int]),
    ("autoloco_last_kernel_ms", C.c_int, [C.c_void_p, C.POINTER(C.c_float)]),
    ("autoloco_set_grid_limit", C.c_int, [C.c_void_p, C.c_int]),
    ("autoloco_launch_shape", C.c_int, [C.c_void_p, C.c_int64, C.c_int32, C.c_int32, C.POINTER(C.c_int32),
                                        C.POINTER(C.c_int32)]),
    ("autoloco_alloc_spread", C.c_int, [C.c_void_p, C.c_int32, C.c_size_t, C.POINTER(C.c_void_p),
                                        C.POINTER(C.c_int32)]),
    ("autoloco_free", C.c_int, [C.c_void_p, C.c_void_p]),
    ("autoloco_round_stats", C.c_int, [C.c_void_p, C.POINTER(Buffers), C.c_double, C.POINTER(Stats)]),
    ("autoloco_outer_step", C.c_int, [C.c_void_p, C.POINTER(Buffers), C.POINTER(OuterCoeffs),
                                      C.c_uint32, C.c_double, C.POINTER(Stats)]),
    ("autoloco_outer_step_int8", C.c_int, [C.c_void_p, C.POINTER(Buffers), C.POINTER(OuterCoeffs),
                                           C.c_uint32, C.c_double, C.POINTER(Stats), C.c_void_p, C.c_void_p]),
    ("autoloco_outer_step_bf16", C.c_int, [C.c_void_p, C.POINTER(Buffers), C.POINTER(OuterCoeffs),
                                           C.c_uint32, C.c_double, C.POINTER(Stats), C.c_void_p]),
    ("autoloco_outer_step_static", C.c_int, [C.c_int, C.c_void_p, C.POINTER(Buffers), C.POINTER(OuterCoeffs),
                                             C.c_uint32, C.c_double, C.POINTER(Stats)]),
    ("autoloco_broadcast_reset", C.c_int, [C.c_void_p, C.POINTER(Buffers)]),
    ("autoloco_traffic_reference", C.c_int, [C.c_void_p, C.POINTER(Buffers)]),
    ("autoloco_traffic_probe", C.c_int, [C.c_void_p, C.c_int64, C.POINTER(ProbeStream), C.c_int32, C.c_int32,
                                         C.c_int32, C.POINTER(C.c_double)]),
    ("autoloco_build_id", C.c_char_p, []),
    ("autoloco_rank_payload", C.c_int, [C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p,
                                        C.POINTER(C.c_double)]),
    ("autoloco_shard_step", C.c_int, [C.c_void_p, C.POINTER(ShardBuffers), C.POINTER(OuterCoeffs), C.c_void_p,
                                      C.POINTER(C.c_double)]),
    ("autoloco_inner_adamw", C.c_int, [C.c_void_p, C.POINTER(AdamWBuffers), C.POINTER(AdamWCoeffs),
                                       C.POINTER(AdamWStats)]),
    ("autoloco_last_adamw_ms", C.c_int, [C.c_void_p, C.POINTER(C.c_float), C.POINTER(C.c_float)]),
    ("autoloco_adamw_traffic_reference", C.c_int, [C.c_void_p, C.POINTER(AdamWBuffers)]),
    ("autoloco_inner_lr", C.c_double, [C.POINTER(Schedule), C.c_int64]),
    ("autoloco_lr_mass", C.c_double, [C.POINTER(Schedule), C.c_int64, C.c_int64]),
    ("autoloco_outer_correction", C.c_int, [C.POINTER(OuterCfg), C.c_double, C.c_double,
                                            C.POINTER(OuterCoeffs)]),
    ("autoloco_controller_default_cfg", None, [C.POINTER(ControllerCfg)]),
    ("autoloco_controller_create", C.c_int, [C.POINTER(ControllerCfg), C.POINTER(C.c_void_p)]),
    ("autoloco_controller_destroy", None, [C.c_void_p]),
    ("autoloco_select_interval", C.c_int, [C.c_void_p, C.POINTER(Observation), C.POINTER(Decision)]),
    ("autoloco_controller_reference", C.c_int, [C.c_void_p, C.POINTER(C.c_double),
                                                C.POINTER(C.c_double), C.POINTER(C.c_double)]),
    ("autoloco_controller_save", C.c_int, [C.c_void_p, C.c_void_p, C.POINTER(C.c_size_t)]),
    ("autoloco_controller_load", C.c_int, [C.c_void_p, C.c_void_p, C.c_size_t]),
]


def check_build_id(handle, expected: str) -> None:
    """Refuses a library built from sources other than the ones beside it."""
    got = handle.autoloco_build_id().decode()
    if got != expected:
        raise RuntimeError(f"{LIB_PATH} was built from other sources (build id {got}, sources {expected}); "
                           "rebuild it: python -m paper_2609_36662_amd.build")


def lib():
    """The loaded library; builds it first if nothing is built yet, and refuses
    one built from other sources than those in this tree."""
    global _lib
    with _lock:
        if _lib is None:
            from . import build as _build
            if not os.path.exists(LIB_PATH):
                _build.build()
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(f"{LIB_PATH} is missing and could not be built")
            handle = C.CDLL(LIB_PATH)
            for name, res, args in SYMBOLS:
                fn = getattr(handle, name)
                fn.restype = res
                fn.argtypes = args
            check_build_id(handle, _build.source_hash())
            _lib = handle
        return _lib


def _check(status: int, what: str, ctx: Optional["Context"] = None):
    if status != 0:
        detail = ""
        if ctx is not None and ctx.handle:
            detail = lib().autoloco_last_error(ctx.handle).decode()
        raise AutolocoError(status, what, detail)


# ----------------------------------------------------------------- context --
class Context:
    """An autoloco_ctx bound to one device and one HIP stream."""

    def __init__(self, device: int = 0, stream=None):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("the AutoLoCo round library needs a GPU; none is visible")
        if stream is None:
            stream = torch.cuda.current_stream(device)
        self.stream = stream
        raw = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
        h = C.c_void_p()
        _check(lib().autoloco_create(device, C.c_void_p(raw), C.byref(h)), "autoloco_create")
        self.handle = h
        self.device = device
        # spread buffers not yet freed; while there are any, close() detaches the
        # handle from the API but keeps the native context for their frees
        self._live = 0
        self._held = None

    def close(self):
        h = getattr(self, "handle", None)
        if h:
            self.handle = None
            if self._live:
                self._held = h
            else:
                lib().autoloco_destroy(h)

    def _buffer_freed(self):
        self._live -= 1
        if self._live == 0 and self._held is not None:
            h, self._held = self._held, None
            lib().autoloco_destroy(h)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def autoloco_create(device: int = 0, stream=None) -> Context:
    return Context(device, stream)


def autoloco_destroy(ctx: Context) -> None:
    ctx.close()


def autoloco_last_error(ctx: Context) -> str:
    return lib().autoloco_last_error(ctx.handle).decode()


def autoloco_set_timing(ctx: Context, enable: bool) -> None:
    _check(lib().autoloco_set_timing(ctx.handle, int(bool(enable))), "autoloco_set_timing", ctx)


def autoloco_last_kernel_ms(ctx: Context) -> float:
    ms = C.c_float()
    _check(lib().autoloco_last_kernel_ms(ctx.handle, C.byref(ms)), "autoloco_last_kernel_ms", ctx)
    return ms.value


def autoloco_set_grid_limit(ctx: Context, max_blocks: int) -> None:
    _check(lib().autoloco_set_grid_limit(ctx.handle, int(max_blocks)), "autoloco_set_grid_limit", ctx)


def autoloco_launch_shape(ctx: Context, n: int, k: int, replica_dtype: int = F32):
    b, t = C.c_int32(), C.c_int32()
    _check(lib().autoloco_launch_shape(ctx.handle, int(n), int(k), int(replica_dtype), C.byref(b), C.byref(t)),
           "autoloco_launch_shape", ctx)
    return b.value, t.value


# -------------------------------------------------------------- placement --
_TYPESTR = {"float32": "<f4", "bfloat16": "<V2"}


class _DeviceBuffer:
    """Owner of one autoloco_alloc_spread buffer; exposes it to torch through
    __cuda_array_interface__ and frees it when the last view is gone."""

    def __init__(self, ctx: "Context", ptr: int, nbytes: int):
        self._ctx = ctx
        self.ptr = ptr
        self.nbytes = nbytes
        ctx._live += 1

    def view(self, n: int, dtype):
        import torch
        if dtype == torch.float32:
            cai = {"shape": (n,), "typestr": "<f4", "data": (self.ptr, False), "version": 2, "strides": None}
            holder = type("_Cai", (), {})()
            holder.__cuda_array_interface__ = cai
            holder.owner = self
            return torch.as_tensor(holder, device=f"cuda:{self._ctx.device}")
        if dtype == torch.bfloat16:
            # bf16 has no array-interface type string: view the bytes as int16, then reinterpret
            cai = {"shape": (n,), "typestr": "<i2", "data": (self.ptr, False), "version": 2, "strides": None}
            holder = type("_Cai", (), {})()
            holder.__cuda_array_interface__ = cai
            holder.owner = self
            return torch.as_tensor(holder, device=f"cuda:{self._ctx.device}").view(torch.bfloat16)
        raise TypeError(dtype)

    def __del__(self):
        ptr, self.ptr = self.ptr, 0
        if not ptr:
            return
        ctx = self._ctx
        try:
            h = ctx.handle or ctx._held
            if h:
                lib().autoloco_free(h, C.c_void_p(ptr))
        except Exception:
            pass
        ctx._buffer_freed()


def autoloco_alloc_spread(ctx: "Context", count: int, nbytes: int):
    """Raw pointers of `count` buffers of `nbytes`, spread in physical memory,
    and whether spreading was possible."""
    out = (C.c_void_p * count)()
    spread = C.c_int32(0)
    _check(lib().autoloco_alloc_spread(ctx.handle, int(count), int(nbytes), out, C.byref(spread)),
           "autoloco_alloc_spread", ctx)
    return [int(p) for p in out], bool(spread.value)


def autoloco_free(ctx: "Context", ptr: int) -> None:
    _check(lib().autoloco_free(ctx.handle, C.c_void_p(ptr)), "autoloco_free", ctx)


def spread_tensors(ctx: "Context", n: int, dtypes):
    """torch tensors of n elements each (one per dtype in `dtypes`), backed by
    autoloco_alloc_spread memory; each frees its memory when collected."""
    import torch
    sizes = [n * (4 if d == torch.float32 else 2) for d in dtypes]
    ptrs, spread = autoloco_alloc_spread(ctx, len(dtypes), max(max(sizes), 16))
    out = []
    for p, d, nb in zip(ptrs, dtypes, sizes):
        out.append(_DeviceBuffer(ctx, p, nb).view(n, d))
    return out, spread


# ----------------------------------------------------------- marshalling --
def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"replicas must be float32 or bfloat16, got {t.dtype}")


def make_buffers(theta, replicas: Sequence, momentum=None, n: Optional[int] = None) -> Buffers:
    """Describe caller-owned device tensors to the library (no copies)."""
    import torch
    reps = list(replicas)
    if not 1 <= len(reps) <= MAX_K:
        raise ValueError(f"need 1..{MAX_K} replicas, got {len(reps)}")
    ts = [theta] + reps + ([momentum] if momentum is not None else [])
    for t in ts:
        if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
            raise TypeError("all buffers must be CUDA (HIP) tensors")
        if not t.is_contiguous():
            raise ValueError("all buffers must be contiguous")
    if theta.dtype != torch.float32 or (momentum is not None and momentum.dtype != torch.float32):
        raise TypeError("theta and momentum must be float32")
    code = _dtype_code(reps[0])
    if any(_dtype_code(r) != code for r in reps):
        raise TypeError("all replicas must share one dtype")
    count = theta.numel() if n is None else int(n)
    if any(t.numel() < count for t in ts):
        raise ValueError("a buffer is shorter than n")
    b = Buffers()
    b.n = count
    b.k = len(reps)
    b.replica_dtype = code
    b.theta = theta.data_ptr()
    b.momentum = momentum.data_ptr() if momentum is not None else None
    for i, r in enumerate(reps):
        b.replicas[i] = r.data_ptr()
    return b


def make_coeffs(mu: float, eta_out: float, rho: float = 1.0, normalize: bool = False,
                kappa: float = float("nan")) -> OuterCoeffs:
    c = OuterCoeffs()
    c.mu, c.eta_out, c.rho, c.kappa, c.normalize = mu, eta_out, rho, kappa, int(bool(normalize))
    return c


def autoloco_round_stats(ctx: Context, theta, replicas, eps: float = 1e-12, n=None) -> Stats:
    b = make_buffers(theta, replicas, None, n)
    out = Stats()
    _check(lib().autoloco_round_stats(ctx.handle, C.byref(b), eps, C.byref(out)), "autoloco_round_stats", ctx)
    return out


def autoloco_outer_step(ctx: Context, theta, momentum, replicas, coeffs: OuterCoeffs,
                        flags: int = FUSE_STATS | FUSE_RESET, eps: float = 1e-12, n=None) -> Optional[Stats]:
    b = make_buffers(theta, replicas, momentum, n)
    out = Stats()
    _check(lib().autoloco_outer_step(ctx.handle, C.byref(b), C.byref(coeffs), flags, eps,
                                     C.byref(out) if flags & FUSE_STATS else None),
           "autoloco_outer_step", ctx)
    return out if flags & FUSE_STATS else None


def autoloco_outer_step_static(theta, momentum, replicas, coeffs: OuterCoeffs, flags: int = FUSE_STATS | FUSE_RESET,
                               eps: float = 1e-12, device: Optional[int] = None, stream=None, n=None) -> Optional[Stats]:
    """autoloco_outer_step without a context: the library allocates nothing
    (its reduction scratch is a static device array)."""
    import torch
    b = make_buffers(theta, replicas, momentum, n)
    if device is None:
        device = theta.device.index if theta.device.index is not None else torch.cuda.current_device()
    if stream is None:
        # an ordinal torch does not know goes to the library as is (it rejects it)
        stream = torch.cuda.current_stream(device) if 0 <= device < torch.cuda.device_count() else 0
    raw = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    st = Stats()
    status = lib().autoloco_outer_step_static(int(device), C.c_void_p(raw), C.byref(b), C.byref(coeffs),
                                              int(flags), float(eps), C.byref(st))
    if status != 0:
        raise AutolocoError(status, "autoloco_outer_step_static")
    return st if flags & FUSE_STATS else None


def autoloco_outer_step_int8(ctx: Context, theta, momentum, replicas, coeffs: OuterCoeffs,
                             flags: int = FUSE_STATS | FUSE_RESET, eps: float = 1e-12, n=None,
                             mean_codes=None, mean_scales=None) -> Optional[Stats]:
    """The corrected step with the worker average taken through the INT8 codec."""
    import torch
    b = make_buffers(theta, replicas, momentum, n)
    if (mean_codes is None) != (mean_scales is None):
        raise ValueError("pass both payload buffers or neither")
    if mean_codes is not None:
        if mean_codes.dtype != torch.int8 or mean_scales.dtype != torch.float32:
            raise TypeError("mean_codes must be int8 and mean_scales float32")
        if mean_codes.device.type != "cuda" or mean_scales.device.type != "cuda":
            raise TypeError("payload buffers must be device tensors")
        nb = (b.n + 4095) // 4096
        if mean_codes.numel() < b.n or mean_scales.numel() < nb:
            raise ValueError("payload buffers too short")
    out = Stats()
    _check(lib().autoloco_outer_step_int8(ctx.handle, C.byref(b), C.byref(coeffs), flags, eps,
                                          C.byref(out) if flags & FUSE_STATS else None,
                                          C.c_void_p(mean_codes.data_ptr()) if mean_codes is not None else None,
                                          C.c_void_p(mean_scales.data_ptr()) if mean_scales is not None else None),
           "autoloco_outer_step_int8", ctx)
    return out if flags & FUSE_STATS else None


def autoloco_outer_step_bf16(ctx: Context, theta, momentum, replicas, coeffs: OuterCoeffs,
                             flags: int = FUSE_STATS | FUSE_RESET, eps: float = 1e-12, mean_bf16=None,
                             n=None) -> Optional[Stats]:
    """The round with BF16 pseudo-gradient payloads; mean_bf16 (a bfloat16 tensor
    of at least n elements) receives the mean every worker receives."""
    import torch
    b = make_buffers(theta, replicas, momentum, n)
    if mean_bf16 is not None:
        if not isinstance(mean_bf16, torch.Tensor) or mean_bf16.device.type != "cuda" \
                or mean_bf16.dtype != torch.bfloat16 or not mean_bf16.is_contiguous() or mean_bf16.numel() < b.n:
            raise ValueError("mean_bf16 must be a contiguous CUDA bfloat16 tensor of at least n elements")
    st = Stats() if flags & FUSE_STATS else None
    _check(lib().autoloco_outer_step_bf16(ctx.handle, C.byref(b), C.byref(coeffs), int(flags), float(eps),
                                          C.byref(st) if st is not None else None,
                                          C.c_void_p(mean_bf16.data_ptr()) if mean_bf16 is not None else None),
           "autoloco_outer_step_bf16", ctx)
    return st


def _cuda_contig(t, dtype, n, what):
    import torch
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or not t.is_contiguous() or t.dtype != dtype:
        raise TypeError(f"{what} must be a contiguous CUDA {dtype} tensor")
    if t.numel() < n:
        raise ValueError(f"{what} is shorter than n")
    return t.data_ptr()


def autoloco_rank_payload(ctx: Context, theta, replica, payload, sq_norm: bool = True, n=None):
    """One worker's BF16 payload (into `payload`) and ||Delta_r||^2 (or None)."""
    import torch
    count = theta.numel() if n is None else int(n)
    code = _dtype_code(replica)
    out = C.c_double() if sq_norm else None
    _check(lib().autoloco_rank_payload(ctx.handle, count, _cuda_contig(theta, torch.float32, count, "theta"),
                                       _cuda_contig(replica, replica.dtype, count, "replica"), code,
                                       _cuda_contig(payload, torch.bfloat16, count, "payload"),
                                       C.byref(out) if out is not None else None), "autoloco_rank_payload", ctx)
    return out.value if out is not None else None


def autoloco_shard_step(ctx: Context, theta, momentum, payloads: Sequence, coeffs: OuterCoeffs, mean_bf16=None,
                        sq_mean: bool = True, n=None):
    """The received mean and the corrected step on one shard; returns the shard's ||mean||^2 (or None)."""
    import torch
    count = theta.numel() if n is None else int(n)
    if not 1 <= len(payloads) <= MAX_K:
        raise ValueError(f"need 1..{MAX_K} payload shards")
    b = ShardBuffers()
    b.n = count
    b.k = len(payloads)
    b.theta = _cuda_contig(theta, torch.float32, count, "theta")
    b.momentum = _cuda_contig(momentum, torch.float32, count, "momentum")
    for i, p in enumerate(payloads):
        b.payloads[i] = _cuda_contig(p, torch.bfloat16, count, "payload")
    mp = _cuda_contig(mean_bf16, torch.bfloat16, count, "mean_bf16") if mean_bf16 is not None else None
    out = C.c_double() if sq_mean else None
    _check(lib().autoloco_shard_step(ctx.handle, C.byref(b), C.byref(coeffs), mp,
                                     C.byref(out) if out is not None else None), "autoloco_shard_step", ctx)
    return out.value if out is not None else None


def autoloco_broadcast_reset(ctx: Context, theta, replicas, n=None) -> None:
    b = make_buffers(theta, replicas, None, n)
    _check(lib().autoloco_broadcast_reset(ctx.handle, C.byref(b)), "autoloco_broadcast_reset", ctx)


def autoloco_traffic_reference(ctx: Context, theta, momentum, replicas, n=None) -> None:
    """The fused round's loads and stores without its arithmetic (buffers unchanged)."""
    b = make_buffers(theta, replicas, momentum, n)
    _check(lib().autoloco_traffic_reference(ctx.handle, C.byref(b)), "autoloco_traffic_reference", ctx)


# -------------------------------------------------------- host scalars --
PROBE_READ, PROBE_WRITE = 1, 2
PROBE_RUN1, PROBE_RUN2, PROBE_SERIAL, PROBE_TILE, PROBE_PHASED, PROBE_RUN8 = 0, 1, 2, 3, 4, 5


def autoloco_traffic_probe(ctx: Context, streams: Sequence, shape: int = PROBE_RUN1, blocks: int = 0,
                           n: Optional[int] = None) -> float:
    """Streaming-pattern probe: streams is a sequence of (tensor, access) with
    access PROBE_READ, PROBE_WRITE or both; returns the bytes moved."""
    import torch
    if not streams:
        raise ValueError("no streams")
    if n is None:
        n = streams[0][0].numel()
    arr = (ProbeStream * len(streams))()
    for i, (t, access) in enumerate(streams):
        if not t.is_cuda or not t.is_contiguous() or t.numel() < n:
            raise ValueError(f"stream {i}: need a contiguous device tensor of at least {n} elements")
        if t.dtype not in (torch.float32, torch.bfloat16, torch.int32, torch.int16):
            raise TypeError(f"stream {i}: 4- or 2-byte elements only")
        arr[i] = ProbeStream(t.data_ptr(), t.element_size(), int(access))
    moved = C.c_double()
    _check(lib().autoloco_traffic_probe(ctx.handle, int(n), arr, len(streams), int(shape), int(blocks),
                                        C.byref(moved)), "autoloco_traffic_probe", ctx)
    return moved.value


def autoloco_build_id() -> str:
    return lib().autoloco_build_id().decode()


def make_adamw_coeffs(lr: float, step: int, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1,
                      max_grad_norm=1.0) -> AdamWCoeffs:
    """Settings of one inner step (defaults: the C4 recipe)."""
    return AdamWCoeffs(float(lr), float(beta1), float(beta2), float(eps), float(weight_decay),
                       float(max_grad_norm), int(step))


def make_adamw_buffers(params: Sequence, exp_avg: Sequence, exp_avg_sq: Sequence, grads: Sequence,
                       model_bf16: Optional[Sequence] = None, n: Optional[int] = None) -> AdamWBuffers:
    """Describe the workers' caller-owned device tensors to the library (no copies)."""
    import torch
    k = len(params)
    if not 1 <= k <= MAX_K:
        raise ValueError(f"need 1..{MAX_K} workers, got {k}")
    groups = [list(params), list(exp_avg), list(exp_avg_sq), list(grads)]
    if any(len(g) != k for g in groups) or (model_bf16 is not None and len(model_bf16) != k):
        raise ValueError("every per-worker list needs one tensor per worker")
    count = params[0].numel() if n is None else int(n)
    for g in groups:
        for t in g:
            if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or not t.is_contiguous():
                raise TypeError("all buffers must be contiguous CUDA (HIP) tensors")
            if t.dtype != torch.float32:
                raise TypeError("params, moments and gradients must be float32")
            if t.numel() < count:
                raise ValueError("a buffer is shorter than n")
    b = AdamWBuffers()
    b.n = count
    b.k = k
    for i in range(k):
        b.params[i] = params[i].data_ptr()
        b.exp_avg[i] = exp_avg[i].data_ptr()
        b.exp_avg_sq[i] = exp_avg_sq[i].data_ptr()
        b.grads[i] = grads[i].data_ptr()
        if model_bf16 is not None:
            t = model_bf16[i]
            if t.dtype != torch.bfloat16 or not t.is_contiguous() or t.numel() < count:
                raise TypeError("model_bf16 must be contiguous bfloat16 tensors of at least n elements")
            b.model_bf16[i] = t.data_ptr()
    return b


def autoloco_inner_adamw(ctx: Context, params, exp_avg, exp_avg_sq, grads, coeffs: AdamWCoeffs,
                         model_bf16=None, stats: bool = True, n=None) -> Optional[AdamWStats]:
    """One AdamW step of every worker; returns the gradient norms (stats=True)
    or None (asynchronous on the context's stream)."""
    b = make_adamw_buffers(params, exp_avg, exp_avg_sq, grads, model_bf16, n)
    out = AdamWStats() if stats else None
    _check(lib().autoloco_inner_adamw(ctx.handle, C.byref(b), C.byref(coeffs),
                                      C.byref(out) if out is not None else None), "autoloco_inner_adamw", ctx)
    return out


def autoloco_adamw_traffic_reference(ctx: Context, params, exp_avg, exp_avg_sq, grads, model_bf16=None,
                                     n=None) -> None:
    """The AdamW update pass's loads and stores without its arithmetic (a
    measurement: every buffer keeps what the last step left in it)."""
    b = make_adamw_buffers(params, exp_avg, exp_avg_sq, grads, model_bf16, n)
    _check(lib().autoloco_adamw_traffic_reference(ctx.handle, C.byref(b)), "autoloco_adamw_traffic_reference", ctx)


def autoloco_last_adamw_ms(ctx: Context):
    """(norm pass ms, update pass ms) of the last timed AdamW step."""
    a, b = C.c_float(), C.c_float()
    _check(lib().autoloco_last_adamw_ms(ctx.handle, C.byref(a), C.byref(b)), "autoloco_last_adamw_ms", ctx)
    return a.value, b.value


def make_schedule(peak=4e-4, min_lr=0.0, warmup=1000, total=50_000) -> Schedule:
    s = Schedule()
    s.peak, s.min_lr, s.warmup, s.total = peak, min_lr, warmup, total
    return s


def autoloco_inner_lr(sched: Schedule, step: int) -> float:
    return lib().autoloco_inner_lr(C.byref(sched), step)


def autoloco_lr_mass(sched: Schedule, start_step: int, steps: int) -> float:
    return lib().autoloco_lr_mass(C.byref(sched), start_step, steps)


def make_outer_cfg(eta_base=0.7, mu_base=0.9, mu_min=0.45, mu_max=0.90, kappa_max=1.6,
                   eps=1e-12, normalize=False) -> OuterCfg:
    c = OuterCfg()
    c.eta_base, c.mu_base, c.mu_min, c.mu_max = eta_base, mu_base, mu_min, mu_max
    c.kappa_max, c.eps, c.normalize = kappa_max, eps, int(bool(normalize))
    return c


def autoloco_outer_correction(cfg: OuterCfg, lambda_sel: float, lambda_base: float) -> OuterCoeffs:
    out = OuterCoeffs()
    _check(lib().autoloco_outer_correction(C.byref(cfg), lambda_sel, lambda_base, C.byref(out)),
           "autoloco_outer_correction")
    return out


def default_controller_cfg(**overrides) -> ControllerCfg:
    c = ControllerCfg()
    lib().autoloco_controller_default_cfg(C.byref(c))
    for key, val in overrides.items():
        if key == "sched":
            c.sched = val
        elif key == "outer":
            c.outer = val
        else:
            setattr(c, key, val)
    return c


class Controller:
    """An autoloco_controller."""

    def __init__(self, cfg: Optional[ControllerCfg] = None):
        cfg = cfg if cfg is not None else default_controller_cfg()
        h = C.c_void_p()
        _check(lib().autoloco_controller_create(C.byref(cfg), C.byref(h)), "autoloco_controller_create")
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            lib().autoloco_controller_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def autoloco_controller_create(cfg: Optional[ControllerCfg] = None) -> Controller:
    return Controller(cfg)


def make_observation(D, C_, lambda_done, tokens, h_step_done, finite=True) -> Observation:
    o = Observation()
    o.D, o.C, o.lambda_done, o.tokens = D, C_, lambda_done, tokens
    o.h_step_done, o.finite = int(h_step_done), int(bool(finite))
    return o


def autoloco_select_interval(ctrl: Controller, obs: Optional[Observation]) -> Decision:
    out = Decision()
    _check(lib().autoloco_select_interval(ctrl.handle, C.byref(obs) if obs is not None else None,
                                          C.byref(out)), "autoloco_select_interval")
    return out


def autoloco_controller_reference(ctrl: Controller):
    d, c, l = C.c_double(), C.c_double(), C.c_double()
    _check(lib().autoloco_controller_reference(ctrl.handle, C.byref(d), C.byref(c), C.byref(l)),
           "autoloco_controller_reference")
    return d.value, c.value, l.value


def autoloco_controller_save(ctrl: Controller) -> bytes:
    n = C.c_size_t(0)
    _check(lib().autoloco_controller_save(ctrl.handle, None, C.byref(n)), "autoloco_controller_save")
    buf = C.create_string_buffer(n.value)
    _check(lib().autoloco_controller_save(ctrl.handle, buf, C.byref(n)), "autoloco_controller_save")
    return buf.raw[: n.value]


def autoloco_controller_load(ctrl: Controller, blob: bytes) -> None:
    buf = C.create_string_buffer(blob, len(blob))
    _check(lib().autoloco_controller_load(ctrl.handle, buf, len(blob)), "autoloco_controller_load")
