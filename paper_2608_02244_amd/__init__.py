"""fsched — batched evaluation of resource-fair LLM batching on AMD MI355X.

Thin Python binding of ``libfsched.so`` (the C ABI declared in
``include/fsched.h``).  Every step of the evaluation runs in the library's HIP
kernels; this module only marshals arguments.  There is no CPU fallback: if the
library has not been built, every call raises.

Inputs may be torch tensors on a ROCm device (the call is enqueued on the
current torch stream; device-pointer mode) or numpy arrays (host mode: the
library stages through device memory and returns when results are back).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfsched.so")

ALPHA_INF = 2**31 - 1
UNLIMITED = 0
POLICIES = {"fcfs": 0, "ljf": 1, "isjl": 2, "sjf": 3}
F_DEVICE_PTRS, F_SYNC, F_BETA_SQRT17, F_RESUME_FILL, F_PREFILL = 1, 4, 8, 16, 32

OK, EINVAL, ERANGE, ENOMEM, EDEVICE, ETOOLARGE, ENOTIMPL, EINTERNAL = 0, -1, -2, -3, -4, -5, -6, -7
ESCRATCH = -8
NOALLOC_SCRATCH_BYTES = 64 << 20  # FSCHED_NOALLOC_SCRATCH_BYTES
T_INVALID, T_RANGE, T_TOOLARGE, T_INTERNAL = -1, -2, -5, -7

METRIC_FIELDS = ("T", "O", "Q", "E", "C", "W", "sum_completion", "sum_latency", "sum_extent",
                 "busy_steps", "peak_kv", "unfair_steps", "max_extent", "max_active")
METRICS_DTYPE = np.dtype([(f, np.int64) for f in METRIC_FIELDS[:12]] +
                         [("max_extent", np.int32), ("max_active", np.int32)])
METRICS_BYTES = 104
EXPORTS = ("fsched_simulate", "fsched_simulate_robust", "fsched_cost_decompose", "fsched_bruteforce_opt",
           "fsched_strerror", "fsched_abi_version", "fsched_last_hip_error",
           "fsched_release_cache", "fsched_simulate_noalloc")


class Params(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("alpha", ctypes.c_int32), ("M_kv", ctypes.c_int64),
                ("policy", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("cost_c", ctypes.c_int64), ("cost_tau", ctypes.c_int64)]


assert ctypes.sizeof(Params) == 40


class FschedError(RuntimeError):
    def __init__(self, code: int, what: str):
        msg = lib().fsched_strerror(code).decode()
        super().__init__(f"{what}: fsched error {code} ({msg})")
        self.code = code


_lib = None


def lib():
    """Load libfsched.so; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first "
                               "(there is no CPU fallback)")
        L = ctypes.CDLL(LIB_PATH)
        P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        L.fsched_simulate.argtypes = [P, I64, I32, P, P, P, P, P, P, P]
        L.fsched_simulate_noalloc.argtypes = [P, I64, I32, P, P, P, P, P, P, P]
        L.fsched_simulate_robust.argtypes = [P, I64, I32, P, P, P, P, P, P, P, P]
        L.fsched_cost_decompose.argtypes = [P, I64, I32, P, P, P, P, P, P, P]
        L.fsched_bruteforce_opt.argtypes = [P, I64, I32, P, P, P, P, P, P]
        for f in (L.fsched_simulate, L.fsched_simulate_noalloc, L.fsched_simulate_robust, L.fsched_cost_decompose, L.fsched_bruteforce_opt,
                  L.fsched_abi_version, L.fsched_last_hip_error, L.fsched_release_cache):
            f.restype = ctypes.c_int
        L.fsched_strerror.restype = ctypes.c_char_p
        L.fsched_strerror.argtypes = [ctypes.c_int]
        _lib = L
    return _lib


def release_cache() -> None:
    """Give the memory the library's scratch pool keeps between calls back to the
    current device (fsched_release_cache)."""
    rc = lib().fsched_release_cache()
    if rc:
        raise FschedError(rc, "fsched_release_cache")


def make_params(policy: str = "isjl", B: int = 0, alpha: int = ALPHA_INF, M_kv: int = 0,
                cost_c: int = 0, cost_tau: int = 1, beta_sqrt17: bool = False,
                device: bool = False, resume_fill: bool = False,
                prefill: bool = False) -> Params:
    flags = (F_DEVICE_PTRS if device else 0) | (F_BETA_SQRT17 if beta_sqrt17 else 0) | \
        (F_RESUME_FILL if resume_fill else 0) | (F_PREFILL if prefill else 0)
    return Params(B=B, alpha=alpha, M_kv=M_kv, policy=POLICIES[policy], flags=flags,
                  cost_c=cost_c, cost_tau=cost_tau)


def metrics_view(raw) -> np.ndarray:
    """Structured numpy view of raw metrics ([n_inst, 13] int64, torch or numpy)."""
    if hasattr(raw, "detach"):
        raw = raw.detach().cpu().numpy()
    raw = np.ascontiguousarray(raw)
    return raw.view(METRICS_DTYPE).reshape(-1)


def _is_torch(x) -> bool:
    return hasattr(x, "data_ptr") and hasattr(x, "is_cuda")


def _torch_tables(*tables):
    import torch
    ts = []
    for x in tables:
        if x.dtype != torch.int32 or not x.is_contiguous() or not x.is_cuda:
            raise ValueError("job tables must be contiguous int32 tensors on the GPU")
        ts.append(x if x.dim() == 2 else x.reshape(1, -1))
    if any(x.shape != ts[0].shape for x in ts):
        raise ValueError("job tables differ in shape")
    return ts


def _np_tables(*tables):
    out = []
    for x in tables:
        a = np.ascontiguousarray(x, dtype=np.int32)
        out.append(a if a.ndim == 2 else a.reshape(1, -1))
    if any(x.shape != out[0].shape for x in out):
        raise ValueError("job tables differ in shape")
    return out


def _stream_handle(torch, stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def simulate(arrival, prompt, output, *, policy: str, B: int, alpha: int, M_kv: int = 0,
             cost_c: int = 0, cost_tau: int = 1, beta_sqrt17: bool = False,
             resume_fill: bool = False, prefill: bool = False, schedule: bool = False,
             stream=None):
    """fsched_simulate over every row (instance) of the job tables (``prefill``:
    the prompt is prefilled at admission, FSCHED_F_PREFILL).

    Torch inputs: returns (metrics [n_inst, 13] int64 tensor, start, finish) with
    start/finish None unless ``schedule``; nothing is synchronised.
    Numpy inputs: returns (metrics structured array, start, finish) in host memory.
    """
    p = make_params(policy, B, alpha, M_kv, cost_c, cost_tau, beta_sqrt17,
                    device=_is_torch(arrival), resume_fill=resume_fill, prefill=prefill)
    return _simulate("fsched_simulate", p, (arrival, prompt, output), schedule, stream)


def simulate_noalloc(arrival, prompt, output, out, *, policy: str, B: int, alpha: int,
                     M_kv: int = 0, cost_c: int = 0, cost_tau: int = 1,
                     beta_sqrt17: bool = False, resume_fill: bool = False,
                     prefill: bool = False, start=None, finish=None, stream=None):
    """fsched_simulate_noalloc: ``simulate`` on torch device tensors into outputs
    the caller allocated beforehand (``out`` [n_inst, 13] int64; ``start`` /
    ``finish`` [n_inst, n_jobs] int32 or None); the library allocates nothing.
    Enqueued on ``stream`` (default: the current torch stream)."""
    import torch
    ts = _torch_tables(arrival, prompt, output)
    n_inst, n = ts[0].shape
    for name, x, shape, dt in (("out", out, (n_inst, 13), torch.int64),
                               ("start", start, (n_inst, n), torch.int32),
                               ("finish", finish, (n_inst, n), torch.int32)):
        if x is None and name != "out":
            continue
        if x is None or tuple(x.shape) != shape or x.dtype != dt or not x.is_contiguous() \
                or not x.is_cuda:
            raise ValueError(f"{name} must be a contiguous {dt} GPU tensor of shape {shape}")
    p = make_params(policy, B, alpha, M_kv, cost_c, cost_tau, beta_sqrt17, device=True,
                    resume_fill=resume_fill, prefill=prefill)
    rc = lib().fsched_simulate_noalloc(ctypes.byref(p), n_inst, n, *[x.data_ptr() for x in ts],
                                       out.data_ptr(),
                                       start.data_ptr() if start is not None else None,
                                       finish.data_ptr() if finish is not None else None,
                                       _stream_handle(torch, stream))
    if rc:
        raise FschedError(rc, "fsched_simulate_noalloc")
    return out, start, finish


def simulate_robust(arrival, prompt, output, upper, *, B: int, alpha: int, M_kv: int = 0,
                    cost_c: int = 0, cost_tau: int = 1, beta_sqrt17: bool = False,
                    resume_fill: bool = False, prefill: bool = False, schedule: bool = False,
                    stream=None):
    """fsched_simulate_robust: Robust-ISJL planned on prompt + upper (upper >= output).

    Same inputs and returns as ``simulate``; ``upper`` is shaped like the tables."""
    p = make_params("isjl", B, alpha, M_kv, cost_c, cost_tau, beta_sqrt17,
                    device=_is_torch(arrival), resume_fill=resume_fill, prefill=prefill)
    return _simulate("fsched_simulate_robust", p, (arrival, prompt, output, upper), schedule,
                     stream)


def _simulate(name, p, tables, schedule, stream):
    fn = getattr(lib(), name)
    if _is_torch(tables[0]):
        import torch
        ts = _torch_tables(*tables)
        n_inst, n = ts[0].shape
        out = torch.empty((n_inst, 13), dtype=torch.int64, device=ts[0].device)
        st = torch.empty((n_inst, n), dtype=torch.int32, device=ts[0].device) if schedule else None
        fi = torch.empty((n_inst, n), dtype=torch.int32, device=ts[0].device) if schedule else None
        rc = fn(ctypes.byref(p), n_inst, n, *[x.data_ptr() for x in ts], out.data_ptr(),
                st.data_ptr() if st is not None else None,
                fi.data_ptr() if fi is not None else None, _stream_handle(torch, stream))
        if rc:
            raise FschedError(rc, name)
        return out, st, fi
    ts = _np_tables(*tables)
    n_inst, n = ts[0].shape
    out = np.zeros(n_inst, dtype=METRICS_DTYPE)
    st = np.empty((n_inst, n), np.int32) if schedule else None
    fi = np.empty((n_inst, n), np.int32) if schedule else None
    rc = fn(ctypes.byref(p), n_inst, n, *[x.ctypes.data for x in ts], out.ctypes.data,
            st.ctypes.data if st is not None else None,
            fi.ctypes.data if fi is not None else None, None)
    if rc:
        raise FschedError(rc, name)
    return out, st, fi


def cost_decompose(arrival, prompt, output, start, *, B: int, alpha: int, M_kv: int = 0,
                   cost_c: int = 0, cost_tau: int = 1, stream=None):
    """fsched_cost_decompose: re-score schedules.  Returns (metrics, violation)."""
    p = make_params("fcfs", B, alpha, M_kv, cost_c, cost_tau, device=_is_torch(arrival))
    if _is_torch(arrival):
        import torch
        a, pr, o = _torch_tables(arrival, prompt, output)
        n_inst, n = a.shape
        if start.dtype != torch.int32 or not start.is_contiguous() or start.numel() != n_inst * n:
            raise ValueError("start must be a contiguous int32 tensor shaped like the tables")
        out = torch.empty((n_inst, 13), dtype=torch.int64, device=a.device)
        viol = torch.empty((n_inst,), dtype=torch.int32, device=a.device)
        rc = lib().fsched_cost_decompose(ctypes.byref(p), n_inst, n, a.data_ptr(), pr.data_ptr(),
                                         o.data_ptr(), start.data_ptr(), out.data_ptr(),
                                         viol.data_ptr(), _stream_handle(torch, stream))
        if rc:
            raise FschedError(rc, "fsched_cost_decompose")
        return out, viol
    a, pr, o = _np_tables(arrival, prompt, output)
    n_inst, n = a.shape
    s = np.ascontiguousarray(start, dtype=np.int32).reshape(n_inst, n)
    out = np.zeros(n_inst, dtype=METRICS_DTYPE)
    viol = np.zeros(n_inst, dtype=np.uint32)
    rc = lib().fsched_cost_decompose(ctypes.byref(p), n_inst, n, a.ctypes.data, pr.ctypes.data,
                                     o.ctypes.data, s.ctypes.data, out.ctypes.data,
                                     viol.ctypes.data, None)
    if rc:
        raise FschedError(rc, "fsched_cost_decompose")
    return out, viol


def bruteforce_opt(arrival, prompt, output, *, B: int, alpha: int, M_kv: int = 0,
                   schedule: bool = False, stream=None):
    """fsched_bruteforce_opt: exact alpha-fair optimum makespan (n_jobs <= 8)."""
    p = make_params("isjl", B, alpha, M_kv, device=_is_torch(arrival))
    if _is_torch(arrival):
        import torch
        a, pr, o = _torch_tables(arrival, prompt, output)
        n_inst, n = a.shape
        T = torch.empty((n_inst,), dtype=torch.int64, device=a.device)
        st = torch.empty((n_inst, n), dtype=torch.int32, device=a.device) if schedule else None
        rc = lib().fsched_bruteforce_opt(ctypes.byref(p), n_inst, n, a.data_ptr(),
                                         pr.data_ptr(), o.data_ptr(), T.data_ptr(),
                                         st.data_ptr() if st is not None else None,
                                         _stream_handle(torch, stream))
        if rc:
            raise FschedError(rc, "fsched_bruteforce_opt")
        return T, st
    a, pr, o = _np_tables(arrival, prompt, output)
    n_inst, n = a.shape
    T = np.zeros(n_inst, dtype=np.int64)
    st = np.empty((n_inst, n), np.int32) if schedule else None
    rc = lib().fsched_bruteforce_opt(ctypes.byref(p), n_inst, n, a.ctypes.data, pr.ctypes.data,
                                     o.ctypes.data, T.ctypes.data,
                                     st.ctypes.data if st is not None else None, None)
    if rc:
        raise FschedError(rc, "fsched_bruteforce_opt")
    return T, st


def build():
    """Compile libfsched.so in-tree (hipcc, gfx950)."""
    from . import buildlib as _b
    global _lib
    _lib = None
    return _b.build()
