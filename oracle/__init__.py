"""ORACLE — test infrastructure only.

Python access to the plain single-threaded C reference in ``oracle.c``.  Only
the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg use
it.  It shares no code with the GPU library: its own struct layout, its own
policy and flag numbers, its own build.

Policies: "fcfs", "ljf", "isjl", "sjf".  ``alpha=ALPHA_INF`` is an infinite
fairness budget; ``B=0`` and ``M_kv=0`` mean "no limit".
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

ALPHA_INF = 2**31 - 1
POLICIES = {"fcfs": 0, "ljf": 1, "isjl": 2, "sjf": 3}
FLAG_BETA_SQRT17 = 8
FLAG_RESUME_FILL = 16
FLAG_PREFILL = 32  # prompt prefilled at admission: service = output, footprint prompt + progress

METRIC_FIELDS = ["T", "O", "Q", "E", "C", "W", "sum_completion", "sum_latency",
                 "sum_extent", "busy_steps", "peak_kv", "unfair_steps",
                 "max_extent", "max_active"]
METRICS_DTYPE = np.dtype([(f, np.int64) for f in METRIC_FIELDS[:12]] +
                         [("max_extent", np.int32), ("max_active", np.int32)])
assert METRICS_DTYPE.itemsize == 104

ERRORS = {0: "ok", -1: "invalid argument", -2: "value out of range", -3: "out of memory",
          -5: "instance too large", -7: "internal error (step bound exceeded)"}

_lib = None


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"oracle error {code}: {ERRORS.get(code, 'unknown')}")
        self.code = code


def build(force: bool = True) -> str:
    global _lib
    if force or not os.path.exists(_LIB):
        subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-o", _LIB + ".tmp",
                        _SRC, "-lm"], check=True)
        os.replace(_LIB + ".tmp", _LIB)
        _lib = None
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(True)
        lib = ctypes.CDLL(_LIB)
        P, I32, I64, U32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
        lib.oracle_simulate_batch.argtypes = [I64, I32, P, P, P, I32, I32, I64, I32, U32, I64,
                                              I64, P, P, P]
        lib.oracle_simulate_robust_batch.argtypes = [I64, I32, P, P, P, P, I32, I32, I64, I32,
                                                     U32, I64, I64, P, P, P]
        lib.oracle_decompose.argtypes = [I32, P, P, P, I32, I32, I64, I64, I64, P, P, P]
        lib.oracle_opt_batch.argtypes = [I64, I32, P, P, P, I32, I32, I64, P, P]
        for f in (lib.oracle_simulate_batch, lib.oracle_simulate_robust_batch,
                  lib.oracle_decompose, lib.oracle_opt_batch):
            f.restype = ctypes.c_int
        lib.oracle_pack_scans_take.restype = ctypes.c_int64
        lib.oracle_pack_scans_take.argtypes = []
        assert lib.oracle_metrics_size() == 104
        _lib = lib
    return _lib


def _tables(arrival, prompt, output):
    a = np.ascontiguousarray(arrival, dtype=np.int32)
    p = np.ascontiguousarray(prompt, dtype=np.int32)
    o = np.ascontiguousarray(output, dtype=np.int32)
    if a.ndim == 1:
        a, p, o = a[None], p[None], o[None]
    assert a.shape == p.shape == o.shape and a.ndim == 2
    return a, p, o


def _ptr(x):
    return None if x is None else x.ctypes.data


def simulate(arrival, prompt, output, *, policy: str, B: int, alpha: int, M_kv: int = 0,
             cost_c: int = 0, cost_tau: int = 1, flags: int = 0, schedule: bool = False):
    """Simulate every row (instance).  Returns metrics (structured array) and,
    with ``schedule=True``, also (start, finish) int32 arrays."""
    a, p, o = _tables(arrival, prompt, output)
    n_inst, n = a.shape
    out = np.zeros(n_inst, dtype=METRICS_DTYPE)
    st = np.empty((n_inst, n), np.int32) if schedule else None
    fi = np.empty((n_inst, n), np.int32) if schedule else None
    rc = _load().oracle_simulate_batch(n_inst, n, a.ctypes.data, p.ctypes.data, o.ctypes.data,
                                       B, alpha, M_kv, POLICIES[policy], flags, cost_c,
                                       cost_tau, out.ctypes.data, _ptr(st), _ptr(fi))
    if rc:
        raise OracleError(rc)
    return (out, st, fi) if schedule else out


def pack_scans_take() -> int:
    """Pack candidates Phase ONE examined on this thread since the last call."""
    return int(_load().oracle_pack_scans_take())


def simulate_robust(arrival, prompt, output, upper, *, policy: str = "isjl", B: int,
                    alpha: int, M_kv: int = 0, cost_c: int = 0, cost_tau: int = 1,
                    flags: int = 0, schedule: bool = False):
    """Simulate with planning sizes prompt + upper (Section 3.4; upper >= output):
    ISJL gives Robust-ISJL.  Returns as ``simulate``."""
    a, p, o = _tables(arrival, prompt, output)
    u = np.ascontiguousarray(upper, dtype=np.int32).reshape(a.shape)
    n_inst, n = a.shape
    out = np.zeros(n_inst, dtype=METRICS_DTYPE)
    st = np.empty((n_inst, n), np.int32) if schedule else None
    fi = np.empty((n_inst, n), np.int32) if schedule else None
    rc = _load().oracle_simulate_robust_batch(n_inst, n, a.ctypes.data, p.ctypes.data,
                                              o.ctypes.data, u.ctypes.data, B, alpha, M_kv,
                                              POLICIES[policy], flags, cost_c, cost_tau,
                                              out.ctypes.data, _ptr(st), _ptr(fi))
    if rc:
        raise OracleError(rc)
    return (out, st, fi) if schedule else out


def decompose(arrival, prompt, output, start, *, B: int, alpha: int, M_kv: int = 0,
              cost_c: int = 0, cost_tau: int = 1):
    """Re-score given schedules.  Returns (metrics, violation_mask)."""
    a, p, o = _tables(arrival, prompt, output)
    s = np.ascontiguousarray(start, dtype=np.int32).reshape(a.shape)
    n_inst, n = a.shape
    out = np.zeros(n_inst, dtype=METRICS_DTYPE)
    viol = np.zeros(n_inst, dtype=np.uint32)
    lib = _load()
    for k in range(n_inst):
        rc = lib.oracle_decompose(n, a[k].ctypes.data, p[k].ctypes.data, o[k].ctypes.data, B,
                                  alpha, M_kv, cost_c, cost_tau, s[k].ctypes.data,
                                  out[k:k + 1].ctypes.data, viol[k:k + 1].ctypes.data)
        if rc:
            raise OracleError(rc)
    return out, viol


def opt(arrival, prompt, output, *, B: int, alpha: int, M_kv: int = 0, schedule: bool = False):
    """Exact alpha-fair optimum makespan per instance (n <= 8)."""
    a, p, o = _tables(arrival, prompt, output)
    n_inst, n = a.shape
    T = np.zeros(n_inst, dtype=np.int64)
    st = np.empty((n_inst, n), np.int32) if schedule else None
    rc = _load().oracle_opt_batch(n_inst, n, a.ctypes.data, p.ctypes.data, o.ctypes.data, B,
                                  alpha, M_kv, T.ctypes.data, _ptr(st))
    if rc:
        raise OracleError(rc)
    return (T, st) if schedule else T


# ---------------------------------------------------------------------------
# Sharded runs: the C oracle keeps no shared state, so contiguous instance
# ranges can run on several host threads at once (ctypes releases the GIL for
# the duration of each call).  Each thread runs the same single-threaded code
# on its own rows; results are identical to one call over all rows.

def host_threads(limit: int = 16) -> int:
    """Threads to use: the cores this process may run on, at most ``limit``."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(limit, n))


def _shards(n_inst: int, threads: int, chunk: int):
    step = max(1, min(chunk, -(-n_inst // (threads * 4))))
    return [(b, min(n_inst, b + step)) for b in range(0, n_inst, step)]


def simulate_parallel(arrival, prompt, output, *, threads: int, chunk: int = 256,
                      progress=None, **kw):
    """``simulate`` over contiguous instance shards on ``threads`` host threads."""
    from concurrent.futures import ThreadPoolExecutor
    a, p, o = _tables(arrival, prompt, output)
    n_inst, n = a.shape
    sched = kw.get("schedule", False)
    out = np.zeros(n_inst, dtype=METRICS_DTYPE)
    st = np.empty((n_inst, n), np.int32) if sched else None
    fi = np.empty((n_inst, n), np.int32) if sched else None

    def run(span):
        b, e = span
        r = simulate(a[b:e], p[b:e], o[b:e], **kw)
        if sched:
            out[b:e], st[b:e], fi[b:e] = r
        else:
            out[b:e] = r
        return e - b

    done = 0
    with ThreadPoolExecutor(max_workers=threads) as ex:
        for k in ex.map(run, _shards(n_inst, threads, chunk)):
            done += k
            if progress:
                progress(done, n_inst)
    return (out, st, fi) if sched else out


def opt_parallel(arrival, prompt, output, *, threads: int, chunk: int = 1024, progress=None,
                 **kw):
    """``opt`` over contiguous instance shards on ``threads`` host threads."""
    from concurrent.futures import ThreadPoolExecutor
    a, p, o = _tables(arrival, prompt, output)
    n_inst = a.shape[0]
    T = np.zeros(n_inst, dtype=np.int64)

    def run(span):
        b, e = span
        T[b:e] = opt(a[b:e], p[b:e], o[b:e], **kw)
        return e - b

    done = 0
    with ThreadPoolExecutor(max_workers=threads) as ex:
        for k in ex.map(run, _shards(n_inst, threads, chunk)):
            done += k
            if progress:
                progress(done, n_inst)
    return T
