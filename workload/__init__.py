"""Seeded synthetic workloads for the batched scheduling evaluator.

This module only produces inputs: integer job tables (arrival step, prompt
tokens, output tokens) drawn from seeded distributions, plus the scheduling
parameters each named workload is run with.  It holds none of the scheduling
method's arithmetic, so both the oracle and the GPU library can consume its
output without sharing any code with each other.

The job model follows the paper's statement of the problem (Section 2): each
request is a number of tokens processed one per step, here split into a prompt
and an output part; arrivals are release steps (the online setting of the
section on online arrivals).  The distributions of the five named workloads are
synthetic stand-ins shaped like the paper's workloads; none reproduces a
dataset.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB = os.path.join(_HERE, "libfsched_gen.so")

ALPHA_INF = 2**31 - 1  # "fairness budget = infinity"
UNLIMITED = 0          # B = 0 -> no count limit; M_kv = 0 -> no KV budget

DIST_UNIFORM, DIST_LOGNORMAL, DIST_PARETO, DIST_TWO_UNIFORM = 0, 1, 2, 3


class _Dist(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("p0", ctypes.c_double), ("p1", ctypes.c_double),
                ("a1", ctypes.c_int64), ("b1", ctypes.c_int64),
                ("a2", ctypes.c_int64), ("b2", ctypes.c_int64),
                ("lo", ctypes.c_int64), ("hi", ctypes.c_int64)]


class _Recipe(ctypes.Structure):
    _fields_ = [("cfg_tag", ctypes.c_uint64), ("seed", ctypes.c_uint64),
                ("rate", ctypes.c_double), ("prompt", _Dist), ("output", _Dist)]


def uniform(a: int, b: int) -> dict:
    return dict(kind=DIST_UNIFORM, a1=a, b1=b)


def lognormal(median: float, sigma: float, lo: int, hi: int) -> dict:
    return dict(kind=DIST_LOGNORMAL, p0=median, p1=sigma, lo=lo, hi=hi)


def pareto(shape: float, xmin: float, cap: int) -> dict:
    return dict(kind=DIST_PARETO, p0=shape, p1=xmin, hi=cap)


def two_uniform(p: float, a1: int, b1: int, a2: int, b2: int) -> dict:
    return dict(kind=DIST_TWO_UNIFORM, p0=p, a1=a1, b1=b1, a2=a2, b2=b2)


def _mk_dist(d: dict) -> _Dist:
    out = _Dist()
    for k, v in d.items():
        setattr(out, k, v)
    return out


@dataclass(frozen=True)
class Workload:
    """A named synthetic workload and the scheduling parameters it runs with."""
    name: str
    tag: int
    n_inst: int
    n_jobs: int
    rate: float                      # Poisson arrivals per step (0: all at step 0)
    prompt: dict
    output: dict
    B: int                           # batch capacity (count of requests)
    M_kv: int                        # KV reservation budget in tokens (0: none)
    alphas: Tuple[int, ...]          # fairness budgets to evaluate
    cost_c: int                      # fixed cost per step (integer units)
    cost_tau: int                    # footprint coefficient (integer units)
    policies: Tuple[str, ...]
    seed: int = 0
    note: str = ""


# The five named workloads.  B, the cost coefficients of the last three and the
# seeds are not fixed by the workload descriptions; the values below are the
# readings recorded in the design notes (B near M_kv / E[len] so that both the
# count guard and the KV guard bind at times).
WORKLOADS: Dict[str, Workload] = {w.name: w for w in [
    Workload("uniform_256x64", 1, 256, 64, 0.0, uniform(1, 16), uniform(1, 32),
             B=8, M_kv=256, alphas=(8,), cost_c=0, cost_tau=1,
             policies=("fcfs", "ljf", "isjl"),
             note="offline; step cost = max active footprint"),
    Workload("lognormal_4096x1000", 2, 4096, 1000, 2.0,
             lognormal(512.0, 1.0, 1, 8192), lognormal(200.0, 1.1, 1, 4096),
             B=64, M_kv=65536, alphas=(64,), cost_c=1000, cost_tau=1,
             policies=("fcfs", "ljf", "isjl")),
    Workload("bimodal_sweep_4096x2000", 3, 4096, 2000, 4.0,
             uniform(32, 2048), two_uniform(0.8, 16, 128, 1024, 4096),
             B=128, M_kv=262144, alphas=(0, 16, 64, 256, 1024, ALPHA_INF),
             cost_c=1000, cost_tau=1, policies=("isjl", "fcfs", "ljf")),
    Workload("pareto_65536x2000", 4, 65536, 2000, 8.0,
             lognormal(1024.0, 0.8, 1, 16384), pareto(1.5, 8.0, 8192),
             B=512, M_kv=1048576, alphas=(128,), cost_c=1000, cost_tau=1,
             policies=("isjl",), note="throughput benchmark"),
    Workload("tiny_opt_1048576x8", 5, 1048576, 8, 0.0,
             uniform(1, 4), two_uniform(0.5, 1, 1, 1, 16),
             B=2, M_kv=16, alphas=(1, 2, 4), cost_c=0, cost_tau=1,
             policies=("isjl",), note="exact optimum by exhaustive search; "
             "also evaluated with no KV budget"),
    # Shaped like the conversation sample of the paper's system-efficiency
    # section (2,000 requests; total tokens with mean 126, median 90, max 905):
    # total tokens LN(median 90, sigma 0.82) clipped to 1..905 (mean 126), all in
    # the output column; Poisson arrivals at 0.25 requests per step (twice the
    # service rate of B = 16 at the mean length).  A synthetic stand-in, not the
    # dataset.
    Workload("lmsys_shaped_256x2000", 6, 256, 2000, 0.25, uniform(0, 0),
             lognormal(90.0, 0.82, 1, 905), B=16, M_kv=0, alphas=(50, 100, 150),
             cost_c=0, cost_tau=1, policies=("fcfs", "sjf", "ljf", "isjl"),
             note="system-efficiency table shape; B = 16 and 32"),
]}

WORKLOAD_ORDER: List[str] = list(WORKLOADS)

_lib = None


def _build() -> None:
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)


def build(force: bool = True) -> str:
    """Compile the generator library in-tree."""
    global _lib
    if force or not os.path.exists(_LIB):
        _build()
        _lib = None
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            _build()
        lib = ctypes.CDLL(_LIB)
        lib.gen_jobs.restype = ctypes.c_int
        lib.gen_jobs.argtypes = [ctypes.POINTER(_Recipe), ctypes.c_int64, ctypes.c_int64,
                                 ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p]
        _lib = lib
    return _lib


def generate(w: Workload | str, n_inst: Optional[int] = None, inst_begin: int = 0,
             n_jobs: Optional[int] = None):
    """Return (arrival, prompt, output), each int32 [n_inst, n_jobs], C-contiguous.

    Instances are generated independently: rows for instances
    inst_begin .. inst_begin + n_inst - 1 are identical whether they are drawn
    alone or as part of the full table.
    """
    if isinstance(w, str):
        w = WORKLOADS[w]
    n_inst = w.n_inst if n_inst is None else int(n_inst)
    n_jobs = w.n_jobs if n_jobs is None else int(n_jobs)
    rec = _Recipe(cfg_tag=w.tag, seed=w.seed, rate=w.rate,
                  prompt=_mk_dist(w.prompt), output=_mk_dist(w.output))
    arr = np.empty((n_inst, n_jobs), dtype=np.int32)
    pro = np.empty((n_inst, n_jobs), dtype=np.int32)
    out = np.empty((n_inst, n_jobs), dtype=np.int32)
    if n_inst == 0:
        return arr, pro, out
    rc = _load().gen_jobs(ctypes.byref(rec), inst_begin, n_inst, n_jobs,
                          arr.ctypes.data, pro.ctypes.data, out.ctypes.data)
    if rc != 0:
        raise ValueError(f"generator rejected recipe for {w.name}")
    return arr, pro, out


def random_tables(rng: np.random.Generator, n_inst: int, n_jobs: int, max_prompt: int,
                  max_output: int, max_arrival: int = 0, sorted_arrivals: bool = False):
    """Small random job tables for property tests (numpy Generator, seeded by caller)."""
    pro = rng.integers(0, max_prompt + 1, size=(n_inst, n_jobs), dtype=np.int32)
    out = rng.integers(1, max_output + 1, size=(n_inst, n_jobs), dtype=np.int32)
    if max_arrival > 0:
        arr = rng.integers(0, max_arrival + 1, size=(n_inst, n_jobs), dtype=np.int32)
        if sorted_arrivals:
            arr = np.sort(arr, axis=1).astype(np.int32)
    else:
        arr = np.zeros((n_inst, n_jobs), dtype=np.int32)
    return np.ascontiguousarray(arr), np.ascontiguousarray(pro), np.ascontiguousarray(out)


# ---------------------------------------------------------------------------
# The linear-pricing experiment of the paper's numerical section on profit and
# cost alignment: n potential requests with lengths uniform on 1..o_max, each
# quoted p0 * o (p0 = p / 500); a request in length bucket b (ten buckets of
# width o_max / 10) accepts with probability max(0, 1 - k_b * price), where
# k_b = 1 / (p0 (2b - 1) o_max / 10).  The accepted requests form one offline
# instance (all released at step 0, no prompt part).  Draws come from
# SplitMix64 keyed by (seed, replication): per request, the length, then the
# acceptance uniform.

_MASK64 = (1 << 64) - 1


def _splitmix64(state: int):
    while True:
        state = (state + 0x9E3779B97F4A7C15) & _MASK64
        z = state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
        yield z ^ (z >> 31)


def pricing_requests(replication: int, seed: int = 0, n: int = 400, o_max: int = 1000,
                     p: float = 1.0):
    """Return (lengths of the n potential requests, accepted mask, p0)."""
    rnd = _splitmix64((seed * 0x100000001B3 + 7919 * replication + 0x5EED) & _MASK64)
    p0 = p / 500.0
    width = o_max // 10
    lens = np.empty(n, dtype=np.int32)
    acc = np.zeros(n, dtype=bool)
    for i in range(n):
        u = (next(rnd) >> 11) * (2.0 ** -53)
        o = 1 + int(u * o_max)
        b = (o + width - 1) // width
        k_b = 1.0 / (p0 * (2 * b - 1) * width)
        prob = max(0.0, 1.0 - k_b * p0 * o)
        v = (next(rnd) >> 11) * (2.0 ** -53)
        lens[i] = o
        acc[i] = v < prob
    return lens, acc, p0


def pricing_instance(replication: int, seed: int = 0, n: int = 400):
    """The accepted requests of one replication as a one-instance job table."""
    lens, acc, _ = pricing_requests(replication, seed, n)
    out = lens[acc].reshape(1, -1).astype(np.int32)
    z = np.zeros_like(out)
    return np.ascontiguousarray(z), np.ascontiguousarray(z), np.ascontiguousarray(out)


def prediction_upper(output, slack: float, seed: int = 0, tight: bool = False) -> np.ndarray:
    """Upper ends u_i >= o_i of output-length prediction intervals (inputs of
    Robust-ISJL): u_i = o_i + floor(U_i * slack * o_i) with U_i uniform on [0, 1)
    from a seeded PCG64 stream, or U_i = 1 with ``tight`` (u_i = floor((1 +
    slack) o_i), the interval of the scale-normalised corollary).  Same shape as
    ``output``, int32."""
    o = np.asarray(output, dtype=np.int64)
    if tight:
        u = np.ones(o.shape)
    else:
        u = np.random.Generator(np.random.PCG64(seed)).random(o.shape)
    e = np.floor(u * float(slack) * o).astype(np.int64)
    return (o + e).astype(np.int32)
