"""GPU parity of the prefill-at-admission variant (FSCHED_F_PREFILL) against the
oracle with the same flag, through the C ABI: every metric, start and finish
step, bit-exact.  All four policies and Robust-ISJL; offline, sorted and
unsorted releases, KV budgets, alpha = 0 / infinity, up to 4,096 jobs and 1,024
workers; the calls that score in the chunked reading refuse the flag."""
import ctypes
import zlib

import numpy as np
import pytest

import oracle
import workload
import paper_2608_02244_amd as fs
from oracle import ALPHA_INF, FLAG_PREFILL
from test_gpu_simulate import assert_same, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def run_gpu(dev, tables, robust=False, **kw):
    import torch
    ts = [torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(dev) for x in tables]
    if robust:
        raw, st, fi = fs.simulate_robust(*ts, prefill=True, schedule=True, **kw)
    else:
        raw, st, fi = fs.simulate(*ts, prefill=True, schedule=True, **kw)
    torch.cuda.synchronize()
    return fs.metrics_view(raw), st.cpu().numpy(), fi.cpu().numpy()


def check(dev, ctx, tables, robust=False, **kw):
    got, gs, gf = run_gpu(dev, tables, robust, **kw)
    if robust:
        ref, rs, rf = oracle.simulate_robust(*tables, flags=FLAG_PREFILL, schedule=True, **kw)
    else:
        ref, rs, rf = oracle.simulate(*tables, flags=FLAG_PREFILL, schedule=True, **kw)
    assert_same(ctx, got, ref, gs, rs, gf, rf)
    return got


CASES = [("fcfs", ALPHA_INF), ("sjf", ALPHA_INF), ("ljf", 0), ("ljf", 5), ("isjl", 0),
         ("isjl", 2), ("isjl", 7), ("isjl", 40), ("isjl", ALPHA_INF)]


@pytest.mark.parametrize("policy,alpha", CASES)
def test_random_small_instances(dev, policy, alpha):
    rng = np.random.default_rng(zlib.crc32(f"prefill:{policy}:{alpha}".encode()))
    for trial in range(12):
        n = int(rng.choice([1, 2, 7, 64, 65, 200, 700]))
        B = int(rng.choice([1, 2, 3, 5, 8, 0]))
        M_kv = int(rng.choice([0, 0, 60, 400]))
        mode = trial % 3  # offline, sorted releases, unsorted releases
        a, p, o = workload.random_tables(rng, 16, n, int(rng.choice([0, 6, 60])),
                                         int(rng.choice([5, 40])),
                                         max_arrival=0 if mode == 0 else int(rng.choice([20, 300])),
                                         sorted_arrivals=(mode == 1))
        ctx = f"prefill {policy} alpha={alpha} n={n} B={B} M={M_kv} mode={mode}"
        log(ctx)
        check(dev, ctx, (a, p, o), policy=policy, B=B, alpha=alpha, M_kv=M_kv,
              cost_c=int(rng.integers(0, 50)), cost_tau=int(rng.integers(1, 4)))


@pytest.mark.parametrize("policy", ["isjl", "fcfs", "ljf", "sjf"])
def test_max_sizes(dev, policy):
    rng = np.random.default_rng(zlib.crc32(f"prefill-max:{policy}".encode()))
    for B, alpha, M in ((1024, 40, 0), (700, 5, 40000)):
        a, p, o = workload.random_tables(rng, 2, 4096, 80, 120, max_arrival=3000,
                                         sorted_arrivals=True)
        log(f"prefill max {policy} B={B}")
        check(dev, f"prefill max {policy} B={B}", (a, p, o), policy=policy, B=B,
              alpha=alpha if policy in ("isjl", "ljf") else ALPHA_INF, M_kv=M, cost_c=7,
              cost_tau=2)


def test_robust_prefill(dev):
    rng = np.random.default_rng(31)
    for trial in range(8):
        n = int(rng.choice([5, 64, 300]))
        a, p, o = workload.random_tables(rng, 16, n, 30, 40, max_arrival=200,
                                         sorted_arrivals=bool(trial % 2))
        u = workload.prediction_upper(o, 1.0, seed=trial)
        B, alpha, M = int(rng.choice([2, 4, 9])), int(rng.choice([0, 3, 20])), int(
            rng.choice([0, 300]))
        ctx = f"robust prefill n={n} B={B} alpha={alpha} M={M}"
        log(ctx)
        check(dev, ctx, (a, p, o, u), robust=True, B=B, alpha=alpha, M_kv=M, cost_c=3,
              cost_tau=1)


def test_lmsys_shaped_with_prompts(dev):
    """The efficiency workload's total tokens split into a prompt and an output
    part (a third prompt, rounded down) under every policy of the table."""
    a, p, o = workload.generate("lmsys_shaped_256x2000", n_inst=8)
    tot = p + o
    p2 = (tot // 3).astype(np.int32)
    o2 = (tot - p2).astype(np.int32)
    for pol, al in (("fcfs", ALPHA_INF), ("sjf", ALPHA_INF), ("ljf", ALPHA_INF), ("isjl", 50)):
        for B in (16, 32):
            log(f"lmsys prefill {pol} B={B}")
            check(dev, f"lmsys prefill {pol} B={B}", (a, p2, o2), policy=pol, B=B, alpha=al,
                  cost_c=0, cost_tau=1)


def test_other_calls_refuse_the_flag(dev):
    a, p, o = workload.random_tables(np.random.default_rng(1), 2, 6, 3, 5)
    prm = fs.make_params("isjl", 2, 3, prefill=True)
    m = np.zeros(2, dtype=fs.METRICS_DTYPE)
    viol = np.zeros(2, dtype=np.uint32)
    st = np.zeros_like(o)
    rc = fs.lib().fsched_cost_decompose(ctypes.byref(prm), 2, 6, a.ctypes.data, p.ctypes.data,
                                        o.ctypes.data, st.ctypes.data, m.ctypes.data,
                                        viol.ctypes.data, None)
    assert rc == fs.ENOTIMPL
    T = np.zeros(2, dtype=np.int64)
    rc = fs.lib().fsched_bruteforce_opt(ctypes.byref(prm), 2, 6, a.ctypes.data, p.ctypes.data,
                                        o.ctypes.data, T.ctypes.data, None, None)
    assert rc == fs.ENOTIMPL
