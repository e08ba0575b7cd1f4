"""GPU parity over whole named workloads, through the C ABI.

Every instance of a contiguous prefix of each workload (all of it with
``FSCHED_FULL_PARITY=1``) runs on the GPU and, sharded over the host's cores,
through the single-threaded oracle; every metric, every start and every finish
must agree exactly.  Policies: every policy of the workload; every fairness
budget for ISJL (the six of the sweep workload included).  FCFS and LJF
schedules do not depend on alpha (only the count of steps with extent above
alpha does), so on the sweep workload they run at alpha = 64.  The exact
optimum of the tiny workload is compared on a prefix of each (alpha, KV budget)
setting, ISJL on it in full.

Default prefixes keep the round's test run short; the full run is the one
recorded in the design notes.
"""
import os
import sys
import time

import numpy as np
import pytest

import oracle
import workload
import paper_2608_02244_amd as fs
from oracle import ALPHA_INF

pytestmark = pytest.mark.gpu

FULL = os.environ.get("FSCHED_FULL_PARITY") == "1"
DEFAULT_PREFIX = {"uniform_256x64": 256, "lognormal_4096x1000": 1024,
                  "bimodal_sweep_4096x2000": 512, "pareto_65536x2000": 1024}
OPT_PREFIX = 65536 if FULL else 2048
ISJL_TINY_PREFIX = 1048576 if FULL else 65536


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _progress(ctx):
    last = [time.time()]

    def cb(done, total):
        if time.time() - last[0] > 20 or done == total:
            last[0] = time.time()
            log(f"  {ctx}: oracle {done}/{total}")
    return cb


def _compare(ctx, gm, gs, gf, rm, rs, rf):
    bad = np.zeros(len(rm), dtype=bool)
    for f in fs.METRIC_FIELDS:
        bad |= gm[f] != rm[f]
    bad |= (gs != rs).any(1) | (gf != rf).any(1)
    nbad = int(bad.sum())
    log(f"  {ctx}: {len(rm)} instances compared, {nbad} differ")
    if nbad:
        i = int(np.nonzero(bad)[0][0])
        diff = [f for f in fs.METRIC_FIELDS if gm[f][i] != rm[f][i]]
        raise AssertionError(f"{ctx}: {nbad} instances differ; first {i}: metrics {diff}, "
                             f"starts equal {bool((gs[i] == rs[i]).all())}")


@pytest.mark.parametrize("name", list(DEFAULT_PREFIX))
def test_every_instance_every_policy(dev, name):
    import torch
    w = workload.WORKLOADS[name]
    n = w.n_inst if FULL else min(w.n_inst, DEFAULT_PREFIX[name])
    threads = oracle.host_threads()
    log(f"{name}: {n} of {w.n_inst} instances, oracle on {threads} host threads")
    a, p, o = workload.generate(w, n_inst=n)
    ta, tp, to = (torch.from_numpy(x).to(dev) for x in (a, p, o))
    for pol in w.policies:
        if pol == "isjl":
            alphas = w.alphas
        elif name == "bimodal_sweep_4096x2000":
            alphas = (64,)
        else:
            alphas = w.alphas if pol == "ljf" else (ALPHA_INF,)
        for alpha in alphas:
            ctx = f"{name} {pol} alpha={alpha}"
            kw = dict(policy=pol, B=w.B, alpha=alpha, M_kv=w.M_kv, cost_c=w.cost_c,
                      cost_tau=w.cost_tau)
            t0 = time.time()
            raw, st, fi = fs.simulate(ta, tp, to, schedule=True, **kw)
            torch.cuda.synchronize()
            gm = fs.metrics_view(raw).copy()
            gs, gf = st.cpu().numpy(), fi.cpu().numpy()
            del raw, st, fi
            log(f"  {ctx}: gpu {time.time() - t0:.2f} s")
            t0 = time.time()
            rm, rs, rf = oracle.simulate_parallel(a, p, o, threads=threads, schedule=True,
                                                  progress=_progress(ctx), **kw)
            log(f"  {ctx}: oracle {time.time() - t0:.1f} s")
            _compare(ctx, gm, gs, gf, rm, rs, rf)
    del ta, tp, to
    torch.cuda.empty_cache()


@pytest.mark.parametrize("M_kv", [16, 0])
def test_tiny_workload_opt_and_isjl(dev, M_kv):
    import torch
    w = workload.WORKLOADS["tiny_opt_1048576x8"]
    threads = oracle.host_threads()
    a, p, o = workload.generate(w, n_inst=ISJL_TINY_PREFIX)
    t = [torch.from_numpy(x).to(dev) for x in (a, p, o)]
    n_opt = min(OPT_PREFIX, ISJL_TINY_PREFIX)
    for alpha in w.alphas:
        ctx = f"tiny M_kv={M_kv} alpha={alpha}"
        kw = dict(B=w.B, alpha=alpha, M_kv=M_kv)
        raw, st, fi = fs.simulate(*t, schedule=True, policy="isjl", cost_c=w.cost_c,
                                  cost_tau=w.cost_tau, **kw)
        torch.cuda.synchronize()
        gm = fs.metrics_view(raw).copy()
        gs, gf = st.cpu().numpy(), fi.cpu().numpy()
        rm, rs, rf = oracle.simulate_parallel(a, p, o, threads=threads, schedule=True,
                                              chunk=8192, progress=_progress(ctx + " isjl"),
                                              policy="isjl", cost_c=w.cost_c,
                                              cost_tau=w.cost_tau, **kw)
        _compare(ctx + " isjl", gm, gs, gf, rm, rs, rf)
        T, _ = fs.bruteforce_opt(*(x[:n_opt] for x in t), schedule=True, **kw)
        torch.cuda.synchronize()
        T = T.cpu().numpy()
        t0 = time.time()
        ref = oracle.opt_parallel(a[:n_opt], p[:n_opt], o[:n_opt], threads=threads,
                                  progress=_progress(ctx + " opt"), **kw)
        nbad = int((T != ref).sum())
        log(f"  {ctx} opt: {n_opt} instances compared, {nbad} differ "
            f"(oracle {time.time() - t0:.1f} s)")
        assert nbad == 0, f"{ctx}: T_opt differs at {np.nonzero(T != ref)[0][:5].tolist()}"
