"""GPU parity of fsched_simulate_robust (Robust-ISJL, Section 3.4) against the
oracle, through the C ABI: every metric, start and finish step, bit-exact.
Small random instances (offline, sorted and unsorted releases, KV budgets,
alpha = 0 / infinity, the two job-bitmap widths and up to 16 worker slots per
lane), exact predictions against fsched_simulate, the full-size pareto_65536x2000
workload with loose predictions (sampled instances against the oracle,
fairness on all), error paths, and the experiment driver against the oracle's.
"""
import ctypes
import zlib

import numpy as np
import pytest

import oracle
import workload
import paper_2608_02244_amd as fs
from oracle import ALPHA_INF
from paper_2608_02244_amd import robust as rb
from test_gpu_simulate import assert_same, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def gpu_rob(dev, a, p, o, u, schedule=True, **kw):
    import torch
    ts = [torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(dev) for x in (a, p, o, u)]
    raw, st, fi = fs.simulate_robust(*ts, schedule=schedule, **kw)
    torch.cuda.synchronize()
    m = fs.metrics_view(raw)
    if schedule:
        return m, st.cpu().numpy(), fi.cpu().numpy()
    return m, None, None


def check(dev, ctx, a, p, o, u, **kw):
    got, gs, gf = gpu_rob(dev, a, p, o, u, **kw)
    ref, rs, rf = oracle.simulate_robust(a, p, o, u, schedule=True, **kw)
    assert_same(ctx, got, ref, gs, rs, gf, rf)
    return got


@pytest.mark.parametrize("alpha", [0, 1, 3, 8, 40, ALPHA_INF])
def test_random_small_instances(dev, alpha):
    rng = np.random.default_rng(zlib.crc32(f"robust:{alpha}".encode()))
    for trial in range(12):
        n = int(rng.choice([1, 3, 7, 64, 65, 200, 700]))
        B = int(rng.choice([1, 2, 3, 5, 8, 0]))
        M_kv = int(rng.choice([0, 0, 60, 400]))
        mode = trial % 3  # offline, sorted releases, unsorted releases
        a, p, o = workload.random_tables(rng, 16, n, int(rng.choice([0, 6])),
                                         int(rng.choice([5, 40])),
                                         max_arrival=0 if mode == 0 else int(rng.choice([20, 300])),
                                         sorted_arrivals=(mode == 1))
        slack = float(rng.choice([0.0, 0.3, 1.0, 4.0]))
        u = workload.prediction_upper(o, slack, seed=trial, tight=bool(trial % 4 == 3))
        ctx = f"robust alpha={alpha} n={n} B={B} M={M_kv} mode={mode} slack={slack}"
        log(ctx)
        check(dev, ctx, a, p, o, u, B=B, alpha=alpha, M_kv=M_kv, cost_c=int(rng.integers(0, 50)),
              cost_tau=1)


def test_max_sizes(dev):
    """4096 jobs (two bitmap words per lane) and up to 1024 workers."""
    rng = np.random.default_rng(77)
    for B, alpha, M in ((1024, 40, 0), (700, 5, 30000), (64, 200, 0)):
        a, p, o = workload.random_tables(rng, 2, 4096, 50, 120, max_arrival=3000,
                                         sorted_arrivals=True)
        u = workload.prediction_upper(o, 0.8, seed=B)
        log(f"robust max sizes B={B}")
        check(dev, f"robust max B={B}", a, p, o, u, B=B, alpha=alpha, M_kv=M, cost_c=7,
              cost_tau=2)


def test_exact_predictions_equal_isjl(dev):
    rng = np.random.default_rng(3)
    a, p, o = workload.random_tables(rng, 64, 300, 10, 60, max_arrival=500,
                                     sorted_arrivals=True)
    for alpha, B, M in ((0, 4, 0), (6, 16, 2000), (ALPHA_INF, 8, 0)):
        r, rs, rf = gpu_rob(dev, a, p, o, o, B=B, alpha=alpha, M_kv=M, cost_c=5, cost_tau=1)
        i, is_, if_ = fs.simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=M, cost_c=5,
                                  cost_tau=1, schedule=True)
        assert_same(f"u = o alpha={alpha}", r, i, rs, is_, rf, if_)


def test_pareto_workload_with_loose_predictions(dev):
    import torch
    w = workload.WORKLOADS["pareto_65536x2000"]
    log("generate pareto_65536x2000")
    a, p, o = workload.generate(w)
    u = workload.prediction_upper(o, 0.5, seed=1)
    ts = [torch.from_numpy(x).to(dev) for x in (a, p, o, u)]
    alpha = w.alphas[0]
    raw, _, _ = fs.simulate_robust(*ts, B=w.B, alpha=alpha, M_kv=w.M_kv, cost_c=w.cost_c,
                                   cost_tau=w.cost_tau)
    torch.cuda.synchronize()
    m = fs.metrics_view(raw)
    lens = p.astype(np.int64) + o
    assert np.array_equal(m["O"], lens.sum(1))
    assert (m["unfair_steps"] == 0).all() and (m["max_extent"] <= alpha).all()
    assert (m["max_active"] <= w.B).all()
    sample = np.array([0, 17, 40000, w.n_inst - 1])
    ref = oracle.simulate_robust(a[sample], p[sample], o[sample], u[sample], B=w.B, alpha=alpha,
                                 M_kv=w.M_kv, cost_c=w.cost_c, cost_tau=w.cost_tau)
    assert_same("pareto robust sample", m[sample], ref)
    del ts
    torch.cuda.empty_cache()


def test_errors(dev):
    import torch
    rng = np.random.default_rng(8)
    a, p, o = workload.random_tables(rng, 4, 30, 5, 20)
    u = workload.prediction_upper(o, 1.0, seed=2)
    u[1, 4] = o[1, 4] - 1            # upper below the output: invalid table
    u[2, 0] = (1 << 20)              # proxy length beyond the kernel limit
    got, _, _ = gpu_rob(dev, a, p, o, u, B=3, alpha=4)
    assert got["T"][1] == fs.T_INVALID and got["T"][2] == fs.T_TOOLARGE
    keep = [0, 3]
    ref = oracle.simulate_robust(a[keep], p[keep], o[keep], u[keep], B=3, alpha=4)
    assert_same("valid rows next to invalid ones", got[keep], ref)
    with pytest.raises(fs.FschedError) as ei:
        fs.simulate_robust(a, p, o, u, B=3, alpha=4)
    assert ei.value.code == fs.EINVAL
    # other policies are not implemented on predicted sizes
    prm = fs.make_params("ljf", 3, 4)
    m = np.zeros(4, dtype=fs.METRICS_DTYPE)
    rc = fs.lib().fsched_simulate_robust(ctypes.byref(prm), 4, 30, a.ctypes.data, p.ctypes.data,
                                         o.ctypes.data, o.ctypes.data, m.ctypes.data, None,
                                         None, None)
    assert rc == fs.ENOTIMPL
    rc = fs.lib().fsched_simulate_robust(ctypes.byref(fs.make_params("isjl", 3, 4)), 4, 30,
                                         a.ctypes.data, p.ctypes.data, o.ctypes.data, None,
                                         m.ctypes.data, None, None, None)
    assert rc == fs.EINVAL


def oracle_quad(a, p, o, u, B, alpha, M_kv=0):
    mr = oracle.simulate_robust(a, p, o, u, B=B, alpha=alpha, M_kv=M_kv, cost_c=0, cost_tau=0)
    T_opt = oracle.opt(a, p, o, B=B, alpha=alpha, M_kv=M_kv)
    mi = oracle.simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=M_kv, cost_c=0,
                         cost_tau=0)
    mu = oracle.simulate(a, p, u, policy="isjl", B=B, alpha=alpha, M_kv=M_kv, cost_c=0,
                         cost_tau=0)
    return mr["T"], mr["unfair_steps"], T_opt, mi["T"], mu["T"]


def test_experiment_matches_oracle(dev):
    a, p, o = workload.generate("tiny_opt_1048576x8", n_inst=120, inst_begin=9000)
    u = workload.prediction_upper(o, 1.0, seed=4)
    got = rb.run(rb.gpu_quad, a, p, o, u, [1, 4, 7], B=2)
    ref = rb.run(oracle_quad, a, p, o, u, [1, 4, 7], B=2)
    assert got == ref
