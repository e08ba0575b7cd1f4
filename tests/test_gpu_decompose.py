"""GPU parity of fsched_cost_decompose against the oracle, through the C ABI.

Metrics and violation masks must match exactly, for schedules produced by every
policy (there the re-scored metrics also equal the simulation's) and for random
start vectors that break capacity, KV, fairness and release constraints.
"""
import sys
import zlib

import numpy as np
import pytest

import oracle
import workload
import paper_2608_02244_amd as fs
from oracle import ALPHA_INF

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_dec(dev, a, p, o, s, **kw):
    import torch
    t = [torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(dev) for x in (a, p, o, s)]
    raw, viol = fs.cost_decompose(*t, **kw)
    torch.cuda.synchronize()
    return fs.metrics_view(raw), viol.cpu().numpy().astype(np.uint32)


def same(ctx, got, ref, gv, rv):
    for f in fs.METRIC_FIELDS:
        if not np.array_equal(got[f], ref[f]):
            bad = np.nonzero(got[f] != ref[f])[0][:5]
            raise AssertionError(f"{ctx}: {f} differs at {bad.tolist()}: gpu "
                                 f"{got[f][bad].tolist()} oracle {ref[f][bad].tolist()}")
    if not np.array_equal(gv, rv):
        bad = np.nonzero(gv != rv)[0][:5]
        raise AssertionError(f"{ctx}: violation differs at {bad.tolist()}: gpu "
                             f"{gv[bad].tolist()} oracle {rv[bad].tolist()}")


@pytest.mark.parametrize("policy,alpha", [("fcfs", ALPHA_INF), ("sjf", ALPHA_INF), ("ljf", 2),
                                          ("isjl", 0), ("isjl", 3), ("isjl", 12)])
def test_policy_schedules(dev, policy, alpha):
    rng = np.random.default_rng(zlib.crc32(f"dec:{policy}:{alpha}".encode()))
    for trial in range(8):
        n = int(rng.choice([1, 5, 33, 64, 100, 257]))
        B = int(rng.choice([1, 2, 4, 9]))
        M = int(rng.choice([0, 30, 200]))
        a, p, o = workload.random_tables(rng, 20, n, 6, 25,
                                         max_arrival=int(rng.choice([0, 50, 300])),
                                         sorted_arrivals=bool(trial % 2))
        kw = dict(B=B, alpha=alpha, M_kv=M, cost_c=int(rng.integers(0, 9)),
                  cost_tau=int(rng.integers(0, 4)))
        sm, st, _ = oracle.simulate(a, p, o, policy=policy, schedule=True, **kw)
        ref, rv = oracle.decompose(a, p, o, st, **kw)
        got, gv = gpu_dec(dev, a, p, o, st, **kw)
        ctx = f"{policy} alpha={alpha} n={n} B={B} M={M} trial={trial}"
        log(ctx)
        same(ctx, got, ref, gv, rv)
        same(ctx + " vs simulate", got, sm, gv, rv)


def test_random_start_vectors(dev):
    """Arbitrary schedules: every violation bit, idle gaps, simultaneous events."""
    rng = np.random.default_rng(77)
    for trial in range(30):
        n = int(rng.choice([1, 2, 6, 40, 64, 65, 300]))
        a, p, o = workload.random_tables(rng, 16, n, 4, 15, max_arrival=20)
        span = int(rng.choice([3, 30, 400]))
        s = rng.integers(0, span, size=a.shape).astype(np.int32)
        if trial % 5 == 0:
            s[0, 0] = -3  # negative start in one instance
        kw = dict(B=int(rng.choice([0, 1, 3, 6])), alpha=int(rng.choice([0, 2, 9, ALPHA_INF])),
                  M_kv=int(rng.choice([0, 10, 40])), cost_c=int(rng.integers(0, 50)),
                  cost_tau=int(rng.integers(0, 5)))
        ref, rv = oracle.decompose(a, p, o, s, **kw)
        got, gv = gpu_dec(dev, a, p, o, s, **kw)
        ctx = f"random starts trial={trial} n={n} {kw}"
        log(ctx)
        same(ctx, got, ref, gv, rv)
    assert True


def test_random_start_vectors_large(dev):
    """Large instances: event groups that span several 64-event chunks, long and
    short jobs mixed, every kind of budget."""
    rng = np.random.default_rng(1234)
    for trial in range(12):
        n = int(rng.choice([500, 1000, 2048, 4096]))
        a, p, o = workload.random_tables(rng, 6, n, 8, int(rng.choice([3, 40, 900])),
                                         max_arrival=int(rng.choice([0, 100])))
        span = int(rng.choice([2, 10, 300, 5000]))
        s = (a + rng.integers(0, span, size=a.shape)).astype(np.int32)
        kw = dict(B=int(rng.choice([0, 16, 300])), alpha=int(rng.choice([0, 5, 200, ALPHA_INF])),
                  M_kv=int(rng.choice([0, 500, 20000])), cost_c=int(rng.integers(0, 50)),
                  cost_tau=int(rng.integers(0, 5)))
        ctx = f"large random starts trial={trial} n={n} span={span} {kw}"
        log(ctx)
        ref, rv = oracle.decompose(a, p, o, s, **kw)
        got, gv = gpu_dec(dev, a, p, o, s, **kw)
        same(ctx, got, ref, gv, rv)


def test_limits_and_host_mode(dev):
    a = np.zeros((2, 3), np.int32)
    p = np.zeros((2, 3), np.int32)
    o = np.full((2, 3), 4, np.int32)
    s = np.array([[0, 1, 2], [0, (1 << 19), 5]], np.int32)
    got, gv = gpu_dec(dev, a, p, o, s, B=2, alpha=1)
    assert got["T"][1] == fs.T_TOOLARGE
    ref, rv = oracle.decompose(a[:1], p[:1], o[:1], s[:1], B=2, alpha=1)
    same("row next to a too-large row", got[:1], ref, gv[:1], rv)
    hm, hv = fs.cost_decompose(a[:1], p[:1], o[:1], s[:1], B=2, alpha=1)
    same("host mode", hm, ref, hv, rv)


@pytest.mark.parametrize("name", ["lognormal_4096x1000", "pareto_65536x2000"])
def test_named_workload_schedules(dev, name):
    """Full-size: the GPU simulation's schedules re-scored on the GPU reproduce its
    metrics for every instance; sampled instances also match the oracle."""
    import torch
    w = workload.WORKLOADS[name]
    a, p, o = workload.generate(w)
    ta, tp, to = (torch.from_numpy(x).to(dev) for x in (a, p, o))
    kw = dict(B=w.B, alpha=w.alphas[0], M_kv=w.M_kv, cost_c=w.cost_c, cost_tau=w.cost_tau)
    log(f"simulate {name}")
    raw, st, _ = fs.simulate(ta, tp, to, policy="isjl", schedule=True, **kw)
    log(f"decompose {name}")
    draw, dv = fs.cost_decompose(ta, tp, to, st, **kw)
    torch.cuda.synchronize()
    sm, dm = fs.metrics_view(raw), fs.metrics_view(draw)
    dv = dv.cpu().numpy()
    assert (dv == 0).all()
    for f in fs.METRIC_FIELDS:
        assert np.array_equal(sm[f], dm[f]), f
    idx = np.array([0, 1, w.n_inst // 2, w.n_inst - 1])
    stn = st.cpu().numpy()[idx]
    ref, rv = oracle.decompose(a[idx], p[idx], o[idx], stn, **kw)
    same(name, dm[idx], ref, dv[idx].astype(np.uint32), rv)


def test_long_jobs_take_the_wide_pass(dev):
    """Jobs of 65,536 tokens or more do not fit the 16-bit lengths of the first
    pass: their instances are scored by the second (32-bit) pass, next to rows
    the first pass finishes; 65,535 and 65,536 sit on either side of the cut."""
    rng = np.random.default_rng(77)
    n = 40
    a = np.zeros((6, n), np.int32)
    p = rng.integers(0, 50, size=(6, n)).astype(np.int32)
    o = rng.integers(1, 3000, size=(6, n)).astype(np.int32)
    o[1, 7] = 65535 - p[1, 7]          # longest job exactly 65,535: first pass
    o[2, 3] = 65536 - p[2, 3]          # exactly 65,536: second pass
    o[3, ::5] = rng.integers(70000, 200000, size=o[3, ::5].shape)
    o[5, 0] = 300000
    s = (a + rng.integers(0, 40000, size=a.shape)).astype(np.int32)
    for kw in (dict(B=4, alpha=ALPHA_INF), dict(B=0, alpha=1000, M_kv=500000, cost_c=3,
                                                cost_tau=1)):
        ref, rv = oracle.decompose(a, p, o, s, **kw)
        got, gv = gpu_dec(dev, a, p, o, s, **kw)
        same(f"long jobs {kw}", got, ref, gv, rv)
        hm, hv = fs.cost_decompose(a, p, o, s, **kw)
        same(f"long jobs host mode {kw}", hm, ref, hv, rv)


def test_start_groups_across_chunks(dev):
    """Schedules built from few start times and few lengths: groups of up to
    hundreds of simultaneous starts and ends that span several 64-event chunks,
    the earliest and the latest active start losing their last job at any
    position of a chunk, and gaps that empty the machine between bursts.  These
    are the cases where the re-scoring sweep switches between its walk-free
    common case and the walk over the group ends."""
    rng = np.random.default_rng(20261202)
    for trial in range(24):
        n = int(rng.choice([70, 130, 400, 1000, 2000]))
        n_times = int(rng.choice([2, 3, 5, 12]))
        n_lens = int(rng.choice([1, 2, 4, 9]))
        gap = int(rng.choice([0, 1, 40]))
        times = np.cumsum(rng.integers(1, 30, size=n_times)) + gap * np.arange(n_times)
        lens = rng.integers(1, 60, size=n_lens)
        inst = 8
        s = rng.choice(times, size=(inst, n)).astype(np.int32)
        o = rng.choice(lens, size=(inst, n)).astype(np.int32)
        p = np.zeros((inst, n), np.int32)
        a = np.zeros((inst, n), np.int32)
        kw = dict(B=int(rng.choice([0, 64, 1000])), alpha=int(rng.choice([0, 7, 50, ALPHA_INF])),
                  M_kv=int(rng.choice([0, 5000])), cost_c=int(rng.integers(0, 9)),
                  cost_tau=int(rng.integers(0, 4)))
        ctx = f"start groups trial={trial} n={n} times={n_times} lens={n_lens} gap={gap} {kw}"
        log(ctx)
        ref, rv = oracle.decompose(a, p, o, s, **kw)
        got, gv = gpu_dec(dev, a, p, o, s, **kw)
        same(ctx, got, ref, gv, rv)
