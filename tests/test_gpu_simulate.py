"""GPU parity of fsched_simulate against the oracle, through the C ABI.

Integers must match exactly: every metric of every instance and the start and
finish step of every job.  Small cases cover every policy, ragged sizes,
releases (sorted and unsorted), KV budgets, alpha = 0 / infinity, B = 1 /
unlimited, the kernel's size limits and the fill sweep (runs of completions
admitting queued jobs, FCFS / SJF / ISJL at alpha >= 2^20 with up to 128
workers).  The named workloads run at full size
in the launch configuration the benchmark times; there the oracle checks
sampled instances and identities that hold at any size check all of them.
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


def gpu_sim(dev, a, p, o, schedule=True, **kw):
    import torch
    ta, tp, to = (torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(dev)
                  for x in (a, p, o))
    raw, st, fi = fs.simulate(ta, tp, to, schedule=schedule, **kw)
    torch.cuda.synchronize()
    m = fs.metrics_view(raw)
    if schedule:
        return m, st.cpu().numpy(), fi.cpu().numpy()
    return m, None, None


def first_divergence(gs, rs):
    """Instance and job of the earliest start at which two schedules differ."""
    rows = np.nonzero((gs != rs).any(1))[0]
    if len(rows) == 0:
        return None
    i = rows[0]
    js = np.nonzero(gs[i] != rs[i])[0]
    j = js[np.argmin(np.minimum(gs[i, js], rs[i, js]))]
    return int(i), int(j)


def assert_same(ctx, got, ref, gs=None, rs=None, gf=None, rf=None):
    if gs is not None:
        d = first_divergence(gs, rs)
        if d is not None:
            i, j = d
            t0 = min(gs[i, j], rs[i, j])
            near = np.nonzero((np.abs(rs[i] - t0) <= 3) | (np.abs(gs[i] - t0) <= 3))[0]
            raise AssertionError(
                f"{ctx}: schedules diverge at instance {i}, job {j} (gpu start {gs[i, j]}, "
                f"oracle start {rs[i, j]}, len {rf[i, j] - rs[i, j]}); jobs starting near "
                f"{t0}: " + "; ".join(f"job {k} len {rf[i, k] - rs[i, k]} gpu {gs[i, k]} "
                                      f"oracle {rs[i, k]}" for k in near[:12]))
    for f in fs.METRIC_FIELDS:
        if not np.array_equal(got[f], ref[f]):
            bad = np.nonzero(got[f] != ref[f])[0][:5]
            raise AssertionError(f"{ctx}: metric {f} differs at instances {bad.tolist()}: "
                                 f"gpu {got[f][bad].tolist()} oracle {ref[f][bad].tolist()}")
    if gs is not None:
        for name, g, r in (("start", gs, rs), ("finish", gf, rf)):
            if not np.array_equal(g, r):
                i, j = np.argwhere(g != r)[0]
                raise AssertionError(f"{ctx}: {name} differs first at instance {i} job {j}: "
                                     f"gpu {g[i, j]} oracle {r[i, j]}")


def check(dev, ctx, a, p, o, **kw):
    got, gs, gf = gpu_sim(dev, a, p, o, **kw)
    kw2 = dict(kw)
    flags = oracle.FLAG_BETA_SQRT17 if kw2.pop("beta_sqrt17", False) else 0
    ref, rs, rf = oracle.simulate(a, p, o, schedule=True, flags=flags, **kw2)
    assert_same(ctx, got, ref, gs, rs, gf, rf)
    return got


CASES = [
    ("fcfs", ALPHA_INF), ("fcfs", 3), ("sjf", ALPHA_INF), ("ljf", 0), ("ljf", 4),
    ("isjl", 0), ("isjl", 1), ("isjl", 2), ("isjl", 3), ("isjl", 6), ("isjl", 15),
    ("isjl", ALPHA_INF),
]


@pytest.mark.parametrize("policy,alpha", CASES)
def test_random_small_instances(dev, policy, alpha):
    rng = np.random.default_rng(zlib.crc32(f"small:{policy}:{alpha}".encode()))
    for trial in range(14):
        n = int(rng.choice([1, 2, 3, 7, 31, 64, 65, 130, 200]))
        B = int(rng.choice([1, 2, 3, 5, 8, 0]))
        if B == 0 and n > 1024:
            B = 64
        M_kv = int(rng.choice([0, 0, 20, 60, 400]))
        mode = trial % 3  # offline, sorted releases, unsorted releases
        a, p, o = workload.random_tables(rng, 24, n, int(rng.choice([0, 4, 30])),
                                         int(rng.choice([4, 20, 90])),
                                         max_arrival=0 if mode == 0 else int(rng.choice([5, 60, 400])),
                                         sorted_arrivals=(mode == 1))
        c, tau = int(rng.integers(0, 100)), int(rng.integers(0, 5))
        ctx = f"{policy} alpha={alpha} n={n} B={B} M={M_kv} mode={mode} trial={trial}"
        log(ctx)
        check(dev, ctx, a, p, o, policy=policy, B=B, alpha=alpha, M_kv=M_kv, cost_c=c,
              cost_tau=tau)


def test_beta_sqrt17_b2(dev):
    rng = np.random.default_rng(5)
    for trial in range(6):
        a, p, o = workload.random_tables(rng, 64, 12, 3, 25)
        for alpha in (1, 2, 4, 8):
            check(dev, f"beta* alpha={alpha}", a, p, o, policy="isjl", B=2, alpha=alpha,
                  beta_sqrt17=True)


def test_paper_examples_on_gpu(dev):
    """The worked examples the oracle is pinned to, run through the GPU path."""
    L, al = 10, 3
    ell = np.array([[L] + [1] * L], np.int32)
    z = np.zeros_like(ell)
    g = check(dev, "quadratic fcfs", z, z, ell, policy="fcfs", B=2, alpha=ALPHA_INF)
    assert g["T"][0] == L and g["E"][0] == L * (L - 1) // 2
    g = check(dev, "quadratic isjl", z, z, ell, policy="isjl", B=2, alpha=al)
    assert g["T"][0] == L + (L - al - 1 + 1) // 2
    ell = np.array([[2 * al + 1, 2 * al + 1, al, al]], np.int32)
    z = np.zeros_like(ell)
    g = check(dev, "over-inserting", z, z, ell, policy="isjl", B=2, alpha=al)
    assert g["T"][0] == 2 * al + 1 + 2 * al
    ell = np.array([[9, 15, 5, 10, 19]], np.int32)
    z = np.zeros_like(ell)
    g = check(dev, "B=3 guard", z, z, ell, policy="isjl", B=3, alpha=8)
    assert g["T"][0] == 40


def test_algorithm3_hand_traces_on_gpu(dev):
    """The hand-traced cases of Algorithm 3's spare and long workers and of the
    plan width under the KV budget (tests/golden/alg3_spare_examples.json)."""
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "alg3_spare_examples.json")
    for c in json.load(open(path)):
        a, p, o = (np.array([c[k]], np.int32) for k in ("arrival", "prompt", "output"))
        g, gs, _ = gpu_sim(dev, a, p, o, policy="isjl", B=c["B"], alpha=c["alpha"],
                           M_kv=c["M_kv"])
        assert int(g["T"][0]) == c["T"], c["name"]
        assert gs[0].tolist() == c["start"], c["name"]
        check(dev, c["name"], a, p, o, policy="isjl", B=c["B"], alpha=c["alpha"],
              M_kv=c["M_kv"])


@pytest.mark.parametrize("policy", ["isjl", "fcfs", "ljf", "sjf"])
def test_max_sizes(dev, policy):
    """n = 4096 jobs (two bitmap words per lane) and 1024 workers (16 slots per lane)."""
    rng = np.random.default_rng(zlib.crc32(policy.encode()))
    for B, alpha, M in ((1024, 40, 0), (700, 5, 30000), (64, 200, 0)):
        a, p, o = workload.random_tables(rng, 3, 4096, 50, 120, max_arrival=3000,
                                         sorted_arrivals=True)
        log(f"max sizes {policy} B={B}")
        check(dev, f"max {policy} B={B}", a, p, o, policy=policy, B=B,
              alpha=alpha if policy in ("isjl", "ljf") else ALPHA_INF, M_kv=M, cost_c=7,
              cost_tau=2)


def test_degenerate_instances(dev):
    z1 = np.zeros((1, 1), np.int32)
    for pol in ("fcfs", "ljf", "isjl", "sjf"):
        g = check(dev, f"single job {pol}", np.array([[5]], np.int32), z1,
                  np.array([[3]], np.int32), policy=pol, B=1, alpha=0)
        assert g["T"][0] == 8 and g["busy_steps"][0] == 3
    # identical jobs, B >= n, every KV budget edge
    ell = np.full((4, 50), 7, np.int32)
    z = np.zeros_like(ell)
    for pol in ("fcfs", "ljf", "isjl", "sjf"):
        for M in (0, 7, 8, 13, 14, 349, 350):
            check(dev, f"identical {pol} M={M}", z, z, ell, policy=pol, B=0, alpha=2, M_kv=M)
    # every job larger than the KV budget: all run alone
    check(dev, "oversized", z, z, ell, policy="isjl", B=4, alpha=3, M_kv=5)
    # long idle gaps between releases
    arr = np.array([[0, 1000, 1000, 50000, 50001]], np.int32)
    ell = np.array([[3, 2, 9, 1, 4]], np.int32)
    for pol in ("fcfs", "ljf", "isjl", "sjf"):
        check(dev, f"gaps {pol}", arr, np.zeros_like(ell), ell, policy=pol, B=2, alpha=1,
              cost_c=3)
    # sorted arrivals beyond 2^20 are within limits
    arr = np.array([[0, 2_000_000, 2_000_000]], np.int32)
    ell = np.array([[4, 4, 4]], np.int32)
    for pol in ("fcfs", "isjl"):
        check(dev, f"late sorted {pol}", arr, np.zeros_like(ell), ell, policy=pol, B=2, alpha=1)


def test_markers_and_host_mode(dev):
    import torch
    rng = np.random.default_rng(9)
    a, p, o = workload.random_tables(rng, 6, 40, 5, 20, max_arrival=30)
    o[1, 3] = 0                      # invalid output length
    p[2, 0] = (1 << 20)              # length beyond the kernel limit
    a[3, :] = a[3, ::-1].copy()
    a[3, 0] = (1 << 20) + 5          # unsorted and beyond 2^20
    got, _, _ = gpu_sim(dev, a, p, o, policy="isjl", B=3, alpha=4)
    assert got["T"][1] == fs.T_INVALID
    assert got["T"][2] == fs.T_TOOLARGE
    assert got["T"][3] == fs.T_TOOLARGE
    for f in fs.METRIC_FIELDS[1:]:
        assert got[f][1] == 0 and got[f][2] == 0
    keep = [0, 4, 5]
    ref = oracle.simulate(a[keep], p[keep], o[keep], policy="isjl", B=3, alpha=4)
    assert_same("valid rows next to invalid ones", got[keep], ref)
    # host mode reports the marker as a return code
    with pytest.raises(fs.FschedError) as ei:
        fs.simulate(a, p, o, policy="isjl", B=3, alpha=4)
    assert ei.value.code == fs.EINVAL
    # host mode results equal device mode results
    hm, hs, hf = fs.simulate(a[keep], p[keep], o[keep], policy="isjl", B=3, alpha=4,
                             schedule=True)
    dm, ds, df = gpu_sim(dev, a[keep], p[keep], o[keep], policy="isjl", B=3, alpha=4)
    assert_same("host vs device mode", hm, dm, hs, ds, hf, df)


def identities(ctx, m, a, p, o, w, alpha, fair):
    lens = p.astype(np.int64) + o
    assert (m["T"] > 0).all(), ctx
    assert np.array_equal(m["O"], lens.sum(1)), ctx
    assert np.array_equal(m["Q"], (lens * (lens + 1) // 2).sum(1)), ctx
    assert np.array_equal(m["C"], w.cost_c * m["T"] + w.cost_tau * (m["Q"] + m["E"])), ctx
    assert (m["max_active"] <= w.B).all(), ctx
    assert (m["busy_steps"] <= m["T"]).all() and (m["T"] >= lens.max(1)).all(), ctx
    assert np.array_equal(m["sum_latency"], m["sum_completion"] - a.astype(np.int64).sum(1)), ctx
    if fair and alpha != ALPHA_INF:
        assert (m["max_extent"] <= alpha).all() and (m["unfair_steps"] == 0).all(), ctx
        assert (m["E"] <= alpha * m["O"]).all(), ctx


@pytest.mark.parametrize("name", ["uniform_256x64", "lognormal_4096x1000",
                                  "bimodal_sweep_4096x2000", "pareto_65536x2000"])
def test_named_workloads_full_size(dev, name):
    import torch
    w = workload.WORKLOADS[name]
    log(f"generate {name}")
    a, p, o = workload.generate(w)
    ta, tp, to = (torch.from_numpy(x).to(dev) for x in (a, p, o))
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    n_sample = w.n_inst if w.n_inst <= 256 else (32 if name == "bimodal_sweep_4096x2000" else 5)
    sample = np.unique(np.concatenate([[0, w.n_inst - 1],
                                       rng.integers(0, w.n_inst, size=n_sample)]))
    alphas = w.alphas
    for pol in w.policies:
        for alpha in (alphas if pol in ("isjl", "ljf") else (ALPHA_INF,)):
            ctx = f"{name} {pol} alpha={alpha}"
            log(ctx)
            raw, _, _ = fs.simulate(ta, tp, to, policy=pol, B=w.B, alpha=alpha, M_kv=w.M_kv,
                                    cost_c=w.cost_c, cost_tau=w.cost_tau)
            torch.cuda.synchronize()
            m = fs.metrics_view(raw)
            identities(ctx, m, a, p, o, w, alpha, pol in ("isjl", "ljf"))
            ref, rs, rf = oracle.simulate(a[sample], p[sample], o[sample], policy=pol, B=w.B,
                                          alpha=alpha, M_kv=w.M_kv, cost_c=w.cost_c,
                                          cost_tau=w.cost_tau, schedule=True)
            assert_same(ctx, m[sample], ref)
            gm, gs, gf = gpu_sim(dev, a[sample], p[sample], o[sample], policy=pol, B=w.B,
                                 alpha=alpha, M_kv=w.M_kv, cost_c=w.cost_c,
                                 cost_tau=w.cost_tau)
            assert_same(ctx + " (schedules)", gm, ref, gs, rs, gf, rf)
    del ta, tp, to
    torch.cuda.empty_cache()


@pytest.mark.parametrize("policy", ["isjl", "ljf"])
def test_long_jobs(dev, policy):
    """Lengths close to 2^20: the drain sweep cannot pack progress under the
    completion key and takes the payload sort."""
    rng = np.random.default_rng(zlib.crc32(f"long:{policy}".encode()))
    n = 40
    for B, alpha in ((3, 1000), (8, 200000), (5, 0)):
        o = rng.integers(1, (1 << 20) - 1, size=(4, n)).astype(np.int32)
        o[:, ::3] = rng.integers(1, 5000, size=o[:, ::3].shape)  # mix in short jobs
        p = np.zeros_like(o)
        a = np.sort(rng.integers(0, 1 << 19, size=(4, n)), axis=1).astype(np.int32)
        a[:2] = 0
        log(f"long jobs {policy} B={B} alpha={alpha}")
        check(dev, f"long {policy} B={B} alpha={alpha}", a, p, o, policy=policy, B=B,
              alpha=alpha, M_kv=0, cost_c=3, cost_tau=1)


def test_resume_fill_reading(dev):
    """The experiment flag (Phase TWO resumes once A_max <= alpha) against the
    oracle with the same flag: small random instances and a full-size sample."""
    rng = np.random.default_rng(zlib.crc32(b"resume"))
    for trial in range(18):
        n = int(rng.choice([7, 64, 130, 300]))
        B = int(rng.choice([3, 5, 8, 0]))
        alpha = int(rng.choice([1, 4, 15, 60]))
        mode = trial % 3
        a, p, o = workload.random_tables(rng, 16, n, int(rng.choice([0, 8])), 40,
                                         max_arrival=0 if mode == 0 else 300,
                                         sorted_arrivals=(mode == 1))
        M_kv = int(rng.choice([0, 0, 400]))
        ctx = f"resume n={n} B={B} alpha={alpha} M={M_kv} mode={mode}"
        log(ctx)
        got, gs, gf = gpu_sim(dev, a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=M_kv,
                              cost_c=3, cost_tau=1, resume_fill=True)
        ref, rs, rf = oracle.simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=M_kv,
                                      cost_c=3, cost_tau=1, schedule=True,
                                      flags=oracle.FLAG_RESUME_FILL)
        assert_same(ctx, got, ref, gs, rs, gf, rf)
    w = workload.WORKLOADS["lognormal_4096x1000"]
    a, p, o = workload.generate(w, n_inst=48)
    log("resume lognormal_4096x1000 sample")
    kw = dict(policy="isjl", B=w.B, alpha=w.alphas[0], M_kv=w.M_kv, cost_c=w.cost_c,
              cost_tau=w.cost_tau)
    got, gs, gf = gpu_sim(dev, a, p, o, resume_fill=True, **kw)
    ref, rs, rf = oracle.simulate(a, p, o, schedule=True, flags=oracle.FLAG_RESUME_FILL, **kw)
    assert_same("resume lognormal sample", got, ref, gs, rs, gf, rf)


def test_kv_budget_cuts_long_admission_batches(dev):
    """Admission batches of more than 8 jobs under a KV budget that stops them at
    every position around 8 (the small-slot kernels scan the first 8 alone):
    offline and with releases, every policy."""
    rng = np.random.default_rng(404)
    for trial in range(6):
        n, B = 180, int(rng.choice([40, 100, 200]))
        a, p, o = workload.random_tables(rng, 24, n, 3, 12,
                                         max_arrival=0 if trial % 2 == 0 else 50,
                                         sorted_arrivals=True)
        for M in (60, 100, 113, 140, 400):
            for pol, al in (("isjl", 2), ("isjl", ALPHA_INF), ("ljf", ALPHA_INF),
                            ("sjf", ALPHA_INF), ("fcfs", ALPHA_INF)):
                ctx = f"kv cut {pol} alpha={al} B={B} M={M} trial={trial}"
                check(dev, ctx, a, p, o, policy=pol, B=B, alpha=al, M_kv=M, cost_c=2,
                      cost_tau=1)


def test_many_slots_with_quiet_sweeps(dev):
    """4 or more worker slots per lane (B > 128) with releases spaced so that the
    machine often runs a few dozen jobs with nothing queued: the completions
    before the next release are swept with the active slots packed through the
    gather buffer (FCFS has one only for this).  Several instances per block, so
    a pack that strayed past its wave's LDS would show up in a neighbour."""
    rng = np.random.default_rng(2024)
    for B in (200, 512, 1024):
        for M in (0, 400):
            a, p, o = workload.random_tables(rng, 12, 600, 3, 14, max_arrival=900,
                                             sorted_arrivals=True)
            for pol, al in (("fcfs", ALPHA_INF), ("sjf", ALPHA_INF), ("isjl", 3),
                            ("isjl", ALPHA_INF), ("ljf", ALPHA_INF)):
                ctx = f"quiet sweeps {pol} alpha={al} B={B} M={M}"
                log(ctx)
                check(dev, ctx, a, p, o, policy=pol, B=B, alpha=al, M_kv=M, cost_c=2,
                      cost_tau=1)


@pytest.mark.parametrize("policy,alpha", [("fcfs", ALPHA_INF), ("sjf", ALPHA_INF),
                                          ("ljf", 30), ("isjl", 30), ("isjl", ALPHA_INF)])
def test_unsorted_arrivals_many_jobs(dev, policy, alpha):
    """The general variant (arrivals not in index order) at two bitmap words per
    lane and up to 16 slots per lane, with and without a KV budget."""
    rng = np.random.default_rng(zlib.crc32(f"unsorted-big:{policy}:{alpha}".encode()))
    for n, B, M in ((4096, 1024, 0), (3000, 300, 20000), (2500, 150, 0)):
        a, p, o = workload.random_tables(rng, 3, n, 40, 100, max_arrival=4000)
        ctx = f"unsorted big {policy} alpha={alpha} n={n} B={B} M={M}"
        log(ctx)
        check(dev, ctx, a, p, o, policy=policy, B=B, alpha=alpha, M_kv=M, cost_c=5,
              cost_tau=1)


@pytest.mark.parametrize("policy,alpha", [("fcfs", ALPHA_INF), ("sjf", ALPHA_INF),
                                          ("isjl", ALPHA_INF), ("isjl", 1 << 20),
                                          ("isjl", (1 << 20) - 1)])
def test_fill_sweep_queued_completions(dev, policy, alpha):
    """Up to 2 slots per lane with a long queue: FCFS, SJF and ISJL with alpha at
    least the length limit take runs of completions at once, each admitting the
    next jobs of the queue (alpha just below the limit takes the variant
    without it).  KV budgets from none to binding, all released at once,
    releases through the run (in index order and not), B from 4 to 128 and one or
    two job-bitmap words per lane."""
    rng = np.random.default_rng(zlib.crc32(f"fill:{policy}:{alpha}".encode()))
    for n, B, M, arr in ((500, 4, 0, 0), (2000, 128, 0, 0), (2000, 100, 6000, 0),
                         (1500, 64, 2500, 0), (2000, 128, 9000, 3000), (900, 37, 1500, 20000),
                         (2000, 128, 0, -6000), (1200, 90, 4000, -2000), (3000, 120, 5000, 0),
                         (4096, 64, 0, 8000)):
        a, p, o = workload.random_tables(rng, 4, n, 60, 200, max_arrival=abs(arr),
                                         sorted_arrivals=arr > 0)
        ctx = f"fill sweep {policy} alpha={alpha} n={n} B={B} M={M} arrivals={arr}"
        log(ctx)
        check(dev, ctx, a, p, o, policy=policy, B=B, alpha=alpha, M_kv=M, cost_c=3,
              cost_tau=2)


def test_rank_scratch_reuse_across_calls_and_streams(dev):
    """Every policy but FCFS takes its rank table from the library's stream-ordered
    pool: back-to-back calls of different sizes on a side stream (no host sync in
    between, the earlier tables freed on the stream) each match the oracle, and a
    call after fsched_release_cache gives the same metrics."""
    import torch
    rng = np.random.default_rng(99)
    side = torch.cuda.Stream()
    jobs = []
    for n_inst, n, B, pol, al in ((40, 700, 64, "isjl", 9), (7, 2000, 128, "sjf", ALPHA_INF),
                                  (25, 300, 16, "ljf", 5), (3, 4096, 300, "isjl", ALPHA_INF)):
        a, p, o = workload.random_tables(rng, n_inst, n, 30, 90, max_arrival=3 * n,
                                         sorted_arrivals=True)
        jobs.append((a, p, o, dict(policy=pol, B=B, alpha=al, M_kv=5000, cost_c=2, cost_tau=1)))
    outs = []
    with torch.cuda.stream(side):
        for a, p, o, kw in jobs:
            ts = [torch.from_numpy(x).to(dev, non_blocking=False) for x in (a, p, o)]
            raw, st, fi = fs.simulate(*ts, schedule=True, **kw)
            outs.append((ts, raw, st, fi))
    side.synchronize()
    fs.release_cache()  # the pool gives its memory back; the next call takes it again
    a, p, o, kw = jobs[0]
    again, _, _ = fs.simulate(*[torch.from_numpy(x).to(dev) for x in (a, p, o)], **kw)
    torch.cuda.synchronize()
    assert np.array_equal(fs.metrics_view(again), fs.metrics_view(outs[0][1]))
    for (a, p, o, kw), (_, raw, st, fi) in zip(jobs, outs):
        ctx = f"rank scratch reuse {kw}"
        log(ctx)
        ref, rs, rf = oracle.simulate(a, p, o, schedule=True, **kw)
        assert_same(ctx, fs.metrics_view(raw), ref, st.cpu().numpy(), rs, fi.cpu().numpy(), rf)


@pytest.mark.parametrize("alpha", [2, 40, 300])
def test_plan_links_in_hbm(dev, alpha):
    """ISJL with up to 8 slots per lane and 2,000 jobs: the plan-queue links would
    cap a CU below 16 waves in LDS, so they go to HBM scratch (also for the
    predicted-size and prefill variants); 4 and 8 slots per lane also take the
    kernels held to 128 VGPRs."""
    rng = np.random.default_rng(zlib.crc32(f"qlinks:{alpha}".encode()))
    for B, M, arr in ((100, 0, 0), (128, 12000, 4000), (70, 6000, -3000), (200, 30000, 3000),
                      (512, 0, 0), (400, 45000, -3000)):
        a, p, o = workload.random_tables(rng, 5, 2000, 60, 200, max_arrival=abs(arr),
                                         sorted_arrivals=arr > 0)
        kw = dict(B=B, alpha=alpha, M_kv=M, cost_c=3, cost_tau=1)
        ctx = f"plan links in HBM alpha={alpha} B={B} M={M} arrivals={arr}"
        log(ctx)
        check(dev, ctx, a, p, o, policy="isjl", **kw)
        log(ctx + " prefill")
        got, gs, gf = gpu_sim(dev, a, p, o, policy="isjl", prefill=True, **kw)
        ref, rs, rf = oracle.simulate(a, p, o, policy="isjl", schedule=True,
                                      flags=oracle.FLAG_PREFILL, **kw)
        assert_same(ctx + " prefill", got, ref, gs, rs, gf, rf)
        log(ctx + " robust")
        u = workload.prediction_upper(o, 0.5, seed=B)
        import torch
        ts = [torch.from_numpy(np.ascontiguousarray(x)).to(dev) for x in (a, p, o, u)]
        raw, st, fi = fs.simulate_robust(*ts, schedule=True, **kw)
        torch.cuda.synchronize()
        ref, rs, rf = oracle.simulate_robust(a, p, o, u, schedule=True, **kw)
        assert_same(ctx + " robust", fs.metrics_view(raw), ref, st.cpu().numpy(), rs,
                    fi.cpu().numpy(), rf)


@pytest.mark.parametrize("policy,alpha", [("fcfs", ALPHA_INF), ("sjf", ALPHA_INF), ("ljf", 4),
                                          ("isjl", 40), ("isjl", ALPHA_INF)])
def test_one_round_and_many_round_launches(dev, policy, alpha):
    """A grid whose waves are all resident at once takes the kernels that turn
    each wave's issue priority with its event count; a larger grid the kernels
    without.  On the same instances both give the same metrics and schedules
    (1, 2, 4 and 8 slots per lane; sorted, unsorted and no releases), and the
    first instances match the oracle."""
    rng = np.random.default_rng(zlib.crc32(f"rounds:{policy}:{alpha}".encode()))
    for B, arr in ((50, 400), (128, -300), (200, 300), (300, 0)):
        a, p, o = workload.random_tables(rng, 12288, 300, 40, 120, max_arrival=abs(arr),
                                         sorted_arrivals=arr > 0)
        kw = dict(policy=policy, B=B, alpha=alpha, M_kv=6000, cost_c=3, cost_tau=1)
        ctx = f"one round vs many policy={policy} alpha={alpha} B={B} arrivals={arr}"
        log(ctx)
        big, bs, bf = gpu_sim(dev, a, p, o, **kw)
        small, ss, sf = gpu_sim(dev, a[:256], p[:256], o[:256], **kw)
        assert_same(ctx, small, big[:256], ss, bs[:256], sf, bf[:256])
        ref, rs, rf = oracle.simulate(a[:6], p[:6], o[:6], schedule=True, **kw)
        assert_same(ctx + " oracle", small[:6], ref, ss[:6], rs, sf[:6], rf)


@pytest.mark.parametrize("variant", ["prefill", "robust", "robust_prefill"])
def test_one_round_and_many_round_launches_variants(dev, variant):
    """The prefill and predicted-size variants of ISJL (alpha = 40) take the
    turning-priority kernels in a grid resident at once too: the same
    instances in a one-round and a many-round launch give the same metrics and
    schedules, and the first instances match the oracle."""
    import torch
    rng = np.random.default_rng(zlib.crc32(f"rounds:{variant}".encode()))
    pre = variant.endswith("prefill")
    rob = variant.startswith("robust")
    for B, arr in ((50, 400), (128, -300), (300, 0)):
        a, p, o = workload.random_tables(rng, 12288, 300, 40, 120, max_arrival=abs(arr),
                                         sorted_arrivals=arr > 0)
        u = workload.prediction_upper(o, 0.5, seed=B)
        kw = dict(B=B, alpha=40, M_kv=6000, cost_c=3, cost_tau=1)
        ctx = f"one round vs many {variant} B={B} arrivals={arr}"
        log(ctx)

        def run(k):
            tabs = (a[:k], p[:k], o[:k]) + ((u[:k],) if rob else ())
            ts = [torch.from_numpy(np.ascontiguousarray(x)).to(dev) for x in tabs]
            if rob:
                raw, st, fi = fs.simulate_robust(*ts, prefill=pre, schedule=True, **kw)
            else:
                raw, st, fi = fs.simulate(*ts, policy="isjl", prefill=pre, schedule=True, **kw)
            torch.cuda.synchronize()
            return fs.metrics_view(raw), st.cpu().numpy(), fi.cpu().numpy()

        big, bs, bf = run(12288)
        small, ss, sf = run(256)
        assert_same(ctx, small, big[:256], ss, bs[:256], sf, bf[:256])
        flags = oracle.FLAG_PREFILL if pre else 0
        if rob:
            ref, rs, rf = oracle.simulate_robust(a[:4], p[:4], o[:4], u[:4], schedule=True,
                                                 flags=flags, **kw)
        else:
            ref, rs, rf = oracle.simulate(a[:4], p[:4], o[:4], policy="isjl", schedule=True,
                                          flags=flags, **kw)
        assert_same(ctx + " oracle", small[:4], ref, ss[:4], rs, sf[:4], rf)


@pytest.mark.parametrize("policy,alpha", [("fcfs", ALPHA_INF), ("sjf", ALPHA_INF),
                                          ("isjl", 25), ("isjl", 300), ("isjl", ALPHA_INF)])
def test_releases_behind_a_blocked_head(dev, policy, alpha):
    """Dense releases while the KV budget holds the queue's head back with slots
    free: FCFS takes no release as an event while something is queued, SJF and
    ISJL in FILL only an arrival that precedes the head and fits (in sorted and
    unsorted release order)."""
    rng = np.random.default_rng(zlib.crc32(f"blocked-head:{policy}:{alpha}".encode()))
    for n, B, M, arr in ((1000, 64, 3000, 600), (700, 16, 900, 1400), (1500, 100, 5000, -900),
                         (300, 40, 400, 2000)):
        a, p, o = workload.random_tables(rng, 6, n, 50, 120, max_arrival=abs(arr),
                                         sorted_arrivals=arr > 0)
        ctx = f"blocked head {policy} alpha={alpha} n={n} B={B} M={M} arrivals={arr}"
        log(ctx)
        check(dev, ctx, a, p, o, policy=policy, B=B, alpha=alpha, M_kv=M, cost_c=1,
              cost_tau=1)
