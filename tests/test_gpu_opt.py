"""GPU parity of fsched_bruteforce_opt against the oracle, through the C ABI.

The optimum makespan is unique and must equal the oracle's exactly.  Optimal
schedules are not unique: the returned one must be valid (the oracle's
re-scoring finds no violation) and reach the optimum.  At full size every
instance is also checked against properties that hold at any size: the optimum
is at most ISJL's makespan and at least the trivial lower bounds, and its
schedule re-scores (on the GPU) to the optimum with no violation.
"""
import sys
import time
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


def gpu_opt(dev, a, p, o, **kw):
    import torch
    t = [torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(dev) for x in (a, p, o)]
    T, st = fs.bruteforce_opt(*t, schedule=True, **kw)
    torch.cuda.synchronize()
    return T.cpu().numpy(), st.cpu().numpy()


def check(dev, ctx, a, p, o, **kw):
    T, st = gpu_opt(dev, a, p, o, **kw)
    ref = oracle.opt(a, p, o, **kw)
    if not np.array_equal(T, ref):
        bad = np.nonzero(T != ref)[0][:5]
        raise AssertionError(f"{ctx}: T_opt differs at {bad.tolist()}: gpu {T[bad].tolist()} "
                             f"oracle {ref[bad].tolist()}; lengths "
                             f"{(p[bad[0]] + o[bad[0]]).tolist()} arrivals {a[bad[0]].tolist()}")
    m, v = oracle.decompose(a, p, o, st, B=kw["B"], alpha=kw["alpha"], M_kv=kw.get("M_kv", 0))
    bad = np.nonzero((v != 0) | (m["T"] != T))[0]
    assert len(bad) == 0, (f"{ctx}: returned schedule invalid or not optimal at {bad[:5].tolist()}:"
                           f" violations {v[bad[:5]].tolist()} T {m['T'][bad[:5]].tolist()}")
    return T


@pytest.mark.parametrize("B", [1, 2, 3, 4, 0])
def test_random_tiny_instances(dev, B):
    rng = np.random.default_rng(zlib.crc32(f"opt:{B}".encode()))
    for trial in range(10):
        n = int(rng.integers(1, 9))
        alpha = int(rng.choice([0, 1, 2, 3, 5, ALPHA_INF]))
        M = int(rng.choice([0, 0, 12, 20]))
        a, p, o = workload.random_tables(rng, 40, n, 3, 12,
                                         max_arrival=int(rng.choice([0, 0, 6, 25])))
        ctx = f"B={B} n={n} alpha={alpha} M={M} trial={trial}"
        log(ctx)
        check(dev, ctx, a, p, o, B=B, alpha=alpha, M_kv=M)


def test_paper_instances(dev):
    for al in (1, 2, 3, 4):
        L = 2 * al + 1
        ell = np.array([[L, L, al, al]], np.int32)
        z = np.zeros_like(ell)
        assert check(dev, "over-inserting", z, z, ell, B=2, alpha=al)[0] == L + al
        ell = np.array([[3 * al - 1, 2 * al, 2 * al]], np.int32)
        z = np.zeros_like(ell)
        assert check(dev, "under-inserting", z, z, ell, B=2, alpha=al)[0] == 4 * al
    L, al = 20, 3
    arr = np.array([[0, al + 1]], np.int32)
    ell = np.array([[L, L]], np.int32)
    assert check(dev, "online adversary", arr, np.zeros_like(ell), ell, B=2, alpha=al)[0] == \
        L + al + 1
    ell = np.array([[9, 15, 5, 10, 19]], np.int32)
    z = np.zeros_like(ell)
    assert check(dev, "B=3 finding", z, z, ell, B=3, alpha=8)[0] == 20


def test_limits(dev):
    import torch
    z = np.zeros((1, 9), np.int32)
    with pytest.raises(fs.FschedError) as ei:
        gpu_opt(dev, z, z, np.ones((1, 9), np.int32), B=2, alpha=1)
    assert ei.value.code == fs.ETOOLARGE
    ell = np.array([[3, 256], [3, 4]], np.int32)
    z = np.zeros_like(ell)
    T, _ = gpu_opt(dev, z, z, ell, B=2, alpha=1)
    assert T[0] == fs.T_TOOLARGE and T[1] == oracle.opt(z[1:], z[1:], ell[1:], B=2, alpha=1)[0]


@pytest.mark.parametrize("M_kv", [16, 0])
def test_tiny_opt_workload_full_size(dev, M_kv):
    """1,048,576 instances x 8 jobs, B = 2, alpha in {1, 2, 4}; M_kv = 16 and none."""
    import torch
    w = workload.WORKLOADS["tiny_opt_1048576x8"]
    a, p, o = workload.generate(w)
    ta, tp, to = (torch.from_numpy(x).to(dev) for x in (a, p, o))
    lens = p.astype(np.int64) + o
    lb = np.maximum(lens.max(1), (lens.sum(1) + 1) // 2)
    rng = np.random.default_rng(M_kv + 1)
    sample = np.unique(np.concatenate([[0, w.n_inst - 1], rng.integers(0, w.n_inst, 150)]))
    for alpha in w.alphas:
        t0 = time.time()
        T, st = fs.bruteforce_opt(ta, tp, to, B=w.B, alpha=alpha, M_kv=M_kv, schedule=True)
        torch.cuda.synchronize()
        log(f"M_kv={M_kv} alpha={alpha}: {w.n_inst} exact optima in {time.time() - t0:.2f} s")
        Tn = T.cpu().numpy()
        raw, _, _ = fs.simulate(ta, tp, to, policy="isjl", B=w.B, alpha=alpha, M_kv=M_kv)
        dm, dv = fs.cost_decompose(ta, tp, to, st, B=w.B, alpha=alpha, M_kv=M_kv)
        torch.cuda.synchronize()
        Ti = fs.metrics_view(raw)["T"]
        dmT = fs.metrics_view(dm)["T"]
        assert (Tn <= Ti).all() and (Tn >= lb).all()
        assert (dv.cpu().numpy() == 0).all() and np.array_equal(dmT, Tn)
        ref = oracle.opt(a[sample], p[sample], o[sample], B=w.B, alpha=alpha, M_kv=M_kv)
        assert np.array_equal(Tn[sample], ref)
        r = Tn / Ti
        log(f"  min T_opt/T_isjl = {r.min():.4f} at instance {int(r.argmin())}")


# Instances of the tiny workload (first 4,096) whose search fills the first
# pass's LDS memo before it ends (B = 3 or 4, large alpha): the second pass with
# its large memo must finish them, at the oracle's optimum.
CAPPED = [(4, 0, 11, 158), (4, 0, 11, 862), (4, 0, 11, 3430), (4, 0, 15, 1189),
          (3, 0, 15, 2273), (4, 16, 11, 1504), (4, 16, 11, 1508)]


def test_searches_beyond_the_first_pass_cap(dev):
    import torch
    a, p, o = workload.generate("tiny_opt_1048576x8", n_inst=4096)
    for B, M, al, i in CAPPED:
        ctx = f"instance {i} B={B} M_kv={M} alpha={al}"
        log(ctx)
        t = [torch.from_numpy(x[i:i + 1].copy()).to(dev) for x in (a, p, o)]
        T, st = fs.bruteforce_opt(*t, B=B, alpha=al, M_kv=M, schedule=True)
        torch.cuda.synchronize()
        T = T.cpu().numpy()
        ref = oracle.opt(a[i:i + 1], p[i:i + 1], o[i:i + 1], B=B, alpha=al, M_kv=M)
        assert int(T[0]) == int(ref[0]), f"{ctx}: gpu {int(T[0])} oracle {int(ref[0])}"
        m, v = oracle.decompose(a[i:i + 1], p[i:i + 1], o[i:i + 1], st.cpu().numpy(), B=B,
                                alpha=al, M_kv=M)
        assert int(v[0]) == 0 and int(m["T"][0]) == int(T[0]), ctx
