"""fsched_simulate_noalloc against fsched_simulate through the C ABI, on the GPU:
metrics, starts and finishes equal element by element on two calls in a row,
the second smaller and of another shape, so the fixed scratch buffer holds the
first call's contents when the second runs."""
import ctypes
import sys

import numpy as np
import pytest

import workload
import paper_2608_02244_amd as fs

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


def both(dev, name, n_inst, **kw):
    import torch
    w = workload.WORKLOADS[name]
    a, p, o = workload.generate(w, n_inst=n_inst)
    t = [torch.from_numpy(x).to(dev) for x in (a, p, o)]
    ref, rs, rf = fs.simulate(*t, schedule=True, B=w.B, M_kv=w.M_kv, cost_c=w.cost_c,
                              cost_tau=w.cost_tau, **kw)
    out = torch.zeros((n_inst, 13), dtype=torch.int64, device=dev)
    st = torch.zeros((n_inst, w.n_jobs), dtype=torch.int32, device=dev)
    fi = torch.zeros((n_inst, w.n_jobs), dtype=torch.int32, device=dev)
    fs.simulate_noalloc(*t, out, start=st, finish=fi, B=w.B, M_kv=w.M_kv, cost_c=w.cost_c,
                        cost_tau=w.cost_tau, **kw)
    torch.cuda.synchronize()
    g, r = fs.metrics_view(out), fs.metrics_view(ref)
    assert (r["T"] > 0).all()
    for f in fs.METRIC_FIELDS:
        assert np.array_equal(g[f], r[f]), f"{name} {kw}: metric {f} differs"
    assert torch.equal(st, rs) and torch.equal(fi, rf), f"{name} {kw}: schedules differ"


def test_noalloc_equals_simulate_two_calls(dev):
    # first call: ISJL at a finite alpha with 128 workers uses both parts of the
    # scratch (rank table and plan-queue links); second: fewer, shorter instances
    log("noalloc call 1: bimodal_sweep 512 instances, ISJL alpha=256")
    both(dev, "bimodal_sweep_4096x2000", 512, policy="isjl", alpha=256)
    log("noalloc call 2: pareto 192 instances, ISJL alpha=128 (8 slots per lane)")
    both(dev, "pareto_65536x2000", 192, policy="isjl", alpha=128)
    log("noalloc call 3: lognormal 96 instances, ISJL alpha=64")
    both(dev, "lognormal_4096x1000", 96, policy="isjl", alpha=64)
    log("noalloc call 4: lognormal 40 instances, SJF")
    both(dev, "lognormal_4096x1000", 40, policy="sjf", alpha=fs.ALPHA_INF)


def test_noalloc_refuses_oversized_scratch(dev):
    import torch
    a = torch.zeros((65536, 2000), dtype=torch.int32, device=dev)
    out = torch.empty((65536, 13), dtype=torch.int64, device=dev)
    with pytest.raises(fs.FschedError) as e:
        fs.simulate_noalloc(a, a, a, out, policy="isjl", B=512, alpha=128, M_kv=1 << 20)
    assert e.value.code == fs.ESCRATCH
