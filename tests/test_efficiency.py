"""The system-efficiency experiment on the CPU: the LMSYS-shaped workload's
moments against the ones the paper states for its sample, the driver's
arithmetic against closed forms, and the driver over the oracle."""
import numpy as np

import oracle
import workload
from paper_2608_02244_amd import efficiency as ef


def osim(a, p, o, pol, B, al, M_kv=0):
    return oracle.simulate(a, p, o, policy=pol, B=B, alpha=al, M_kv=M_kv, cost_c=0, cost_tau=1)


def test_workload_shape():
    """Mean 126, median 90, max 905 (stated for the paper's 2,000-conversation
    sample); total tokens in the output column; Poisson arrivals at 0.25 per step."""
    a, p, o = workload.generate("lmsys_shaped_256x2000", n_inst=32)
    L = p.astype(np.int64) + o
    assert (p == 0).all() and L.min() >= 1 and L.max() <= 905
    assert 118 <= L.mean() <= 134 and 86 <= np.median(L) <= 94
    assert 12000 <= L.var() <= 17000
    gaps = np.diff(a, axis=1)
    assert (gaps >= 0).all()
    assert abs(a[:, -1].mean() - 1999 / 0.25) < 0.03 * 8000


def test_paper_ratios():
    r = ef.paper_ratios()
    assert abs(r[16]["ISJL(150)"][0] - 276 / 243) < 1e-12
    assert abs(r[32]["ISJL(50)"][1] - 62 / 78) < 1e-12
    assert r[16]["LJF"] == (1.0, 1.0)


def test_unlimited_batch_closed_form():
    """B = n, every request at step 0: FCFS, SJF and LJF start everything at 0,
    so throughput = O / max len and AEL = mean len exactly."""
    _, p, o = workload.generate("lmsys_shaped_256x2000", n_inst=3, n_jobs=300)
    z = np.zeros_like(o)
    pols = (("fcfs", None), ("sjf", None), ("ljf", None))
    tab = ef.run_table(osim, z, p, o, Bs=(300,), policies=pols)
    L = (p + o).astype(np.int64)
    for k in ("FCFS", "SJF", "LJF"):
        r = tab[300][k]
        assert abs(r["throughput"] - np.mean(L.sum(1) / L.max(1))) < 1e-9
        assert abs(r["ael"] - L.mean()) < 1e-9


def test_driver_over_the_oracle():
    a, p, o = workload.generate("lmsys_shaped_256x2000", n_inst=2, n_jobs=600)
    for arr in (a, np.zeros_like(a)):
        tab = ef.run_table(osim, arr, p, o)
        for B, rows in tab.items():
            assert set(rows) == {"FCFS", "SJF", "LJF", "ISJL(50)", "ISJL(100)", "ISJL(150)"}
            for k, r in rows.items():
                assert 0 < r["throughput"] <= B
                if k == "LJF":  # batches start together at an empty machine
                    assert r["max_extent"] == 0
                if k.startswith("ISJL"):
                    al = int(k[5:-1])
                    assert r["unfair_steps"] == 0 and r["max_extent"] <= al
            assert rows["LJF"]["throughput_vs_ljf"] == 1.0
    lines = ef.format_table(tab)
    assert len(lines) == 2 + 12
