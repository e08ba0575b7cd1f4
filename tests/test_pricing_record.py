"""The linear-pricing table of Section 5.2 under the adopted ISJL reading, as a
pinned outcome: ``tests/golden/pricing_record.json`` (written by
``tests/golden/make_pricing_record.py`` from the oracle only) holds 200
replications of LJF, FCFS and ISJL and the means of the alternative readings of
``oracle/readings.py``.  These tests check the record against the oracle, pin
what it says, and keep the paper's ISJL rows as an expected failure."""
import json
import os

import numpy as np
import pytest

import oracle
import workload
from oracle import readings

HERE = os.path.dirname(os.path.abspath(__file__))
REC = json.load(open(os.path.join(HERE, "golden", "pricing_record.json")))
ALPHAS = REC["alphas"]
A = REC["adopted"]


def _ratios():
    TL = np.array(A["T_ljf"], dtype=float)
    return np.array(A["isjl"]["T"], dtype=float) / TL[:, None]


@pytest.mark.parametrize("rep", [0, 1])
def test_readings_module_defaults_are_the_oracle(rep):
    """With the default switches ``readings.simulate`` is the oracle's ISJL, and
    ``brk="resume"`` is the oracle's resume flag (schedules equal job by job)."""
    a, p, o = workload.pricing_instance(rep)
    lens = [int(x) for x in o[0]]
    for al in (50, 300):
        for flags, kw in ((0, {}), (oracle.FLAG_RESUME_FILL, {"brk": "resume"})):
            _, st, _ = oracle.simulate(a, p, o, policy="isjl", B=50, alpha=al, flags=flags,
                                       schedule=True)
            assert readings.simulate(lens, 50, al, **kw) == st[0].tolist()


def test_record_rows_equal_the_oracle():
    for rep in range(3):
        a, p, o = workload.pricing_instance(rep)
        assert int(o.shape[1]) == A["n"][rep]
        lj = oracle.simulate(a, p, o, policy="ljf", B=50, alpha=0)
        assert int(lj["T"][0]) == A["T_ljf"][rep] and int(lj["Q"][0]) == A["Q"][rep]
        fc = oracle.simulate(a, p, o, policy="fcfs", B=50, alpha=oracle.ALPHA_INF)
        assert int(fc["T"][0]) == A["fcfs"]["T"][rep] and int(fc["E"][0]) == A["fcfs"]["E"][rep]
        for k, al in enumerate(ALPHAS):
            m = oracle.simulate(a, p, o, policy="isjl", B=50, alpha=al)
            assert int(m["T"][0]) == A["isjl"]["T"][rep][k]
            assert int(m["E"][0]) == A["isjl"]["E"][rep][k]
            mr = oracle.simulate(a, p, o, policy="isjl", B=50, alpha=al,
                                 flags=oracle.FLAG_RESUME_FILL)
            assert int(mr["T"][0]) == A["isjl_resume"]["T"][rep][k]


def test_schedule_free_terms_and_baselines_agree_with_the_paper():
    """What does not depend on the ISJL reading matches the printed table within
    its five-replication sampling error: tau Q (32.07), FCFS against LJF
    (throughput ratio 39.78 / 39.83) and FCFS's average extent (566.26)."""
    n = len(A["T_ljf"])
    q = np.array(A["Q"], dtype=float) * 1e-6
    assert abs(q.mean() - 32.07) < 3 * q.std() / np.sqrt(5)
    f = np.array(A["fcfs"]["T"], dtype=float) / np.array(A["T_ljf"], dtype=float)
    assert abs(f.mean() - 39.83 / 39.78) < 3 * f.std() / np.sqrt(5)
    ext = np.array(A["fcfs"]["sum_extent"], dtype=float) / np.array(A["fcfs"]["busy_steps"])
    assert abs(ext.mean() - 566.26) < 3 * ext.std() / np.sqrt(5)
    assert n == REC["replications_adopted"] >= 200


def test_isjl_rows_pinned_outcome():
    """Under the adopted reading ISJL is fair at every step and finishes later
    than LJF at every alpha, by the recorded margins (mean T_ISJL / T_LJF over
    200 replications); the paper prints ISJL ahead of LJF."""
    r = _ratios().mean(0)
    np.testing.assert_allclose(r, [1.342, 1.388, 1.386, 1.675, 1.658, 1.607, 1.412], atol=5e-4)
    assert all(u == 0 for u in A["isjl"]["unfair_steps_total"])
    assert all(x > 1.3 for x in r)
    assert all(x < 1 for x in REC["paper"]["T_over_T_LJF"])
    ext = np.array(A["isjl"]["avg_extent"]).mean(0)
    assert all(e <= al for e, al in zip(ext, ALPHAS))


@pytest.mark.xfail(strict=True, reason="the paper's ISJL rows are not reproduced under the "
                                       "adopted reading (Section 5.2); see the readings record")
def test_paper_isjl_rows_within_sampling_error():
    r = _ratios()
    se5 = r.std(0) / np.sqrt(5)
    assert np.all(np.abs(r.mean(0) - np.array(REC["paper"]["T_over_T_LJF"])) <= 3 * se5)


def test_no_reading_reaches_the_paper_and_no_bound_excludes_it():
    """Recorded over 40 replications: every fair reading stays above the paper's
    T / T_LJF at alpha = 500 (0.819); the hand-built fair cohort schedule reaches
    about 0.9, as fast as the best fair reading and far ahead of the adopted one;
    and the volume bound O / (B T_LJF) lies below 0.819, so it cannot show the
    paper's number unreachable by a fair schedule."""
    rd = REC["readings"]
    fair = {k: v for k, v in rd.items() if max(v["unfair_step_fraction"]) == 0.0}
    assert "adopted" in fair and "resume" in fair
    cohort = rd["fair cohort construction (not ISJL)"]["T_over_T_LJF"][-1]
    for name, v in fair.items():
        assert v["T_over_T_LJF"][-1] > REC["paper"]["T_over_T_LJF"][-1], name
        assert cohort <= v["T_over_T_LJF"][-1] + 1e-3, name
    assert cohort < 0.9 < rd["adopted"]["T_over_T_LJF"][-1]
    vol = np.mean(np.array(A["O"], dtype=float) / (50 * np.array(A["T_ljf"], dtype=float)))
    assert vol < REC["paper"]["T_over_T_LJF"][-1]


def test_cohort_schedule_is_fair_on_the_oracle_rescorer():
    a, p, o = workload.pricing_instance(0)
    lens = [int(x) for x in o[0]]
    for al in (50, 500):
        st = np.array(readings.cohort_schedule(lens, 50, al), np.int32).reshape(1, -1)
        m, viol = oracle.decompose(a, p, o, st, B=50, alpha=al)
        assert int(viol[0]) == 0 and int(m["unfair_steps"][0]) == 0
