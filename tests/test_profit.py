"""The linear-pricing experiment (profit and cost alignment), on the CPU: the
acceptance draws against their expectation and the paper's printed averages,
and the driver run over the oracle against the properties the paper states."""
import math
import zlib

import numpy as np
import pytest

import oracle
import workload
from paper_2608_02244_amd import profit


def oracle_simulate(a, p, o, policy, B, alpha):
    return oracle.simulate(a, p, o, policy=policy, B=B, alpha=alpha, M_kv=0, cost_c=0,
                           cost_tau=0)


def acceptance_expectation(n=400, o_max=1000):
    o = np.arange(1, o_max + 1)
    b = np.ceil(o / (o_max // 10))
    pr = np.maximum(0.0, 1.0 - o / ((2 * b - 1) * (o_max // 10)))
    q = o * (o + 1) / 2
    return (n * pr.mean(), n * (pr * o).mean(), n * (pr * q).mean(),
            n * (pr * q * q).mean() - n * (pr * q).mean() ** 2)


def test_acceptance_draws_match_their_expectation():
    """Many replications: accepted count and Q average to the model's expectation
    (summed directly over the 1,000 lengths)."""
    en, eo, eq, vq = acceptance_expectation()
    R = 400
    ns, qs = [], []
    for r in range(R):
        _, _, o = workload.pricing_instance(r, seed=11)
        ns.append(o.shape[1])
        qs.append(float((o.astype(np.int64) * (o + 1) // 2).sum()))
    assert abs(np.mean(ns) - en) < 4 * math.sqrt(en / R)
    assert abs(np.mean(qs) - eq) < 4 * math.sqrt(vq / R)


def test_acceptance_draws_match_the_papers_averages():
    """The paper prints 5-replication averages tau*Q = 32.07 and revenue
    (profit + cost of any row) = 197.14 (Table of the profit and cost
    decomposition, n = 400, B = 50): the model's expectation lies within three
    standard errors of a 5-replication mean of them."""
    _, eo, eq, vq = acceptance_expectation()
    tau, p0 = 1e-6, 1 / 500
    assert abs(tau * eq - 32.07) < 3 * tau * math.sqrt(vq / 5)
    assert abs(p0 * eo - (128.73 + 68.41)) < 0.05 * p0 * eo


def test_length_buckets_and_probabilities():
    """Edge lengths of the buckets: probability 1 - o / ((2b - 1) 100)."""
    lens, acc, p0 = workload.pricing_requests(0)
    assert p0 == 1 / 500 and lens.min() >= 1 and lens.max() <= 1000
    # a length of 100 sits in bucket 1 (probability 0), 101 in bucket 2
    o = np.array([100, 101, 200, 901, 1000])
    b = (o + 99) // 100
    pr = np.maximum(0, 1 - o / ((2 * b - 1) * 100))
    assert pr[0] == 0.0 and abs(pr[1] - (1 - 101 / 300)) < 1e-15 and pr[4] == 1 - 1000 / 1900


@pytest.fixture(scope="module")
def table():
    return profit.run_table(oracle_simulate, replications=3)


def test_intrinsic_term_and_revenue_are_schedule_free(table):
    """Profit-decomposition theorem (Section 5): Q does not depend on the schedule (nor does the revenue)."""
    for r in range(3):
        rows = [table["metrics"][k][r] for k in table["metrics"]]
        assert len({int(x["Q"]) for x in rows}) == 1
        assert len({int(x["O"]) for x in rows}) == 1


def test_ljf_has_no_externality(table):
    v = table["table"]["LJF"]
    assert v["tauE"] == 0.0 and v["avg_extent"] == 0.0


def test_isjl_extent_within_alpha_and_ordering(table):
    """Fairness bounds every step's extent by alpha, so its average too; FCFS has
    no fairness guard and the largest extent; profit FCFS < LJF."""
    t = table["table"]
    ext = [t[f"ISJL(alpha={a})"]["avg_extent"] for a in profit.ALPHAS]
    for a, e in zip(profit.ALPHAS, ext):
        assert e <= a
    assert t["FCFS"]["avg_extent"] > max(ext)
    assert t["FCFS"]["profit"] < t["LJF"]["profit"]
    # LJF has the largest profit of all rows, as in the paper's table (its E is 0
    # and c is small).
    assert max(v["profit"] for v in t.values()) == t["LJF"]["profit"]
    # ISJL's makespan is pinned against LJF's: on these replications ISJL under
    # the adopted reading finishes after LJF at every alpha (the paper prints it
    # ahead); test_pricing_record.py pins the 200-replication means and keeps
    # the paper's rows as an expected failure.
    for a in profit.ALPHAS:
        assert t[f"ISJL(alpha={a})"]["throughput"] < t["LJF"]["throughput"]


def test_cost_identity_in_integers():
    """C = c T + tau (Q + E) exactly, with integer c and tau (Section 5)."""
    a, p, o = workload.pricing_instance(0)
    for pol, al in profit.POLICIES:
        m = oracle.simulate(a, p, o, policy=pol, B=50,
                            alpha=profit.ALPHA_INF if al is None else al, M_kv=0,
                            cost_c=7, cost_tau=3)
        assert int(m["C"][0]) == 7 * int(m["T"][0]) + 3 * (int(m["Q"][0]) + int(m["E"][0]))


def test_pairwise_profit_difference_and_break_even():
    """Section 5's pairwise comparison: with the same accepted requests,
    profit(A) - profit(B) = c (T_B - T_A) + tau (E_B - E_A); against LJF (E = 0)
    the difference vanishes at c* = tau E_A / (T_LJF - T_A) and changes sign
    there (the side depends on the sign of T_LJF - T_A)."""
    a, p, o = workload.pricing_instance(1)
    rows = {f"{pol}{al}": oracle_simulate(a, p, o, pol, 50, profit.ALPHA_INF if al is None else al)[0]
            for pol, al in profit.POLICIES}
    lj = rows["ljfNone"]
    rng = np.random.default_rng(3)
    for name, r in rows.items():
        for _ in range(3):
            c, tau = float(rng.uniform(0, 0.05)), float(rng.uniform(0, 1e-5))
            d = profit.row_terms(r, c, tau, 1 / 500)["profit"] - \
                profit.row_terms(lj, c, tau, 1 / 500)["profit"]
            want = c * (int(lj["T"]) - int(r["T"])) + tau * (int(lj["E"]) - int(r["E"]))
            assert abs(d - want) <= 1e-9 * max(1.0, abs(want))
        dT = int(lj["T"]) - int(r["T"])
        if dT != 0 and int(r["E"]) > 0:
            c_star = 1e-6 * int(r["E"]) / dT
            if c_star > 0:
                for c, sgn in ((c_star * 1.01, 1), (c_star * 0.99, -1)):
                    d = profit.row_terms(r, c, 1e-6, 1 / 500)["profit"] - \
                        profit.row_terms(lj, c, 1e-6, 1 / 500)["profit"]
                    assert np.sign(d) == sgn * np.sign(dT)


def oracle_simulate_batch(a, p, o, alpha, B, M_kv):
    m, _, fi = oracle.simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=M_kv,
                               cost_c=0, cost_tau=0, schedule=True)
    return m, fi


def test_q_over_o_matches_the_token_sum():
    """Q / O from the token-level sums (r = a + 1): sum_k k over each job."""
    o = np.array([[1, 2, 3, 10]], np.int32)
    p = np.zeros_like(o)
    want = sum(sum(range(1, x + 1)) for x in (1, 2, 3, 10)) / 16
    assert profit.q_over_o(p, o) == want
    assert profit.alpha_cost(0.5, p, o) == 0.5 * want


def test_alpha_calibration_replay_on_the_oracle():
    """Every alpha-fair schedule has E <= alpha O, so at alpha = delta Q / O the
    externality stays within delta Q; the chosen alpha minimises c T + tau E
    among the grid points that meet the targets."""
    a, p, o = workload.generate("lognormal_4096x1000", n_inst=6, n_jobs=120)
    deltas = (0.0, 0.05, 0.1, 0.2, 0.5, 1.0)
    res = profit.calibrate_alpha(oracle_simulate_batch, a, p, o, deltas, B=16, M_kv=20000)
    for g in res["grid"]:
        assert g["E_within_alpha_O"] and g["externality_within_delta"]
    best = min(res["grid"], key=lambda g: (g["sched_cost"], g["alpha"]))
    assert res["alpha_star"] == best["alpha"]
    # a throughput target above every grid point leaves nothing to choose
    top = max(g["throughput"] for g in res["grid"])
    assert profit.calibrate_alpha(oracle_simulate_batch, a, p, o, deltas, B=16, M_kv=20000,
                                  min_throughput=top * 1.01)["alpha_star"] is None
