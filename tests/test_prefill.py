"""The prefill-at-admission variant in the oracle: the prompt is processed when
the job is admitted, the job then runs one step per output token, its KV
footprint is prompt + decode progress (the Section 5 batch cost takes the
largest footprint), fairness (eq. (1)) is over decode progress, and a job
reserves prompt + output of the KV budget.

Pins: hand-traced examples, the chunked reading at zero prompts, the profit-decomposition
identity (Section 5) C = c T + tau (Q + E) with Q computed from the lengths alone, the
single-worker case (no externality), fairness, and the schedule's validity
against the budget and capacity."""
import json
import os

import numpy as np
import pytest

import oracle
import workload
from oracle import ALPHA_INF, FLAG_PREFILL

HERE = os.path.dirname(os.path.abspath(__file__))
POLS = [("fcfs", ALPHA_INF), ("sjf", ALPHA_INF), ("ljf", 0), ("isjl", 0), ("isjl", 3),
        ("isjl", 12), ("isjl", ALPHA_INF)]


def test_hand_traced_examples():
    for c in json.load(open(os.path.join(HERE, "golden", "prefill_examples.json"))):
        t = [np.array([c[k]], np.int32) for k in ("arrival", "prompt", "output")]
        m, s, f = oracle.simulate(*t, policy=c["policy"], B=c["B"], alpha=c["alpha"],
                                  M_kv=c["M_kv"], cost_c=c["cost_c"], cost_tau=c["cost_tau"],
                                  flags=FLAG_PREFILL, schedule=True)
        assert s[0].tolist() == c["start"] and f[0].tolist() == c["finish"]
        for k, v in c["metrics"].items():
            assert int(m[k][0]) == v, k


def _tables(seed, n_inst=30, n=20, max_arrival=40):
    rng = np.random.default_rng(seed)
    return workload.random_tables(rng, n_inst, n, 15, 30, max_arrival=max_arrival)


@pytest.mark.parametrize("policy,alpha", POLS)
def test_zero_prompts_are_the_chunked_reading(policy, alpha):
    a, _, o = _tables(1)
    z = np.zeros_like(o)
    for M in (0, 90):
        r = oracle.simulate(a, z, o, policy=policy, B=4, alpha=alpha, M_kv=M, cost_c=3,
                            cost_tau=1, flags=FLAG_PREFILL, schedule=True)
        b = oracle.simulate(a, z, o, policy=policy, B=4, alpha=alpha, M_kv=M, cost_c=3,
                            cost_tau=1, schedule=True)
        for x, y in zip(r, b):
            assert (x == y).all()


@pytest.mark.parametrize("policy,alpha", POLS)
def test_identities_fairness_and_validity(policy, alpha):
    a, p, o = _tables(2 + alpha % 50)
    B, M, c, tau = 4, 150, 7, 2
    m, s, f = oracle.simulate(a, p, o, policy=policy, B=B, alpha=alpha, M_kv=M, cost_c=c,
                              cost_tau=tau, flags=FLAG_PREFILL, schedule=True)
    P, O = p.astype(np.int64), o.astype(np.int64)
    assert (f - s == O).all() and (s >= a).all()
    assert (m["O"] == (P + O).sum(1)).all()
    assert (m["Q"] == (O * P + O * (O + 1) // 2).sum(1)).all()
    assert (m["C"] == c * m["T"] + tau * (m["Q"] + m["E"])).all()
    assert (m["E"] >= 0).all() and (m["sum_completion"] == f.sum(1)).all()
    if policy in ("ljf", "isjl"):
        assert (m["unfair_steps"] == 0).all() and (m["max_extent"] <= alpha).all()
    for i in range(len(m)):
        T = int(m["T"][i])
        assert T == f[i].max()
        for t in range(T):
            act = (s[i] <= t) & (t < f[i])
            assert act.sum() <= B
            if act.sum() >= 2:
                assert (P[i][act] + O[i][act]).sum() <= M


def test_single_worker_has_no_externality():
    a, p, o = _tables(9)
    m = oracle.simulate(a, p, o, policy="fcfs", B=1, alpha=ALPHA_INF, cost_c=0, cost_tau=1,
                        flags=FLAG_PREFILL)
    assert (m["E"] == 0).all() and (m["C"] == m["Q"]).all() and (m["W"] == m["Q"]).all()
