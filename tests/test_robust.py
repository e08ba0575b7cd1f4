"""Robust-ISJL (Section 3.4) in the oracle, and the experiment driver on the CPU.

Pins: hand-traced examples (tests/golden/robust_examples.json), exact
predictions reduce to ISJL, the fairness theorem (any upper bounds), the
schedules' validity by the independent re-scorer, the packable residual error
against brute force over set partitions and the remark's closed form, and the
guarantee T_R <= 4/3 (T_OPT + Delta_pack) with its corollary on a sample of tiny
offline instances.  The first step of the guarantee's proof (T_R <= T_ISJL on the
proxy instance) does not hold for every instance: a recorded case checks that.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
import workload
from oracle import ALPHA_INF
from paper_2608_02244_amd import robust as rb

HERE = os.path.dirname(os.path.abspath(__file__))


def oracle_quad(a, p, o, u, B, alpha, M_kv=0):
    mr = oracle.simulate_robust(a, p, o, u, B=B, alpha=alpha, M_kv=M_kv, cost_c=0, cost_tau=0)
    T_opt = oracle.opt(a, p, o, B=B, alpha=alpha, M_kv=M_kv)
    mi = oracle.simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=M_kv, cost_c=0,
                         cost_tau=0)
    mu = oracle.simulate(a, p, u, policy="isjl", B=B, alpha=alpha, M_kv=M_kv, cost_c=0,
                         cost_tau=0)
    return mr["T"], mr["unfair_steps"], T_opt, mi["T"], mu["T"]


def test_hand_traced_examples():
    cases = json.load(open(os.path.join(HERE, "golden", "robust_examples.json")))
    for c in cases:
        t = [np.array([c[k]], np.int32) for k in ("arrival", "prompt", "output", "upper")]
        m, s, f = oracle.simulate_robust(*t, B=c["B"], alpha=c["alpha"], M_kv=c["M_kv"],
                                         schedule=True)
        assert m["T"][0] == c["T_robust"]
        assert s[0].tolist() == c["start_robust"] and f[0].tolist() == c["finish_robust"]
        m, s, f = oracle.simulate(*t[:3], policy="isjl", B=c["B"], alpha=c["alpha"],
                                  M_kv=c["M_kv"], schedule=True)
        assert m["T"][0] == c["T_isjl"]
        assert s[0].tolist() == c["start_isjl"] and f[0].tolist() == c["finish_isjl"]


def _random(seed, n_inst=40, n=24):
    rng = np.random.default_rng(seed)
    a, p, o = workload.random_tables(rng, n_inst, n, 12, 40, max_arrival=60)
    u = workload.prediction_upper(o, 1.5, seed=seed)
    return a, p, o, u


@pytest.mark.parametrize("alpha,B,M", [(0, 3, 0), (3, 4, 0), (9, 6, 200), (25, 0, 0),
                                       (ALPHA_INF, 5, 150)])
def test_exact_predictions_are_isjl(alpha, B, M):
    a, p, o, _ = _random(11 + alpha % 97)
    r, rs, rf = oracle.simulate_robust(a, p, o, o, B=B, alpha=alpha, M_kv=M, cost_c=3,
                                       cost_tau=1, schedule=True)
    i, is_, if_ = oracle.simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=M, cost_c=3,
                                  cost_tau=1, schedule=True)
    assert (r == i).all() and (rs == is_).all() and (rf == if_).all()


@pytest.mark.parametrize("alpha,B,M", [(0, 3, 0), (2, 4, 0), (7, 6, 220), (30, 0, 0)])
def test_fair_and_valid_for_any_upper_bound(alpha, B, M):
    """Fairness theorem: no step with a progress range above alpha whatever the
    upper bounds; the schedule re-scored from its start steps alone is valid
    (releases, B, true reservations within M) and gives the same metrics."""
    a, p, o, u = _random(5 + alpha)
    m, s, f = oracle.simulate_robust(a, p, o, u, B=B, alpha=alpha, M_kv=M, cost_c=2, cost_tau=1,
                                     schedule=True)
    assert (m["unfair_steps"] == 0).all() and (m["max_extent"] <= alpha).all()
    assert (f - s == p + o).all()
    d, viol = oracle.decompose(a, p, o, s, B=B, alpha=alpha, M_kv=M, cost_c=2, cost_tau=1)
    assert (viol == 0).all()
    for k in ("T", "E", "C", "W", "sum_completion", "peak_kv", "max_extent"):
        assert (d[k] == m[k]).all(), k


def test_upper_below_output_is_rejected():
    a, p, o, u = _random(3, n_inst=1, n=6)
    u = u.copy()
    u[0, 2] = o[0, 2] - 1
    with pytest.raises(oracle.OracleError):
        oracle.simulate_robust(a, p, o, u, B=2, alpha=3)


def _delta_pack_brute(length, slack, alpha, B):
    """Every set partition of the jobs (restricted growth strings)."""
    n = len(length)
    best = None
    for rgs in itertools.product(range(n), repeat=n):
        if rgs[0] != 0 or any(rgs[i] > max(rgs[:i]) + 1 for i in range(1, n)):
            continue
        groups = {}
        for j, g in enumerate(rgs):
            groups.setdefault(g, []).append(j)
        ok = all(len(G) <= (B or n) and max(length[j] for j in G) - min(length[j] for j in G)
                 <= alpha for G in groups.values())
        if ok:
            v = sum(max(slack[j] for j in G) for G in groups.values())
            best = v if best is None else min(best, v)
    return best


def test_delta_pack_against_set_partitions():
    rng = np.random.default_rng(4)
    for _ in range(60):
        n = int(rng.integers(1, 7))
        L = rng.integers(1, 12, n)
        e = rng.integers(0, 6, n)
        al = int(rng.integers(0, 8))
        B = int(rng.integers(0, 4))
        assert rb.delta_pack(L[None], e[None], al, B)[0] == _delta_pack_brute(L, e, al, B)


def test_delta_pack_closed_forms():
    """All lengths in one alpha-window with equal slack e: ceil(n / B) e (the
    remark after the corollary); alpha = 0 with distinct lengths: the summed
    slack Delta (only singletons); B unlimited and one window: the largest slack."""
    L = np.array([[10, 11, 12, 13, 14, 10, 12]])
    for B in (1, 2, 3, 7):
        assert rb.delta_pack(L, np.full_like(L, 5), 4, B)[0] == -(-7 // B) * 5
    e = np.array([[3, 0, 2, 7, 1, 4, 4]])
    assert rb.delta_pack(np.array([[1, 2, 3, 4, 5, 6, 7]]), e, 0, 3)[0] == e.sum()
    assert rb.delta_pack(L, e, 4, 0)[0] == e.max()


def test_guarantee_and_corollary_on_tiny_instances():
    """T_R <= 4/3 (T_OPT + Delta_pack) and the corollary on a sample of the tiny
    offline workload at several slacks; fairness holds throughout."""
    a, p, o = workload.generate("tiny_opt_1048576x8", n_inst=120)
    for slack in (0.0, 0.5, 2.0):
        u = workload.prediction_upper(o, slack, seed=21)
        res = rb.run(oracle_quad, a, p, o, u, [1, 3, 7], B=2)
        for r in res["rows"]:
            assert r["unfair"] == 0
            assert r["thm_violations"] == 0 and r["cor_violations"] == 0, r
            if slack == 0.0:
                assert r["mean_r_over_isjl"] == 1.0 and r["mean_delta_pack"] == 0.0


def test_proof_first_step_can_fail():
    """The guarantee's proof bounds T_R by ISJL on the proxy instance (the same
    decisions run with shorter jobs).  Robust-ISJL's guard reads true progress,
    so an early completion changes later decisions: on this instance (B = 2,
    alpha = 7, one job 2 steps shorter than predicted) T_R = 38 > 36 = T_ISJL(I_u),
    while T_OPT = 35 and the guarantee holds (3 * 38 <= 4 * (35 + 2))."""
    o = np.array([[11, 13, 4, 12, 2, 10, 12, 5]], np.int32)
    u = o.copy()
    u[0, 3] += 2
    z = np.zeros_like(o)
    T_r, unfair, T_opt, T_i, T_u = oracle_quad(z, z, o, u, 2, 7)
    assert (int(T_r[0]), int(T_u[0]), int(T_opt[0])) == (38, 36, 35)
    assert unfair[0] == 0
    assert rb.delta_pack(o, u - o, 7, 2)[0] == 2
    _, s, _ = oracle.simulate_robust(z, z, o, u, B=2, alpha=7, schedule=True)
    _, viol = oracle.decompose(z, z, o, s, B=2, alpha=7)
    assert viol[0] == 0
