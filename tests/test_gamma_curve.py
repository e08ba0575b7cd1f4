"""The competitive-ratio experiment on the CPU: the curve's stated properties,
the exact integer comparison, and the driver over the oracle (which must flag
the recorded counterexample to the curve)."""
import json
import math
import os
from fractions import Fraction

import numpy as np

import oracle
import workload
from paper_2608_02244_amd import gamma_curve as gc

HERE = os.path.dirname(os.path.abspath(__file__))


def oracle_pair(a, p, o, B, alpha, flags):
    T_opt = oracle.opt(a, p, o, B=B, alpha=alpha, M_kv=0)
    m = oracle.simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=0, cost_c=0, cost_tau=0,
                        flags=flags)
    return np.asarray(T_opt, np.int64), m["T"].astype(np.int64)


def test_curve_shape_as_stated():
    """Minimum 3/4 at gamma = 1/2 (both branches agree there), 4/5 at 1/3,
    decreasing then increasing, tending to 1 at both ends."""
    assert gc.cr_gamma(50, 100) == Fraction(3, 4)
    assert Fraction(100 + 50, 100 + 100) == Fraction(2 * 100 - 50, 3 * 100 - 100)
    assert gc.cr_gamma(1, 3) == Fraction(4, 5)
    vals = [gc.cr_gamma(a, 1000) for a in range(1, 1000)]
    k = vals.index(min(vals))
    assert k + 1 == 500
    assert all(vals[i] > vals[i + 1] for i in range(k))
    assert all(vals[i] < vals[i + 1] for i in range(k, len(vals) - 1))
    assert vals[0] > Fraction(99, 100) and vals[-1] > Fraction(99, 100)


def test_beta_star_constant():
    """(25 + sqrt 17) / 38 is the B = 2 bound at beta* = (sqrt 17 - 1) alpha / 4:
    min{(alpha + 2 beta)/(alpha + 3 beta), 4 alpha / (6 alpha - beta)} there."""
    b = (math.sqrt(17) - 1) / 4
    v = min((1 + 2 * b) / (1 + 3 * b), 4 / (6 - b))
    assert abs(v - gc.CR_BETA_STAR) < 1e-12 and abs(gc.CR_BETA_STAR - 0.7664) < 1e-4


def test_recorded_counterexample_is_below_the_curve():
    """The B = 2 instance {18, 13, 13, 8, 1}, alpha = 7 (ISJL 35, optimum 27)."""
    rec = json.load(open(os.path.join(HERE, "golden", "cr_findings.json")))
    case = next(c for c in rec if c["B"] == 2)
    o = np.array([case["lengths"]], np.int32)
    z = np.zeros_like(o)
    res = gc.run(oracle_pair, z, z, o, [case["alpha"]], B=2)
    assert sum(r["below"] for r in res["bins"]) == 1
    assert res["min_ratio"] == Fraction(27, 35)


def test_driver_on_a_sample_of_the_tiny_workload():
    a, p, o = workload.generate("tiny_opt_1048576x8", n_inst=60)
    res = gc.run(oracle_pair, a, p, o, [1, 3, 6], B=2)
    assert sum(r["n"] for r in res["bins"]) > 0
    for r in res["bins"]:
        if r["n"]:
            assert r["min_ratio"] <= 1 and r["curve_min"] >= Fraction(3, 4)
