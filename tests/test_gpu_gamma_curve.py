"""The competitive-ratio experiment through the HIP library equals the one over
the oracle (exact optimum and ISJL makespans, so every bin)."""
import numpy as np
import pytest

import oracle
import workload
from paper_2608_02244_amd import gamma_curve as gc

pytestmark = pytest.mark.gpu


def oracle_pair(a, p, o, B, alpha, flags):
    T_opt = oracle.opt(a, p, o, B=B, alpha=alpha, M_kv=0)
    m = oracle.simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=0, cost_c=0, cost_tau=0,
                        flags=flags)
    return np.asarray(T_opt, np.int64), m["T"].astype(np.int64)


@pytest.mark.parametrize("beta_star", [False, True])
def test_gamma_curve_matches_oracle(beta_star):
    a, p, o = workload.generate("tiny_opt_1048576x8", n_inst=150, inst_begin=4096)
    alphas = [1, 2, 4, 7, 11]
    got = gc.run(gc.gpu_pair, a, p, o, alphas, B=2, beta_star=beta_star)
    ref = gc.run(oracle_pair, a, p, o, alphas, B=2, beta_star=beta_star)
    assert got == ref
