"""The linear-pricing experiment through the HIP library: every integer metric of
every (replication, policy) equals the oracle's, hence the whole table."""
import numpy as np
import pytest

import oracle
from paper_2608_02244_amd import profit

pytestmark = pytest.mark.gpu


def oracle_simulate(a, p, o, policy, B, alpha):
    return oracle.simulate(a, p, o, policy=policy, B=B, alpha=alpha, M_kv=0, cost_c=0,
                           cost_tau=0)


def test_profit_table_matches_oracle():
    got = profit.run_table(profit.gpu_simulate, replications=5)
    ref = profit.run_table(oracle_simulate, replications=5)
    for k in ref["metrics"]:
        for g, r in zip(got["metrics"][k], ref["metrics"][k]):
            for f in r.dtype.names:
                assert int(g[f]) == int(r[f]), (k, f)
    assert got["table"] == ref["table"]
    assert got["breakeven"] == ref["breakeven"]


def oracle_simulate_batch(a, p, o, alpha, B, M_kv):
    m, _, fi = oracle.simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=M_kv,
                               cost_c=0, cost_tau=0, schedule=True)
    return m, fi


def test_alpha_calibration_matches_oracle():
    import workload
    a, p, o = workload.generate("bimodal_sweep_4096x2000", n_inst=8, n_jobs=400)
    deltas = (0.0, 0.02, 0.05, 0.1, 0.3, 1.0)
    got = profit.calibrate_alpha(profit.gpu_simulate_batch, a, p, o, deltas, B=128,
                                 M_kv=262144)
    ref = profit.calibrate_alpha(oracle_simulate_batch, a, p, o, deltas, B=128, M_kv=262144)
    assert got == ref
