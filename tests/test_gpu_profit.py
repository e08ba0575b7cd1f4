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
