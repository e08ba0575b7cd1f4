"""The system-efficiency experiment through the HIP library equals the run over
the oracle (every integer metric it averages is exact)."""
import numpy as np
import pytest

import oracle
import workload
from paper_2608_02244_amd import efficiency as ef

pytestmark = pytest.mark.gpu


def osim(a, p, o, pol, B, al, M_kv=0):
    return oracle.simulate(a, p, o, policy=pol, B=B, alpha=al, M_kv=M_kv, cost_c=0, cost_tau=1)


def test_table_matches_oracle():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    a, p, o = workload.generate("lmsys_shaped_256x2000", n_inst=6, inst_begin=100)
    for arr in (a, np.zeros_like(a)):
        got = ef.run_table(ef.gpu_simulate, arr, p, o)
        ref = ef.run_table(osim, arr, p, o)
        assert got == ref


def test_table_matches_oracle_resume_reading():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")

    def osim_resume(a, p, o, pol, B, al, M_kv=0):
        return oracle.simulate(a, p, o, policy=pol, B=B, alpha=al, M_kv=M_kv, cost_c=0,
                               cost_tau=1,
                               flags=oracle.FLAG_RESUME_FILL if pol == "isjl" else 0)

    def gsim_resume(*x):
        return ef.gpu_simulate(*x, resume_fill=True)

    a, p, o = workload.generate("lmsys_shaped_256x2000", n_inst=6, inst_begin=200)
    got = ef.run_table(gsim_resume, a, p, o)
    ref = ef.run_table(osim_resume, a, p, o)
    assert got == ref
