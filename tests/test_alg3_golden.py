"""Hand-traced cases of Algorithm 3's spare-worker and long-worker branches
(Section 3.3) and of the plan width under the KV budget, checked against the
oracle; then each plausible mistake in those branches is planted in a copy of
the oracle (built on the CPU) to show that one of the cases catches it."""
import ctypes
import json
import os
import subprocess

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
CASES = json.load(open(os.path.join(HERE, "golden", "alg3_spare_examples.json")))
SRC = os.path.join(os.path.dirname(HERE), "oracle", "oracle.c")


def _tables(c):
    return (np.array([c["arrival"]], np.int32), np.array([c["prompt"]], np.int32),
            np.array([c["output"]], np.int32))


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_oracle_matches_hand_trace(case):
    a, p, o = _tables(case)
    m, st, fi = oracle.simulate(a, p, o, policy="isjl", B=case["B"], alpha=case["alpha"],
                                M_kv=case["M_kv"], schedule=True)
    assert int(m["T"][0]) == case["T"]
    assert st[0].tolist() == case["start"]
    assert (fi[0] - st[0]).tolist() == [x + y for x, y in zip(case["prompt"], case["output"])]
    # eq. (1) holds at every step, and the re-scorer sees no violation
    assert int(m["unfair_steps"][0]) == 0
    _, viol = oracle.decompose(a, p, o, st, B=case["B"], alpha=case["alpha"], M_kv=case["M_kv"])
    assert int(viol[0]) == 0


# (name, text in oracle.c, replacement): each is a reading of Algorithm 3 that a
# careless implementation could take instead of the adopted one.
MUTATIONS = [
    ("spare caps of 2 alpha", "if (S->load[w] + L <= a) {", "if (S->load[w] + L <= 2 * a) {"),
    ("worker 1 idles on the sum of all packs",
     "if (S->load[w] > pmax) pmax = S->load[w];", "pmax += S->load[w];"),
    ("no KV cut of the plan width", "if (I->M != 0 && q > 0 && resv + L > I->M) break;",
     "if (0) break;"),
    ("long workers scanned in ascending index", "for (int64_t w = m - 1; w >= 1; --w)",
     "for (int64_t w = 1; w < m; ++w)"),
    ("no spare workers", "for (int64_t w = m; w < Bp; ++w)", "for (int64_t w = Bp; w < Bp; ++w)"),
]


def _build_variant(tmp_path, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, old
    path = tmp_path / "variant.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / "libvariant.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-o", str(so), str(path),
                    "-lm"], check=True)
    lib = ctypes.CDLL(str(so))
    P, I32, I64, U32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
    lib.oracle_simulate_batch.argtypes = [I64, I32, P, P, P, I32, I32, I64, I32, U32, I64, I64,
                                          P, P, P]
    lib.oracle_simulate_batch.restype = ctypes.c_int
    return lib


def _variant_schedule(lib, c):
    a, p, o = _tables(c)
    n = a.shape[1]
    out = np.zeros(1, dtype=oracle.METRICS_DTYPE)
    st = np.empty((1, n), np.int32)
    fi = np.empty((1, n), np.int32)
    rc = lib.oracle_simulate_batch(1, n, a.ctypes.data, p.ctypes.data, o.ctypes.data, c["B"],
                                   c["alpha"], c["M_kv"], oracle.POLICIES["isjl"], 0, 0, 1,
                                   out.ctypes.data, st.ctypes.data, fi.ctypes.data)
    assert rc == 0
    return int(out["T"][0]), st[0].tolist()


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(tmp_path, name, old, new):
    lib = _build_variant(tmp_path, old, new)
    caught = [c["name"] for c in CASES if _variant_schedule(lib, c) != (c["T"], c["start"])]
    assert caught, f"no golden case catches: {name}"
