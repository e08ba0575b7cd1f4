"""The named workloads are the recorded bytes: the SHA-256 of each one's job
tables (arrival, prompt, output in that order) equals the value stored in
tests/golden/workload_sha256.json and quoted in the benchmark spec."""
import hashlib
import json
import os

import pytest

import workload

REC = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "workload_sha256.json")))


@pytest.mark.parametrize("name", list(REC["workloads"]))
def test_workload_tables_hash(name):
    a, p, o = workload.generate(name)
    h = hashlib.sha256()
    for x in (a, p, o):
        h.update(x.tobytes())
    assert list(a.shape) == REC["workloads"][name]["shape"]
    assert h.hexdigest() == REC["workloads"][name]["sha256"]
