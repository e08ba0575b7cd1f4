"""Writes roofline_counts.json: the unit counts of the simulate kernel's
algorithmic operation model, measured with the oracle on the first instances of
each benchmarked workload (the kernel plays no part in them).

For one instance of n jobs under a policy, the method's work is counted in
int32 lane operations as
  * ordering: a bitonic network on NP = 2^ceil(log2 n) keys, NP/2 L (L + 1) / 2
    compare-exchanges of 2 operations (a min and a max), L = log2 NP; not for
    FCFS with arrivals already in index order;
  * events: every job starts once and completes once (2n events); at each one
    the active set S is passed over once (the next completion, the span's
    reductions): ceil(|S| / 64) wave operations of 64 lanes;
  * Phase ONE (ISJL): every pack candidate it examines is placed first-fit over
    the B worker loads by one ballot per 64 workers, ceil(B / 64) wave
    operations of 64 lanes.
This file records, per (workload, policy, alpha), the means over the sampled
instances of the event term (sum of ceil(|S| / 64) over the 2n events) and of
the candidates examined; the sort term is a closed form.

Run from the repository root:  python tests/golden/make_roofline_counts.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
import oracle  # noqa: E402
import workload  # noqa: E402

SAMPLE = 128
INF = oracle.ALPHA_INF
RUNS = [("pareto_65536x2000", "isjl", 128)] + [
    ("bimodal_sweep_4096x2000", "isjl", al) for al in (0, 16, 64, 256, 1024, INF)] + [
    ("bimodal_sweep_4096x2000", "fcfs", INF), ("bimodal_sweep_4096x2000", "ljf", 64),
    ("uniform_256x64", "fcfs", INF), ("uniform_256x64", "ljf", 8), ("uniform_256x64", "isjl", 8),
    ("lognormal_4096x1000", "fcfs", INF), ("lognormal_4096x1000", "ljf", 64),
    ("lognormal_4096x1000", "isjl", 64)] + [
    ("tiny_opt_1048576x8", "isjl", al) for al in (1, 2, 4)]


def event_wave_ops(start, finish):
    """Sum over the 2n start / completion events of ceil(|S| / 64), |S| being
    the number of active jobs at the event (the job itself included)."""
    s = np.sort(start)
    f = np.sort(finish)

    def active(t):  # jobs with start <= t < finish
        return np.searchsorted(s, t, side="right") - np.searchsorted(f, t, side="right")

    at_start = active(start)
    at_end = active(finish - 1)
    return int(((at_start + 63) // 64).sum() + ((at_end + 63) // 64).sum())


def measure(name, policy, alpha, sample=SAMPLE):
    w = workload.WORKLOADS[name]
    a, p, o = workload.generate(w, n_inst=sample)
    ev, scans = [], []
    oracle.pack_scans_take()
    for k in range(sample):
        m, st, fi = oracle.simulate(a[k:k + 1], p[k:k + 1], o[k:k + 1], policy=policy, B=w.B,
                                    alpha=alpha, M_kv=w.M_kv, cost_c=w.cost_c,
                                    cost_tau=w.cost_tau, schedule=True)
        scans.append(oracle.pack_scans_take())
        ev.append(event_wave_ops(st[0].astype(np.int64), fi[0].astype(np.int64)))
    return {"workload": name, "policy": policy,
            "alpha": "inf" if alpha == oracle.ALPHA_INF else alpha, "sample": sample,
            "event_wave_ops_per_instance": float(np.mean(ev)),
            "pack_candidates_per_instance": float(np.mean(scans))}


def main():
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=oracle.host_threads()) as ex:
        rows = list(ex.map(lambda r: measure(*r), RUNS))
    with open(os.path.join(ROOT, "tests", "golden", "roofline_counts.json"), "w") as fh:
        json.dump({"cite": "survey of the hot path, measurement: work terms of the sort, "
                           "the events and Phase ONE's first-fit ballots",
                   "runs": rows}, fh, indent=1)
        fh.write("\n")
    for r in rows:
        print(r)


if __name__ == "__main__":
    main()
