"""Profit and cost alignment of schedules: the paper's linear-pricing experiment.

Host post-processing of the exact integer metrics of ``fsched_simulate`` (the
derived real-valued quantities are fp64 on the host):

* revenue under linear token pricing: ``R = p0 * O`` (O = total tokens served);
* cost by the decomposition of Section 5 (Theorem 5.1):
  ``C = tau * Q + c * T + tau * E``, Q the intrinsic (schedule-free) term, T the
  makespan, E the batching externality;
* profit ``R - C``; throughput ``O / T``; average within-batch extent
  ``sum_extent / busy_steps``;
* break-even fixed cost of ISJL(alpha) against LJF (whose E is 0):
  ``c*_alpha = tau * E_alpha / (T_LJF - T_alpha)``.

The workload (accepted requests of each replication) comes from
``workload.pricing_instance``; every policy of a replication serves the same
accepted requests, so revenue and tau * Q are the same for all of them.
"""
from __future__ import annotations

from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

ALPHAS = (50, 100, 150, 250, 300, 400, 500)
POLICIES = [("fcfs", None), ("ljf", None)] + [("isjl", a) for a in ALPHAS]
ALPHA_INF = 2**31 - 1


def label(policy: str, alpha: Optional[int]) -> str:
    return policy.upper() if alpha is None else f"{policy.upper()}(alpha={alpha})"


def gpu_simulate(a, p, o, policy: str, B: int, alpha: int):
    """One instance through the HIP library (host buffers)."""
    from . import simulate
    m, _, _ = simulate(a, p, o, policy=policy, B=B, alpha=alpha, M_kv=0, cost_c=0, cost_tau=0)
    return m


def row_terms(m, c: float, tau: float, p0: float) -> Dict[str, float]:
    """Real-valued terms of one instance's metrics (a structured row)."""
    T, O, Q, E = (float(m[f]) for f in ("T", "O", "Q", "E"))
    busy = float(m["busy_steps"])
    revenue = p0 * O
    cost = tau * Q + c * T + tau * E
    return {"T": T, "O": O, "Q": Q, "E": E, "revenue": revenue, "cost": cost,
            "profit": revenue - cost, "tauQ": tau * Q, "cT": c * T, "tauE": tau * E,
            "throughput": O / T, "avg_extent": float(m["sum_extent"]) / busy if busy else 0.0}


def run_table(simulate: Callable = gpu_simulate, replications: int = 5, seed: int = 0,
              n: int = 400, B: int = 50, c: float = 0.0005, tau: float = 1e-6,
              policies: Sequence = POLICIES) -> Dict:
    """The profit / cost decomposition table and the break-even table, averaged
    over replications (the paper's design: n = 400, B = 50, c = 0.0005,
    tau = 1e-6, p0 = 1/500)."""
    import workload
    per: Dict[str, List[Dict[str, float]]] = {label(*pa): [] for pa in policies}
    metrics: Dict[str, list] = {label(*pa): [] for pa in policies}
    p0 = None
    for r in range(replications):
        a, p, o = workload.pricing_instance(r, seed, n)
        _, _, p0 = workload.pricing_requests(r, seed, n)
        for pol, al in policies:
            m = simulate(a, p, o, pol, B, ALPHA_INF if al is None else al)
            row = m[0]
            per[label(pol, al)].append(row_terms(row, c, tau, p0))
            metrics[label(pol, al)].append(row)
    keys = ("profit", "cost", "tauQ", "cT", "tauE", "throughput", "avg_extent", "T", "E")
    avg = {k: {f: float(np.mean([x[f] for x in v])) for f in keys} for k, v in per.items()}
    base = avg[label("ljf", None)]
    for k, v in avg.items():
        v["gain_vs_ljf"] = v["throughput"] / base["throughput"] - 1.0
    breakeven = {}
    for pol, al in policies:
        if pol != "isjl":
            continue
        v = avg[label(pol, al)]
        saving = base["T"] - v["T"]
        breakeven[al] = {"time_saving": saving, "tauE": v["tauE"],
                         "c_star": v["tauE"] / saving if saving > 0 else float("inf")}
    return {"n": n, "B": B, "c": c, "tau": tau, "p0": p0, "replications": replications,
            "seed": seed, "table": avg, "breakeven": breakeven, "metrics": metrics}


def format_table(res: Dict) -> str:
    lines = ["policy | profit | cost | tauQ | cT | tauE | throughput | gain vs LJF | avg extent"]
    for k, v in res["table"].items():
        lines.append(f"{k} | {v['profit']:.2f} | {v['cost']:.2f} | {v['tauQ']:.2f} | "
                     f"{v['cT']:.2f} | {v['tauE']:.2f} | {v['throughput']:.2f} | "
                     f"{100 * v['gain_vs_ljf']:.2f}% | {v['avg_extent']:.2f}")
    lines.append("alpha | time saving vs LJF | tauE | c*")
    for al, v in res["breakeven"].items():
        lines.append(f"{al} | {v['time_saving']:.1f} | {v['tauE']:.2f} | {v['c_star']:.4f}")
    return "\n".join(lines)


if __name__ == "__main__":
    import sys
    import os
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    print(format_table(run_table()))
