"""Profit and cost alignment of schedules: the paper's linear-pricing experiment.

Host post-processing of the exact integer metrics of ``fsched_simulate`` (the
derived real-valued quantities are fp64 on the host):

* revenue under linear token pricing: ``R = p0 * O`` (O = total tokens served);
* cost by the decomposition of Section 5 (the profit-decomposition theorem):
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


# ---------------------------------------------------------------------------
# Calibration of the fairness budget by replay (the paper's practical
# calibration procedure): every alpha-fair schedule has E <= alpha * O, so
# alpha <= alpha_cost(delta) = delta * Q / O keeps the externality cost within
# delta times the intrinsic cost; the operator replays a workload under ISJL on
# a grid of alpha values scaled by Q / O and picks the alpha with the smallest
# schedule-dependent cost c T + tau E, subject to service targets.


def q_over_o(prompt, output) -> float:
    """Q / O of a workload: sum len (len + 1) / 2 over sum len."""
    ln = np.asarray(prompt, dtype=np.int64) + np.asarray(output, dtype=np.int64)
    return float((ln * (ln + 1) // 2).sum()) / float(ln.sum())


def alpha_cost(delta: float, prompt, output) -> float:
    return delta * q_over_o(prompt, output)


def gpu_simulate_batch(a, p, o, alpha: int, B: int, M_kv: int):
    """All instances through the HIP library: (metrics, finish) on the host."""
    from . import simulate
    m, _, fi = simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=M_kv, cost_c=0,
                        cost_tau=0, schedule=True)
    return m, fi


def calibrate_alpha(simulate_batch: Callable, a, p, o, deltas: Sequence[float], B: int,
                    M_kv: int = 0, c: float = 0.0005, tau: float = 1e-6,
                    min_throughput: Optional[float] = None,
                    latency_q: float = 0.95, max_latency_q: Optional[float] = None) -> Dict:
    """Replay the workload (every instance) under ISJL for alpha = round(delta Q/O)
    and return the grid with the chosen alpha.

    Per alpha: schedule cost c * sum T + tau * sum E, throughput sum O / sum T,
    the latency quantile over every job (finish - arrival), and whether
    tau E <= delta tau Q holds (it must when alpha <= alpha_cost(delta))."""
    qo = q_over_o(p, o)
    arr = np.asarray(a, dtype=np.int64)
    grid = []
    for d in deltas:
        al = int(d * qo)
        m, fi = simulate_batch(a, p, o, al, B, M_kv)
        T, O, Q, E = (float(m[f].astype(np.int64).sum()) for f in ("T", "O", "Q", "E"))
        lat = np.asarray(fi, dtype=np.int64) - arr
        grid.append({"delta": d, "alpha": al, "sched_cost": c * T + tau * E,
                     "throughput": O / T, "latency_q": float(np.quantile(lat, latency_q)),
                     "tauE": tau * E, "tauQ": tau * Q,
                     "externality_within_delta": E <= d * Q,
                     "E_within_alpha_O": bool((m["E"].astype(np.int64) <=
                                               al * m["O"].astype(np.int64)).all())})
    ok = [g for g in grid
          if (min_throughput is None or g["throughput"] >= min_throughput)
          and (max_latency_q is None or g["latency_q"] <= max_latency_q)]
    best = min(ok, key=lambda g: (g["sched_cost"], g["alpha"])) if ok else None
    return {"q_over_o": qo, "grid": grid, "alpha_star": None if best is None else best["alpha"]}
