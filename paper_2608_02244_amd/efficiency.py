"""The system-efficiency experiment (the paper's section on system efficiency
under resource-fair scheduling): throughput and average end-to-end latency of
FCFS, SJF, LJF and ISJL (alpha = 50, 100, 150) at B = 16 and 32 on a workload of
2,000 requests per instance.

Per instance, throughput is the tokens served over the makespan (tokens per
step: the paper's time unit is not stated, so only ratios between policies
compare with its table) and AEL the mean over requests of completion minus
release (equal to the mean completion when every request is released at step 0).
Both are averaged over the instances of the batch; the integer metrics they come
from are the library's, exact.
"""
from __future__ import annotations

from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

ALPHA_INF = 2**31 - 1
POLICIES: Tuple[Tuple[str, Optional[int]], ...] = (
    ("fcfs", None), ("sjf", None), ("ljf", None), ("isjl", 50), ("isjl", 100), ("isjl", 150))
# the paper's printed table: (throughput, AEL) per batch size and policy
PAPER = {16: {"FCFS": (216, 62), "SJF": (196, 60), "LJF": (243, 66), "ISJL(50)": (262, 53),
              "ISJL(100)": (270, 56), "ISJL(150)": (276, 54)},
         32: {"FCFS": (278, 70), "SJF": (259, 67), "LJF": (323, 78), "ISJL(50)": (357, 62),
              "ISJL(100)": (369, 63), "ISJL(150)": (378, 65)}}


def label(policy: str, alpha: Optional[int]) -> str:
    return policy.upper() if alpha is None else f"{policy.upper()}({alpha})"


def gpu_simulate(a, p, o, policy: str, B: int, alpha: int, M_kv: int = 0,
                 resume_fill: bool = False):
    """Every instance through the HIP library on cuda:0; metrics on the host
    (``resume_fill``: ISJL's other reading of Phase TWO's stop)."""
    import torch
    from . import metrics_view, simulate
    dev = torch.device("cuda:0")
    ta, tp, to = (torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(dev)
                  for x in (a, p, o))
    raw, _, _ = simulate(ta, tp, to, policy=policy, B=B, alpha=alpha, M_kv=M_kv, cost_c=0,
                         cost_tau=1, resume_fill=resume_fill and policy == "isjl")
    return metrics_view(raw).copy()


def run_table(simulate: Callable, a, p, o, Bs: Sequence[int] = (16, 32),
              policies: Sequence = POLICIES, M_kv: int = 0) -> Dict:
    """Per batch size and policy: mean throughput (tokens / step), mean AEL
    (steps), both relative to LJF, the largest within-batch progress range and
    whether any step broke the fairness budget."""
    n = np.asarray(o).shape[1]
    table: Dict[int, Dict[str, Dict]] = {}
    for B in Bs:
        rows: Dict[str, Dict] = {}
        for pol, al in policies:
            m = simulate(a, p, o, pol, B, ALPHA_INF if al is None else al, M_kv)
            if (m["T"] < 0).any():
                raise RuntimeError("an instance reported an error marker")
            T = m["T"].astype(np.float64)
            rows[label(pol, al)] = {
                "throughput": float(np.mean(m["O"] / T)),
                "ael": float(np.mean(m["sum_latency"] / n)),
                "T": float(np.mean(T)),
                "max_extent": int(m["max_extent"].max()),
                "unfair_steps": int(m["unfair_steps"].sum()),
            }
        base = rows["LJF"]
        for r in rows.values():
            r["throughput_vs_ljf"] = r["throughput"] / base["throughput"]
            r["ael_vs_ljf"] = r["ael"] / base["ael"]
        table[B] = rows
    return table


def paper_ratios() -> Dict[int, Dict[str, Tuple[float, float]]]:
    """The printed table relative to LJF: (throughput ratio, AEL ratio)."""
    return {B: {k: (v[0] / t["LJF"][0], v[1] / t["LJF"][1]) for k, v in t.items()}
            for B, t in PAPER.items()}


def format_table(table: Dict) -> List[str]:
    lines = ["| B | policy | throughput (tok/step) | AEL (steps) | thr / LJF | AEL / LJF | "
             "paper thr / LJF | paper AEL / LJF |", "|---|---|---|---|---|---|---|---|"]
    pr = paper_ratios()
    for B, rows in table.items():
        for k, r in rows.items():
            pt, pa = pr.get(B, {}).get(k, (float("nan"), float("nan")))
            lines.append(f"| {B} | {k} | {r['throughput']:.2f} | {r['ael']:.0f} | "
                         f"{r['throughput_vs_ljf']:.3f} | {r['ael_vs_ljf']:.3f} | {pt:.3f} | "
                         f"{pa:.3f} |")
    return lines
