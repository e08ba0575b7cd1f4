"""The Robust-ISJL experiment (Section 3.4): ISJL planned on the upper ends u_i of
output-length prediction intervals, run on the true lengths.

On tiny offline instances (all releases at 0, no KV budget) it checks, per
instance and in integers:

* fairness on the true run (no step with a progress range above alpha);
* the competitive guarantee under interval uncertainty,
  T_R <= 4/3 (T_OPT + Delta_pack)  <=>  3 T_R <= 4 (T_OPT + Delta_pack),
  with T_OPT the exact alpha-fair optimum and Delta_pack the packable residual
  error: the least, over partitions of the jobs into groups of at most B jobs
  whose true lengths span at most alpha, of the summed per-group largest slack
  e_i = u_i - o_i;
* the scale-normalised corollary, T_OPT / T_R >= 3/4 / (1 + B eps_bar) with
  eps_bar = Delta / O (Delta the summed slack, O the summed true length)
  <=>  4 T_OPT (O + B Delta) >= 3 T_R O;
* the first step of the guarantee's proof, T_R <= T_ISJL(I_u) (ISJL run on the
  proxy instance whose lengths are the upper bounds).

Job length here is prompt + output (the tokens a job holds a slot for); the
slack is on the output part, so a job's proxy length is prompt + u_i.
"""
from __future__ import annotations

from typing import Callable, Dict, List, Sequence

import numpy as np


def delta_pack(length, slack, alpha: int, B: int, chunk: int = 4096) -> np.ndarray:
    """Packable residual prediction error per instance (rows of ``length`` and
    ``slack``; at most 12 jobs): the least summed group maximum of the slack over
    partitions into groups of at most B jobs whose lengths span at most alpha.
    Exact, by dynamic programming over job subsets (each subset's best partition
    takes the group holding its lowest job, then the best partition of the rest)."""
    L = np.asarray(length, dtype=np.int64)
    E = np.asarray(slack, dtype=np.int64)
    if L.ndim == 1:
        L, E = L[None], E[None]
    n_inst, n = L.shape
    if n > 12:
        raise ValueError("delta_pack: at most 12 jobs per instance")
    if (E < 0).any():
        raise ValueError("delta_pack: negative slack")
    Bc = n if B == 0 else min(B, n)
    full = (1 << n) - 1
    pop = np.array([bin(m).count("1") for m in range(1 << n)])
    out = np.empty(n_inst, dtype=np.int64)
    big = np.iinfo(np.int64).max // 4
    for c0 in range(0, n_inst, chunk):
        l, e = L[c0:c0 + chunk].T, E[c0:c0 + chunk].T  # [n, m]
        m = l.shape[1]
        lo = np.empty((1 << n, m), np.int64)
        hi = np.empty((1 << n, m), np.int64)
        me = np.empty((1 << n, m), np.int64)
        lo[0], hi[0], me[0] = big, -big, 0
        for s in range(1, 1 << n):
            b = (s & -s).bit_length() - 1
            r = s & (s - 1)
            lo[s] = np.minimum(lo[r], l[b])
            hi[s] = np.maximum(hi[r], l[b])
            me[s] = np.maximum(me[r], e[b])
        ok = (hi - lo <= alpha) & (pop[:, None] <= Bc)
        ok[0] = True
        cost = np.where(ok, me, big)
        dp = np.empty((1 << n, m), np.int64)
        dp[0] = 0
        for s in range(1, 1 << n):
            low = s & -s
            rest = s ^ low
            best = np.full(m, big, np.int64)
            g = rest
            while True:  # every subset g of the rest: group = g + the lowest job
                grp = g | low
                best = np.minimum(best, cost[grp] + dp[s ^ grp])
                if g == 0:
                    break
                g = (g - 1) & rest
            dp[s] = best
        out[c0:c0 + m] = dp[full]
    return out


def gpu_quad(a, p, o, u, B: int, alpha: int, M_kv: int = 0):
    """Through the HIP library on cuda:0: T_R, its unfair steps, T_OPT,
    T_ISJL(I) and T_ISJL(I_u) per instance.  T_OPT is negative (a marker) for an
    instance whose exhaustive search gave up (its push limit)."""
    import torch
    from . import bruteforce_opt, simulate, simulate_robust
    mr, _, _ = simulate_robust(a, p, o, u, B=B, alpha=alpha, M_kv=M_kv, cost_c=0, cost_tau=0)
    dev = torch.device("cuda:0")
    ta, tp, to = (torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(dev)
                  for x in (a, p, o))
    T_opt, _ = bruteforce_opt(ta, tp, to, B=B, alpha=alpha, M_kv=M_kv)
    T_opt = T_opt.cpu().numpy()
    mi, _, _ = simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=M_kv, cost_c=0,
                        cost_tau=0)
    mu, _, _ = simulate(a, p, u, policy="isjl", B=B, alpha=alpha, M_kv=M_kv, cost_c=0,
                        cost_tau=0)
    return (mr["T"].astype(np.int64), mr["unfair_steps"].astype(np.int64),
            np.asarray(T_opt, np.int64), mi["T"].astype(np.int64), mu["T"].astype(np.int64))


def run(quad: Callable, a, p, o, u, alphas: Sequence[int], B: int = 2) -> Dict:
    """Per alpha: instances, fairness violations, violations of the guarantee,
    of the corollary and of the proof's first step (with the worst instance of
    each), the smallest T_OPT / T_R and the mean T_R / T_ISJL.  Instances whose
    optimum was not found (negative T_OPT) are left out and counted."""
    P = np.asarray(p, np.int64)
    O = np.asarray(o, np.int64)
    U = np.asarray(u, np.int64)
    if (U < O).any():
        raise ValueError("upper bounds below the true outputs")
    length = P + O
    slack = U - O
    tot_len = length.sum(axis=1)
    tot_slack = slack.sum(axis=1)
    Bc = length.shape[1] if B == 0 else min(B, length.shape[1])
    rows: List[Dict] = []
    for al in alphas:
        T_r, unfair, T_opt, T_i, T_u = (np.asarray(x, np.int64) for x in quad(a, p, o, u, B, al))
        if (T_r < 0).any() or (T_i < 0).any() or (T_u < 0).any():
            raise RuntimeError("an instance reported an error marker")
        solved = T_opt >= 0
        dp = delta_pack(length, slack, al, B)
        thm = solved & (3 * T_r > 4 * (T_opt + dp))
        cor = solved & (4 * T_opt * (tot_len + Bc * tot_slack) < 3 * T_r * tot_len)
        step1 = T_r > T_u

        def worst(mask, gap):
            if not mask.any():
                return None
            q = np.nonzero(mask)[0]
            j = int(q[np.argmax(gap[q])])
            return {"instance": j, "T_r": int(T_r[j]), "T_opt": int(T_opt[j]),
                    "delta_pack": int(dp[j]), "T_isjl": int(T_i[j]), "T_isjl_u": int(T_u[j]),
                    "lengths": length[j].tolist(), "slack": slack[j].tolist()}

        rows.append({
            "alpha": int(al), "n": int(len(T_r)), "opt_unsolved": int((~solved).sum()),
            "unfair": int((unfair > 0).sum()),
            "thm_violations": int(thm.sum()),
            "thm_worst": worst(thm, (3 * T_r - 4 * (T_opt + dp)) / np.maximum(T_r, 1)),
            "cor_violations": int(cor.sum()),
            "step1_violations": int(step1.sum()),
            "step1_worst": worst(step1, (T_r - T_u) / np.maximum(T_u, 1)),
            "min_opt_over_r": float((T_opt[solved] / T_r[solved]).min()),
            "mean_r_over_isjl": float((T_r / T_i).mean()),
            "mean_delta_pack": float(dp.mean()), "mean_delta": float(tot_slack.mean()),
        })
    return {"B": B, "rows": rows}
