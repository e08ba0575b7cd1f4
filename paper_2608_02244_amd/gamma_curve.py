"""The competitive-ratio experiment: exact optimum against ISJL on tiny offline
instances (B = 2 by default), binned by gamma = alpha / o_1 (o_1 the longest
job), against the paper's lower-bound curve (Theorem on the competitive ratio
as a function of gamma):

    CR(gamma) = (1 + gamma) / (1 + 2 gamma)    for 0 < gamma <= 1/2,
                (2 - gamma) / (3 - 2 gamma)    for 1/2 <= gamma < 1,

and, with beta* (the B = 2 choice beta = (sqrt 17 - 1) alpha / 4), against the
constant (25 + sqrt 17) / 38 of the B = 2 theorem.  Every comparison is done in
integers: with gamma = alpha / o_1 the curve is (o_1 + alpha) / (o_1 + 2 alpha)
or (2 o_1 - alpha) / (3 o_1 - 2 alpha), and an instance falls below it when
T_OPT * den < T_ISJL * num.  Only instances with 0 < alpha < o_1 are on the curve.
"""
from __future__ import annotations

import math
from fractions import Fraction
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

FLAG_BETA_SQRT17 = 8
CR_BETA_STAR = (25 + math.sqrt(17)) / 38  # B = 2, beta = beta*


def cr_gamma(alpha: int, o1: int) -> Fraction:
    """The curve at gamma = alpha / o_1 as an exact fraction (0 < alpha < o_1)."""
    if 2 * alpha <= o1:
        return Fraction(o1 + alpha, o1 + 2 * alpha)
    return Fraction(2 * o1 - alpha, 3 * o1 - 2 * alpha)


def gpu_pair(a, p, o, B: int, alpha: int, flags: int):
    """(T_OPT, T_ISJL) per instance through the HIP library (host buffers)."""
    from . import bruteforce_opt, simulate
    T_opt, _ = bruteforce_opt(a, p, o, B=B, alpha=alpha, M_kv=0)
    m, _, _ = simulate(a, p, o, policy="isjl", B=B, alpha=alpha, M_kv=0, cost_c=0, cost_tau=0,
                       beta_sqrt17=bool(flags & FLAG_BETA_SQRT17))
    return np.asarray(T_opt, dtype=np.int64), m["T"].astype(np.int64)


def run(pair: Callable, a, p, o, alphas: Sequence[int], B: int = 2, beta_star: bool = False,
        bins: Sequence[float] = (0.0, 0.1, 0.2, 0.3, 1 / 3, 0.4, 0.5, 0.6, 0.7, 0.8, 0.9, 1.0)
        ) -> Dict:
    """Per gamma bin: instances, the smallest T_OPT / T_ISJL (exact), the curve's
    smallest value over the bin's instances, and the instances below the curve
    (with the worst one).  With beta_star also the count below the beta* constant."""
    ln = np.asarray(p, dtype=np.int64) + np.asarray(o, dtype=np.int64)
    o1 = ln.max(axis=1)
    flags = FLAG_BETA_SQRT17 if beta_star else 0
    nb = len(bins) - 1
    rows: List[Dict] = [dict(lo=bins[k], hi=bins[k + 1], n=0, min_ratio=None, curve_min=None,
                             below=0, worst=None) for k in range(nb)]
    below_const = 0
    overall = None
    edges = np.asarray(bins, dtype=np.float64)
    for al in alphas:
        T_opt, T_isjl = pair(a, p, o, B, al, flags)
        T_opt = np.asarray(T_opt, np.int64)
        T_isjl = np.asarray(T_isjl, np.int64)
        ok = (al > 0) & (al < o1)
        if not ok.any():
            continue
        idx = np.nonzero(ok)[0]
        g = al / o1[idx]
        kb = np.clip(np.searchsorted(edges, g, side="left") - 1, 0, nb - 1)
        small = 2 * al <= o1[idx]
        num = np.where(small, o1[idx] + al, 2 * o1[idx] - al)
        den = np.where(small, o1[idx] + 2 * al, 3 * o1[idx] - 2 * al)
        to, ti = T_opt[idx], T_isjl[idx]
        below = to * den < ti * num
        r = to / ti
        c = num / den
        if beta_star:
            below_const += int((r < CR_BETA_STAR).sum())
        for k in range(nb):
            sel = kb == k
            if not sel.any():
                continue
            row = rows[k]
            row["n"] += int(sel.sum())
            q = np.nonzero(sel)[0]
            jr = q[np.argmin(r[q])]
            fr = Fraction(int(to[jr]), int(ti[jr]))
            if row["min_ratio"] is None or fr < row["min_ratio"]:
                row["min_ratio"] = fr
            jc = q[np.argmin(c[q])]
            fc = Fraction(int(num[jc]), int(den[jc]))
            if row["curve_min"] is None or fc < row["curve_min"]:
                row["curve_min"] = fc
            qb = q[below[q]]
            row["below"] += int(len(qb))
            if len(qb):
                jw = qb[np.argmax(c[qb] - r[qb])]
                gap = Fraction(int(num[jw]), int(den[jw])) - Fraction(int(to[jw]), int(ti[jw]))
                if row["worst"] is None or gap > row["worst"]["gap"]:
                    row["worst"] = {"gap": gap, "instance": int(idx[jw]), "alpha": int(al),
                                    "o1": int(o1[idx[jw]]), "T_opt": int(to[jw]),
                                    "T_isjl": int(ti[jw])}
        jm = np.argmin(r)
        fm = Fraction(int(to[jm]), int(ti[jm]))
        if overall is None or fm < overall:
            overall = fm
    return {"B": B, "beta_star": beta_star, "alphas": list(alphas), "bins": rows,
            "min_ratio": overall, "below_beta_star_constant": below_const if beta_star else None}


def to_json(res: Dict) -> Dict:
    def f(x):
        return None if x is None else [x.numerator, x.denominator, float(x)]
    out = dict(res)
    out["min_ratio"] = f(res["min_ratio"])
    out["bins"] = []
    for r in res["bins"]:
        rr = dict(r)
        rr["min_ratio"] = f(r["min_ratio"])
        rr["curve_min"] = f(r["curve_min"])
        if r["worst"] is not None:
            rr["worst"] = dict(r["worst"], gap=float(r["worst"]["gap"]))
        out["bins"].append(rr)
    return out
