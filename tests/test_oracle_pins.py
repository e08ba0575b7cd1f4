"""Pins for the oracle: checks against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: every expected value is a value
the paper prints or derives for a worked example, a closed form, an identity,
an invariant, a textbook routine (LPT list scheduling, P||Cmax, optimal batch
grouping) implemented independently below, or brute force over all start
vectors on tiny instances.
"""
import heapq
import itertools
import json
import os
import zlib
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import ALPHA_INF
from workload import random_tables

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
# smallest T_OPT / T_ISJL (beta = alpha, beta*) on the fixed B = 2 sample below
WORST_B2_SAMPLE = (Fraction(35, 44), Fraction(29, 37))


def z(n):
    return np.zeros(n, np.int32)


def arr(x):
    return np.asarray(x, dtype=np.int32)


def sim1(lengths, policy, B, alpha, arrival=None, prompt=None, M_kv=0, c=0, tau=1, flags=0):
    n = len(lengths)
    a = arr(arrival) if arrival is not None else z(n)
    p = arr(prompt) if prompt is not None else z(n)
    m, s, f = oracle.simulate(a, p, arr(lengths), policy=policy, B=B, alpha=alpha, M_kv=M_kv,
                              cost_c=c, cost_tau=tau, flags=flags, schedule=True)
    return m[0], s[0], f[0]


# ---------------------------------------------------------------------------
# Worked examples of the paper


@pytest.mark.parametrize("L", [2, 3, 5, 10, 31])
def test_quadratic_externality_fcfs_ljf(L):
    """Proposition on FCFS's quadratic externality (Section 5): B = 2, one job of
    length L then L unit jobs.  FCFS: T = L, E = L(L-1)/2.  LJF: T = L + ceil((L-1)/2),
    E = 0."""
    lengths = [L] + [1] * L
    m, _, _ = sim1(lengths, "fcfs", 2, ALPHA_INF)
    assert m["T"] == L and m["E"] == L * (L - 1) // 2
    m, _, _ = sim1(lengths, "ljf", 2, 0)
    assert m["T"] == L + (L - 1 + 1) // 2 and m["E"] == 0


@pytest.mark.parametrize("L,alpha", [(4, 1), (6, 2), (7, 3), (10, 3), (20, 5)])
def test_quadratic_instance_isjl(L, alpha):
    """ISJL on the same instance (hand-derived from Phase TWO): o_2 = 1 <= alpha, so
    the unit jobs are filled next to the long job at steps 0..alpha, then the
    remaining unit jobs run in pairs: T = L + ceil((L-alpha-1)/2), E = alpha(alpha+1)/2."""
    lengths = [L] + [1] * L
    m, _, _ = sim1(lengths, "isjl", 2, alpha)
    assert m["T"] == L + (L - alpha - 1 + 1) // 2
    assert m["E"] == alpha * (alpha + 1) // 2
    if L + 1 <= 8:
        assert oracle.opt(z(L + 1), z(L + 1), arr(lengths), B=2, alpha=alpha)[0] == m["T"]


@pytest.mark.parametrize("alpha", [1, 2, 3, 4, 6])
def test_over_inserting_family(alpha):
    """Lemma 'cost of over-inserting' (Section 3.2): at S = L and P = Q = alpha the
    ratio (L+P)/(S+P+Q) is reached.  Instance {L, L, alpha, alpha}, L = 2 alpha + 1:
    T_ISJL = L + 2 alpha, T_OPT = L + alpha."""
    L = 2 * alpha + 1
    lengths = [L, L, alpha, alpha]
    m, _, _ = sim1(lengths, "isjl", 2, alpha)
    assert m["T"] == L + 2 * alpha
    assert oracle.opt(z(4), z(4), arr(lengths), B=2, alpha=alpha)[0] == L + alpha


@pytest.mark.parametrize("alpha", [1, 2, 3, 4, 5])
def test_under_inserting_family(alpha):
    """Lemma 'cost of under-inserting': the tight point S = P = 2 alpha, L just
    below S + P - beta.  Instance {3 alpha - 1, 2 alpha, 2 alpha}: T_ISJL = 5 alpha - 1,
    T_OPT = 4 alpha (ratio 4 alpha / (5 alpha - 1) -> 4/5)."""
    lengths = [3 * alpha - 1, 2 * alpha, 2 * alpha]
    m, _, _ = sim1(lengths, "isjl", 2, alpha)
    assert m["T"] == 5 * alpha - 1
    assert oracle.opt(z(3), z(3), arr(lengths), B=2, alpha=alpha)[0] == 4 * alpha


@pytest.mark.parametrize("L,alpha", [(10, 2), (20, 3), (40, 7)])
def test_online_adversary(L, alpha):
    """Proposition on the online lower bound (Section 3.5): J1 of length L at 0 and
    J2 of length L at alpha + 1 (s = 0 for a policy that starts J1 at once).  A
    policy that starts J1 at 0 cannot co-run J2: T = 2L; FCFS has no fairness guard
    and co-runs them: T = L + alpha + 1; the clairvoyant optimum waits: L + alpha + 1."""
    lengths, arrivals = [L, L], [0, alpha + 1]
    assert sim1(lengths, "isjl", 2, alpha, arrival=arrivals)[0]["T"] == 2 * L
    assert sim1(lengths, "ljf", 2, alpha, arrival=arrivals)[0]["T"] == 2 * L
    assert sim1(lengths, "fcfs", 2, ALPHA_INF, arrival=arrivals)[0]["T"] == L + alpha + 1
    assert oracle.opt(arr(arrivals), z(2), arr(lengths), B=2, alpha=alpha)[0] == L + alpha + 1


def test_isjl_b2_plan_timing():
    """Algorithm 2 on {10, 8, 3, 1}, alpha = 2 (hand trace): q = min{10-8+2, 4} = 4,
    pack [3, 1] (P = 4 > alpha) runs alone for P - alpha = 2 steps, o_1 starts at 2,
    the pack continues next to o_1, o_2 starts when the pack ends (step 4)."""
    m, s, f = sim1([10, 8, 3, 1], "isjl", 2, 2)
    assert list(s) == [2, 4, 0, 3]
    assert m["T"] == 12 and m["max_extent"] <= 2


def test_fcfs_strict_order_with_kv():
    """FCFS admits in arrival order and stops at the first job that does not fit
    (no skipping): lengths [3, 4, 1], KV budget 5, B = 3."""
    m, s, _ = sim1([3, 4, 1], "fcfs", 3, ALPHA_INF, M_kv=5)
    assert list(s) == [0, 3, 3] and m["T"] == 7


def test_sjf_order_and_kv():
    """SJF admits shortest first: B = 1 gives starts 1, 3, 0 for lengths [3, 1, 2];
    with B = 3, KV budget 4, the job of length 3 waits until it fits or is alone."""
    m, s, _ = sim1([3, 1, 2], "sjf", 1, ALPHA_INF)
    assert list(s) == [3, 0, 1] and m["T"] == 6
    m, s, _ = sim1([3, 1, 2], "sjf", 3, ALPHA_INF, M_kv=4)
    assert list(s) == [2, 0, 0] and m["T"] == 5


def test_oversized_job_runs_alone():
    """A job whose reservation exceeds the KV budget may run only alone."""
    m, s, _ = sim1([2, 9, 2], "fcfs", 3, ALPHA_INF, M_kv=5)
    assert list(s) == [0, 2, 11] and m["T"] == 13 and m["max_active"] == 1


def test_prompt_counts_as_service():
    """Section 2: o_i counts prompt and output tokens, one per step; a job of
    prompt p and output o runs p + o steps."""
    m, s, f = sim1([3, 2], "fcfs", 2, ALPHA_INF, prompt=[4, 0])
    assert list(f - s) == [7, 2]
    assert m["O"] == 9


def test_idle_steps_count_and_cost_c():
    """Idle steps waiting for a release count in T and cost c each."""
    m, s, _ = sim1([2], "fcfs", 1, ALPHA_INF, arrival=[5], c=7, tau=1)
    assert m["T"] == 7 and s[0] == 5
    assert m["C"] == 7 * 7 + (1 + 2)
    assert m["busy_steps"] == 2


def test_single_batch_closed_forms():
    """LJF, one batch of lengths {5, 3, 2} started together, (c, tau) = (0, 1):
    max r at step t is t + 1, so W = 5*6/2; E_t = sum of gaps to the longest job;
    peak KV occupancy sum r is reached at the last step with three jobs (t = 1)."""
    m, s, _ = sim1([5, 3, 2], "ljf", 3, 0)
    assert list(s) == [0, 0, 0]
    assert m["W"] == 15
    assert m["E"] == 0  # equal progress: no externality
    assert m["peak_kv"] == max(3 * 1, 3 * 2, 2 * 3, 1 * 4, 1 * 5)
    assert m["sum_completion"] == 5 + 3 + 2


# ---------------------------------------------------------------------------
# Identities and invariants on random instances


def q_by_definition(lengths):
    """Q = sum_i sum_{k=1}^{o_i} k (the profit-decomposition theorem, Section 5), by explicit summation."""
    return sum(sum(range(1, int(l) + 1)) for l in lengths)


POLICY_ALPHAS = [("fcfs", ALPHA_INF), ("sjf", ALPHA_INF), ("ljf", 0), ("ljf", 3),
                 ("isjl", 0), ("isjl", 1), ("isjl", 3), ("isjl", 8), ("isjl", ALPHA_INF)]


@pytest.mark.parametrize("policy,alpha", POLICY_ALPHAS)
def test_decomposition_identity_and_invariants(policy, alpha):
    """Profit-decomposition theorem (Section 5): C = cT + tau Q + tau E exactly; each job runs its length once so
    sum_t |S_t| = O; fair policies keep every step within alpha and E <= alpha O;
    capacity and the KV budget hold at every step."""
    rng = np.random.default_rng(zlib.crc32(f"{policy}:{alpha}".encode()))
    for trial in range(60):
        n = int(rng.integers(1, 14))
        B = int(rng.integers(1, 5))
        M_kv = int(rng.choice([0, 0, 12, 25]))
        a, p, o = random_tables(rng, 1, n, 4, 12, max_arrival=int(rng.choice([0, 6, 30])))
        c, tau = int(rng.integers(0, 50)), int(rng.integers(0, 4))
        m, s, f = oracle.simulate(a, p, o, policy=policy, B=B, alpha=alpha, M_kv=M_kv,
                                  cost_c=c, cost_tau=tau, schedule=True)
        m, s, f = m[0], s[0], f[0]
        lengths = (p[0].astype(np.int64) + o[0])
        Q = q_by_definition(lengths)
        assert m["Q"] == Q and m["O"] == lengths.sum()
        assert m["C"] == c * m["T"] + tau * Q + tau * m["E"]
        assert (s >= a[0]).all() and (f - s == lengths).all() and m["T"] == f.max()
        occ = np.zeros(m["T"], np.int64)
        res = np.zeros(m["T"], np.int64)
        for i in range(n):
            occ[s[i]:f[i]] += 1
            res[s[i]:f[i]] += lengths[i]
        assert occ.sum() == lengths.sum()
        assert occ.max() <= B
        if M_kv:
            assert ((res <= M_kv) | (occ <= 1)).all()
        if policy in ("ljf", "isjl"):
            assert m["unfair_steps"] == 0
            if alpha != ALPHA_INF:
                assert m["max_extent"] <= alpha
                assert m["E"] <= alpha * m["O"]
        if policy == "ljf":
            assert m["E"] == 0


def test_ljf_closed_form_and_ratio():
    """Proof of the LJF theorem (Section 3.1): offline, no KV budget, LJF's makespan is
    o_1 + o_{B+1} + o_{2B+1} + ... over the sorted lengths, E_LJF = 0 (Prop. on
    pairwise profit), and T_OPT / T_LJF >= B / (2B - 1)."""
    rng = np.random.default_rng(7)
    for trial in range(80):
        n = int(rng.integers(1, 8))
        B = int(rng.integers(1, 4))
        lengths = rng.integers(1, 15, size=n).astype(np.int32)
        srt = sorted(lengths.tolist(), reverse=True)
        m = sim1(lengths, "ljf", B, 2)[0]
        assert m["T"] == sum(srt[::B]) and m["E"] == 0
        T_opt = oracle.opt(z(n), z(n), lengths, B=B, alpha=2)[0]
        assert Fraction(int(T_opt), int(m["T"])) >= Fraction(B, 2 * B - 1)


def lpt_schedule(lengths, B):
    """Graham's LPT list scheduling: jobs in (-len, index) order, each on the
    machine that frees first.  Returns start steps."""
    order = sorted(range(len(lengths)), key=lambda i: (-lengths[i], i))
    free = [0] * B
    heapq.heapify(free)
    start = [0] * len(lengths)
    for i in order:
        t = heapq.heappop(free)
        start[i] = t
        heapq.heappush(free, t + lengths[i])
    return start


def pcmax_bruteforce(lengths, B):
    """P||Cmax by enumerating every assignment of jobs to B machines."""
    best = None
    for assign in itertools.product(range(B), repeat=len(lengths)):
        loads = [0] * B
        for i, w in enumerate(assign):
            loads[w] += lengths[i]
        mk = max(loads)
        best = mk if best is None else min(best, mk)
    return best


def batch_grouping_bruteforce(lengths, B):
    """Least sum of batch maxima over every partition into batches of at most B
    jobs (a 0-fair schedule is a sequence of simultaneous-start batches)."""
    items = list(lengths)
    best = [None]

    def rec(rest, acc):
        if not rest:
            best[0] = acc if best[0] is None else min(best[0], acc)
            return
        first, others = rest[0], rest[1:]
        for k in range(0, min(B - 1, len(others)) + 1):
            for comb in itertools.combinations(range(len(others)), k):
                grp = [first] + [others[c] for c in comb]
                left = [others[c] for c in range(len(others)) if c not in comb]
                rec(left, acc + max(grp))

    rec(items, 0)
    return best[0]


def test_alpha_zero_is_ljf_and_optimal():
    """alpha = 0 is LJF's endpoint (Corollary on certified profit): ISJL produces
    LJF's schedule (also with releases and a KV budget), and offline the optimum
    equals the best grouping into batches."""
    rng = np.random.default_rng(11)
    for trial in range(60):
        n = int(rng.integers(1, 16))
        B = int(rng.integers(1, 6))
        a, p, o = random_tables(rng, 1, n, 5, 12, max_arrival=int(rng.choice([0, 8, 40])))
        M_kv = int(rng.choice([0, 15, 30]))
        _, si, _ = oracle.simulate(a, p, o, policy="isjl", B=B, alpha=0, M_kv=M_kv,
                                   schedule=True)
        _, sl, _ = oracle.simulate(a, p, o, policy="ljf", B=B, alpha=0, M_kv=M_kv,
                                   schedule=True)
        assert (si == sl).all()
    for trial in range(60):
        n = int(rng.integers(1, 8))
        B = int(rng.integers(1, 4))
        lengths = rng.integers(1, 12, size=n).astype(np.int32)
        mi, si, _ = sim1(lengths, "isjl", B, 0)
        ml, sl, _ = sim1(lengths, "ljf", B, 0)
        assert list(si) == list(sl)
        T_opt = oracle.opt(z(n), z(n), lengths, B=B, alpha=0)[0]
        assert T_opt == batch_grouping_bruteforce(lengths.tolist(), B) == ml["T"]


def test_large_alpha_is_lpt_and_graham():
    """alpha >= max length: the fairness guard never binds, ISJL's Phase TWO is LPT
    list scheduling, its makespan is within (4/3 - 1/(3B)) of P||Cmax, which is
    also the fair optimum (the proposition quoting Graham 1969, Section 3.2)."""
    rng = np.random.default_rng(12)
    for trial in range(60):
        n = int(rng.integers(1, 8))
        B = int(rng.integers(1, 4))
        lengths = rng.integers(1, 12, size=n).astype(np.int32)
        alpha = int(lengths.max()) + int(rng.integers(0, 3))
        m, s, _ = sim1(lengths, "isjl", B, alpha)
        assert list(s) == lpt_schedule(lengths.tolist(), B)
        opt_p = pcmax_bruteforce(lengths.tolist(), B)
        assert Fraction(int(m["T"])) <= (Fraction(4, 3) - Fraction(1, 3 * B)) * opt_p
        assert oracle.opt(z(n), z(n), lengths, B=B, alpha=alpha)[0] == opt_p
        # alpha = max length - 1 already makes fairness vacuous
        assert oracle.opt(z(n), z(n), lengths, B=B,
                          alpha=int(lengths.max()) - 1)[0] == opt_p


# ---------------------------------------------------------------------------
# Exact optimum against its definition (brute force over start vectors)


def opt_by_enumeration(arrival, lengths, B, alpha, M_kv):
    n = len(lengths)
    H = int(max(arrival)) + int(sum(lengths))
    ranges = [np.arange(arrival[i], H - lengths[i] + 1) for i in range(n)]
    grids = np.meshgrid(*ranges, indexing="ij")
    S = np.stack([g.ravel() for g in grids], axis=1)  # [V, n]
    L = np.asarray(lengths)[None, :]
    ok = np.ones(len(S), bool)
    for t in range(H):
        act = (S <= t) & (t < S + L)
        cnt = act.sum(1)
        ok &= cnt <= B
        if M_kv:
            ok &= ((act * L).sum(1) <= M_kv) | (cnt <= 1)
        prog = np.where(act, t - S, -1)
        mx = prog.max(1)
        mn = np.where(act, prog, 1 << 30).min(1)
        ok &= (cnt == 0) | (mx - mn <= alpha)
    mk = (S + L).max(1)
    return int(mk[ok].min())


def test_opt_matches_definition_bruteforce():
    """The exact search equals the least makespan over every start vector that
    meets the constraints of the Appendix A program (plus releases and KV)."""
    rng = np.random.default_rng(13)
    for trial in range(45):
        n = int(rng.integers(1, 5))
        B = int(rng.integers(1, 4))
        alpha = int(rng.integers(0, 4))
        lengths = rng.integers(1, 4, size=n).astype(np.int32)
        arrival = rng.integers(0, 3, size=n).astype(np.int32) if trial % 2 else z(n)
        M_kv = int(rng.choice([0, 4, 6]))
        T, s = oracle.opt(arrival, z(n), lengths, B=B, alpha=alpha, M_kv=M_kv, schedule=True)
        assert T[0] == opt_by_enumeration(arrival, lengths, B, alpha, M_kv)
        m, v = oracle.decompose(arrival, z(n), lengths, s, B=B, alpha=alpha, M_kv=M_kv)
        assert v[0] == 0 and m["T"][0] == T[0]


def test_opt_monotone_in_alpha():
    """The alpha-fair feasible sets are nested (Section 5.1, calibration), so
    T*_alpha is non-increasing in alpha."""
    rng = np.random.default_rng(14)
    for trial in range(30):
        n = int(rng.integers(2, 7))
        lengths = rng.integers(1, 15, size=n).astype(np.int32)
        Ts = [int(oracle.opt(z(n), z(n), lengths, B=2, alpha=a)[0]) for a in range(0, 16, 2)]
        assert all(x >= y for x, y in zip(Ts, Ts[1:]))


# ---------------------------------------------------------------------------
# Competitive-ratio claims (checked, not assumed)


def theorem1_bound(alpha, beta):
    a, b = Fraction(alpha), Fraction(beta)
    if b <= a:
        return min((a + 2 * b) / (a + 3 * b), 4 * a / (6 * a - b))
    return min((2 * a + b) / (2 * a + 2 * b), 4 * a / (6 * a - b))


def floor_beta_star(alpha):
    k = 0
    while (4 * (k + 1) + alpha) ** 2 <= 17 * alpha * alpha:
        k += 1
    return k


def test_b2_competitive_ratio_bounds():
    """B = 2 on 400 random instances of at most 6 jobs.  LJF's ratio T_OPT/T is at
    least B/(2B-1) = 2/3: the LJF theorem of Section 3.1, which holds in general
    and is asserted on every instance.  ISJL's ratios are not guarantees: the
    3/4 of the remark on beta = alpha (Section 3.2) and the B = 2 theorem's bound
    at beta* both fail on recorded 8-job instances (tests/golden/cr_findings.json).
    So the smallest ISJL ratios on this fixed sample are pinned as regression
    values (exact fractions), not checked against those claims."""
    rng = np.random.default_rng(15)
    worst_a, worst_b = Fraction(1), Fraction(1)
    for trial in range(400):
        n = int(rng.integers(2, 7))
        alpha = int(rng.integers(1, 9))
        lengths = rng.integers(1, 25, size=n).astype(np.int32)
        T_opt = int(oracle.opt(z(n), z(n), lengths, B=2, alpha=alpha)[0])
        T_i = int(sim1(lengths, "isjl", 2, alpha)[0]["T"])
        T_b = int(sim1(lengths, "isjl", 2, alpha, flags=oracle.FLAG_BETA_SQRT17)[0]["T"])
        T_l = int(sim1(lengths, "ljf", 2, alpha)[0]["T"])
        assert Fraction(T_opt, T_l) >= Fraction(2, 3)
        assert T_opt <= min(T_i, T_b, T_l)
        worst_a = min(worst_a, Fraction(T_opt, T_i))
        worst_b = min(worst_b, Fraction(T_opt, T_b))
    assert (worst_a, worst_b) == WORST_B2_SAMPLE


def test_beta_star_floor_values():
    """floor((sqrt(17)-1) alpha / 4) for a few alphas."""
    assert [floor_beta_star(a) for a in (1, 2, 4, 8, 50)] == [0, 1, 3, 6, 39]


def test_recorded_findings():
    """Counterexamples found by this oracle to two of the paper's claims, each
    traced by hand (tests/golden/cr_findings.json has the traces):
    - the gamma-curve CR(gamma) (Section 4) is not a lower bound at B = 2, beta = alpha;
    - with B = 3, where Algorithm 3's plan is fair only pairwise with o_1 and every
      plan start is guarded, T_OPT/T_ISJL falls to 1/2 < 3/4 (the claim of the
      general-B theorem, Section 3.3);
    - at B = 2 with beta = alpha the ratio falls to 26/35 < 3/4 (the B = 2 theorem's
      bound at beta = alpha)."""
    with open(os.path.join(GOLDEN, "cr_findings.json")) as fh:
        cases = json.load(fh)
    for c in cases:
        n = len(c["lengths"])
        lengths = arr(c["lengths"])
        m, s, _ = sim1(lengths, "isjl", c["B"], c["alpha"])
        assert m["T"] == c["T_isjl"] and list(s) == c["isjl_starts"]
        T, so = oracle.opt(z(n), z(n), lengths, B=c["B"], alpha=c["alpha"], schedule=True)
        assert T[0] == c["T_opt"]
        mm, v = oracle.decompose(z(n), z(n), lengths, so, B=c["B"], alpha=c["alpha"])
        assert v[0] == 0 and mm["T"][0] == c["T_opt"]


# ---------------------------------------------------------------------------
# Re-scoring a schedule


@pytest.mark.parametrize("policy,alpha", POLICY_ALPHAS)
def test_decompose_agrees_with_simulate(policy, alpha):
    rng = np.random.default_rng(21)
    for trial in range(25):
        n = int(rng.integers(1, 12))
        B = int(rng.integers(1, 4))
        M_kv = int(rng.choice([0, 20]))
        a, p, o = random_tables(rng, 3, n, 3, 10, max_arrival=10)
        m, s, f = oracle.simulate(a, p, o, policy=policy, B=B, alpha=alpha, M_kv=M_kv,
                                  cost_c=5, cost_tau=2, schedule=True)
        md, v = oracle.decompose(a, p, o, s, B=B, alpha=alpha, M_kv=M_kv, cost_c=5, cost_tau=2)
        assert (md == m).all()
        if policy in ("ljf", "isjl") or alpha == ALPHA_INF:
            assert (v == 0).all()


def test_decompose_violation_bits():
    L = arr([3, 3, 3])
    zz = z(3)
    _, v = oracle.decompose(arr([1, 0, 0]), zz, L, arr([0, 0, 5]), B=3, alpha=9)
    assert v[0] == 1
    _, v = oracle.decompose(zz, zz, L, arr([0, 0, 0]), B=2, alpha=9)
    assert v[0] == 2
    _, v = oracle.decompose(zz, zz, L, arr([0, 0, 3]), B=3, alpha=9, M_kv=5)
    assert v[0] == 4
    _, v = oracle.decompose(zz, zz, L, arr([0, 2, 6]), B=3, alpha=1)
    assert v[0] == 8
    _, v = oracle.decompose(zz, zz, L, arr([0, -1, 6]), B=3, alpha=1)
    assert v[0] & 16


def test_invalid_inputs_rejected():
    with pytest.raises(oracle.OracleError):
        oracle.simulate(z(2), arr([0, -1]), arr([1, 1]), policy="fcfs", B=1, alpha=0)
    with pytest.raises(oracle.OracleError):
        oracle.simulate(z(2), z(2), arr([1, 0]), policy="fcfs", B=1, alpha=0)
    with pytest.raises(oracle.OracleError):
        oracle.opt(z(9), z(9), np.ones(9, np.int32), B=2, alpha=1)


def test_resume_fill_reading():
    """The experiment flag that resumes Phase TWO once A_max <= alpha: with B = 2
    it changes nothing (the job left running keeps A_max > alpha until it ends),
    every step stays within alpha, and for B > 2 it can only admit more."""
    rng = np.random.default_rng(16)
    changed = 0
    for trial in range(40):
        n = int(rng.integers(2, 40))
        a, p, o = random_tables(rng, 8, n, 3, 30,
                                         max_arrival=int(rng.choice([0, 40])),
                                         sorted_arrivals=bool(trial % 2))
        for B in (1, 2, 3, 6):
            alpha = int(rng.integers(0, 25))
            kw = dict(policy="isjl", B=B, alpha=alpha, M_kv=int(rng.choice([0, 60])),
                      cost_c=1, cost_tau=1)
            m0 = oracle.simulate(a, p, o, **kw)
            m1 = oracle.simulate(a, p, o, flags=oracle.FLAG_RESUME_FILL, **kw)
            assert (m1["unfair_steps"] == 0).all() and (m1["max_extent"] <= alpha).all()
            if B <= 2:
                for f in m0.dtype.names:
                    assert np.array_equal(m0[f], m1[f]), (B, f)
            else:
                changed += int((m0["T"] != m1["T"]).sum())
    assert changed > 0
