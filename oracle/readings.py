"""ORACLE — test infrastructure only.

Alternative readings of ISJL (Section 3.3, Algorithm 3, and Section 3.5's
"return to Phase ONE") on offline instances (every job released at step 0, no
prompt part, no KV budget), written as a plain per-step loop in Python so that
each reading is a switch a reader can check against the text.  Used only to
measure how far each reading is from the paper's linear-pricing table
(Section 5.2), never by the GPU library.  With the default switches it is the
adopted reading and agrees with ``oracle.c`` (checked in the tests).

Switches (the adopted reading first):
  guard  True  : every planned start waits for A_max(t) <= alpha (eq. (1) at
                 every step); False: the plan starts regardless (the listing).
  brk  "drain" : after Phase TWO meets A_max > alpha nothing is filled until the
                 machine is empty, then Phase ONE; "resume": filling resumes as
                 soon as A_max(t) <= alpha again.
  epoch "empty": Phase ONE only at an empty machine with no plan pending;
        "break": Phase ONE also as soon as Phase TWO breaks, on the queued jobs
                 and the idle workers, while the running jobs continue.
  oj "worker"  : long job o_j runs on worker j after its pack; "phase2": o_j is
                 not planned and Phase TWO takes it (the listing never places it).
  cap "paper"  : cap_j = min{2 alpha, o_1 - o_j + beta}; "alpha": min{alpha, ...}.
  beta         : None for beta = alpha (Section 3.3), or an integer.
  skip True    : a pack candidate that fits no worker is skipped (the listing's
                 "continue"); False: the scan stops there (Section 3.2's prose).

``cohort_schedule`` is not a reading of ISJL: it is a fair schedule built by
hand (cohorts whose every start lies in their first alpha steps, then guarded
longest-first fill), used as an upper bound on the alpha-fair optimum.
"""
from __future__ import annotations


def simulate(lens, B, alpha, guard=True, brk="drain", epoch="empty", oj="worker",
             cap="paper", beta=None, skip=True):
    """Start step of every job under ISJL read with the given switches."""
    n = len(lens)
    order = sorted(range(n), key=lambda i: (-lens[i], i))
    state = [0] * n  # 0 waiting, 1 running, 2 done
    planned = [False] * n
    start = [-1] * n
    cur = [-1] * B  # job on each worker
    queues = [[] for _ in range(B)]
    hold = {}  # o_1's earliest start (worker 1's idle time)
    draining = False
    done, t = 0, 0
    b = alpha if beta is None else beta
    while done < n:
        for w in range(B):
            j = cur[w]
            if j >= 0 and start[j] + lens[j] == t:
                state[j], cur[w] = 2, -1
                done += 1
        if done == n:
            break
        running = [j for j in cur if j >= 0]
        amax = max((t - start[j] for j in running), default=0)
        pending = any(queues)
        if epoch == "empty":
            phase_one = not running and not pending
        else:
            phase_one = not pending and (not running or draining)
        idle = [w for w in range(B) if cur[w] < 0]
        pool = [j for j in order if state[j] == 0 and not planned[j]]
        if phase_one and pool and idle:
            draining = False
            Bp = len(idle)
            if not (len(pool) == 1 or Bp == 1 or lens[pool[1]] <= alpha):
                m = min(Bp, sum(1 for j in pool if lens[j] > alpha))
                o1 = lens[pool[0]]
                caps = [alpha] * Bp
                for w in range(1, m):
                    top = 2 * alpha if cap == "paper" else alpha
                    caps[w] = min(top, o1 - lens[pool[w]] + b)
                load = [0] * Bp
                packs = [[] for _ in range(Bp)]
                for q in range(m, len(pool)):
                    j, L = pool[q], lens[pool[q]]
                    w = next((w for w in range(m, Bp) if load[w] + L <= alpha), -1)
                    if w < 0:
                        w = next((w for w in range(m - 1, 0, -1) if load[w] + L <= caps[w]), -1)
                    if w >= 0:
                        packs[w].append(j)
                        load[w] += L
                    elif not skip:
                        break
                for w in range(Bp):
                    for j in packs[w]:
                        queues[idle[w]].append(j)
                        planned[j] = True
                    if 1 <= w < m and oj == "worker":
                        queues[idle[w]].append(pool[w])
                        planned[pool[w]] = True
                queues[idle[0]].append(pool[0])
                planned[pool[0]] = True
                pmax = max(load[1:]) if Bp > 1 else 0
                hold[pool[0]] = t + min(max(pmax - alpha, 0), alpha)
        for w in range(B):  # planned starts, workers in index order
            if cur[w] >= 0 or not queues[w]:
                continue
            j = queues[w][0]
            if t >= hold.get(j, 0) and (not guard or amax <= alpha):
                queues[w].pop(0)
                start[j], state[j], cur[w] = t, 1, j
        if draining and brk == "resume" and amax <= alpha:
            draining = False
        if not draining:  # Phase TWO: longest unplanned job on each idle worker
            for w in range(B):
                if cur[w] >= 0 or queues[w]:
                    continue
                j = next((j for j in order if state[j] == 0 and not planned[j]), -1)
                if j < 0:
                    break
                if amax > alpha:
                    draining = True
                    break
                start[j], state[j], cur[w] = t, 1, j
        t += 1
    return start


def cohort_schedule(lens, B, alpha, theta=1.0):
    """A fair schedule (every pair of co-running jobs starts within alpha):
    while a job longer than theta * alpha remains, a cohort starts at an empty
    machine with the B longest remaining jobs, each but the first preceded on
    its worker by short jobs (at most alpha long, longest first, total at most
    min{alpha, o_1 - L_j}), so every start lies in the cohort's first alpha
    steps; the rest run longest first on idle workers whenever A_max <= alpha."""
    n = len(lens)
    rem = sorted(range(n), key=lambda i: (-lens[i], i))
    start = [0] * n
    t = 0
    while rem and lens[rem[0]] > theta * alpha:
        finals, rest = rem[:B], rem[B:]
        o1 = lens[finals[0]]
        shorts = sorted((j for j in rest if lens[j] <= alpha), key=lambda i: (-lens[i], i))
        used = set()
        end = t
        for k, j in enumerate(finals):
            room = min(alpha, o1 - lens[j]) if k else 0
            p = 0
            for s in shorts:
                if s not in used and p + lens[s] <= room:
                    start[s] = t + p
                    p += lens[s]
                    used.add(s)
            start[j] = t + p
            end = max(end, start[j] + lens[j])
        t = end
        rem = [j for j in rest if j not in used]
    cur = [-1] * B
    queue = list(rem)
    while queue:
        for w in range(B):
            if cur[w] >= 0 and start[cur[w]] + lens[cur[w]] <= t:
                cur[w] = -1
        if max((t - start[j] for j in cur if j >= 0), default=0) <= alpha:
            for w in range(B):
                if cur[w] < 0 and queue:
                    j = queue.pop(0)
                    start[j], cur[w] = t, j
        t += 1
    return start
