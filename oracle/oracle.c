/*
 * ORACLE — test infrastructure only.
 *
 * A plain, slow, single-threaded CPU implementation of what the batched
 * scheduling evaluator computes.  It exists to check the GPU library: only the
 * tests, the smoke check and the benchmark's CPU-baseline leg may load it, and
 * it shares no code, header or table with the GPU path.
 *
 * Everything follows "Efficiency and Cost Alignment in Batched LLM Serving via
 * Resource-Fair Scheduling" (Yao & Zhou):
 *   - the token-step model, capacity B and fairness constraint: Section 2,
 *     eq. (1) and the scheduling-policy definition;
 *   - LJF: Section 3.1, Algorithm 1 (static batches, longest first);
 *   - ISJL: Section 3.2 Algorithm 2 (B = 2) and Section 3.3 Algorithm 3 (B >= 2),
 *     run on the released queue as in Section 3.5 (Online-ISJL);
 *   - FCFS / SJF: the examples of Section 2.1 and the continuous-batching remark
 *     that follows them;
 *   - cost accounting: Section 5, eq. (batch cost c + tau |S| max r), the
 *     intrinsic term Q and the batching externality E of the profit-decomposition
 *     theorem;
 *   - exact optimum: Appendix A (the integer program), extended with release
 *     steps and the KV budget.
 * Where the paper is silent or inconsistent the readings recorded in the design
 * notes are used; each one is marked "reading:" below.
 *
 * Style: a literal per-step loop.  At every step the active set is scanned for
 * its max / min / sum; nothing is skipped or done in closed form.  All integer
 * arithmetic is int64.
 *
 * Parity pins for this file are in tests/test_oracle_pins.py; every function
 * here is pinned (none is "parity unpinned").
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

#define OR_OK 0
#define OR_EINVAL -1
#define OR_ERANGE -2
#define OR_ENOMEM -3
#define OR_ETOOLARGE -5
#define OR_EINTERNAL -7

#define POL_FCFS 0
#define POL_LJF 1
#define POL_ISJL 2
#define POL_SJF 3

#define FLAG_BETA_SQRT17 8u
#define FLAG_RESUME_FILL 16u
#define FLAG_PREFILL 32u

#define ALPHA_INF_SENTINEL 2147483647

/* Per-instance results; 104 bytes, all exact integers. */
typedef struct {
  int64_t T, O, Q, E, C, W;
  int64_t sum_completion, sum_latency;
  int64_t sum_extent, busy_steps;
  int64_t peak_kv, unfair_steps;
  int32_t max_extent, max_active;
} or_metrics;

typedef struct {
  int32_t n;
  int64_t B;          /* effective capacity (n when unlimited)   */
  int64_t M;          /* KV budget, 0 = none                      */
  int64_t alpha;      /* INT64_MAX when infinite                  */
  int64_t c, tau;
  const int32_t* arrival;
  int64_t* len;       /* service length = prompt + output         */
  int64_t* plan;      /* planning size: len, or prompt + the predicted upper
                         bound of the output (Robust-ISJL, Section 3.4) */
  int64_t* resv;      /* KV reservation while active: plan, or prompt + plan in
                         the prefill-at-admission variant */
  int64_t* pre;       /* footprint offset: NULL (chunked prompt), or the prompt
                         when it is prefilled at admission */
} or_inst;

/* ------------------------------------------------------------------ */
/* Accounting of one step (Section 5).  r_i = a_i + 1 is the index of the
 * token being processed; the step costs c + tau * |S| * max r; the
 * externality of the step is sum over S of (max r - r_i).  An empty step
 * costs c so that the total equals c T + tau Q + tau E with T the makespan. */
typedef struct {
  int64_t E, C, W, sum_extent, busy, peak_kv, unfair;
  int64_t max_extent, max_active;
} or_acc;

static void account_step(or_acc* a, const or_inst* I, int64_t t, const int64_t* start,
                         const int32_t* act, int32_t nact) {
  if (nact == 0) {
    a->C += I->c;
    a->W += I->c;
    return;
  }
  /* footprint r = progress (+ the prompt when it was prefilled at admission);
   * the fairness range is over progress (eq. (1)) */
  int64_t mx = INT64_MIN, sr = 0, amx = INT64_MIN, amn = INT64_MAX;
  for (int32_t k = 0; k < nact; ++k) {
    int64_t a_k = t - start[act[k]] + 1;
    int64_t r = a_k + (I->pre ? I->pre[act[k]] : 0);
    if (r > mx) mx = r;
    sr += r;
    if (a_k > amx) amx = a_k;
    if (a_k < amn) amn = a_k;
  }
  a->E += (int64_t)nact * mx - sr;
  a->C += I->c + I->tau * (int64_t)nact * mx;
  a->W += I->c + I->tau * mx;
  int64_t ext = amx - amn;
  a->sum_extent += ext;
  a->busy += 1;
  if (ext > I->alpha) a->unfair += 1;
  if (ext > a->max_extent) a->max_extent = ext;
  if (nact > a->max_active) a->max_active = nact;
  if (sr > a->peak_kv) a->peak_kv = sr;
}

static void finish_metrics(or_metrics* m, const or_inst* I, const or_acc* a, int64_t T,
                           const int64_t* start) {
  memset(m, 0, sizeof(*m));
  int64_t O = 0, Q = 0, sc = 0, sl = 0;
  for (int32_t i = 0; i < I->n; ++i) {
    int64_t l = I->len[i], q = I->pre ? I->pre[i] : 0;
    O += q + l; /* tokens served */
    /* Q = sum_i of the footprint summed over the job's own steps (profit
     * decomposition, Section 5):
     * sum_{k=1..l_i} (q_i + k) */
    Q += l * q + l * (l + 1) / 2;
    sc += start[i] + l;
    sl += start[i] + l - I->arrival[i];
  }
  m->T = T;
  m->O = O;
  m->Q = Q;
  m->E = a->E;
  m->C = a->C;
  m->W = a->W;
  m->sum_completion = sc;
  m->sum_latency = sl;
  m->sum_extent = a->sum_extent;
  m->busy_steps = a->busy;
  m->peak_kv = a->peak_kv;
  m->unfair_steps = a->unfair;
  m->max_extent = (int32_t)a->max_extent;
  m->max_active = (int32_t)a->max_active;
}

/* ------------------------------------------------------------------ */
/* Orders.  Keys are unique because the job index breaks ties. */
/* Comparator keys for qsort, one set per thread so that several threads may
 * each run the oracle on their own instances at once. */
static _Thread_local const int64_t* g_key1;
static _Thread_local const int32_t* g_key1i;
static _Thread_local int g_key_mode; /* 0: (arrival, i)  1: (len, i)  2: (-len, i) */

static int cmp_order(const void* pa, const void* pb) {
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  int64_t ka, kb;
  if (g_key_mode == 0) {
    ka = g_key1i[a];
    kb = g_key1i[b];
  } else if (g_key_mode == 1) {
    ka = g_key1[a];
    kb = g_key1[b];
  } else {
    ka = -g_key1[a];
    kb = -g_key1[b];
  }
  if (ka != kb) return ka < kb ? -1 : 1;
  return a < b ? -1 : (a > b ? 1 : 0);
}

static void make_order(int32_t* ord, const or_inst* I, int mode) {
  for (int32_t i = 0; i < I->n; ++i) ord[i] = i;
  g_key1 = I->plan;
  g_key1i = I->arrival;
  g_key_mode = mode;
  qsort(ord, (size_t)I->n, sizeof(int32_t), cmp_order);
}

/* ------------------------------------------------------------------ */
/* Simulation state shared by the policies. */
enum { ST_WAIT = 0, ST_ACTIVE = 1, ST_DONE = 2 };

typedef struct {
  const or_inst* I;
  int64_t* start;
  int8_t* st;
  int32_t* act;
  int32_t nact;
  int64_t res; /* sum of reserved lengths of the active jobs */
  /* ISJL only */
  int32_t* cur;      /* job on worker w, or -1 */
  int32_t* wk;       /* worker of job i        */
  int32_t* qhead;
  int32_t* qtail;
  int32_t* qnext;
  int8_t* planned;
  int64_t* load;
  int64_t* cap;
  int32_t* pool;
  int mode; /* 0 FILL, 1 DRAIN */
  int64_t t_w1;
} or_sim;

/* KV guard (reading: clairvoyant reservation of the full length at admission;
 * a job that would run alone is always admissible). */
static int kv_ok(const or_sim* S, int32_t j) {
  if (S->I->M == 0 || S->nact == 0) return 1;
  return S->res + S->I->resv[j] <= S->I->M;
}

static void admit(or_sim* S, int32_t j, int64_t t) {
  S->st[j] = ST_ACTIVE;
  S->start[j] = t;
  S->act[S->nact++] = j;
  S->res += S->I->resv[j];
}

static int released(const or_inst* I, int32_t j, int64_t t) { return I->arrival[j] <= t; }

/* FCFS (order (arrival, i)) and SJF (order (len, i)): continuous batching in a
 * strict priority order; admission stops at the first released job that does
 * not fit.  No fairness guard (these are the paper's unfair baselines). */
static void admit_strict(or_sim* S, const int32_t* ord, int64_t t, int stop_on_unreleased) {
  const or_inst* I = S->I;
  for (int32_t k = 0; k < I->n; ++k) {
    int32_t j = ord[k];
    if (S->st[j] != ST_WAIT) continue;
    if (!released(I, j, t)) {
      if (stop_on_unreleased) break;
      continue;
    }
    if (S->nact >= I->B) break;
    if (!kv_ok(S, j)) break;
    admit(S, j, t);
  }
}

/* LJF, Algorithm 1: only at an empty machine, start the longest-first prefix of
 * the released jobs, at most B of them, stopping at the first that does not fit
 * the KV budget; the batch then runs until every member has finished. */
static void admit_ljf(or_sim* S, const int32_t* ord_long, int64_t t) {
  const or_inst* I = S->I;
  if (S->nact != 0) return;
  for (int32_t k = 0; k < I->n; ++k) {
    int32_t j = ord_long[k];
    if (S->st[j] != ST_WAIT || !released(I, j, t)) continue;
    if (S->nact >= I->B) break;
    if (!kv_ok(S, j)) break;
    admit(S, j, t);
  }
}

/* ---------------- ISJL ---------------- */
/* Count of pack candidates examined by Phase ONE on this thread (a measure of
 * the method's work, read by the roofline's operation count; no effect on any
 * result). */
static _Thread_local int64_t g_pack_scans;
int64_t oracle_pack_scans_take(void) {
  int64_t v = g_pack_scans;
  g_pack_scans = 0;
  return v;
}

static void enqueue(or_sim* S, int32_t w, int32_t j) {
  S->qnext[j] = -1;
  if (S->qtail[w] < 0) S->qhead[w] = j;
  else S->qnext[S->qtail[w]] = j;
  S->qtail[w] = j;
  S->planned[j] = 1;
}

static int any_queue(const or_sim* S) {
  for (int64_t w = 0; w < S->I->B; ++w)
    if (S->qhead[w] >= 0) return 1;
  return 0;
}

/* floor of beta* = (sqrt(17) - 1) alpha / 4, the B = 2 choice of Section 3.2:
 * the largest integer k >= 0 with (4k + alpha)^2 <= 17 alpha^2. */
static int64_t beta_sqrt17(int64_t alpha) {
  int64_t k = (int64_t)floor((sqrt(17.0) - 1.0) * (double)alpha / 4.0);
  if (k < 0) k = 0;
  for (;;) {
    __int128 a = (__int128)(4 * (k + 1) + alpha);
    if (a * a <= (__int128)17 * alpha * alpha) k++;
    else break;
  }
  for (;;) {
    __int128 a = (__int128)(4 * k + alpha);
    if (k > 0 && a * a > (__int128)17 * alpha * alpha) k--;
    else break;
  }
  return k;
}

/* Phase ONE (Algorithms 2 and 3) on the released queue (Online-ISJL).
 * pool = released, unstarted, unplanned jobs in order (-len, i). */
static void phase_one(or_sim* S, const int32_t* ord_long, int64_t t, uint32_t flags) {
  const or_inst* I = S->I;
  int32_t k = 0;
  for (int32_t q = 0; q < I->n; ++q) {
    int32_t j = ord_long[q];
    if (S->st[j] == ST_WAIT && !S->planned[j] && released(I, j, t)) S->pool[k++] = j;
  }
  if (k == 0) return;
  S->mode = 0; /* FILL */
  const int64_t a = I->alpha;
  /* Reading (the paper has no KV budget): the plan uses only as many workers as
   * the longest queued jobs can occupy together, Bp = the largest k <= B whose k
   * longest jobs' reservations fit M_kv (at least one).  At alpha = 0 this keeps
   * ISJL identical to LJF. */
  int64_t Bp = 0, resv = 0;
  for (int32_t q = 0; q < k && Bp < I->B; ++q) {
    int64_t L = I->resv[S->pool[q]];
    if (I->M != 0 && q > 0 && resv + L > I->M) break;
    resv += L;
    Bp++;
  }
  /* "if o_2 <= alpha, go to Phase TWO" (also: a single job, or one worker) */
  if (k == 1 || Bp == 1 || I->plan[S->pool[1]] <= a) return;
  /* M = min{B, #{o_i > alpha}}; o_1 > o_2 > alpha so M >= 2 */
  int64_t m = 0;
  for (int32_t q = 0; q < k; ++q)
    if (I->plan[S->pool[q]] > a) m++;
  if (m > Bp) m = Bp;
  const int64_t beta = (flags & FLAG_BETA_SQRT17) ? beta_sqrt17(a) : a;
  const int64_t o1 = I->plan[S->pool[0]];
  /* cap_j = min{2 alpha, o_1 - o_j + beta} for the long workers j = 2..M;
   * the spare workers j = M+1..Bp take packs of total at most alpha. */
  for (int64_t w = 0; w < Bp; ++w) {
    S->load[w] = 0;
    if (w >= 1 && w < m) {
      int64_t c1 = 2 * a, c2 = o1 - I->plan[S->pool[w]] + beta;
      S->cap[w] = c1 < c2 ? c1 : c2;
    } else {
      S->cap[w] = a;
    }
  }
  /* Scan the shorter jobs in decreasing length (reading: only ranks after the
   * M long jobs; a job that fits no worker is skipped and stays queued).  Each
   * goes to the first spare worker with room, else to the long worker of
   * largest index with room. */
  /* Algorithm 3 visits the candidates from o_k, the longest within the largest
   * cap (spare caps alpha included); only those are counted. */
  int64_t cap_top = Bp > m ? a : 0;
  for (int64_t w = 1; w < m; ++w)
    if (S->cap[w] > cap_top) cap_top = S->cap[w];
  for (int32_t q = (int32_t)m; q < k; ++q) {
    int32_t j = S->pool[q];
    int64_t L = I->plan[j];
    int64_t placed = -1;
    if (L <= cap_top) g_pack_scans++;
    for (int64_t w = m; w < Bp; ++w)
      if (S->load[w] + L <= a) {
        placed = w;
        break;
      }
    if (placed < 0)
      for (int64_t w = m - 1; w >= 1; --w)
        if (S->load[w] + L <= S->cap[w]) {
          placed = w;
          break;
        }
    if (placed >= 0) {
      enqueue(S, (int32_t)placed, j);
      S->load[placed] += L;
    }
  }
  /* Worker j in 2..M runs its pack and then o_j; worker 1 holds o_1. */
  for (int64_t w = 1; w < m; ++w) enqueue(S, (int32_t)w, S->pool[w]);
  enqueue(S, 0, S->pool[0]);
  /* Worker 1 idles for min{max{max_j P_j - alpha, 0}, alpha} (reading: the
   * largest pack sum; exact for B = 2, where it is Algorithm 2's delay). */
  int64_t pmax = 0;
  for (int64_t w = 1; w < Bp; ++w)
    if (S->load[w] > pmax) pmax = S->load[w];
  int64_t idle = pmax - a;
  if (idle < 0) idle = 0;
  if (idle > a) idle = a;
  S->t_w1 = t + idle;
}

static int32_t longest_pool_job(const or_sim* S, const int32_t* ord_long, int64_t t) {
  const or_inst* I = S->I;
  for (int32_t q = 0; q < I->n; ++q) {
    int32_t j = ord_long[q];
    if (S->st[j] == ST_WAIT && !S->planned[j] && released(I, j, t)) return j;
  }
  return -1;
}

static void admit_isjl(or_sim* S, const int32_t* ord_long, int64_t t, int64_t amax,
                       uint32_t flags) {
  const or_inst* I = S->I;
  /* Epoch: the machine is empty and no plan is pending -> Phase ONE. */
  if (S->nact == 0 && !any_queue(S)) phase_one(S, ord_long, t, flags);
  /* Plan starts, workers in index order.  Each start is guarded by the
   * fairness check A_max(t) <= alpha and the KV budget (reading: for B > 2 the
   * plan alone does not keep every pair within alpha). */
  for (int64_t w = 0; w < I->B; ++w) {
    if (S->cur[w] >= 0 || S->qhead[w] < 0) continue;
    if (w == 0 && t < S->t_w1) continue;
    int32_t j = S->qhead[w];
    if (amax <= I->alpha && kv_ok(S, j)) {
      S->qhead[w] = S->qnext[j];
      if (S->qhead[w] < 0) S->qtail[w] = -1;
      admit(S, j, t);
      S->cur[w] = j;
      S->wk[j] = (int32_t)w;
    }
  }
  /* Phase TWO: an idle worker with nothing planned takes the longest released
   * unplanned job while A_max(t) <= alpha; otherwise stop admitting (DRAIN)
   * until the machine is empty and Phase ONE runs again. */
  if (S->mode != 0) {
    /* Reading flag (experiments only): resume as soon as A_max(t) <= alpha. */
    if ((flags & FLAG_RESUME_FILL) && amax <= I->alpha) S->mode = 0;
    else return;
  }
  for (int64_t w = 0; w < I->B; ++w) {
    if (S->cur[w] >= 0 || S->qhead[w] >= 0) continue;
    int32_t j = longest_pool_job(S, ord_long, t);
    if (j < 0) break;
    if (amax > I->alpha) {
      S->mode = 1;
      break;
    }
    if (!kv_ok(S, j)) break;
    admit(S, j, t);
    S->cur[w] = j;
    S->wk[j] = (int32_t)w;
  }
}

/* ------------------------------------------------------------------ */
static int check_table(int32_t n, const int32_t* arrival, const int32_t* prompt,
                       const int32_t* output) {
  if (n < 1 || !arrival || !prompt || !output) return OR_EINVAL;
  for (int32_t i = 0; i < n; ++i) {
    if (arrival[i] < 0 || prompt[i] < 0 || output[i] < 1) return OR_EINVAL;
    if ((int64_t)prompt[i] + output[i] > (1 << 30)) return OR_ERANGE;
  }
  return OR_OK;
}

static int make_inst(or_inst* I, int32_t n, const int32_t* arrival, const int32_t* prompt,
                     const int32_t* output, int32_t B, int32_t alpha, int64_t M_kv,
                     int64_t c, int64_t tau) {
  int rc = check_table(n, arrival, prompt, output);
  if (rc) return rc;
  if (B < 0 || alpha < 0 || M_kv < 0 || c < 0 || tau < 0) return OR_EINVAL;
  I->n = n;
  I->B = B == 0 ? n : B;
  I->M = M_kv;
  I->alpha = alpha == ALPHA_INF_SENTINEL ? INT64_MAX : alpha;
  I->c = c;
  I->tau = tau;
  I->arrival = arrival;
  I->len = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
  if (!I->len) return OR_ENOMEM;
  for (int32_t i = 0; i < n; ++i) I->len[i] = (int64_t)prompt[i] + output[i];
  I->plan = I->len;
  I->resv = I->len;
  I->pre = NULL;
  return OR_OK;
}

/* Simulate one instance under one policy, step by step.
 * Step t (0-based): retire jobs whose last token was processed at t-1; compute
 * A_max(t) = max progress of the still-active jobs; let the policy admit jobs
 * released by t (they start with progress 0); account the step.  The run ends
 * when every job has finished; T is the makespan (idle steps included). */
static int simulate_impl(int32_t n, const int32_t* arrival, const int32_t* prompt,
                         const int32_t* output, const int32_t* upper, int32_t B, int32_t alpha,
                         int64_t M_kv, int32_t policy, uint32_t flags, int64_t cost_c,
                         int64_t cost_tau, or_metrics* out, int32_t* start_out,
                         int32_t* finish_out) {
  if (!out) return OR_EINVAL;
  if (policy < 0 || policy > 3) return OR_EINVAL;
  or_inst I;
  int rc = make_inst(&I, n, arrival, prompt, output, B, alpha, M_kv, cost_c, cost_tau);
  if (rc) return rc;
  int64_t* extra = NULL; /* plan, resv and pre of the variants */
  const int prefill = (flags & FLAG_PREFILL) != 0;
  if (upper || prefill) {
    extra = (int64_t*)malloc(sizeof(int64_t) * 3 * (size_t)n);
    if (!extra) {
      free(I.len);
      return OR_ENOMEM;
    }
    I.plan = extra;
    I.resv = extra + n;
    for (int32_t i = 0; i < n; ++i) {
      if (upper && (upper[i] < output[i] || (int64_t)prompt[i] + upper[i] > (1 << 30))) {
        const int code = upper[i] < output[i] ? OR_EINVAL : OR_ERANGE;
        free(extra);
        free(I.len);
        return code;
      }
      /* Robust-ISJL (Section 3.4): the sizes used for ordering, packing, M, the
       * caps and (reading) the KV reservation take the predicted upper bound of
       * the output; jobs still run their true length. */
      const int64_t out_plan = upper ? upper[i] : output[i];
      if (prefill) {
        /* Prefill at admission (reading of Section 1 with eq. (1)'s decode
         * progress): the prompt is processed when the job is admitted, the job
         * then runs one step per output token, its footprint is prompt +
         * progress, and it reserves prompt + output. */
        I.len[i] = output[i];
        I.plan[i] = out_plan;
        I.resv[i] = (int64_t)prompt[i] + out_plan;
      } else {
        I.plan[i] = (int64_t)prompt[i] + out_plan;
        I.resv[i] = I.plan[i];
      }
    }
    if (prefill) {
      I.pre = extra + 2 * (size_t)n;
      for (int32_t i = 0; i < n; ++i) I.pre[i] = prompt[i];
    }
  }
  size_t nn = (size_t)n, nb = (size_t)I.B;
  or_sim S;
  memset(&S, 0, sizeof(S));
  S.I = &I;
  S.start = (int64_t*)malloc(sizeof(int64_t) * nn);
  S.st = (int8_t*)calloc(nn, 1);
  S.act = (int32_t*)malloc(sizeof(int32_t) * nn);
  int32_t* ord = (int32_t*)malloc(sizeof(int32_t) * nn);
  int32_t* scratch_act = (int32_t*)malloc(sizeof(int32_t) * nn);
  int ok = S.start && S.st && S.act && ord && scratch_act;
  if (policy == POL_ISJL) {
    S.cur = (int32_t*)malloc(sizeof(int32_t) * nb);
    S.qhead = (int32_t*)malloc(sizeof(int32_t) * nb);
    S.qtail = (int32_t*)malloc(sizeof(int32_t) * nb);
    S.load = (int64_t*)malloc(sizeof(int64_t) * nb);
    S.cap = (int64_t*)malloc(sizeof(int64_t) * nb);
    S.wk = (int32_t*)malloc(sizeof(int32_t) * nn);
    S.qnext = (int32_t*)malloc(sizeof(int32_t) * nn);
    S.planned = (int8_t*)calloc(nn, 1);
    S.pool = (int32_t*)malloc(sizeof(int32_t) * nn);
    ok = ok && S.cur && S.qhead && S.qtail && S.load && S.cap && S.wk && S.qnext && S.planned &&
         S.pool;
    if (ok) {
      for (size_t w = 0; w < nb; ++w) S.cur[w] = S.qhead[w] = S.qtail[w] = -1;
      for (size_t i = 0; i < nn; ++i) S.wk[i] = S.qnext[i] = -1;
    }
  }
  if (!ok) {
    rc = OR_ENOMEM;
    goto done;
  }
  for (size_t i = 0; i < nn; ++i) S.start[i] = -1;
  if (policy == POL_FCFS) make_order(ord, &I, 0);
  else if (policy == POL_SJF) make_order(ord, &I, 1);
  else make_order(ord, &I, 2);

  int64_t max_r = 0, sum_len = 0, max_len = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (arrival[i] > max_r) max_r = arrival[i];
    sum_len += I.plan[i];
    if (I.plan[i] > max_len) max_len = I.plan[i];
  }
  int64_t a_cap = I.alpha < max_len ? I.alpha : max_len;
  const int64_t bound = max_r + 2 * sum_len + (int64_t)n * a_cap + 2;

  or_acc acc;
  memset(&acc, 0, sizeof(acc));
  int32_t ndone = 0;
  int64_t t = 0;
  for (;;) {
    /* (1) retire */
    int32_t keep = 0;
    for (int32_t k = 0; k < S.nact; ++k) {
      int32_t j = S.act[k];
      if (S.start[j] + I.len[j] == t) {
        S.st[j] = ST_DONE;
        S.res -= I.resv[j];
        ndone++;
        if (policy == POL_ISJL) S.cur[S.wk[j]] = -1;
      } else {
        scratch_act[keep++] = j;
      }
    }
    memcpy(S.act, scratch_act, sizeof(int32_t) * (size_t)keep);
    S.nact = keep;
    if (ndone == n) break;
    /* (2) releases are implicit: job i is in the queue iff arrival_i <= t. */
    /* (3) A_max(t): largest progress among active jobs (0 if none). */
    int64_t amax = 0;
    for (int32_t k = 0; k < S.nact; ++k) {
      int64_t a = t - S.start[S.act[k]];
      if (a > amax) amax = a;
    }
    /* (4) admissions */
    switch (policy) {
      case POL_FCFS: admit_strict(&S, ord, t, 1); break;
      case POL_SJF: admit_strict(&S, ord, t, 0); break;
      case POL_LJF: admit_ljf(&S, ord, t); break;
      default: admit_isjl(&S, ord, t, amax, flags); break;
    }
    /* (5) account step t */
    account_step(&acc, &I, t, S.start, S.act, S.nact);
    t++;
    if (t > bound) {
      rc = OR_EINTERNAL;
      goto done;
    }
  }
  finish_metrics(out, &I, &acc, t, S.start);
  if (start_out)
    for (int32_t i = 0; i < n; ++i) start_out[i] = (int32_t)S.start[i];
  if (finish_out)
    for (int32_t i = 0; i < n; ++i) finish_out[i] = (int32_t)(S.start[i] + I.len[i]);
  rc = OR_OK;
done:
  free(S.start);
  free(S.st);
  free(S.act);
  free(ord);
  free(scratch_act);
  free(S.cur);
  free(S.qhead);
  free(S.qtail);
  free(S.load);
  free(S.cap);
  free(S.wk);
  free(S.qnext);
  free(S.planned);
  free(S.pool);
  free(extra);
  free(I.len);
  return rc;
}

/* ------------------------------------------------------------------ */
/* Re-score a given schedule (start steps) from the schedule alone: check the
 * constraints at every step and accumulate the Section 5 cost terms.
 * violation bits: 1 start before release, 2 more than B active, 4 KV budget
 * exceeded with two or more active, 8 fairness range above alpha,
 * 16 negative start (nothing else is evaluated then). */
int oracle_decompose(int32_t n, const int32_t* arrival, const int32_t* prompt,
                     const int32_t* output, int32_t B, int32_t alpha, int64_t M_kv,
                     int64_t cost_c, int64_t cost_tau, const int32_t* start_in,
                     or_metrics* out, uint32_t* violation) {
  if (!out || !violation || !start_in) return OR_EINVAL;
  or_inst I;
  int rc = make_inst(&I, n, arrival, prompt, output, B, alpha, M_kv, cost_c, cost_tau);
  if (rc) return rc;
  uint32_t v = 0;
  int64_t* start = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
  int32_t* act = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
  if (!start || !act) {
    free(start);
    free(act);
    free(I.len);
    return OR_ENOMEM;
  }
  int64_t T = 0;
  for (int32_t i = 0; i < n; ++i) {
    start[i] = start_in[i];
    if (start[i] < 0) v |= 16u;
    if (start[i] < arrival[i]) v |= 1u;
    if (start[i] + I.len[i] > T) T = start[i] + I.len[i];
  }
  or_acc acc;
  memset(&acc, 0, sizeof(acc));
  if (v & 16u) {
    memset(out, 0, sizeof(*out));
    *violation = v;
    free(start);
    free(act);
    free(I.len);
    return OR_OK;
  }
  for (int64_t t = 0; t < T; ++t) {
    int32_t nact = 0;
    int64_t res = 0;
    for (int32_t i = 0; i < n; ++i)
      if (start[i] <= t && t < start[i] + I.len[i]) {
        act[nact++] = i;
        res += I.len[i];
      }
    if (nact > I.B) v |= 2u;
    if (I.M != 0 && nact >= 2 && res > I.M) v |= 4u;
    if (nact > 0) {
      int64_t mx = INT64_MIN, mn = INT64_MAX;
      for (int32_t k = 0; k < nact; ++k) {
        int64_t a = t - start[act[k]];
        if (a > mx) mx = a;
        if (a < mn) mn = a;
      }
      if (mx - mn > I.alpha) v |= 8u;
    }
    account_step(&acc, &I, t, start, act, nact);
  }
  finish_metrics(out, &I, &acc, T, start);
  *violation = v;
  free(start);
  free(act);
  free(I.len);
  return OR_OK;
}

/* ------------------------------------------------------------------ */
/* Exact alpha-fair optimum (Appendix A's integer program, plus release steps
 * and the KV budget): the least makespan over every start vector with
 * s_i >= r_i, at most B jobs active per step, reservations within M_kv unless a
 * job runs alone, and |s_i - s_j| <= alpha for every pair active at a common
 * step (for contiguous non-preemptive jobs that is the IP's fairness row).
 *
 * Plain exhaustive search: at every step branch over every admissible subset of
 * released unstarted jobs, including the empty subset (deliberate waiting),
 * memoised on (step clipped to the last release, unstarted set, progress of
 * each active job).  The only pruning: at an empty machine with every
 * remaining job released, waiting one step is never better (the rest of the
 * schedule can be shifted one step earlier), so the empty subset is skipped
 * there.  n <= 8 and lengths <= 65535. */
typedef struct {
  uint64_t k0, k1, k2;
  int64_t val;
  int32_t used;
} or_memo_e;

typedef struct {
  or_memo_e* tab;
  size_t cap, cnt;
  const or_inst* I;
  int64_t rmax;
} or_opt;

static uint64_t h64(uint64_t x) {
  x ^= x >> 33;
  x *= 0xff51afd7ed558ccdULL;
  x ^= x >> 33;
  x *= 0xc4ceb9fe1a85ec53ULL;
  x ^= x >> 33;
  return x;
}

static int memo_grow(or_opt* P);

static or_memo_e* memo_find(or_opt* P, uint64_t k0, uint64_t k1, uint64_t k2, int create) {
  if (create && (P->cnt + 1) * 2 > P->cap) {
    if (memo_grow(P)) return NULL;
  }
  if (P->cap == 0) return NULL;
  size_t mask = P->cap - 1;
  size_t h = (size_t)(h64(k0 ^ h64(k1 ^ h64(k2)))) & mask;
  for (;;) {
    or_memo_e* e = &P->tab[h];
    if (!e->used) {
      if (!create) return NULL;
      e->used = 1;
      e->k0 = k0;
      e->k1 = k1;
      e->k2 = k2;
      e->val = -1;
      P->cnt++;
      return e;
    }
    if (e->k0 == k0 && e->k1 == k1 && e->k2 == k2) return e;
    h = (h + 1) & mask;
  }
}

static int memo_grow(or_opt* P) {
  size_t ncap = P->cap ? P->cap * 2 : 1024;
  or_memo_e* old = P->tab;
  size_t ocap = P->cap;
  P->tab = (or_memo_e*)calloc(ncap, sizeof(or_memo_e));
  if (!P->tab) {
    P->tab = old;
    return -1;
  }
  P->cap = ncap;
  P->cnt = 0;
  for (size_t i = 0; i < ocap; ++i)
    if (old[i].used) {
      or_memo_e* e = memo_find(P, old[i].k0, old[i].k1, old[i].k2, 1);
      e->val = old[i].val;
    }
  free(old);
  return 0;
}

/* prog[i]: 0 = not active, else steps already processed (>= 1). */
static int64_t opt_rec(or_opt* P, int64_t t, uint32_t U, const uint16_t* prog, int* err) {
  const or_inst* I = P->I;
  const int32_t n = I->n;
  int nA = 0;
  for (int32_t i = 0; i < n; ++i)
    if (prog[i]) nA++;
  if (U == 0 && nA == 0) return 0;
  uint64_t tk = (uint64_t)(t < P->rmax ? t : P->rmax);
  uint64_t k1 = 0, k2 = 0;
  for (int32_t i = 0; i < n && i < 4; ++i) k1 |= (uint64_t)prog[i] << (16 * i);
  for (int32_t i = 4; i < n; ++i) k2 |= (uint64_t)prog[i] << (16 * (i - 4));
  uint64_t k0 = (tk << 8) | U;
  or_memo_e* e = memo_find(P, k0, k1, k2, 0);
  if (e && e->val >= 0) return e->val;

  uint32_t rel = 0;
  for (int32_t i = 0; i < n; ++i)
    if ((U >> i & 1u) && I->arrival[i] <= t) rel |= 1u << i;
  int64_t amax = 0, resA = 0;
  for (int32_t i = 0; i < n; ++i)
    if (prog[i]) {
      if (prog[i] > amax) amax = prog[i];
      resA += I->len[i];
    }
  int64_t best = INT64_MAX;
  /* iterate over all subsets X of rel, including the empty one */
  uint32_t X = rel;
  for (;;) {
    int okX = 1;
    if (X == 0) {
      if (nA == 0 && rel == U) okX = 0;
    } else {
      int cnt = nA;
      int64_t res = resA;
      for (int32_t i = 0; i < n; ++i)
        if (X >> i & 1u) {
          cnt++;
          res += I->len[i];
        }
      if (cnt > I->B) okX = 0;
      if (amax > I->alpha) okX = 0;
      if (I->M != 0 && cnt >= 2 && res > I->M) okX = 0;
    }
    if (okX) {
      uint16_t np[8];
      for (int32_t i = 0; i < n; ++i) {
        int64_t p = prog[i];
        if (X >> i & 1u) p = 1;
        else if (p) p = p + 1;
        if (p && p >= I->len[i]) p = 0; /* finished at the end of step t */
        np[i] = (uint16_t)p;
      }
      /* a job of length 1 started now finishes now; it is no longer unstarted */
      int64_t r = opt_rec(P, t + 1, U & ~X, np, err);
      if (*err) return 0;
      if (r != INT64_MAX && r + 1 < best) best = r + 1;
    }
    if (X == 0) break;
    X = (X - 1) & rel;
  }
  e = memo_find(P, k0, k1, k2, 1);
  if (!e) {
    *err = OR_ENOMEM;
    return 0;
  }
  e->val = best;
  return best;
}

int oracle_opt(int32_t n, const int32_t* arrival, const int32_t* prompt, const int32_t* output,
               int32_t B, int32_t alpha, int64_t M_kv, int64_t* T_opt, int32_t* start_opt) {
  if (!T_opt) return OR_EINVAL;
  if (n > 8) return OR_ETOOLARGE;
  or_inst I;
  int rc = make_inst(&I, n, arrival, prompt, output, B, alpha, M_kv, 0, 0);
  if (rc) return rc;
  for (int32_t i = 0; i < n; ++i)
    if (I.len[i] > 65535) {
      free(I.len);
      return OR_ETOOLARGE;
    }
  or_opt P;
  memset(&P, 0, sizeof(P));
  P.I = &I;
  for (int32_t i = 0; i < n; ++i)
    if (arrival[i] > P.rmax) P.rmax = arrival[i];
  uint16_t prog[8] = {0};
  int err = 0;
  uint32_t U = (n == 32) ? 0xffffffffu : ((1u << n) - 1u);
  int64_t R = opt_rec(&P, 0, U, prog, &err);
  if (err) {
    free(P.tab);
    free(I.len);
    return err;
  }
  *T_opt = R;
  if (start_opt) {
    /* Walk the memo: at each step take the first subset (in the enumeration
     * order above) that attains the optimum from the current state. */
    int64_t t = 0;
    uint32_t Ucur = U;
    uint16_t pc[8] = {0};
    for (int32_t i = 0; i < n; ++i) start_opt[i] = -1;
    while (Ucur != 0) {
      int64_t here = opt_rec(&P, t, Ucur, pc, &err);
      uint32_t rel = 0;
      int nA = 0;
      int64_t amax = 0, resA = 0;
      for (int32_t i = 0; i < n; ++i) {
        if ((Ucur >> i & 1u) && arrival[i] <= t) rel |= 1u << i;
        if (pc[i]) {
          nA++;
          if (pc[i] > amax) amax = pc[i];
          resA += I.len[i];
        }
      }
      uint32_t X = rel, chosen = 0xffffffffu;
      for (;;) {
        int okX = 1;
        if (X == 0) {
          if (nA == 0 && rel == Ucur) okX = 0;
        } else {
          int cnt = nA;
          int64_t res = resA;
          for (int32_t i = 0; i < n; ++i)
            if (X >> i & 1u) {
              cnt++;
              res += I.len[i];
            }
          if (cnt > I.B || amax > I.alpha || (I.M != 0 && cnt >= 2 && res > I.M)) okX = 0;
        }
        if (okX) {
          uint16_t np[8];
          for (int32_t i = 0; i < n; ++i) {
            int64_t p = pc[i];
            if (X >> i & 1u) p = 1;
            else if (p) p = p + 1;
            if (p && p >= I.len[i]) p = 0;
            np[i] = (uint16_t)p;
          }
          int64_t r = opt_rec(&P, t + 1, Ucur & ~X, np, &err);
          if (r != INT64_MAX && r + 1 == here) {
            chosen = X;
            memcpy(pc, np, sizeof(np));
            break;
          }
        }
        if (X == 0) break;
        X = (X - 1) & rel;
      }
      if (chosen == 0xffffffffu || err) {
        free(P.tab);
        free(I.len);
        return err ? err : OR_EINTERNAL;
      }
      for (int32_t i = 0; i < n; ++i)
        if (chosen >> i & 1u) start_opt[i] = (int32_t)t;
      Ucur &= ~chosen;
      t++;
    }
  }
  free(P.tab);
  free(I.len);
  return OR_OK;
}

int oracle_simulate(int32_t n, const int32_t* arrival, const int32_t* prompt,
                    const int32_t* output, int32_t B, int32_t alpha, int64_t M_kv,
                    int32_t policy, uint32_t flags, int64_t cost_c, int64_t cost_tau,
                    or_metrics* out, int32_t* start_out, int32_t* finish_out) {
  return simulate_impl(n, arrival, prompt, output, NULL, B, alpha, M_kv, policy, flags, cost_c,
                       cost_tau, out, start_out, finish_out);
}

/* Robust-ISJL and the other policies on predicted sizes: upper[i] >= output[i]
 * is the upper end of output i's prediction interval. */
int oracle_simulate_robust(int32_t n, const int32_t* arrival, const int32_t* prompt,
                           const int32_t* output, const int32_t* upper, int32_t B,
                           int32_t alpha, int64_t M_kv, int32_t policy, uint32_t flags,
                           int64_t cost_c, int64_t cost_tau, or_metrics* out,
                           int32_t* start_out, int32_t* finish_out) {
  if (!upper) return OR_EINVAL;
  return simulate_impl(n, arrival, prompt, output, upper, B, alpha, M_kv, policy, flags, cost_c,
                       cost_tau, out, start_out, finish_out);
}

/* Convenience loops over instances (still single-threaded). */
int oracle_simulate_batch(int64_t n_inst, int32_t n, const int32_t* arrival,
                          const int32_t* prompt, const int32_t* output, int32_t B,
                          int32_t alpha, int64_t M_kv, int32_t policy, uint32_t flags,
                          int64_t cost_c, int64_t cost_tau, or_metrics* out,
                          int32_t* start_out, int32_t* finish_out) {
  for (int64_t k = 0; k < n_inst; ++k) {
    size_t off = (size_t)k * (size_t)n;
    int rc = oracle_simulate(n, arrival + off, prompt + off, output + off, B, alpha, M_kv,
                             policy, flags, cost_c, cost_tau, out + k,
                             start_out ? start_out + off : NULL,
                             finish_out ? finish_out + off : NULL);
    if (rc) return rc;
  }
  return OR_OK;
}

int oracle_simulate_robust_batch(int64_t n_inst, int32_t n, const int32_t* arrival,
                                 const int32_t* prompt, const int32_t* output,
                                 const int32_t* upper, int32_t B, int32_t alpha, int64_t M_kv,
                                 int32_t policy, uint32_t flags, int64_t cost_c,
                                 int64_t cost_tau, or_metrics* out, int32_t* start_out,
                                 int32_t* finish_out) {
  for (int64_t k = 0; k < n_inst; ++k) {
    size_t off = (size_t)k * (size_t)n;
    int rc = oracle_simulate_robust(n, arrival + off, prompt + off, output + off, upper + off,
                                    B, alpha, M_kv, policy, flags, cost_c, cost_tau, out + k,
                                    start_out ? start_out + off : NULL,
                                    finish_out ? finish_out + off : NULL);
    if (rc) return rc;
  }
  return OR_OK;
}

int oracle_opt_batch(int64_t n_inst, int32_t n, const int32_t* arrival, const int32_t* prompt,
                     const int32_t* output, int32_t B, int32_t alpha, int64_t M_kv,
                     int64_t* T_opt, int32_t* start_opt) {
  for (int64_t k = 0; k < n_inst; ++k) {
    size_t off = (size_t)k * (size_t)n;
    int rc = oracle_opt(n, arrival + off, prompt + off, output + off, B, alpha, M_kv, T_opt + k,
                        start_opt ? start_opt + off : NULL);
    if (rc) return rc;
  }
  return OR_OK;
}

int oracle_metrics_size(void) { return (int)sizeof(or_metrics); }
