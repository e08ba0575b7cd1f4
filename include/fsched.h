/*
 * fsched — batched evaluation of resource-fair LLM batching on AMD Instinct
 * MI355X (gfx950).  C ABI of libfsched.so.
 *
 * The library evaluates many independent instances of the scheduling model of
 * "Efficiency and Cost Alignment in Batched LLM Serving via Resource-Fair
 * Scheduling" (Yao & Zhou):
 *   - Section 2: n requests, request i processes prompt_i + output_i tokens one
 *     per step (chunked prefill: the paper's o_i counts prompt and output
 *     tokens); at most B requests run per step; the fairness constraint,
 *     eq. (1), bounds the spread of the progress a_i(t) of co-running requests
 *     by alpha;
 *   - Section 3: the policies LJF (Algorithm 1) and ISJL (Algorithm 2 for B = 2,
 *     Algorithm 3 for B >= 2), run on the released queue (Section 3.5,
 *     Online-ISJL), plus the unfair baselines FCFS and SJF of Section 2.1;
 *   - Section 5: the cost of step t is c + tau |S_t| max_{S_t} r_i with
 *     r_i = a_i + 1, and the profit-decomposition theorem splits the total into
 *     tau Q + c T + tau E.
 * In addition to the paper's model every call takes a KV budget M_kv: the
 * reservations (full lengths) of co-running requests must fit in M_kv unless a
 * request runs alone.
 *
 * Conventions shared by every call
 *   - Job tables are row-major [n_inst][n_jobs] int32: arrival step (>= 0),
 *     prompt tokens (>= 0) and output tokens (>= 1) of every job.
 *   - Steps are 0-based.  A job started at step s is active on steps
 *     s .. s + len - 1 (len = prompt + output) and completes at s + len; the
 *     makespan T is the latest completion, idle steps included.
 *   - Pointers: with FSCHED_F_DEVICE_PTRS every array argument is a device
 *     pointer and the call only enqueues work on `stream` (a hipStream_t, or
 *     NULL for the null stream); outputs are valid once the stream reaches the
 *     call.  Without the flag every array is host memory; the library stages
 *     through device memory it allocates and frees itself and returns after
 *     the results are back in host memory.
 *   - The caller owns every buffer.  The library keeps no pointer after the
 *     call (host mode) or after the stream passes the call (device mode).
 *   - fsched_simulate, fsched_simulate_robust and fsched_bruteforce_opt (every
 *     policy but FCFS) also take a scratch table of 2 bytes per job (rows
 *     rounded up to 64 jobs) on `stream`, from a memory pool the library creates
 *     once per device and keeps for the process: freed on the stream after the
 *     call's kernels, it stays in the pool for the next call (else the
 *     device's default pool is used).  If neither can supply it the call
 *     returns FSCHED_ENOMEM before enqueuing any kernel.
 *   - Return codes are FSCHED_OK or a negative FSCHED_E* code; outputs are
 *     undefined on error.  Argument errors (null pointers, bad sizes or
 *     parameters) are detected before any work is enqueued.  In device mode the
 *     job tables are not read on the host: an instance whose table is invalid
 *     (or exceeds a kernel limit) gets T = FSCHED_T_INVALID / FSCHED_T_RANGE /
 *     FSCHED_T_TOOLARGE in its metrics and every other field zero; host mode
 *     checks the tables first and returns the matching error code instead.
 *   - Kernel limits: n_jobs <= 4096; min(B, n_jobs) <= 1024; len < 2^20; when
 *     the arrivals of an instance are not non-decreasing in job index, every
 *     arrival < 2^20.  Beyond them: FSCHED_ETOOLARGE / FSCHED_T_TOOLARGE.
 */
#ifndef FSCHED_H
#define FSCHED_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FSCHED_ABI_VERSION 1

#define FSCHED_ALPHA_INF INT32_MAX /* fairness budget = infinity             */
#define FSCHED_UNLIMITED 0         /* B = 0: no count limit; M_kv = 0: none   */

enum { FSCHED_FCFS = 0, FSCHED_LJF = 1, FSCHED_ISJL = 2, FSCHED_SJF = 3 };

enum {
  FSCHED_OK = 0,
  FSCHED_EINVAL = -1,    /* bad argument or job table                        */
  FSCHED_ERANGE = -2,    /* an int64 accumulator could overflow              */
  FSCHED_ENOMEM = -3,    /* device or host allocation failed                 */
  FSCHED_EDEVICE = -4,   /* a HIP call failed (see fsched_last_hip_error)     */
  FSCHED_ETOOLARGE = -5, /* beyond a kernel limit                            */
  FSCHED_ENOTIMPL = -6,
  FSCHED_EINTERNAL = -7, /* an instance found no next event, or its exact search hit its cap */
  FSCHED_ESCRATCH = -8   /* fsched_simulate_noalloc: the call needs more scratch than
                            FSCHED_NOALLOC_SCRATCH_BYTES                         */
};

/* Per-instance markers written into fsched_metrics.T in device mode. */
#define FSCHED_T_INVALID (-1)
#define FSCHED_T_RANGE (-2)
#define FSCHED_T_TOOLARGE (-5)
#define FSCHED_T_INTERNAL (-7)

enum {
  FSCHED_F_DEVICE_PTRS = 1u, /* array arguments are device pointers            */
  FSCHED_F_SYNC = 4u,        /* device mode: synchronize the stream before return */
  FSCHED_F_BETA_SQRT17 = 8u, /* ISJL: beta = floor((sqrt(17)-1) alpha / 4), the
                                B = 2 choice of Section 3.2; default beta = alpha
                                (Section 3.3)                                   */
  FSCHED_F_RESUME_FILL = 16u, /* ISJL, experiments only: after Phase TWO stops on
                                A_max > alpha, it resumes as soon as A_max <= alpha
                                again instead of waiting for the machine to empty
                                (the other reading of "repeat from Phase ONE"
                                with busy workers, Algorithms 2 and 3)          */
  FSCHED_F_PREFILL = 32u     /* simulate / simulate_robust: the prompt is
                                prefilled when the job is admitted (Section 1's
                                prefill pass; eq. (1)'s progress counts decode
                                tokens): a job runs output_i steps, reserves
                                prompt_i + output_i of M_kv, its footprint in the
                                Section 5 batch cost is prompt_i + progress, and
                                fairness, extent and A_max stay on progress.
                                O counts prompt + output tokens; Q is the
                                footprint summed over the job's own steps.
                                Default: the chunked reading of Section 2 (a job
                                runs prompt_i + output_i steps, footprint =
                                progress).  The other calls return ENOTIMPL
                                with it.                                        */
};

/* Scheduling and cost parameters (40 bytes, no padding). */
typedef struct {
  int32_t B;        /* max requests per step (paper's B), >= 1, or FSCHED_UNLIMITED */
  int32_t alpha;    /* fairness budget on progress, >= 0, or FSCHED_ALPHA_INF        */
  int64_t M_kv;     /* KV reservation budget in tokens, >= 1, or FSCHED_UNLIMITED    */
  int32_t policy;   /* FSCHED_FCFS | FSCHED_LJF | FSCHED_ISJL | FSCHED_SJF           */
  uint32_t flags;   /* FSCHED_F_*                                                    */
  int64_t cost_c;   /* fixed cost of one step, c >= 0 (integer units)                */
  int64_t cost_tau; /* footprint coefficient tau >= 0 (integer units)                */
} fsched_params;

/* Per-instance results (104 bytes); every field is exact.
 *   T               makespan (steps, idle steps included)
 *   O               sum of lengths (tokens)
 *   Q               intrinsic term sum_i len_i (len_i + 1) / 2   (profit decomposition, Section 5)
 *   E               batching externality sum_t sum_S (max r - r_i)  (profit decomposition, Section 5)
 *   C               total cost sum_t (c + tau |S_t| max r); equals c T + tau (Q + E)
 *   W               max-driven step cost sum_t (c + tau max r) (no |S| factor)
 *   sum_completion  sum_i (s_i + len_i)
 *   sum_latency     sum_i (s_i + len_i - arrival_i)
 *   sum_extent      sum over busy steps of (max r - min r)
 *   busy_steps      steps with at least one active job
 *   peak_kv         max over steps of sum_S r_i (tokens held)
 *   unfair_steps    steps whose extent exceeds alpha
 *   max_extent      max over steps of the extent
 *   max_active      max over steps of |S_t|                                     */
typedef struct {
  int64_t T, O, Q, E, C, W;
  int64_t sum_completion, sum_latency;
  int64_t sum_extent, busy_steps;
  int64_t peak_kv, unfair_steps;
  int32_t max_extent, max_active;
} fsched_metrics;

/* fsched_simulate — run every instance under p->policy and report its metrics.
 *
 * Policies (Sections 2.1 and 3):
 *   FCFS  continuous batching in (arrival, index) order; admission stops at the
 *         first released job that does not fit B or M_kv; no fairness guard.
 *   SJF   the same in (length, index) order.
 *   LJF   Algorithm 1: at an empty machine start the longest released jobs, at
 *         most B and stopping at the first that does not fit M_kv; admit nothing
 *         else until the machine is empty again.
 *   ISJL  Algorithms 2/3 on the released queue: Phase ONE builds a plan around
 *         the longest job (short-job packs under the caps min{2 alpha,
 *         o_1 - o_j + beta}, spare workers with packs up to alpha, worker 1
 *         delayed by min{max{max pack - alpha, 0}, alpha}); every plan start and
 *         every Phase TWO admission is guarded by A_max(t) <= alpha; when Phase
 *         TWO finds A_max(t) > alpha it drains until the machine is empty and
 *         Phase ONE runs again.  The plan uses at most as many workers as the
 *         longest queued jobs can fill within M_kv.
 *
 * Arguments
 *   p        parameters (host pointer, read during the call).
 *   n_inst   number of instances, >= 0 (0: nothing is done).
 *   n_jobs   jobs per instance, >= 1.
 *   arrival, prompt, output   job tables [n_inst][n_jobs].
 *   out      [n_inst] metrics.
 *   start, finish   nullable [n_inst][n_jobs] int32: start step and completion
 *            step of every job.
 *   stream   hipStream_t (device mode) or NULL.
 * Errors: EINVAL (null required pointer, n_jobs < 1, n_inst < 0, B < 0,
 *   alpha < 0, M_kv < 0, cost < 0, unknown policy or flag, invalid table in host
 *   mode), ERANGE (host mode: an accumulator could exceed int64), ETOOLARGE,
 *   ENOMEM, EDEVICE. */
int fsched_simulate(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                    const int32_t* arrival, const int32_t* prompt, const int32_t* output,
                    fsched_metrics* out, int32_t* start, int32_t* finish, void* stream);

/* fsched_simulate_robust — Robust-ISJL (Section 3.4): ISJL run with the proxy
 * size prompt_i + upper_i wherever a job size is used to plan — the priority
 * order, Phase ONE's M, caps and packs, worker 1's delay — and (reading: the
 * size known at admission) for the KV reservation against M_kv.  Each job
 * still runs prompt_i + output_i steps, and the fairness guard A_max(t) <=
 * alpha uses the true progress, so the schedule is alpha-fair for any upper
 * (the fairness theorem of Section 3.4).
 * With upper == output the result equals fsched_simulate under ISJL.
 *   upper    [n_inst][n_jobs] int32, upper_i >= output_i (upper end of the
 *            prediction interval of output i; a smaller one is an invalid
 *            table: EINVAL in host mode, T = FSCHED_T_INVALID in device mode).
 *            prompt_i + upper_i is subject to the same length limit as the
 *            true length (ETOOLARGE / FSCHED_T_TOOLARGE beyond it).
 * p->policy must be FSCHED_ISJL (ENOTIMPL otherwise).  All other arguments,
 * outputs and errors as fsched_simulate; metrics describe the true run. */
int fsched_simulate_robust(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                           const int32_t* arrival, const int32_t* prompt,
                           const int32_t* output, const int32_t* upper,
                           fsched_metrics* out, int32_t* start, int32_t* finish,
                           void* stream);

/* fsched_cost_decompose — re-score given schedules (start steps) from the
 * schedule alone (Section 5 terms as in fsched_metrics) and check them.
 *   start      [n_inst][n_jobs] int32 start steps.
 *   violation  [n_inst] uint32 bit mask: 1 a start before its arrival;
 *              2 more than B jobs active at some step; 4 reservations above
 *              M_kv with two or more jobs active; 8 progress range above alpha
 *              (eq. (1)); 16 a negative start (metrics are zero then).
 * p->policy and p->flags other than DEVICE_PTRS / SYNC are ignored, except
 * FSCHED_F_PREFILL (ENOTIMPL: schedules are scored in the chunked reading).
 * Errors as fsched_simulate. */
int fsched_cost_decompose(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                          const int32_t* arrival, const int32_t* prompt,
                          const int32_t* output, const int32_t* start, fsched_metrics* out,
                          uint32_t* violation, void* stream);

/* fsched_bruteforce_opt — exact alpha-fair optimum makespan (Appendix A's
 * integer program with release steps and M_kv added): the least makespan over
 * every start vector with s_i >= arrival_i, at most B active jobs per step,
 * reservations within M_kv unless a job runs alone, and |s_i - s_j| <= alpha for
 * every pair active at a common step.  Exhaustive search over schedules in start
 * order with a memo and lower bounds, started from the ISJL schedule of the
 * instance (which is returned when nothing beats it).  A first pass keeps the
 * search's memo in LDS and stops a search after 2^22 steps; the searches it
 * stops are run again by a second pass with a memo of 2^20 entries per wave in
 * device scratch (256 MiB from the library's pool, with the instance list;
 * stream-ordered, released after the call) and a cap of 2^28 steps.  Only a
 * search past that cap gets T_opt = FSCHED_T_INTERNAL (host mode: EINTERNAL);
 * on the tiny workload (4,096 instances, B = 3 and 4, alpha up to 19, with and
 * without a KV budget) none does.  If the scratch cannot be had, the second
 * pass is skipped and the searches the first pass stopped get the marker.
 *   n_jobs     <= 8 (ETOOLARGE otherwise); every length <= 255 and every
 *              arrival <= 4095 (else T = FSCHED_T_TOOLARGE / ETOOLARGE).
 *   T_opt      [n_inst] int64 optimum makespan.
 *   start_opt  nullable [n_inst][n_jobs] int32: one optimal schedule.
 * p->policy, p->flags other than DEVICE_PTRS / SYNC, cost_c and cost_tau are
 * ignored, except FSCHED_F_PREFILL (ENOTIMPL). */
int fsched_bruteforce_opt(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                          const int32_t* arrival, const int32_t* prompt, const int32_t* output,
                          int64_t* T_opt, int32_t* start_opt, void* stream);

/* fsched_simulate_noalloc — fsched_simulate for callers that cannot allocate
 * device memory during the call: code being captured into a HIP graph, tight
 * serving loops, harnesses that forbid hipMalloc.  It allocates nothing: no
 * hipMalloc / hipFree / pool allocation and no host staging.  Its scratch (the
 * rank table of 2 bytes per job, rows rounded up to 64 jobs, for every policy
 * but FCFS; for ISJL with at most 512 workers and a finite alpha, when the
 * plan-queue links do not fit LDS, 4 bytes per job rounded up to a power of two
 * (at least 64)) is a fixed buffer of FSCHED_NOALLOC_SCRATCH_BYTES per device,
 * part of the library's image and held by each device the library runs on
 * until the process ends; its device address is looked up once per device, on
 * that device's first call.
 *   - p->flags must include FSCHED_F_DEVICE_PTRS (EINVAL otherwise); every
 *     array is a device pointer on the current device, and outputs as in
 *     fsched_simulate.  FSCHED_F_SYNC synchronises the stream before return.
 *   - A call whose scratch would exceed FSCHED_NOALLOC_SCRATCH_BYTES returns
 *     FSCHED_ESCRATCH before enqueuing anything (e.g. at 2,000 jobs per
 *     instance, B = 512 and a finite alpha, 12 KiB per instance: 5,461
 *     instances fit 64 MiB).
 *   - Every call on one device shares that device's buffer: calls that overlap
 *     in time on one device (on different streams, or from several threads)
 *     race and give undefined results.  Calls in order on one stream are safe.
 *     No part of the buffer needs to start cleared (each instance writes its
 *     rows before it reads them), so the last call's contents do no harm.
 * Arguments, results and the other errors as fsched_simulate. */
#define FSCHED_NOALLOC_SCRATCH_BYTES (64u << 20)
int fsched_simulate_noalloc(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                            const int32_t* arrival, const int32_t* prompt,
                            const int32_t* output, fsched_metrics* out, int32_t* start,
                            int32_t* finish, void* stream);

/* Text for a return code (static storage). */
const char* fsched_strerror(int code);

/* FSCHED_ABI_VERSION of the loaded library. */
int fsched_abi_version(void);

/* The hipError_t of the last FSCHED_EDEVICE return on the calling thread. */
int fsched_last_hip_error(void);

/* Returns to the current device the memory that the library's scratch pool on
 * it keeps between calls (the rank tables, see the conventions above); later
 * calls take it from the device again.  Memory of calls still in flight on a
 * stream is not released.  FSCHED_OK (also when the pool was never created),
 * or FSCHED_EDEVICE. */
int fsched_release_cache(void);

#ifdef __cplusplus
}
#endif

#endif /* FSCHED_H */
