// Batched evaluation of the token-step scheduling model: one wavefront per
// instance.
//
// Model (Section 2): job i needs len_i = prompt_i + output_i steps; a job
// started at step s is active on s .. s+len-1; at most B jobs per step; the
// fairness constraint eq. (1) bounds the progress spread of co-running jobs by
// alpha; a KV budget M_kv bounds the summed reservations of co-running jobs.
// Policies: FCFS / SJF (Section 2.1 baselines), LJF (Algorithm 1) and ISJL
// (Algorithms 2 and 3 on the released queue, Section 3.5).  Costs: Section 5.
//
// The kernel is event driven.  Between two events (a completion, a release, a
// delayed plan start, or the step at which A_max(t) crosses alpha while Phase
// TWO waits on the KV budget) the active set is fixed and every active job
// advances one token per step, so the per-step terms of Section 5 are
// arithmetic series summed in closed form:
//   max r over [t, t+D): m_t = t - min_s + 1, sum = D m_t + D(D-1)/2
//   E per step  = sum_S (m_t - r_i) = sum_s - |S| min_s       (constant)
//   extent      = max_s - min_s                               (constant)
//   sum_S r     = |S| (t+1) - sum_s                            (largest at t+D-1)
// Decisions are taken only at events; the step-by-step definition gives the
// same decisions at the steps in between because nothing they depend on
// changes there.  (With the prompt prefilled at admission the largest
// footprint is t + max(prompt_j - start_j) + 1 and E per step is
// |S| G - sum_S (prompt_j - start_j), both constant between events.)
//
// Per-wave state:
//   LDS   W[r]     jobs in the policy's priority order, packed (len << 12 | id)
//         ARR[r]   arrival of rank r (general variant only)
//         QN[r]    next job in the same ISJL plan queue (uint16, ISJL)
//         STG[j]   gather buffer of the first queued ranks (uint16, not FCFS)
//         PEND[i]  released ranks on their way into the bitmap (aliases STG)
//   The drain sweep sorts the active slots in registers; up to 64 of them are
//   first packed into one register through the gather buffer.
//   VGPR  K worker slots per lane: worker w lives in slot w/64 of lane w%64
//         (start, end, ISJL plan-queue head|tail); a bitmap of queued jobs over
//         ranks (bit r%32 of word r/2048 in lane (r/32)%64).
//   SGPR  time, counters, cost accumulators.
#pragma once
#include <type_traits>

#include "sim_common.hpp"
#include "regsort.hpp"
#include "wave.hpp"

namespace fs {

constexpr int POL_FCFS = FSCHED_FCFS, POL_LJF = FSCHED_LJF, POL_ISJL = FSCHED_ISJL,
              POL_SJF = FSCHED_SJF;
constexpr int IDLE = 0x7FFFFFFF;
constexpr uint32_t QNONE = 0xFFFFu;
constexpr uint32_t LMASK = 0xFFFFFu;

__device__ __forceinline__ int plen(uint32_t w) { return (int)(w >> 12); }
__device__ __forceinline__ int pid(uint32_t w) { return (int)(w & 0xFFFu); }

// Bitonic sort of NP (power of two) keys in LDS, ascending, by one wave.
__device__ inline void wave_bitonic_sort(uint32_t* W, int NP, int lane) {
  for (int k = 2; k <= NP; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = lane; i < (NP >> 1); i += WAVE) {
        int lo = ((i & ~(j - 1)) << 1) | (i & (j - 1));
        int hi = lo + j;
        bool up = (lo & k) == 0;
        uint32_t x = W[lo], y = W[hi];
        if ((x > y) == up) {
          W[lo] = y;
          W[hi] = x;
        }
      }
      wave_lds_sync();
    }
  }
}

__device__ inline void write_marker(fsched_metrics* out, int64_t* out_T, int64_t inst,
                                    int64_t code, int lane) {
  if (lane == 0 && out_T) {
    out_T[inst] = code;
  } else if (lane == 0) {
    fsched_metrics m;
    m.T = code;
    m.O = m.Q = m.E = m.C = m.W = 0;
    m.sum_completion = m.sum_latency = m.sum_extent = m.busy_steps = 0;
    m.peak_kv = m.unfair_steps = 0;
    m.max_extent = m.max_active = 0;
    out[inst] = m;
  }
}

template <int NW>
struct PoolBits {
  uint32_t w[NW];

  __device__ __forceinline__ void clear_all() {
#pragma unroll
    for (int i = 0; i < NW; ++i) w[i] = 0u;
  }
  // first set rank, -1 if none
  __device__ __forceinline__ int first() const {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      uint64_t m = ballot(w[i] != 0u);
      if (m) {
        int L = __builtin_ctzll(m);
        uint32_t x = (uint32_t)readlane((int)w[i], L);
        return ((i * WAVE + L) << 5) + __builtin_ctz(x);
      }
    }
    return -1;
  }
  __device__ __forceinline__ void reset(int r, int lane) {
    int L = (r >> 5) & (WAVE - 1), wi = r >> 11;
    uint32_t b = 1u << (r & 31);
#pragma unroll
    for (int i = 0; i < NW; ++i)
      if (i == wi && lane == L) w[i] &= ~b;
  }
  // clear every rank <= r
  __device__ __forceinline__ void clear_upto(int r, int lane) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      int base = (i * WAVE + lane) << 5;
      if (base + 31 <= r) w[i] = 0u;
      else if (base <= r) w[i] &= ~((2u << (r - base)) - 1u);
    }
  }
  __device__ __forceinline__ int count() const {
    int c = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) c += __builtin_popcount(w[i]);
    return wave_sum(c);
  }
};

// Wave-uniform scalars of one instance.
struct SimState {
  int t, ndone, nact, min_s, max_s, min_end;
  int64_t res, sum_s, sum_comp;
  // prefill variant: largest prompt - start and summed prompt of the active jobs
  // (the largest footprint at step t is t + G + 1)
  int G;
  int64_t sp;
};

// ROB: Robust-ISJL (Section 3.4): ordering, packs, caps and the KV reservation
// use prompt + the predicted upper bound of the output; each job still runs its
// true length, and fairness is checked on true progress.
// PRE: the prompt is prefilled at admission (Section 1 with eq. (1)'s decode
// progress): a job runs one step per output token, reserves prompt + output and
// its footprint in the batch cost is prompt + progress; fairness stays on
// progress.  The sweeps are off (completions are taken one event at a time).
// FILL: with the fill sweep (below), for up to 2 slots per lane.
// QH: ISJL with up to 8 slots per lane whose plan-queue links are in HBM
// scratch (else in LDS).  Every kernel with up to 8 slots per lane but FCFS's
// is held to 128 VGPRs, so that 4 waves share a SIMD where the LDS allows 16
// per CU (FCFS's 4- and 8-slot kernels ran slower that way and keep 3).
template <int POL, int K, int NW, bool GEN, bool ROB, bool PRE, bool FILL, bool QH = false,
          bool FAIR = false>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(FILL || K <= 2 || (K <= 8 && POL != POL_FCFS) ? 4 : (K <= 8 ? 3 : 1)))) void simulate_kernel(SimArgs a) {
  static_assert(!ROB || POL == POL_ISJL, "predicted sizes: ISJL only");
  static_assert(!FILL || (K <= 2 && !ROB && !PRE && POL != POL_LJF), "fill sweep variants");
  extern __shared__ uint32_t lds_raw[];
  // With 4 or 8 slots per lane (but FCFS) the wave's index in its block is
  // taken into a scalar register: every row pointer derived from the instance
  // is then scalar, which is what brings those kernels under 128 VGPRs (the
  // narrower kernels ran slower with it, their scalar registers being the
  // scarcer ones).
  constexpr bool WIB_S = (K == 4 || K == 8) && POL != POL_FCFS;
  const int wib = WIB_S ? __builtin_amdgcn_readfirstlane(threadIdx.x >> 6)
                        : (int)(threadIdx.x >> 6);
  const int64_t inst = (int64_t)blockIdx.x * (blockDim.x >> 6) + wib;
  if (inst >= a.n_inst) return;
  const int lane = lane_id();
  const int n = a.n;
  uint32_t* W = lds_raw + (size_t)wib * (size_t)a.wave_words;
  int32_t* ARR = (int32_t*)(W + a.off_arr);
  uint16_t* QN = (uint16_t*)(W + a.off_q);
  // ISJL with up to 8 slots per lane: the plan-queue links live in HBM scratch
  // when that lets more waves share a CU (agent-scope accesses, so one lane's
  // link is seen by the others), else in LDS; the launch picks the kernel for
  // the place (a branch on it at every link would cost the event loop more)
  constexpr bool QGLOBAL = POL == POL_ISJL && K <= 8 && QH;
  uint32_t* QG = QGLOBAL ? a.qlink + inst * (int64_t)a.q_stride : nullptr;
  auto qn_set = [&](int r, uint32_t v) {
    if constexpr (QGLOBAL) __hip_atomic_store(QG + r, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else QN[r] = (uint16_t)v;
  };
  auto qn_get = [&](int r) -> uint32_t {
    if constexpr (QGLOBAL) return __hip_atomic_load(QG + r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else return QN[r];
  };
  uint16_t* STG = (uint16_t*)(W + a.off_stage);
  // Released ranks on their way into the bitmap (not FCFS); shares the gather
  // buffer, which is dead while releases are processed.
  uint32_t* PEND = W + a.off_stage;
  const int64_t row = inst * (int64_t)n;
  const int32_t* A = a.arrival + row;
  const int32_t* P = a.prompt + row;
  const int32_t* O = a.output + row;
  const int32_t* U = ROB ? a.upper + row : nullptr;  // predicted upper bounds of the outputs
  // true service length of job j (ROB: the length that plans used was larger)
  auto true_len = [&](int j, int plan) -> int {
    return ROB ? (PRE ? O[j] : P[j] + O[j]) : plan;
  };
  // KV reservation of job j planned with size `plan`
  auto resv_len = [&](int j, int plan) -> int { return PRE ? P[j] + plan : plan; };

  if (GEN) {  // only instances the sorted-arrival kernel deferred
    const int64_t prev = a.out_T ? a.out_T[inst] : a.out[inst].T;
    if (prev != T_DEFERRED) return;
  }

  // ---- load, validate, instance constants --------------------------------
  // One pass over the job table: validation, instance totals and the
  // priority keys (LJF / ISJL: (-len, index); SJF: (len, index); FCFS:
  // (arrival, index), or (len, index) in arrival order when arrivals are
  // sorted); padding keys sort last.
  const int NP = a.NP;
  int bad = 0, big = 0, unsorted = 0, maxlen = 0, maxfoot = 0, maxarr = 0;
  int64_t osum = 0, qsum = 0, rsum = 0;
  uint64_t q2 = 0;  // twice the footprint sum Q: one 32 x 32 -> 64 product per job
  int carry_ar = 0;
  // The rows are software-pipelined: the loads of row r + PF are issued
  // while row r is processed, so PF rows of loads are in flight (clamped
  // indices keep every load in bounds; the rows past NP are never used).
  constexpr int PF = 4;
  int pf_a[PF], pf_p[PF], pf_o[PF], pf_u[PF];
#pragma unroll
  for (int d = 0; d < PF; ++d) {
    const int ic = min(d * WAVE + lane, n - 1);
    pf_a[d] = A[ic];
    pf_p[d] = P[ic];
    pf_o[d] = O[ic];
    pf_u[d] = ROB ? U[ic] : 0;
  }
  for (int r0 = 0; r0 < NP; r0 += PF * WAVE) {
#pragma unroll
  for (int d = 0; d < PF; ++d) {
    const int i0 = r0 + d * WAVE;
    if (i0 >= NP) break;
    const int i = i0 + lane;
    const bool in = i < n;
    const int ar0 = pf_a[d], p0 = pf_p[d], o0 = pf_o[d], u0 = ROB ? pf_u[d] : o0;
    {
      const int ic = min(i + PF * WAVE, n - 1);
      pf_a[d] = A[ic];
      pf_p[d] = P[ic];
      pf_o[d] = O[ic];
      if (ROB) pf_u[d] = U[ic];
    }
    const int ar = in ? ar0 : 0x7FFFFFFF, p = in ? p0 : 0, o = in ? o0 : 1;
    const int u = in ? u0 : o;
    int prev = __shfl_up(ar, 1);
    if (lane == 0) prev = i0 > 0 ? carry_ar : ar;
    carry_ar = readlane(ar, WAVE - 1);
    uint32_t key = 0xFFFFFFFFu;
    if (in) {
      bad |= (ar < 0) | (p < 0) | (o < 1) | (u < o);
      // service length, planning size and largest footprint
      const int64_t len = PRE ? (int64_t)o : (int64_t)p + (int64_t)o;
      const int64_t plan_len = PRE ? (int64_t)u : (int64_t)p + (int64_t)u;
      const int64_t foot = (int64_t)p + (int64_t)u;
      big |= (foot >= LEN_LIMIT);
      unsorted |= (prev > ar);
      if (foot < LEN_LIMIT && len > maxlen) maxlen = (int)len;
      if (foot < LEN_LIMIT && foot > maxfoot) maxfoot = (int)foot;
      if (ar > maxarr) maxarr = ar;
      osum += (int64_t)p + (int64_t)o;  // tokens served
      // Q: the footprint summed over the job's own steps (Section 5), doubled:
      // len (len + 1), or o (2 p + o + 1) with the prompt prefilled; both
      // factors are below 2^22 in every instance that is simulated (a larger
      // footprint returns the too-large marker before Q is used)
      q2 += PRE ? (uint64_t)(uint32_t)o * (uint32_t)(2 * p + o + 1)
                : (uint64_t)(uint32_t)len * (uint32_t)(len + 1);
      rsum += ar;
      const uint32_t l32 = (uint32_t)(ROB ? plan_len : len) & LMASK;
      if (POL == POL_LJF || POL == POL_ISJL) key = ((LMASK - l32) << 12) | (uint32_t)i;
      else if (POL == POL_SJF) key = (l32 << 12) | (uint32_t)i;
      else if (GEN) key = (((uint32_t)ar & LMASK) << 12) | (uint32_t)i;
      else key = (l32 << 12) | (uint32_t)i;
    }
    W[i] = key;
  }
  }
  bad = ballot(bad != 0) != 0;
  big = ballot(big != 0) != 0;
  unsorted = ballot(unsorted != 0) != 0;
  if (bad) {
    write_marker(a.out, a.out_T, inst, FSCHED_T_INVALID, lane);
    return;
  }
  if (big) {
    write_marker(a.out, a.out_T, inst, FSCHED_T_TOOLARGE, lane);
    return;
  }
  if (!GEN && unsorted) {
    write_marker(a.out, a.out_T, inst, T_DEFERRED, lane);
    return;
  }
  maxlen = wave_max(maxlen);
  maxfoot = wave_max(maxfoot);
  maxarr = wave_max(maxarr);
  osum = wave_sum64(osum);
  qsum = (int64_t)((uint64_t)wave_sum64((int64_t)q2) >> 1);  // every term is even
  rsum = wave_sum64(rsum);
  if (GEN && maxarr >= ARR_LIMIT) {
    write_marker(a.out, a.out_T, inst, FSCHED_T_TOOLARGE, lane);
    return;
  }
  {
    // Largest makespan any policy here can reach: all work serialised after the
    // last release, plus one delayed plan start (<= alpha) per job.
    double amin = a.alpha < maxlen ? (double)a.alpha : (double)maxlen;
    double tb = (double)maxarr + (double)osum + (double)n * amin + 1.0;
    if (tb >= 2147483000.0) {
      write_marker(a.out, a.out_T, inst, FSCHED_T_TOOLARGE, lane);
      return;
    }
    double cb = (double)a.c * tb + (double)a.tau * (double)osum * (double)maxfoot;
    double wb = (double)a.c * tb + (double)a.tau * tb * (double)maxfoot;
    if (cb > 4.0e18 || wb > 4.0e18) {
      write_marker(a.out, a.out_T, inst, FSCHED_T_RANGE, lane);
      return;
    }
  }

  // ---- priority order -----------------------------------------------------
  if (!(POL == POL_FCFS && !GEN)) {
    wave_lds_sync();
    switch (NP) {
      case 64: wave_reg_sort<1, true>(W, lane); break;
      case 128: wave_reg_sort<2, true>(W, lane); break;
      case 256: wave_reg_sort<4, true>(W, lane); break;
      case 512: wave_reg_sort<8, true>(W, lane); break;
      case 1024: wave_reg_sort<16, true>(W, lane); break;
      case 2048: wave_reg_sort<32, true>(W, lane); break;
      default: wave_bitonic_sort(W, NP, lane); break;
    }
    wave_lds_sync();
    // sorted-arrival kernel: each job's rank goes to the rank table for the
    // release chunks (only this wave touches its row)
    uint16_t* RKw = (!GEN && POL != POL_FCFS) ? a.rank + inst * (int64_t)a.rank_stride : nullptr;
    for (int r = lane; r < n; r += WAVE) {
      uint32_t key = W[r];
      int id = (int)(key & 0xFFFu);
      uint32_t len;
      if (POL == POL_LJF || POL == POL_ISJL) len = LMASK - (key >> 12);
      else if (POL == POL_SJF) len = key >> 12;
      else len = (uint32_t)(PRE ? O[id] : P[id] + O[id]);
      W[r] = (len << 12) | (uint32_t)id;
      if (GEN) ARR[r] = A[id];
      else if (RKw) RKw[id] = (uint16_t)r;
    }
    if (RKw) __threadfence_block();  // the stores complete before the row is read
  }
  wave_lds_sync();

  // ---- state ---------------------------------------------------------------
  const int Beff = a.Beff;
  const int alpha = a.alpha;
  const int64_t M = a.M;
  int ws_start[K], ws_end[K];
  int ws_plan[K];  // ROB: KV reservation of the running job (from its planning size)
  int ws_p[K];     // PRE: prompt of the running job (its footprint offset)
  uint32_t ws_q[K];
  uint32_t ws_qn[K];  // links in HBM: the link of the queue's head, loaded ahead
  bool valid[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    ws_plan[k] = 0;
    ws_p[k] = 0;
    ws_start[k] = IDLE;
    ws_end[k] = IDLE;
    ws_q[k] = QNONE | (QNONE << 16);
    ws_qn[k] = QNONE;
    valid[k] = (k * WAVE + lane) < Beff;
  }
  PoolBits<NW> pool;
  pool.clear_all();
  PoolBits<NW> unrel;  // general variant, non-FCFS: ranks not yet released
  unrel.clear_all();
  if (GEN && POL != POL_FCFS) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      int base = (i * WAVE + lane) << 5;
      uint32_t m = 0u;
      if (base + 32 <= n) m = 0xFFFFFFFFu;
      else if (base < n) m = (1u << (n - base)) - 1u;
      unrel.w[i] = m;
    }
  }
  int relk = 0;           // release cursor
  int qcount = 0;         // queued jobs: released, not admitted, not planned
  int chunk = -1;         // release chunk loaded in rel_t / rel_r
  int rel_t = IDLE, rel_r = 0;
  int next_rel = 0;       // general variant, non-FCFS
  int head = 0;           // FCFS: first waiting rank
  // ISJL
  int mode = 0;           // 0 FILL, 1 DRAIN
  int planned = 0;        // planned jobs not yet started
  int t_w1 = 0;           // earliest start of worker 0's planned job

  SimState S;
  S.t = 0;
  S.ndone = 0;
  S.nact = 0;
  S.min_s = IDLE;
  S.max_s = -1;
  S.min_end = IDLE;
  S.res = 0;
  S.sum_s = 0;
  S.sum_comp = 0;
  S.G = -IDLE;
  S.sp = 0;
  // C = c T + tau sum_t |S_t| m_t and W = c T + tau sum_t m_t (m_t: the largest
  // footprint at step t, 0 when idle): c and tau are applied once at the end
  // (every step 0 .. T-1 is accounted exactly once)
  int64_t acc_E = 0, acc_SM = 0, acc_SSM = 0, acc_ext = 0, acc_busy = 0, acc_peak = 0,
          acc_unfair = 0;
  int acc_maxext = 0, acc_maxact = 0;
  // With up to 2 slots per lane the sweeps' per-lane partial sums (and the
  // largest footprint) of their span terms carry over from sweep to sweep and
  // are summed over the wave once after the event loop: integer sums, so the
  // deferral changes no result, and a sweep ends without a reduction.  The
  // wider kernels have no registers to spare for them and reduce per sweep.
  constexpr bool DEFER = K <= 2;
  int64_t pE = 0, pSM = 0, pSSM = 0, pX = 0, pP = 0;
  int pU = 0;
  int32_t* st_out = a.start ? a.start + row : nullptr;
  int32_t* fi_out = a.finish ? a.finish + row : nullptr;
  const int iter_max = 8 * n + 64;
  int iter = 0;
  bool failed = false;

  // rank of each job in the priority order (sorted-arrival kernel, not FCFS)
  const uint16_t* RK =
      (!GEN && POL != POL_FCFS) ? a.rank + inst * (int64_t)a.rank_stride : nullptr;
  // Load release chunk `c` (64 consecutive jobs in arrival order; the general
  // variant releases through ARR and loads chunks only under FCFS).
  auto load_chunk = [&](int c) {
    int j = c * WAVE + lane;
    rel_t = IDLE;
    rel_r = 0;
    if (POL == POL_FCFS) {
      if (j < n) rel_t = GEN ? ARR[j] : A[j];
      rel_r = j;
    } else if (j < n) {
      rel_t = A[j];
      rel_r = RK[j];
    }
    chunk = c;
  };

  // Schedule output of one admitted job.
  auto emit = [&](int id, int t, int len) {
    if (st_out) st_out[id] = t;
    if (fi_out) fi_out[id] = t + len;
  };

  // Whether the first queued job (in priority order) cannot join the running
  // ones under the KV budget: then a strict-prefix admission admits nothing,
  // and the gather is skipped.  Checked with up to 4 slots per lane (B <= 256),
  // where a blocked head is common and the gather is a large share of an event;
  // the 8- and 16-slot kernels (at their register limit) gather regardless.
  auto head_blocked = [&]() -> bool {
    if (K > 4 || M == 0 || S.nact == 0) return false;
    const int r = pool.first();
    if (r < 0) return false;
    const uint32_t wv = W[r];
    return S.res + resv_len(pid(wv), plen(wv)) > M;
  };

  // The first G queued ranks, in priority order, into STG[0..G).  Each lane
  // writes its own word's ranks in turn; with up to 4 slots per lane, one bitmap
  // word per lane and more than 8 ranks, lane L instead finds the rank at
  // position c + L directly: the lane holding it by a binary search over the
  // lanes' inclusive counts, then the right set bit of that lane's word.
  auto gather_first = [&](int G) {
    if constexpr (K <= 4 && NW == 1) {
      if (G > 8) {
        const uint32_t x = pool.w[0];
        const int cnt = __builtin_popcount(x);
        const int incl = wave_scan_incl(cnt);
        for (int c0 = 0; c0 < G; c0 += WAVE) {
          const int P = c0 + lane;
          int lo = 0;  // number of lanes whose count ends at or before P
#pragma unroll
          for (int step = WAVE / 2; step >= 1; step >>= 1) {
            const int v = __shfl(incl, lo + step - 1);
            if (v <= P) lo += step;
          }
          const int owner = lo < WAVE ? lo : WAVE - 1;
          uint32_t w = (uint32_t)__shfl((int)x, owner);
          int k = P - (__shfl(incl, owner) - __builtin_popcount(w));
          // the k-th set bit of w (k < popcount(w) for every P < G)
          int bit = 0;
#pragma unroll
          for (int half = 16; half >= 1; half >>= 1) {
            const int c = __builtin_popcount(w & ((1u << half) - 1u));
            if (k >= c) {
              k -= c;
              bit += half;
              w >>= half;
            }
          }
          if (P < G) STG[P] = (uint16_t)((owner << 5) + bit);
        }
        wave_lds_sync();
        return;
      }
    }
    int gbase = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int cnt = __builtin_popcount(pool.w[i]);
      const int incl = wave_scan_incl(cnt);
      int pos = gbase + incl - cnt;
      uint32_t x = pool.w[i];
      const int base = (i * WAVE + lane) << 5;
      while ((x != 0u) & (pos < G)) {
        const int b = __builtin_ctz(x);
        x &= x - 1u;
        STG[pos] = (uint16_t)(base + b);
        pos++;
      }
      gbase += readlane(incl, 63);
    }
    wave_lds_sync();
  };

  // Admit at step t the longest prefix of STG[0..G) that fits the KV budget
  // (strict order; a job that would run alone always fits), onto the first
  // eligible idle workers in index order (ISJL Phase TWO also needs an empty
  // plan queue).  Returns the number admitted.
  auto admit_prefix = [&](int t, int G, bool need_empty_queue, int& adm, int64_t& adm_len,
                          int& adm_minlen) -> int {
    int na = G;
    int64_t tot64 = -1;  // summed length of the admitted jobs, when the KV scan found it
    if (M != 0) {
      int64_t run = S.res;
      for (int c0 = 0; c0 < G; c0 += WAVE) {
        const int j = c0 + lane;
        int len = 0;
        if (j < G) {
          const uint32_t wv = W[STG[j]];
          len = resv_len(pid(wv), plen(wv));
        }
        const int pre = wave_scan_incl(len);
        const bool fail = (j < G) & ((j > 0) | (S.nact > 0)) & (run + pre > M);
        const uint64_t fm = ballot(fail);
        if (fm) {
          const int f = __builtin_ctzll(fm);
          na = c0 + f;
          if (f > 0) run += readlane(pre, f - 1);
          break;
        }
        run += readlane(pre, 63);
      }
      tot64 = run - S.res;
    }
    // the count in a scalar register, so the walk over the slot registers
    // below branches on it rather than masking lanes (measured on the kernels
    // with more than 2 slots per lane; the narrower ones ran no faster)
    if constexpr (K > 2) na = uni(na);
    if (na == 0) return 0;
    int base = 0, lsum = 0, lplan = 0, lmin = IDLE, lp = 0, lpmax = -IDLE;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      if (base < na) {
        const bool el = valid[k] & (ws_end[k] == IDLE) &
                        (!need_empty_queue | ((ws_q[k] & 0xFFFFu) == QNONE));
        const uint64_t bm = ballot(el);
        const int idx = base + mbcnt(bm);
        if (el & (idx < na)) {
          const uint32_t wv = W[STG[idx]];
          const int plan = plen(wv);
          const int len = true_len(pid(wv), plan);
          ws_start[k] = t;
          ws_end[k] = t + len;
          emit(pid(wv), t, len);
          lsum += len;
          if (ROB || PRE) {
            const int rv = resv_len(pid(wv), plan);
            ws_plan[k] = rv;
            lplan += rv;
            lmin = min(lmin, len);
          }
          if (PRE) {
            const int pp = P[pid(wv)];
            ws_p[k] = pp;
            lp += pp;
            lpmax = max(lpmax, pp);
          }
        }
        base += __builtin_popcountll(bm);
      }
    }
    int tot, ptot;  // true lengths and reservations admitted
    if (ROB || PRE) {
      tot = wave_sum(lsum);
      ptot = tot64 >= 0 ? (int)tot64 : wave_sum(lplan);
      adm_minlen = min(adm_minlen, wave_min(lmin));
    } else {
      tot = ptot = tot64 >= 0 ? (int)tot64 : wave_sum(lsum);
      // the gathered jobs are in priority order, so the shortest admitted one
      // is the last (longest first) or the first (SJF)
      adm_minlen = min(adm_minlen, plen(W[STG[POL == POL_SJF ? 0 : na - 1]]));
    }
    if (PRE) {
      S.sp += wave_sum(lp);
      S.G = max(S.G, wave_max(lpmax) - t);  // na >= 1 jobs were admitted
    }
    pool.clear_upto(STG[na - 1], lane);  // the first na queued ranks
    qcount -= na;
    adm += na;
    adm_len += tot;
    S.res += ptot;
    S.nact += na;
    return na;
  };

  // Gather and admit the strict prefix of the first G queued jobs.  With up to 4
  // slots per lane and a binding KV budget, the first 8 are gathered and scanned
  // alone and the rest only if all 8 fit: admitting those 8 and then the prefix
  // of the next G - 8 is the same strict prefix, and a budget that stops early
  // spares the gather of all G.
  auto admit_first = [&](int t, int G, bool need_empty_queue, int& adm, int64_t& adm_len,
                         int& adm_minlen) -> int {
    constexpr int G0 = 8;
    if (K <= 4 && M != 0 && S.nact > 0 && G > G0) {
      gather_first(G0);
      const int na = admit_prefix(t, G0, need_empty_queue, adm, adm_len, adm_minlen);
      if (na < G0) return na;
      gather_first(G - G0);
      return G0 + admit_prefix(t, G - G0, need_empty_queue, adm, adm_len, adm_minlen);
    }
    gather_first(G);
    return admit_prefix(t, G, need_empty_queue, adm, adm_len, adm_minlen);
  };

  // FAIR: launched when every wave of the grid is resident at once, so that the
  // launch lasts as long as its slowest wave.  A SIMD's arbiter issues for its
  // oldest wave first, which leaves the youngest to finish alone, one
  // dependent instruction at a time; turning each wave's priority with its
  // event count shares the issue slots among the SIMD's waves instead.
  int fair_turn = FAIR ? __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)) : 0;
  while (true) {
    const int t = S.t;
    if constexpr (FAIR) {
      switch (fair_turn++ & 3) {
        case 0: __builtin_amdgcn_s_setprio(0); break;
        case 1: __builtin_amdgcn_s_setprio(1); break;
        case 2: __builtin_amdgcn_s_setprio(2); break;
        default: __builtin_amdgcn_s_setprio(3); break;
      }
    }
    // (1) retire the jobs whose last token was processed at t-1
    if (S.min_end == t) {
      // the earliest / latest start is searched again only if a job holding
      // it retires
      int nret = 0, lsum = 0, lplan = 0, lp = 0, me = IDLE;
      bool hmin = false, hmax = false, hG = false;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const bool r = ws_end[k] == t;
        nret += __builtin_popcountll(ballot(r));
        if (r) {
          lsum += ws_end[k] - ws_start[k];
          if (ROB || PRE) lplan += ws_plan[k];
          if (PRE) {
            lp += ws_p[k];
            hG |= ws_p[k] - ws_start[k] == S.G;
          }
          hmin |= ws_start[k] == S.min_s;
          hmax |= ws_start[k] == S.max_s;
          ws_end[k] = IDLE;
          ws_start[k] = IDLE;
        }
        me = min(me, ws_end[k]);
      }
      int lret = wave_sum(lsum);
      S.min_end = wave_min(me);
      if (ballot(hmin)) {
        int mn = IDLE;
#pragma unroll
        for (int k = 0; k < K; ++k) mn = min(mn, ws_start[k]);
        S.min_s = wave_min(mn);
      }
      if (ballot(hmax)) {
        int mx = -1;
#pragma unroll
        for (int k = 0; k < K; ++k)
          if (ws_start[k] != IDLE) mx = max(mx, ws_start[k]);
        S.max_s = wave_max(mx);
      }
      if (PRE) {
        S.sp -= wave_sum(lp);
        if (ballot(hG)) {
          int g = -IDLE;
#pragma unroll
          for (int k = 0; k < K; ++k)
            if (ws_end[k] != IDLE) g = max(g, ws_p[k] - ws_start[k]);
          S.G = wave_max(g);
        }
      }
      S.ndone += nret;
      S.nact -= nret;
      S.res -= (ROB || PRE) ? wave_sum(lplan) : lret;
      S.sum_s -= (int64_t)nret * t - (int64_t)lret;
    }
    if (S.ndone == n) break;

    // (2) releases.  Arrivals are non-decreasing in job order here, so the
    // jobs released by t are the next lanes of the loaded chunk up to the
    // first later arrival; their pool bits are scattered with LDS atomics and
    // folded into the register bitmap once.
    if (POL == POL_FCFS || !GEN) {
      bool any = false;
      while (relk < n) {
        if ((relk >> 6) != chunk) load_chunk(relk >> 6);
        const int off = relk & (WAVE - 1);
        const uint64_t late = ballot((lane >= off) & (rel_t > t));
        const int hi = late ? __builtin_ctzll(late) : WAVE;
        if (POL != POL_FCFS && hi > off) {
          if (!any) {
#pragma unroll
            for (int i = 0; i < NW; ++i) PEND[i * WAVE + lane] = 0u;
            wave_lds_sync();
            any = true;
          }
          if ((lane >= off) & (lane < hi)) atomicOr(&PEND[rel_r >> 5], 1u << (rel_r & 31));
          qcount += hi - off;
        }
        relk += hi - off;
        if (hi < WAVE) break;
      }
      if (POL != POL_FCFS && any) {
        wave_lds_sync();
#pragma unroll
        for (int i = 0; i < NW; ++i) pool.w[i] |= PEND[i * WAVE + lane];
        wave_lds_sync();
      }
    } else if (next_rel <= t) {
      int nr = IDLE, ng = 0;
#pragma unroll
      for (int i = 0; i < NW; ++i) {
        uint32_t u = unrel.w[i], got = 0u;
        int base = (i * WAVE + lane) << 5;
        while (u) {
          int b = __builtin_ctz(u);
          u &= u - 1u;
          int ar = ARR[base + b];
          if (ar <= t) got |= 1u << b;
          else nr = min(nr, ar);
        }
        unrel.w[i] &= ~got;
        pool.w[i] |= got;
        ng += __builtin_popcount(got);
      }
      qcount += wave_sum(ng);
      next_rel = wave_min(nr);
    }

    // (3) A_max(t): largest progress among the jobs still active
    const int amax = S.nact > 0 ? t - S.min_s : 0;
    const int nact0 = S.nact;
    int adm = 0, adm_minlen = IDLE;
    int64_t adm_len = 0;
    bool kv_block = false;
    int free_empty = 0;  // ISJL: idle workers with nothing planned, after this step's admissions

    // (4) admissions
    if (POL == POL_FCFS) {
      int cnt = min(relk - head, Beff - S.nact);
      int done = 0;
      while (done < cnt) {
        int c = min(WAVE, cnt - done);
        int r = head + done + lane;
        uint32_t wv = lane < c ? W[r] : 0u;
        int len = plen(wv), id = pid(wv);
        const int pp = (PRE && lane < c) ? P[id] : 0;  // prompt (prefill variant)
        int pre = wave_scan_incl(len + pp);            // reservations
        bool fit = (M == 0) | ((int64_t)(S.res + pre) <= M) |
                   ((S.nact == 0) & (done == 0) & (lane == 0));
        uint64_t fm = ballot((lane < c) & !fit);
        int take = fm ? __builtin_ctzll(fm) : c;
        if (take > 0) {
          int base = 0;
#pragma unroll
          for (int k = 0; k < K; ++k) {
            if (base < take) {
              bool idle = valid[k] & (ws_end[k] == IDLE);
              uint64_t bm = ballot(idle);
              int idx = base + mbcnt(bm);
              int src = min(idx, WAVE - 1);
              int l2 = __shfl(len, src), id2 = __shfl(id, src);
              const int p2 = PRE ? __shfl(pp, src) : 0;
              if (idle & (idx < take)) {
                ws_start[k] = t;
                ws_end[k] = t + l2;
                if (PRE) {
                  ws_p[k] = p2;
                  ws_plan[k] = p2 + l2;
                }
                emit(id2, t, l2);
              }
              base += __builtin_popcountll(bm);
            }
          }
          int tl = readlane(pre, take - 1);  // reservations admitted
          adm_minlen = min(adm_minlen, wave_min(lane < take ? len : IDLE));
          adm += take;
          if (PRE) {
            const int lp = wave_sum(lane < take ? pp : 0);
            adm_len += tl - lp;
            S.sp += lp;
            S.G = max(S.G, wave_max(lane < take ? pp : -IDLE) - t);
          } else {
            adm_len += tl;
          }
          S.res += tl;
          S.nact += take;
        }
        done += take;
        if (take < c) break;
      }
      head += done;
    } else if (POL == POL_LJF || POL == POL_SJF) {
      if (POL == POL_SJF || S.nact == 0) {
        const int freew = Beff - S.nact;
        if (freew > 0) {
          const int kp = qcount;
          const int G = min(freew, kp);
          if (G > 0 && !head_blocked()) admit_first(t, G, false, adm, adm_len, adm_minlen);
        }
      }
    } else {  // ISJL
      // Epoch: empty machine, nothing planned, jobs queued -> Phase ONE.
      if (S.nact == 0 && planned == 0) {
        int kp = qcount;
        if (kp > 0) {
          mode = 0;
          int G = min(Beff, kp);
          gather_first(G);  // longest first
          // lengths of the gathered jobs: job j in chunk j / 64, lane j % 64
          // (worker w's long job is gathered job w, in the same place)
          int glen[K];
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const int j = k * WAVE + lane;
            glen[k] = j < G ? plen(W[STG[j]]) : 0;
          }
          // Bp: largest prefix of the longest jobs that fits the KV budget
          int Bp = G;
          if (M != 0) {
            int64_t run = 0;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              if (k * WAVE < G && Bp == G) {
                const int j = k * WAVE + lane;
                // reservation of gathered job j (prefill variant: + prompt)
                const int rv = (PRE && j < G) ? glen[k] + P[pid(W[STG[j]])] : glen[k];
                const int pre = wave_scan_incl(rv);
                const uint64_t fm = ballot((j < G) & (j >= 1) & (run + pre > M));
                if (fm) Bp = k * WAVE + __builtin_ctzll(fm);
                else run += readlane(pre, 63);
              }
            }
            if (Bp < 1) Bp = 1;
          }
          const int o1 = readlane(glen[0], 0);
          const int o2 = kp > 1 ? readlane(glen[0], 1) : 0;
          if (kp > 1 && Bp > 1 && o2 > alpha) {
            // m = min{Bp, #{len > alpha}}: the lengths are non-increasing, so it
            // is the first gathered job with len <= alpha, capped at Bp
            int m = Bp;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              if (k * WAVE < Bp && m == Bp) {
                const int j = k * WAVE + lane;
                const uint64_t fm = ballot((j < Bp) & (glen[k] <= alpha));
                if (fm) m = min(Bp, k * WAVE + __builtin_ctzll(fm));
              }
            }
            if constexpr (K <= 4) m = uni(m);  // scalar (measured: the 8-slot kernel ran slower)
            const int beta = a.beta;
            int cap[K], load[K];
#pragma unroll
            for (int k = 0; k < K; ++k) {
              int w = k * WAVE + lane;
              load[k] = 0;
              if ((w >= 1) & (w < m)) {
                cap[k] = min(2 * alpha, o1 - glen[k] + beta);
              } else if ((w >= m) & (w < Bp)) {
                cap[k] = alpha;
              } else {
                cap[k] = -1;
              }
            }
            // the m long jobs are the first m queued ranks
            const int rlast = STG[m - 1];
            pool.clear_upto(rlast, lane);
            qcount -= m;
            planned += m;
            // Pack scan (Algorithm 3): remaining queued jobs in decreasing length;
            // each goes to the first spare worker with room, else to the long
            // worker of largest index with room; a job that fits nowhere stays.
            const bool has_spare = uni(Bp) > m;
            // Each worker choice below is one ballot per slot register, built
            // from plain comparisons (no short-circuit, which the compiler
            // turns into lane-masked branches and leaves the worker index in a
            // vector register).  With up to 4 slots per lane the spare and long
            // workers' lane masks are kept; the wider kernels, short of scalar
            // registers, test the ranges in the ballot itself.
            uint64_t spare_m[K], long_m[K];
            if constexpr (K <= 4) {
#pragma unroll
              for (int k = 0; k < K; ++k) {
                const int w = k * WAVE + lane;
                spare_m[k] = ballot((w >= m) & (w < Bp));
                long_m[k] = ballot((w >= 1) & (w < m));
              }
            }
            // the ranks still to visit: the queued ranks after rlast (pool was
            // cleared up to it), each cleared once visited
            PoolBits<NW> scan = pool;
            while (true) {
              const int r = scan.first();
              if (r < 0) break;
              scan.reset(r, lane);
              const int len = plen(W[r]);
              int wsel = -1;
              if (has_spare) {  // spare workers, ascending
#pragma unroll
                for (int k = 0; k < K; ++k) {
                  const int w = k * WAVE + lane;
                  const uint64_t ms = K <= 4 ? ballot(cap[k] - load[k] >= len) & spare_m[k]
                                             : ballot((w >= m) & (w < Bp) & (cap[k] - load[k] >= len));
                  if (ms) {
                    wsel = k * WAVE + __builtin_ctzll(ms);
                    break;
                  }
                }
              }
              if (wsel < 0) {  // long workers, largest index first
#pragma unroll
                for (int k = K - 1; k >= 0; --k) {
                  const int w = k * WAVE + lane;
                  const uint64_t ml = K <= 4 ? ballot(cap[k] - load[k] >= len) & long_m[k]
                                             : ballot((w >= 1) & (w < m) & (cap[k] - load[k] >= len));
                  if (ml) {
                    wsel = k * WAVE + 63 - __builtin_clzll(ml);
                    break;
                  }
                }
              }
              if (wsel < 0) {
                // r fits nowhere: skip to the first rank whose length fits the
                // largest room left (lengths are non-increasing in rank)
                int rm = -1;
#pragma unroll
                for (int k = 0; k < K; ++k) rm = max(rm, cap[k] - load[k]);
                const int remmax = wave_max(rm);
                if (remmax <= 0) break;
                const int span = n - r;
                const int sstep = (span + WAVE - 1) / WAVE;
                const int p = r + lane * sstep;
                const uint64_t fm = ballot(p < n && plen(W[p]) <= remmax);
                int lo, hi;
                if (fm) {
                  const int L1 = __builtin_ctzll(fm);
                  hi = r + L1 * sstep;
                  lo = L1 > 0 ? r + (L1 - 1) * sstep + 1 : r;
                } else {
                  // after the last probe inside [r, n)
                  lo = r + ((span - 1) / sstep) * sstep + 1;
                  hi = n;
                }
                const int q = lo + lane;
                const uint64_t fm2 = ballot(q < hi && plen(W[q]) <= remmax);
                const int b = fm2 ? lo + __builtin_ctzll(fm2) : hi;
                if (b >= n) break;
                scan.clear_upto(b - 1, lane);
                continue;
              }
              // append r to worker wsel's queue
              wsel = uni(wsel);  // the same in every lane (kept in a scalar register)
              int qt = (int)QNONE;
#pragma unroll
              for (int k = 0; k < K; ++k)
                if (k == (wsel >> 6)) qt = readlane((int)(ws_q[k] >> 16), wsel & 63);
              if (lane == 0) {
                if (qt != (int)QNONE) qn_set(qt, (uint32_t)r);
                qn_set(r, QNONE);
              }
#pragma unroll
              for (int k = 0; k < K; ++k)
                if ((k == (wsel >> 6)) & (lane == (wsel & 63))) {
                  load[k] += len;
                  uint32_t h = ws_q[k] & 0xFFFFu;
                  if (h == QNONE) h = (uint32_t)r;
                  ws_q[k] = h | ((uint32_t)r << 16);
                }
              pool.reset(r, lane);
              --qcount;
              planned++;
            }
            wave_lds_sync();
            // worker j in 2..M: its pack, then o_j; worker 1: o_1
            int pmax = 0;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              int w = k * WAVE + lane;
              if ((w >= 1) & (w < Bp)) pmax = max(pmax, load[k]);
              if ((w >= 1) & (w < m)) {
                uint32_t r = STG[w];
                uint32_t h = ws_q[k] & 0xFFFFu, tl = ws_q[k] >> 16;
                if (tl != QNONE) qn_set((int)tl, r);
                else h = r;
                qn_set((int)r, QNONE);
                ws_q[k] = h | (r << 16);
              }
              if (w == 0) {
                uint32_t r = STG[0];
                qn_set((int)r, QNONE);
                ws_q[k] = r | (r << 16);
              }
            }
            wave_lds_sync();
            // HBM links: every store is done before a plan start reads them
            if constexpr (QGLOBAL) {
              __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
              // each head's link, loaded now for when it starts
#pragma unroll
              for (int k = 0; k < K; ++k) {
                const uint32_t h = ws_q[k] & 0xFFFFu;
                ws_qn[k] = h != QNONE ? qn_get((int)h) : QNONE;
              }
            }
            pmax = wave_max(pmax);
            int idle1 = pmax - alpha;
            if (idle1 < 0) idle1 = 0;
            if (idle1 > alpha) idle1 = alpha;
            t_w1 = t + idle1;
          }
        }
      }
      // Plan starts (workers in index order), each guarded by
      // A_max(t) <= alpha and the KV budget.
      if (planned > 0 && amax <= alpha) {
        bool cand[K];
        int clen[K];
        uint32_t cwv[K];
        int csum = 0, ccnt = 0;
#pragma unroll
        for (int k = 0; k < K; ++k) {
          int w = k * WAVE + lane;
          uint32_t h = ws_q[k] & 0xFFFFu;
          cand[k] = valid[k] & (ws_end[k] == IDLE) & (h != QNONE) & !((w == 0) & (t < t_w1));
          clen[k] = 0;  // reservation
          cwv[k] = 0u;
          if (cand[k]) {
            const uint32_t wv = W[h];
            cwv[k] = wv;
            clen[k] = resv_len(pid(wv), plen(wv));
          }
          csum += clen[k];
          ccnt += cand[k] ? 1 : 0;
        }
        int tot = wave_sum(csum);
        int ncand = wave_sum(ccnt);
        if (ncand > 0) {
          bool all = (M == 0) || (S.res + tot <= M) || (S.nact == 0 && ncand == 1);
          if (!all) {
            // Sequential KV check in worker order; a blocked worker waits and
            // later workers are still tried.
            int nk = 0;
            int64_t rres = S.res;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              uint64_t mk = ballot(cand[k]);
              uint64_t keep = 0;
              while (mk) {
                int L = __builtin_ctzll(mk);
                mk &= mk - 1;
                int len = readlane(clen[k], L);
                if (S.nact + nk == 0 || rres + len <= M) {
                  keep |= 1ull << L;
                  rres += len;
                  nk++;
                }
              }
              cand[k] = cand[k] && ((keep >> lane) & 1ull);
            }
            tot = (int)(rres - S.res);
            ncand = nk;
          }
          int mlen = IDLE, ltrue = 0, lp = 0, lpmax = -IDLE;
#pragma unroll
          for (int k = 0; k < K; ++k) {
            if (cand[k]) {
              uint32_t h = ws_q[k] & 0xFFFFu;
              const uint32_t wv = cwv[k];
              const int plan = plen(wv);
              const int len = true_len(pid(wv), plan);
              ws_start[k] = t;
              ws_end[k] = t + len;
              if (ROB || PRE) {
                ws_plan[k] = clen[k];
                ltrue += len;
              }
              if (PRE) {
                const int pp = P[pid(wv)];
                ws_p[k] = pp;
                lp += pp;
                lpmax = max(lpmax, pp);
              }
              mlen = min(mlen, len);
              emit(pid(wv), t, len);
              uint32_t nx;
              if constexpr (QGLOBAL) {  // loaded ahead; the new head's link is loaded now
                nx = ws_qn[k];
                ws_qn[k] = nx != QNONE ? qn_get((int)nx) : QNONE;
              } else {
                nx = qn_get((int)h);
              }
              ws_q[k] = (nx == QNONE) ? (QNONE | (QNONE << 16)) : (nx | (ws_q[k] & 0xFFFF0000u));
            }
          }
          adm_minlen = min(adm_minlen, wave_min(mlen));
          adm += ncand;
          adm_len += (ROB || PRE) ? wave_sum(ltrue) : tot;
          S.res += tot;
          if (PRE) {
            // the KV check may have dropped every candidate
            const int gm = wave_max(lpmax);
            if (gm != -IDLE) S.G = max(S.G, gm - t);
            S.sp += wave_sum(lp);
          }
          S.nact += ncand;
          planned -= ncand;
        }
      }
      // Phase TWO (FILL): idle workers with nothing planned take the longest
      // queued unplanned job while A_max(t) <= alpha; otherwise DRAIN (until
      // the machine is empty, or with the resume reading until A_max <= alpha).
      if (mode == 1 && a.resume && amax <= alpha) mode = 0;
      if (mode == 0) {
        // idle workers with an empty plan queue (all idle ones when nothing is planned)
        int nie = Beff - S.nact;
        if (planned > 0) {
          nie = 0;
#pragma unroll
          for (int k = 0; k < K; ++k)
            nie += __builtin_popcountll(
                ballot(valid[k] & (ws_end[k] == IDLE) & ((ws_q[k] & 0xFFFFu) == QNONE)));
        }
        free_empty = nie;
        if (nie > 0) {
          const int kp = qcount;
          if (kp > 0) {
            if (amax > alpha) {
              mode = 1;
            } else if (head_blocked()) {
              kv_block = true;
            } else {
              const int G = min(nie, kp);
              const int na = admit_first(t, G, true, adm, adm_len, adm_minlen);
              free_empty = nie - na;
              if (na < G) kv_block = true;
            }
          }
        }
      }
    }
    if (adm > 0) {
      S.sum_s += (int64_t)adm * t;
      S.sum_comp += (int64_t)adm * t + adm_len;
      S.min_end = min(S.min_end, t + adm_minlen);
      if (nact0 == 0) S.min_s = t;
      S.max_s = t;
    }

    // Fill sweep (up to 2 slots per lane; FCFS, SJF, and ISJL in FILL with
    // nothing planned; jobs queued).  Each coming completion admits the next
    // jobs of the queue's strict prefix that fit the freed slots and the KV
    // budget.  While no job admitted meanwhile completes, nothing is released
    // and (ISJL) A_max stays within alpha at each completion, the admissions
    // follow from counts: after the completions at the sorted positions <= p,
    // the first
    //   A(p) = min(G, free + p + 1, #{j : PQ_j <= M - res + RR_p})
    // queued jobs are in (PQ_j: summed reservations of the queued jobs 0..j in
    // priority order; RR_p: of the completed positions 0..p; A is
    // non-decreasing), and queued job j starts at the completion of the first
    // position with A(p) > j.  The spans are accounted in parallel as in the
    // drain sweep, with the admitted jobs added to the suffix sums, up to the
    // first completion, admitted job's completion, release or (ISJL, KV budget
    // blocking an idle worker) alpha crossing that the counts do not decide;
    // the event loop takes it from there.  The last group of completions is
    // always left to the event loop, so every counted event has a job of the
    // sorted set still active.
    if constexpr (FILL) {
      const int Qn = POL == POL_FCFS ? relk - head : qcount;
      if (S.nact >= 2 && Qn > 0 && (POL != POL_ISJL || (mode == 0 && planned == 0))) {
        int H = IDLE;  // next release
        if (POL == POL_FCFS || !GEN) {
          if (relk < n) {
            if ((relk >> 6) != chunk) load_chunk(relk >> 6);
            H = readlane(rel_t, relk & (WAVE - 1));
          }
        } else {
          H = next_rel;
        }
        // taken when a few completions come before the first queued job could
        // finish after being admitted at the first of them (ISJL: and before
        // A_max surely exceeds alpha: some job started by max_s stays active)
        const int r0 = POL == POL_FCFS ? head : pool.first();
        int64_t lim0 = min((int64_t)H, (int64_t)S.min_end + plen(W[r0]));
        if (POL == POL_ISJL) lim0 = min(lim0, (int64_t)S.max_s + alpha + 1);
        int ahead = 0;
#pragma unroll
        for (int k = 0; k < K; ++k)
          ahead += __builtin_popcountll(ballot((ws_end[k] != IDLE) & ((int64_t)ws_end[k] < lim0)));
        if (ahead >= 4) {
          const int N = S.nact;
          const int Gq = min(Qn, Beff);
          constexpr int NS = K * WAVE;
          // queued job j (register j / 64, lane j % 64) and sorted position q
          // (lane q / K, register q % K); the shuffles run on every lane
          auto at_job = [&](const int(&v)[K], int j) -> int {
            if constexpr (K == 1) {
              return __shfl(v[0], j & (WAVE - 1));
            } else {
              const int v0 = __shfl(v[0], j & (WAVE - 1)), v1 = __shfl(v[1], j & (WAVE - 1));
              return (j >> 6) ? v1 : v0;
            }
          };
          auto at_pos = [&](const int(&v)[K], int q) -> int {
            if constexpr (K == 1) {
              return __shfl(v[0], q & (WAVE - 1));
            } else {
              const int v0 = __shfl(v[0], (q >> 1) & (WAVE - 1));
              const int v1 = __shfl(v[1], (q >> 1) & (WAVE - 1));
              return (q & 1) ? v1 : v0;
            }
          };
          auto at_pos_u = [&](const int(&v)[K], int q) -> int {  // q uniform
            if constexpr (K == 1) {
              return readlane(v[0], q);
            } else {
              const int v0 = readlane(v[0], q >> 1), v1 = readlane(v[1], q >> 1);
              return (q & 1) ? v1 : v0;
            }
          };
          // active jobs sorted by completion: end - t, progress t - start
          uint32_t dk[K];
          int dg[K];
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const bool act = ws_end[k] != IDLE;
            dk[k] = act ? (uint32_t)(ws_end[k] - t) : 0xFFFFFFFFu;
            dg[k] = act ? t - ws_start[k] : 0;
          }
          reg_sort_payload<K>(dk, dg, lane);
          int de[K];  // completion - t of each position (IDLE past N)
#pragma unroll
          for (int k = 0; k < K; ++k) de[k] = lane * K + k < N ? (int)dk[k] : IDLE;
          const int e_up = dpp<DPP_WAVE_SHL1>(de[0], de[0]);  // first position of the next lane
          // progress sum / max / min of the positions of the lanes above
          int xs_g, xs_max, xs_min;
          {
            int lg = 0, lmx = -1, lmn = IDLE;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              if (lane * K + k < N) {
                lg += dg[k];
                lmx = max(lmx, dg[k]);
                lmn = min(lmn, dg[k]);
              }
            }
            const int incl = wave_scan_incl(lg);
            xs_g = readlane(incl, WAVE - 1) - incl;
            const int rmx = wave_scan_incl_max(__shfl(lmx, (WAVE - 1) - lane));
            const int rmn = wave_scan_incl_min(__shfl(lmn, (WAVE - 1) - lane));
            const int src = lane < WAVE - 1 ? (WAVE - 2) - lane : 0;
            xs_max = __shfl(rmx, src);
            xs_min = __shfl(rmn, src);
            if (lane == WAVE - 1) {
              xs_max = -1;
              xs_min = IDLE;
            }
          }
          // ISJL: completions before the first one after which A_max exceeds
          // alpha, or (with a KV budget, which may block an idle worker) whose
          // following span the alpha crossing may cut; fewer than 3 are left
          // to the event loop
          bool go = true;
          if (POL == POL_ISJL) {
            int lfail = IDLE, lcutq = IDLE;
            int cg_max = xs_max;
#pragma unroll
            for (int k = K - 1; k >= 0; --k) {
              const int q = lane * K + k;
              const int e = de[k];
              const int e_nx = (k + 1 < K) ? de[k + 1 < K ? k + 1 : k] : e_up;
              if ((q < N) & ((q + 1 >= N) | (e_nx > e))) {
                if ((q + 1 >= N) | (e + cg_max > alpha)) lfail = q;
                else if ((M != 0) & (alpha != IDLE) & (alpha + 1 - cg_max < e_nx)) lcutq = q;
              }
              if (q < N) cg_max = max(cg_max, dg[k]);
            }
            const int qc = wave_min(lcutq);
            const int qf = min(wave_min(lfail), qc == IDLE ? IDLE : qc + 1);
            int lbelow = 0;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const int q = lane * K + k;
              const int e_nx = (k + 1 < K) ? de[k + 1 < K ? k + 1 : k] : e_up;
              if ((q < qf) & (e_nx > de[k])) lbelow++;
            }
            go = wave_sum(lbelow) >= 3;
          }
          if (go) {
          if (POL != POL_FCFS) gather_first(Gq);
          // queued jobs: length and summed reservations in priority order
          int qlen[K], pq[K];
          {
            int carry = 0;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const int j = k * WAVE + lane;
              int L = 0;
              if (j < Gq) L = plen(W[POL == POL_FCFS ? head + j : (int)STG[j]]);
              qlen[k] = L;
              const int inc = wave_scan_incl(L);
              pq[k] = j < Gq ? carry + inc : IDLE;
              carry += readlane(inc, WAVE - 1);
            }
          }
          // A(q): queued jobs admitted once the positions <= q have completed
          int ap[K];
          {
            int rr[K], run = 0;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              if (lane * K + k < N) run += de[k] + dg[k];  // lengths (= reservations)
              rr[k] = run;
            }
            const int rbase = wave_scan_incl(run) - run;
            const int64_t bud0 = (int64_t)M - S.res;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const int q = lane * K + k;
              int v = min(Gq, Beff - N + q + 1);
              if (M != 0) {
                const int64_t b = bud0 + rbase + rr[k];
                const int bb = b < 0 ? -1 : (b >= (int64_t)IDLE ? IDLE - 1 : (int)b);
                int lo = 0;  // queued jobs whose summed reservations fit
#pragma unroll
                for (int step = NS; step >= 1; step >>= 1) {
                  const int x = at_job(pq, min(lo + step, NS) - 1);
                  if ((lo + step <= NS) & (x <= bb)) lo += step;
                }
                v = min(v, lo);
              }
              ap[k] = q < N ? v : IDLE;
            }
          }
          // start of queued job j relative to t (IDLE: not admitted at these
          // positions), the earliest completion among jobs 0..j and their
          // summed starts
          int sg[K], pm[K], sa[K];
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const int j = k * WAVE + lane;
            int lo = 0;  // positions with A <= j
#pragma unroll
            for (int step = NS; step >= 1; step >>= 1) {
              const int x = at_pos(ap, min(lo + step, NS) - 1);
              if ((lo + step <= NS) & (x <= j)) lo += step;
            }
            const int e = at_pos(de, min(lo, NS - 1));
            sg[k] = lo < N ? e : IDLE;
          }
          {
            int cm = IDLE, cs = 0;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const int im = wave_scan_incl_min(sg[k] == IDLE ? IDLE : sg[k] + qlen[k]);
              pm[k] = min(cm, im);
              cm = min(cm, readlane(im, WAVE - 1));
              const int is = wave_scan_incl(sg[k] == IDLE ? 0 : sg[k]);
              sa[k] = cs + is;
              cs += readlane(is, WAVE - 1);
            }
          }
          const int Hr = H == IDLE ? IDLE : H - t;
          // Which completions the counts decide: the event at group end q is
          // taken if nothing is released by then, no admitted job has completed
          // by then and (ISJL) A_max after it is within alpha; the span after it
          // ends early (lim) at an admitted job's completion or, with an idle
          // worker blocked by the KV budget, at the alpha crossing.
          int lbad = IDLE, lcut = IDLE, lim[K];
          uint32_t gem = 0u;
          {
            int cg_max = xs_max;
#pragma unroll
            for (int k = K - 1; k >= 0; --k) {
              const int q = lane * K + k;
              const bool vq = q < N;
              const int e = de[k];
              const int e_nx = (k + 1 < K) ? de[k + 1 < K ? k + 1 : k] : e_up;
              const bool ge = vq & ((q + 1 >= N) | (e_nx > e));
              const int A = vq ? ap[k] : 0;
              const int pmA = at_job(pm, max(A - 1, 0));
              lim[k] = IDLE;
              if (ge) {
                gem |= 1u << k;
                bool ok = (q + 1 < N) & (e < Hr) & ((A == 0) | (pmA > e));
                if (POL == POL_ISJL) ok = ok && e + cg_max <= alpha;
                if (!ok) {
                  lbad = q;
                } else {
                  int cut = A > 0 ? pmA : IDLE;
                  if (POL == POL_ISJL && alpha != IDLE && N - 1 - q + A < Beff && A < Qn)
                    cut = min(cut, alpha + 1 - cg_max);
                  if (cut < e_nx) lcut = q;
                  lim[k] = min(min(e_nx, Hr), cut);
                }
              }
              if (vq) cg_max = max(cg_max, dg[k]);
            }
          }
          const int pe = wave_min(lbad), pc = wave_min(lcut);
          int p_m;
          {
            int lpm = -1;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const int q = lane * K + k;
              if (((gem >> k) & 1u) & (q < pe) & (q <= pc)) lpm = q;
            }
            p_m = wave_max(lpm);
          }
          const int e_first = readlane(de[0], 0);
          if (POL == POL_ISJL && kv_block && alpha != IDLE && S.min_s + alpha + 1 - t < e_first)
            p_m = -1;  // the crossing comes first
          int tau_rel;
          if (p_m >= 0) {
            tau_rel = at_pos_u(lim, p_m);
          } else {
            tau_rel = min(e_first, Hr);
            if (POL == POL_ISJL && kv_block && alpha != IDLE)
              tau_rel = min(tau_rel, S.min_s + alpha + 1 - t);
          }
          const int A_m = p_m >= 0 ? at_pos_u(ap, p_m) : 0;
          // spans after each counted event, with the jobs at the positions
          // above and the admitted jobs 0..A-1
          int64_t qE = 0, qSM = 0, qSSM = 0, qX = 0, qP = 0;
          int qU = 0;
          int64_t &lE = DEFER ? pE : qE, &lSM = DEFER ? pSM : qSM, &lSSM = DEFER ? pSSM : qSSM,
                  &lX = DEFER ? pX : qX, &lP = DEFER ? pP : qP;
          int& lU = DEFER ? pU : qU;
          int lmx = 0, lma = 0;
          {
            int cg = xs_g, cg_max = xs_max, cg_min = xs_min;
#pragma unroll
            for (int k = K - 1; k >= 0; --k) {
              const int q = lane * K + k;
              const bool vq = q < N;
              const int e = de[k];
              const int e_nx = (k + 1 < K) ? de[k + 1 < K ? k + 1 : k] : e_up;
              const int A = vq ? ap[k] : 0;
              const int saA = at_job(sa, max(A - 1, 0)), sgA = at_job(sg, max(A - 1, 0));
              if (((gem >> k) & 1u) & (q <= p_m)) {
                const int Er = q == p_m ? tau_rel : e_nx;
                const int64_t D = (int64_t)(Er - e);
                const int64_t so = N - 1 - q, s = so + A;
                const int min_s = t - cg_max;
                const int max_s = A > 0 ? t + sgA : t - cg_min;
                const int64_t sum_s = s * (int64_t)t - cg + (A > 0 ? saA : 0);
                const int64_t m0 = (int64_t)(t + e - min_s) + 1;
                const int64_t sm = D * m0 + D * (D - 1) / 2;
                lE += D * (sum_s - s * (int64_t)min_s);
                lSM += sm;
                lSSM += s * sm;
                const int ext = max_s - min_s;
                lX += D * ext;
                if (ext > alpha) lU += (int)D;
                lP = max(lP, s * (int64_t)(t + Er) - sum_s);
                lmx = max(lmx, ext);
                lma = max(lma, (int)s);
              }
              if (vq) {
                cg += dg[k];
                cg_max = max(cg_max, dg[k]);
                cg_min = min(cg_min, dg[k]);
              }
            }
          }
          // span [t, first event): the jobs active now
          {
            const int64_t D = (int64_t)(p_m >= 0 ? e_first : tau_rel), s = N;
            const int64_t m0 = (int64_t)(t - S.min_s) + 1;
            const int64_t sm = D * m0 + D * (D - 1) / 2;
            acc_E += D * (S.sum_s - s * (int64_t)S.min_s);
            acc_SM += sm;
            acc_SSM += s * sm;
            const int ext = S.max_s - S.min_s;
            acc_ext += D * ext;
            if (ext > alpha) acc_unfair += D;
            acc_peak = max(acc_peak, s * (int64_t)(t + D) - S.sum_s);
            lmx = max(lmx, ext);
            lma = max(lma, N);
          }
          if constexpr (!DEFER) {
            acc_E += wave_sum64(lE);
            acc_SM += wave_sum64(lSM);
            acc_SSM += wave_sum64(lSSM);
            acc_ext += wave_sum64(lX);
            acc_unfair += wave_sum(lU);
            acc_peak = max(acc_peak, wave_max64(lP));
          }
          acc_busy += (int64_t)tau_rel;
          acc_maxext = max(acc_maxext, wave_max(lmx));
          acc_maxact = max(acc_maxact, wave_max(lma));
          // completions of the admitted jobs
          {
            int lsc = 0;
#pragma unroll
            for (int k = 0; k < K; ++k)
              if (k * WAVE + lane < A_m) lsc += sg[k] + qlen[k];
            S.sum_comp += (int64_t)A_m * t + wave_sum(lsc);
          }
          // retire every job done by tau, then seat the admitted ones that are
          // still running
          const int tau = t + tau_rel;
          int lret = 0;
#pragma unroll
          for (int k = 0; k < K; ++k) {
            if (ws_end[k] <= tau) {
              lret++;
              ws_end[k] = IDLE;
              ws_start[k] = IDLE;
            }
          }
          if (A_m > 0) {
            int base = 0;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const bool idle = valid[k] & (ws_end[k] == IDLE);
              const uint64_t bm = ballot(idle);
              const int idx = base + mbcnt(bm);
              const int jc = min(idx, A_m - 1);
              const int s_rel = at_job(sg, jc), L = at_job(qlen, jc);
              if (idle & (idx < A_m)) {
                const int rk = POL == POL_FCFS ? head + idx : (int)STG[idx];
                const int st = t + s_rel;
                emit(pid(W[rk]), st, L);
                if (st + L > tau) {
                  ws_start[k] = st;
                  ws_end[k] = st + L;
                } else {
                  lret++;
                }
              }
              base += __builtin_popcountll(bm);
            }
            if (POL == POL_FCFS) {
              head += A_m;
            } else {
              pool.clear_upto(STG[A_m - 1], lane);
              qcount -= A_m;
            }
          }
          S.ndone += wave_sum(lret);
          {
            int cnt = 0, lres = 0, mn = IDLE, mx = -1, me = IDLE;
            int64_t ss = 0;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              if (ws_end[k] != IDLE) {
                cnt++;
                lres += ws_end[k] - ws_start[k];
                ss += ws_start[k];
                mn = min(mn, ws_start[k]);
                mx = max(mx, ws_start[k]);
                me = min(me, ws_end[k]);
              }
            }
            S.nact = wave_sum(cnt);
            S.res = wave_sum(lres);
            S.sum_s = wave_sum64(ss);
            S.min_s = S.nact > 0 ? wave_min(mn) : IDLE;
            S.max_s = S.nact > 0 ? wave_max(mx) : -1;
            S.min_end = wave_min(me);
          }
          S.t = tau;
          if (++iter > iter_max) {
            failed = true;
            break;
          }
          continue;
          }
        }
      }
    }

    // Drain sweep.  LJF between batches and ISJL in DRAIN admit nothing through
    // Phase TWO, and a planned ISJL job can start only at a step where
    // A_max(t) <= alpha, which (A_max grows between completions) can first hold
    // right after a completion, or when the machine is empty.  Every completion
    // before that carries no decision: the active jobs are sorted by
    // completion (in registers) and each span between consecutive completions
    // is accounted in parallel, the jobs active after position i being the
    // positions > i (their count, progress sum and progress range are suffix
    // scans).  The sweep stops at the first completion after which a planned
    // job could start; the jobs still active there stay in their slots.
    // The same holds for FCFS, SJF and ISJL in FILL with nothing queued or
    // planned: no completion before the next release carries a decision, so
    // those completions are swept too (when there are a few of them).
    const bool w0_timer = POL == POL_ISJL && planned > 0 && t_w1 > t &&
                          readlane(ws_end[0], 0) == IDLE &&
                          ((uint32_t)readlane((int)ws_q[0], 0) & 0xFFFFu) != QNONE;
    int quiet = 0;  // completions up to the next release, when nothing waits
    if (!PRE && POL != POL_LJF && S.nact > 0 &&
        (POL == POL_FCFS ? head == relk
                         : (qcount == 0 && (POL != POL_ISJL || (mode == 0 && planned == 0))))) {
      int r_next = IDLE;
      if (POL == POL_FCFS || !GEN) {
        if (relk < n) {
          if ((relk >> 6) != chunk) load_chunk(relk >> 6);
          r_next = readlane(rel_t, relk & (WAVE - 1));
        }
      } else {
        r_next = next_rel;
      }
      if (S.min_end <= r_next) {
#pragma unroll
        for (int k = 0; k < K; ++k)
          quiet += __builtin_popcountll(ballot((ws_end[k] != IDLE) & (ws_end[k] <= r_next)));
      }
    }
    // ISJL in FILL (or waiting on worker 1's timer) with A_max(t) > alpha: no
    // planned start, no Phase TWO admission and no epoch can come before the
    // first completion after which A_max <= alpha (A_max only grows between
    // completions, and every start needs it within alpha).  The only decision
    // meanwhile is Phase TWO's switch to DRAIN, at the first event with an idle
    // worker that has nothing planned and a queued job; both only appear over
    // the span, so it is settled from their first times after the sweep.  Taken
    // when at least two completions come before the last of the oldest active
    // jobs ends (A_max stays above alpha until then); compiled into the kernels
    // with up to 2 slots per lane (on the wider ones it did not fire on the
    // measured workloads and only added code).
    bool amax_sweep = false;
    if (POL == POL_ISJL && K <= 2 && !PRE && !FILL && S.nact > 0 && t - S.min_s > alpha &&
        !(mode == 1 && !w0_timer) && quiet < 3) {
      int oe = -1;
#pragma unroll
      for (int k = 0; k < K; ++k)
        if (ws_start[k] == S.min_s) oe = max(oe, ws_end[k]);
      oe = wave_max(oe);
      int before = 0;
#pragma unroll
      for (int k = 0; k < K; ++k) before += __builtin_popcountll(ballot(ws_end[k] < oe));
      amax_sweep = before >= 2;
    }
    bool sweep = !PRE &&
                 (POL == POL_LJF || (POL == POL_ISJL && mode == 1 && !w0_timer) || quiet >= 3 ||
                  amax_sweep) &&
                 S.nact > 0;
    if (sweep) {
      const int N = S.nact;
      // Progress is at most t - min_s and end - t at most the longest job:
      // when both fit one word together the progress rides in the low bits
      // of the key and the sort moves keys only.
      const int gbits = 32 - __builtin_clz((uint32_t)(t - S.min_s) | 1u);
      const bool packed = gbits < 32 && (int64_t)maxlen < (int64_t)(0xFFFFFFFFu >> gbits);
      int stop = 0, e0 = 0, st_g = 0, st_gmax = -1, st_gmin = IDLE, tau_end = 0;
      int64_t qE = 0, qSM = 0, qSSM = 0, qX = 0, qP = 0;
      int qU = 0;
      int64_t &lE = DEFER ? pE : qE, &lSM = DEFER ? pSM : qSM, &lSSM = DEFER ? pSSM : qSSM,
              &lX = DEFER ? pX : qX, &lP = DEFER ? pP : qP;
      int& lU = DEFER ? pU : qU;
      // Sort the N completions into KS registers per lane (position
      // p = lane * KS + k holds the p-th) and account the spans.  KS = K sorts
      // every slot in place; KS = 1 first packs up to 64 active slots into one
      // register through the gather buffer (for K >= 4).
      auto sweep_body = [&](auto ks_tag) {
        constexpr int KS = decltype(ks_tag)::value;
        uint32_t dk[KS];  // end - t (unused positions: all ones, sorted last)
        int dg[KS];       // progress t - start, carried with its key
        if (packed) {
          if constexpr (KS == K) {
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const bool act = ws_end[k] != IDLE;
              dk[k] = act ? ((uint32_t)(ws_end[k] - t) << gbits) | (uint32_t)(t - ws_start[k])
                          : 0xFFFFFFFFu;
            }
          } else {
            int base = 0;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const bool act = ws_end[k] != IDLE;
              const uint64_t bm = ballot(act);
              if (act)
                PEND[base + mbcnt(bm)] =
                    ((uint32_t)(ws_end[k] - t) << gbits) | (uint32_t)(t - ws_start[k]);
              base += __builtin_popcountll(bm);
            }
            wave_lds_sync();
            dk[0] = lane < N ? PEND[lane] : 0xFFFFFFFFu;
            wave_lds_sync();
          }
          reg_sort_keys<KS, true>(dk, lane);
          const uint32_t gmask = (1u << gbits) - 1u;
#pragma unroll
          for (int k = 0; k < KS; ++k) {
            dg[k] = (int)(dk[k] & gmask);
            dk[k] = dk[k] == 0xFFFFFFFFu ? 0xFFFFFFFFu : dk[k] >> gbits;
          }
        } else if constexpr (KS == K) {
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const bool act = ws_end[k] != IDLE;
            dk[k] = act ? (uint32_t)(ws_end[k] - t) : 0xFFFFFFFFu;
            dg[k] = act ? t - ws_start[k] : 0;
          }
          reg_sort_payload<K>(dk, dg, lane);
        }
        // Suffix state of the lanes above this one (positions >= (lane+1)*KS):
        // progress sum, max and min.
        int xs_g, xs_max, xs_min;
        {
          int lg = 0, lmx = -1, lmn = IDLE;
#pragma unroll
          for (int k = 0; k < KS; ++k) {
            if (lane * KS + k < N) {
              lg += dg[k];
              lmx = max(lmx, dg[k]);
              lmn = min(lmn, dg[k]);
            }
          }
          const int incl = wave_scan_incl(lg);
          xs_g = readlane(incl, WAVE - 1) - incl;
          const int rmx = wave_scan_incl_max(__shfl(lmx, (WAVE - 1) - lane));
          const int rmn = wave_scan_incl_min(__shfl(lmn, (WAVE - 1) - lane));
          const int src = lane < WAVE - 1 ? (WAVE - 2) - lane : 0;
          xs_max = __shfl(rmx, src);
          xs_min = __shfl(rmn, src);
          if (lane == WAVE - 1) {
            xs_max = -1;
            xs_min = IDLE;
          }
        }
        // completion time of the first position of the next lane
        const int e_up = t + dpp<DPP_WAVE_SHL1>((int)dk[0], (int)dk[0]);
        // Stop position: the lowest position ending a tie group after which
        // the machine is empty or A_max <= alpha (A_max right after the
        // completions at e is e - t + the largest progress still active).
        stop = quiet >= 3 ? quiet - 1 : N - 1;
        if (POL == POL_ISJL && (planned > 0 || (a.resume && mode == 1) || amax_sweep)) {
          int cg_max = xs_max, lfound = IDLE;
#pragma unroll
          for (int k = KS - 1; k >= 0; --k) {
            const int pos = lane * KS + k;
            const bool valid = pos < N;
            const int e = t + (int)dk[k];
            const int e_next = (k + 1 < KS) ? t + (int)dk[k + 1 < KS ? k + 1 : k] : e_up;
            const bool group_end = valid & ((pos + 1 >= N) | (e_next > e));
            if (group_end & ((pos + 1 >= N) | (e - t + cg_max <= alpha))) lfound = pos;
            if (valid) cg_max = max(cg_max, dg[k]);
          }
          stop = min(stop, wave_min(lfound));
        }
        // Spans between consecutive completions below `stop`, each with the
        // jobs at the positions above (count N - 1 - p, progress suffix sums).
        int sg = 0, sgmax = -1, sgmin = IDLE, se = 0;
        {
          int cg = xs_g, cg_max = xs_max, cg_min = xs_min;
#pragma unroll
          for (int k = KS - 1; k >= 0; --k) {
            const int pos = lane * KS + k;
            const bool valid = pos < N;
            const int e = t + (int)dk[k];
            const int e_next = (k + 1 < KS) ? t + (int)dk[k + 1 < KS ? k + 1 : k] : e_up;
            if (valid & (pos < stop) & (e_next > e)) {
              const int64_t D = (int64_t)(e_next - e);
              const int64_t s = N - 1 - pos;
              const int min_s = t - cg_max, max_s = t - cg_min;
              const int64_t sum_s = s * (int64_t)t - cg;
              const int64_t m0 = (int64_t)(e - min_s) + 1;
              const int64_t sm = D * m0 + D * (D - 1) / 2;
              lE += D * (sum_s - s * (int64_t)min_s);
              lSM += sm;
              lSSM += s * sm;
              const int ext = max_s - min_s;
              lX += D * ext;
              if (ext > alpha) lU += (int)D;
              lP = max(lP, s * (int64_t)e_next - sum_s);
            }
            if (pos == stop) {
              sg = cg;
              sgmax = cg_max;
              sgmin = cg_min;
              se = e;
            }
            if (valid) {
              cg += dg[k];
              cg_max = max(cg_max, dg[k]);
              cg_min = min(cg_min, dg[k]);
            }
          }
        }
        const int Ls = stop / KS;
        st_g = readlane(sg, Ls);
        st_gmax = readlane(sgmax, Ls);
        st_gmin = readlane(sgmin, Ls);
        tau_end = readlane(se, Ls);
        e0 = t + readlane((int)dk[0], 0);
      };
      if constexpr (K >= 4) {
        // the packing goes through the gather buffer: only when it holds 64 words
        if (packed && N <= WAVE && a.wave_words - a.off_stage >= WAVE)
          sweep_body(std::integral_constant<int, 1>{});
        else sweep_body(std::integral_constant<int, K>{});
      } else {
        sweep_body(std::integral_constant<int, K>{});
      }
      // span [t, e_0): every job still active; the set only shrinks after it,
      // so it also carries the largest extent and count of the sweep
      {
        const int64_t D = (int64_t)(e0 - t), s = N;
        const int64_t m0 = (int64_t)(t - S.min_s) + 1;
        const int64_t sm = D * m0 + D * (D - 1) / 2;
        acc_E += D * (S.sum_s - s * (int64_t)S.min_s);
        acc_SM += sm;
        acc_SSM += s * sm;
        const int ext = S.max_s - S.min_s;
        acc_ext += D * ext;
        if (ext > alpha) acc_unfair += D;
        acc_peak = max(acc_peak, s * (int64_t)e0 - S.sum_s);
        acc_maxext = max(acc_maxext, ext);
        acc_maxact = max(acc_maxact, N);
      }
      if constexpr (!DEFER) {
        acc_E += wave_sum64(lE);
        acc_SM += wave_sum64(lSM);
        acc_SSM += wave_sum64(lSSM);
        acc_ext += wave_sum64(lX);
        acc_unfair += wave_sum(lU);
        acc_peak = max(acc_peak, wave_max64(lP));
      }
      acc_busy += (int64_t)(tau_end - t);
      if (POL == POL_ISJL && amax_sweep && mode == 0) {
        // Phase TWO switches to DRAIN at the first event before tau_end with an
        // idle worker that has nothing planned (from its first completion, or
        // now) and a queued job (now, or from the next release)
        int tn_free = IDLE;
        if (planned == 0 && S.nact < Beff) {
          tn_free = t;
        } else {
          int fe = IDLE;
          bool idle_empty = false;
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const bool empty_q = (ws_q[k] & 0xFFFFu) == QNONE;
            if (valid[k] & empty_q) {
              if (ws_end[k] == IDLE) idle_empty = true;
              else fe = min(fe, ws_end[k]);
            }
          }
          tn_free = ballot(idle_empty) ? t : wave_min(fe);
        }
        int tn_queued = IDLE;
        if (qcount > 0) {
          tn_queued = t;
        } else if (POL == POL_FCFS || !GEN) {
          if (relk < n) {
            if ((relk >> 6) != chunk) load_chunk(relk >> 6);
            tn_queued = readlane(rel_t, relk & (WAVE - 1));
          }
        } else {
          tn_queued = next_rel;
        }
        if (max(tn_free, tn_queued) < tau_end) mode = 1;
      }
      // retire every job that completed by tau_end
      int rc = 0, rl = 0, me = IDLE;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        if (ws_end[k] <= tau_end) {
          rc++;
          rl += ROB ? ws_plan[k] : ws_end[k] - ws_start[k];
          ws_end[k] = IDLE;
          ws_start[k] = IDLE;
        }
        me = min(me, ws_end[k]);
      }
      const int nret = wave_sum(rc);
      S.ndone += nret;
      S.res -= wave_sum(rl);
      S.nact = N - nret;
      S.min_end = wave_min(me);
      if (S.nact > 0) {
        S.sum_s = (int64_t)S.nact * t - st_g;
        S.min_s = t - st_gmax;
        S.max_s = t - st_gmin;
      } else {
        S.sum_s = 0;
        S.min_s = IDLE;
        S.max_s = -1;
      }
      S.t = tau_end;
      if (++iter > iter_max) {
        failed = true;
        break;
      }
      continue;
    }

    // (5) next event.  A release is an event only if the job could be admitted
    // before anything else happens: ISJL with an idle worker that has nothing
    // planned in Phase TWO, or an empty machine with no plan; LJF at an empty
    // machine; SJF with a free slot; FCFS with a free slot and nothing queued
    // (a queued job left waiting with a slot free is blocked by the KV budget,
    // which changes only at a completion, and it precedes every later arrival).  Otherwise it is folded into the
    // next event (the queue is only read there).
    int tn = S.min_end;
    bool rel_matters;
    if (POL == POL_ISJL) rel_matters = (mode == 0 && free_empty > 0) || (S.nact == 0 && planned == 0);
    else if (POL == POL_LJF) rel_matters = S.nact == 0;
    else if (POL == POL_FCFS)  // a queued head blocks every later arrival in FCFS order
      rel_matters = S.nact < Beff && head == relk;
    else rel_matters = S.nact < Beff;
    // ISJL in FILL (with up to 2 slots per lane) and SJF, with a slot free and
    // jobs queued: the queue's head is held back by the KV budget, which stays
    // fixed until a completion.  An arrival before then is an event only if it
    // precedes that head in the policy's order and fits beside the running jobs;
    // the first such arrival bounds the span.
    const bool blocked_head =
        !GEN && !PRE && !ROB && qcount > 0 && S.nact > 0 &&
        ((POL == POL_SJF && S.nact < Beff) ||
         (POL == POL_ISJL && K <= 2 && mode == 0 && free_empty > 0 && kv_block));
    if (blocked_head) {
      rel_matters = false;
      const int hr = pool.first();
      int r = relk;
      while (r < n) {
        if ((r >> 6) != chunk) load_chunk(r >> 6);
        const int off = r & (WAVE - 1);
        const bool in = (lane >= off) & (rel_t < tn);
        const bool m = in && rel_r < hr && S.res + (int64_t)plen(W[rel_r]) <= M;
        const uint64_t mm = ballot(m);
        if (mm) {
          tn = min(tn, readlane(rel_t, __builtin_ctzll(mm)));
          break;
        }
        if (ballot((lane >= off) & (rel_t >= tn))) break;  // the rest arrive after the span
        r = (r & ~(WAVE - 1)) + WAVE;
      }
    }
    if (rel_matters) {
      if (POL == POL_FCFS || !GEN) {
        if (relk < n) {
          if ((relk >> 6) != chunk) load_chunk(relk >> 6);
          tn = min(tn, readlane(rel_t, relk & 63));
        }
      } else {
        tn = min(tn, next_rel);
      }
    }
    if (POL == POL_ISJL) {
      if (planned > 0 && t_w1 > t) {
        bool w0_wait = readlane(ws_end[0], 0) == IDLE &&
                       ((uint32_t)readlane((int)ws_q[0], 0) & 0xFFFFu) != QNONE;
        if (w0_wait) tn = min(tn, t_w1);
      }
      if (mode == 0 && kv_block && alpha != IDLE) tn = min(tn, S.min_s + alpha + 1);
    }
    if (tn == IDLE || tn <= t || ++iter > iter_max) {
      failed = true;
      break;
    }

    // (6) account steps t .. tn-1 (Section 5)
    const int64_t D = (int64_t)(tn - t);
    if (S.nact != 0) {
      const int64_t s = S.nact;
      // largest footprint at step t (it grows by one per step of the span) and
      // the span's externality: each active job pays the largest footprint
      // minus its own, a constant over the span
      int64_t m0, xe;
      if (PRE) {
        m0 = (int64_t)t + S.G + 1;
        xe = s * (int64_t)S.G - (S.sp - S.sum_s);
      } else {
        m0 = (int64_t)(t - S.min_s) + 1;
        xe = S.sum_s - s * (int64_t)S.min_s;
      }
      const int64_t sm = D * m0 + D * (D - 1) / 2;
      acc_E += D * xe;
      acc_SM += sm;
      acc_SSM += s * sm;
      const int ext = S.max_s - S.min_s;
      acc_ext += D * ext;
      acc_busy += D;
      if (ext > alpha) acc_unfair += D;
      acc_maxext = max(acc_maxext, ext);
      acc_maxact = max(acc_maxact, S.nact);
      acc_peak = max(acc_peak, s * (int64_t)tn - S.sum_s + (PRE ? S.sp : 0));
    }
    S.t = tn;
  }
  if constexpr (DEFER) {
    acc_E += wave_sum64(pE);
    acc_SM += wave_sum64(pSM);
    acc_SSM += wave_sum64(pSSM);
    acc_ext += wave_sum64(pX);
    acc_unfair += wave_sum(pU);
    acc_peak = max(acc_peak, wave_max64(pP));
  }

  if (failed) {
    write_marker(a.out, a.out_T, inst, T_INTERNAL, lane);
    return;
  }
  if (lane == 0 && a.out_T) {
    a.out_T[inst] = S.t;
  } else if (lane == 0) {
    fsched_metrics m;
    m.T = S.t;
    m.O = osum;
    m.Q = qsum;
    m.E = acc_E;
    m.C = a.c * (int64_t)S.t + a.tau * acc_SSM;
    m.W = a.c * (int64_t)S.t + a.tau * acc_SM;
    m.sum_completion = S.sum_comp;
    m.sum_latency = S.sum_comp - rsum;
    m.sum_extent = acc_ext;
    m.busy_steps = acc_busy;
    m.peak_kv = acc_peak;
    m.unfair_steps = acc_unfair;
    m.max_extent = acc_maxext;
    m.max_active = acc_maxact;
    a.out[inst] = m;
  }
}

// Whether a grid of `blocks` blocks of `wpb` waves fits the device at once
// (every block resident from the start); false when the runtime cannot tell.
inline bool resident_at_once(const void* kern, int64_t blocks, int wpb, size_t lds) {
  int per_cu = 0, dev = 0, n_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, wpb * WAVE, lds) != hipSuccess ||
      hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return blocks <= (int64_t)per_cu * n_cu;
}

// The fill sweep serves FCFS and SJF with up to 2 slots per lane, and ISJL there
// when alpha is at least the length limit (A_max, below every length, never
// exceeds it).  With a finite budget ISJL's completions mostly meet the guard
// one at a time, and its event loop runs faster without the sweep's code.
template <int POL, bool ROB = false, bool PRE = false>
hipError_t launch_sim(const SimArgs& a, int K, int NW, bool general, int wpb, size_t lds,
                      hipStream_t s) {
  const int64_t blocks = (a.n_inst + wpb - 1) / wpb;
  dim3 grid((unsigned)blocks), block((unsigned)(wpb * WAVE));
  constexpr bool FILL_OK = !ROB && !PRE && POL != POL_LJF;
  constexpr bool FILL_ALWAYS = FILL_OK && POL != POL_ISJL;
  const bool fill = FILL_OK && K <= 2 && (FILL_ALWAYS || a.alpha >= (int)LEN_LIMIT);
  // ISJL plan-queue links in HBM scratch (a kernel of its own, up to 8 slots per
  // lane; the fill-sweep kernels run with alpha at least every length, so
  // nothing is planned there)
  const bool qh = POL == POL_ISJL && K <= 8 && !fill && a.qlink != nullptr;
#define FS_LAUNCH(KK, NN, GG, FF, QQ)                                                     \
  if (K == KK && NW == NN && general == GG && fill == FF && qh == QQ) {                   \
    if constexpr (!GG && KK <= 8) {                                                       \
      if (resident_at_once((const void*)simulate_kernel<POL, KK, NN, GG, ROB, PRE, FF, QQ, true>, \
                           blocks, wpb, lds)) {                                           \
        hipLaunchKernelGGL((simulate_kernel<POL, KK, NN, GG, ROB, PRE, FF, QQ, true>), grid, block, \
                           lds, s, a);                                                    \
        return hipGetLastError();                                                         \
      }                                                                                   \
    }                                                                                     \
    hipLaunchKernelGGL((simulate_kernel<POL, KK, NN, GG, ROB, PRE, FF, QQ>), grid, block, lds, \
                       s, a);                                                             \
    return hipGetLastError();                                                             \
  }
#define FS_LAUNCH_K(KK, FF, QQ)                                                             \
  FS_LAUNCH(KK, 1, false, FF, QQ) FS_LAUNCH(KK, 2, false, FF, QQ) FS_LAUNCH(KK, 1, true, FF, QQ) \
  FS_LAUNCH(KK, 2, true, FF, QQ)
  if constexpr (FILL_OK) {
    FS_LAUNCH_K(1, true, false)
    FS_LAUNCH_K(2, true, false)
  }
  if constexpr (!FILL_ALWAYS) {
    FS_LAUNCH_K(1, false, false)
    FS_LAUNCH_K(2, false, false)
  }
  if constexpr (POL == POL_ISJL) {
    FS_LAUNCH_K(1, false, true)
    FS_LAUNCH_K(2, false, true)
    FS_LAUNCH_K(4, false, true)
    FS_LAUNCH_K(8, false, true)
  }
  FS_LAUNCH_K(4, false, false)
  FS_LAUNCH_K(8, false, false)
  FS_LAUNCH_K(16, false, false)
#undef FS_LAUNCH_K
#undef FS_LAUNCH
  return hipErrorInvalidValue;
}

}  // namespace fs
