// Re-scoring of given schedules (Section 5, Theorem 5.1; eq. (1) checks):
// one wavefront per instance.
//
// The 2n start/end events are sorted in LDS as packed keys
//   time << 13 | kind << 12 | index      (kind 0 = end, 1 = start)
// so that at equal times completions come before starts, matching the step
// model (a job ending at t frees its slot for a job starting at t).  A sweep
// over the sorted events keeps |S|, sum of starts and sum of reservations as
// scalars; the earliest and latest start among the active jobs are found by
// wave-parallel scans over the sorted events (forward from the previous
// earliest, backward from the latest start event seen), 64 events per step.
// Between two event times the active set is fixed and the Section 5 terms are
// summed in closed form, as in the simulation kernel.
#include "dec_common.hpp"
#include "wave.hpp"

namespace fs {

namespace {

constexpr int IDLE32 = 0x7FFFFFFF;

__device__ inline void dec_sort(uint32_t* W, int NP, int lane) {
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

__device__ inline void dec_marker(fsched_metrics* out, uint32_t* viol, int64_t inst, int64_t code,
                                  uint32_t v, int lane) {
  if (lane == 0) {
    fsched_metrics m;
    m.T = code;
    m.O = m.Q = m.E = m.C = m.W = 0;
    m.sum_completion = m.sum_latency = m.sum_extent = m.busy_steps = 0;
    m.peak_kv = m.unfair_steps = 0;
    m.max_extent = m.max_active = 0;
    out[inst] = m;
    viol[inst] = v;
  }
}

}  // namespace

__global__ __launch_bounds__(256) void decompose_kernel(DecArgs a) {
  extern __shared__ uint32_t lds_raw[];
  const int wib = threadIdx.x >> 6;
  const int64_t inst = (int64_t)blockIdx.x * (blockDim.x >> 6) + wib;
  if (inst >= a.n_inst) return;
  const int lane = lane_id();
  const int n = a.n;
  uint32_t* EV = lds_raw + (size_t)wib * (size_t)a.wave_words;
  uint8_t* ST = (uint8_t*)(EV + a.NP2);  // per job: 0 not started, 1 active, 2 ended
  const int64_t row = inst * (int64_t)n;
  const int32_t* A = a.arrival + row;
  const int32_t* P = a.prompt + row;
  const int32_t* O = a.output + row;
  const int32_t* S0 = a.start + row;

  int bad = 0, neg = 0, early = 0, big = 0, maxlen = 0;
  int64_t osum = 0, qsum = 0, csum = 0, lsum = 0, tmax = 0;
  for (int i = lane; i < n; i += WAVE) {
    int ar = A[i], p = P[i], o = O[i], s = S0[i];
    bad |= (ar < 0) | (p < 0) | (o < 1);
    int64_t len = (int64_t)p + (int64_t)o;
    big |= (len >= (1 << 20));
    neg |= (s < 0);
    early |= (s < ar);
    int64_t e = (int64_t)s + len;
    if (e > tmax) tmax = e;
    if (len < (1 << 20) && len > maxlen) maxlen = (int)len;
    osum += len;
    qsum += len * (len + 1) / 2;
    csum += e;
    lsum += e - ar;
  }
  bad = ballot(bad != 0) != 0;
  neg = ballot(neg != 0) != 0;
  early = ballot(early != 0) != 0;
  big = ballot(big != 0) != 0;
  if (bad) {
    dec_marker(a.out, a.viol, inst, FSCHED_T_INVALID, 0u, lane);
    return;
  }
  if (neg) {
    // a negative start: nothing else is evaluated (bit 16, plus bit 1)
    if (lane == 0) {
      fsched_metrics m;
      m.T = m.O = m.Q = m.E = m.C = m.W = 0;
      m.sum_completion = m.sum_latency = m.sum_extent = m.busy_steps = 0;
      m.peak_kv = m.unfair_steps = 0;
      m.max_extent = m.max_active = 0;
      a.out[inst] = m;
      a.viol[inst] = 16u | 1u;
    }
    return;
  }
  if (big) {
    dec_marker(a.out, a.viol, inst, FSCHED_T_TOOLARGE, 0u, lane);
    return;
  }
  // tmax via two 32-bit reductions (all ends are >= 0 here)
  {
    int hi = wave_max((int)(tmax >> 31));
    int lo = wave_max((int)(((tmax >> 31) == hi) ? (tmax & 0x7FFFFFFF) : 0));
    tmax = ((int64_t)hi << 31) | lo;
  }
  maxlen = wave_max(maxlen);
  osum = wave_sum64(osum);
  qsum = wave_sum64(qsum);
  csum = wave_sum64(csum);
  lsum = wave_sum64(lsum);
  if (tmax >= DEC_TIME_LIMIT) {
    dec_marker(a.out, a.viol, inst, FSCHED_T_TOOLARGE, 0u, lane);
    return;
  }
  {
    double cb = (double)a.c * (double)tmax + (double)a.tau * (double)osum * (double)maxlen;
    double wb = (double)a.c * (double)tmax + (double)a.tau * (double)tmax * (double)maxlen;
    if (cb > 4.0e18 || wb > 4.0e18) {
      dec_marker(a.out, a.viol, inst, FSCHED_T_RANGE, 0u, lane);
      return;
    }
  }

  // ---- events ---------------------------------------------------------------
  const int NE = 2 * n, NP2 = a.NP2;
  for (int e = lane; e < NP2; e += WAVE) {
    uint32_t key = 0xFFFFFFFFu;
    if (e < NE) {
      int i = e >> 1;
      int s = S0[i];
      if (e & 1) key = ((uint32_t)s << 13) | (1u << 12) | (uint32_t)i;
      else key = ((uint32_t)(s + P[i] + O[i]) << 13) | (uint32_t)i;
    }
    EV[e] = key;
  }
  for (int i = lane; i < n; i += WAVE) ST[i] = 0;
  wave_lds_sync();
  dec_sort(EV, NP2, lane);

  // ---- sweep ----------------------------------------------------------------
  int cnt = 0, min_s = IDLE32, max_s = -1;
  int pmin = 0;   // events before pmin hold no start of an active job
  int pmax = -1;  // index of the latest start event processed
  bool dirty_min = false, dirty_max = false;
  int64_t sum_s = 0, res = 0;
  int cur_t = 0;
  uint32_t v = early ? 1u : 0u;
  int64_t acc_E = 0, acc_C = 0, acc_W = 0, acc_ext = 0, acc_busy = 0, acc_peak = 0, acc_unf = 0;
  int acc_maxext = 0, acc_maxact = 0;
  const int alpha = a.alpha;
  const int64_t M = a.M;
  const int Bcap = a.B;

  for (int base = 0; base < NE; base += WAVE) {
    const int e = base + lane;
    const uint32_t key = e < NE ? EV[e] : 0xFFFFFFFFu;
    const int kt = (int)(key >> 13), kid = (int)(key & 0xFFFu);
    const int klen = e < NE ? P[kid] + O[kid] : 0;
    const int cnum = min(WAVE, NE - base);
    for (int q = 0; q < cnum; ++q) {
      const int t = readlane(kt, q);
      if (t > cur_t) {
        // refresh the earliest / latest active start if their holders ended
        if (cnt > 0 && dirty_min) {
          while (true) {
            int ee = pmin + lane;
            bool hit = false;
            int st_time = 0;
            if (ee < NE) {
              uint32_t kk = EV[ee];
              hit = ((kk >> 12) & 1u) && ST[kk & 0xFFFu] == 1;
              st_time = (int)(kk >> 13);
            }
            uint64_t m = ballot(hit);
            if (m) {
              int L = __builtin_ctzll(m);
              pmin += L;
              min_s = readlane(st_time, L);
              break;
            }
            pmin += WAVE;
            if (pmin >= NE) break;  // unreachable while cnt > 0
          }
          dirty_min = false;
        }
        if (cnt > 0 && dirty_max) {
          while (true) {
            int ee = pmax - lane;
            bool hit = false;
            int st_time = 0;
            if (ee >= 0) {
              uint32_t kk = EV[ee];
              hit = ((kk >> 12) & 1u) && ST[kk & 0xFFFu] == 1;
              st_time = (int)(kk >> 13);
            }
            uint64_t m = ballot(hit);
            if (m) {
              int L = __builtin_ctzll(m);
              pmax -= L;
              max_s = readlane(st_time, L);
              break;
            }
            pmax -= WAVE;
            if (pmax < 0) break;  // unreachable while cnt > 0
          }
          dirty_max = false;
        }
        // account steps cur_t .. t-1 (Section 5)
        const int64_t D = (int64_t)(t - cur_t);
        if (cnt == 0) {
          acc_C += a.c * D;
          acc_W += a.c * D;
        } else {
          const int64_t s = cnt;
          const int64_t m0 = (int64_t)(cur_t - min_s) + 1;
          const int64_t sm = D * m0 + D * (D - 1) / 2;
          acc_E += D * (sum_s - s * (int64_t)min_s);
          acc_C += a.c * D + a.tau * s * sm;
          acc_W += a.c * D + a.tau * sm;
          const int ext = max_s - min_s;
          acc_ext += D * ext;
          acc_busy += D;
          if (ext > alpha) {
            acc_unf += D;
            v |= 8u;
          }
          acc_maxext = max(acc_maxext, ext);
          acc_maxact = max(acc_maxact, cnt);
          acc_peak = max(acc_peak, s * (int64_t)t - sum_s);
          if (Bcap > 0 && cnt > Bcap) v |= 2u;
          if (M != 0 && cnt >= 2 && res > M) v |= 4u;
        }
        cur_t = t;
      }
      const uint32_t kq = (uint32_t)readlane((int)key, q);
      const int id = (int)(kq & 0xFFFu);
      const int len = readlane(klen, q);
      if ((kq >> 12) & 1u) {  // start
        if (cnt == 0) {
          min_s = t;
          pmin = base + q;
          dirty_min = false;
        }
        cnt++;
        sum_s += t;
        res += len;
        max_s = t;
        pmax = base + q;
        dirty_max = false;
        if (lane == 0) ST[id] = 1;
      } else {  // end
        const int s = t - len;
        cnt--;
        sum_s -= s;
        res -= len;
        if (lane == 0) ST[id] = 2;
        if (s == min_s) dirty_min = true;
        if (s == max_s) dirty_max = true;
        if (cnt == 0) {
          min_s = IDLE32;
          max_s = -1;
          dirty_min = dirty_max = false;
        }
      }
      wave_lds_sync();
    }
  }

  if (lane == 0) {
    fsched_metrics m;
    m.T = tmax;
    m.O = osum;
    m.Q = qsum;
    m.E = acc_E;
    m.C = acc_C;
    m.W = acc_W;
    m.sum_completion = csum;
    m.sum_latency = lsum;
    m.sum_extent = acc_ext;
    m.busy_steps = acc_busy;
    m.peak_kv = acc_peak;
    m.unfair_steps = acc_unf;
    m.max_extent = acc_maxext;
    m.max_active = acc_maxact;
    a.out[inst] = m;
    a.viol[inst] = v;
  }
}

hipError_t launch_decompose(const DecArgs& a, int wpb, size_t lds, hipStream_t s) {
  const int64_t blocks = (a.n_inst + wpb - 1) / wpb;
  hipLaunchKernelGGL(decompose_kernel, dim3((unsigned)blocks), dim3((unsigned)(wpb * WAVE)), lds,
                     s, a);
  return hipGetLastError();
}

}  // namespace fs
