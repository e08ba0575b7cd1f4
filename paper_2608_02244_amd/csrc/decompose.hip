// Re-scoring of given schedules (Section 5, profit decomposition; eq. (1) checks):
// one wavefront per instance.
//
// The 2n start/end events are sorted (in registers, or in LDS beyond 4,096
// events) as packed keys
//   time << 13 | kind << 12 | index      (kind 0 = end, 1 = start)
// so that at equal times completions come before starts, matching the step
// model (a job ending at t frees its slot for a job starting at t).  Between
// two event times the active set is fixed and the Section 5 terms are summed
// in closed form, as in the simulation kernel; the sweep itself is described
// where it runs.
#include <type_traits>

#include "dec_common.hpp"
#include "regsort.hpp"
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

// NARROW: lengths are kept as 16-bit values (an instance with a job of 65,536
// tokens or more is left to the wide pass).
template <bool NARROW>
__global__ __launch_bounds__(256) void decompose_kernel(DecArgs a) {
  extern __shared__ uint32_t lds_raw[];
  const int wib = threadIdx.x >> 6;
  const int64_t inst = (int64_t)blockIdx.x * (blockDim.x >> 6) + wib;
  if (inst >= a.n_inst) return;
  const int lane = lane_id();
  const int n = a.n;
  uint32_t* EV = lds_raw + (size_t)wib * (size_t)a.wave_words;
  using len_t = typename std::conditional<NARROW, uint16_t, int32_t>::type;
  len_t* LEN = (len_t*)(EV + a.NP2);  // per job: prompt + output
  if (!NARROW && a.deferred_only && a.out[inst].T != DEC_DEFERRED) return;
  const int64_t row = inst * (int64_t)n;
  const int32_t* A = a.arrival + row;
  const int32_t* P = a.prompt + row;
  const int32_t* O = a.output + row;
  const int32_t* S0 = a.start + row;

  // One pass over the job table: validation, instance totals, the two event
  // keys of every job (end: (s + len, 0, i), start: (s, 1, i); they are only
  // sorted once the table is known to be valid) and the lengths.  The rows are
  // software-pipelined: the loads of row r + PF are issued while row r is
  // processed (clamped indices keep every load in bounds).
  const int NE = 2 * n, NP2 = a.NP2;
  int bad = 0, neg = 0, early = 0, big = 0, maxlen = 0;
  int64_t osum = 0, qsum = 0, csum = 0, lsum = 0, tmax = 0;
  constexpr int PF = 4;
  int pf_a[PF], pf_p[PF], pf_o[PF], pf_s[PF];
#pragma unroll
  for (int d = 0; d < PF; ++d) {
    const int ic = min(d * WAVE + lane, n - 1);
    pf_a[d] = A[ic];
    pf_p[d] = P[ic];
    pf_o[d] = O[ic];
    pf_s[d] = S0[ic];
  }
  for (int r0 = 0; r0 < n; r0 += PF * WAVE) {
#pragma unroll
    for (int d = 0; d < PF; ++d) {
      const int i0 = r0 + d * WAVE;
      if (i0 >= n) break;
      const int i = i0 + lane;
      const int ar = pf_a[d], p = pf_p[d], o = pf_o[d], s = pf_s[d];
      {
        const int ic = min(i + PF * WAVE, n - 1);
        pf_a[d] = A[ic];
        pf_p[d] = P[ic];
        pf_o[d] = O[ic];
        pf_s[d] = S0[ic];
      }
      if (i < n) {
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
        EV[2 * i] = ((uint32_t)(s + p + o) << 13) | (uint32_t)i;
        EV[2 * i + 1] = ((uint32_t)s << 13) | (1u << 12) | (uint32_t)i;
        LEN[i] = (len_t)(p + o);
      }
    }
  }
  for (int e = NE + lane; e < NP2; e += WAVE) EV[e] = 0xFFFFFFFFu;
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
  if (NARROW && maxlen >= 65536) {
    dec_marker(a.out, a.viol, inst, DEC_DEFERRED, 0u, lane);
    return;
  }
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

  // ---- events (keys written above) ---------------------------------------------
  wave_lds_sync();
  switch (NP2) {  // register sort up to 64 keys per lane, LDS network beyond
    case 64: wave_reg_sort<1, true>(EV, lane); break;
    case 128: wave_reg_sort<2, true>(EV, lane); break;
    case 256: wave_reg_sort<4, true>(EV, lane); break;
    case 512: wave_reg_sort<8, true>(EV, lane); break;
    case 1024: wave_reg_sort<16, true>(EV, lane); break;
    case 2048: wave_reg_sort<32, true>(EV, lane); break;
    case 4096: wave_reg_sort<64, true>(EV, lane); break;
    default: dec_sort(EV, NP2, lane); break;
  }
  wave_lds_sync();

  // ---- sweep ----------------------------------------------------------------
  // 64 sorted events at a time: |S|, the start sum and the reservation sum
  // after each event are prefix scans of the events' deltas.  A group is the
  // events of one time; the span after a group end lasts to the next event
  // time.  The earliest / latest active start after a group end changes only
  // when the group starts jobs or when the last active job holding it ends, so
  // only those group ends are visited one by one: the earliest start is kept
  // with the number of active jobs that started then (nmin; the same for the
  // latest, nmax), and a group end is visited when it has starts or when the
  // ends since the last visit use up nmin or nmax.  A start event is active at
  // time t when its job ends after t; a new earliest (latest) start is searched
  // forward (backward) from the previous one, 64 events per step.  The values
  // in force at every group end are then spread by lane and the span terms of
  // all group ends of the chunk are summed at once.
  const int alpha = a.alpha;
  const int64_t M = a.M;
  const int Bcap = a.B;
  uint32_t v = early ? 1u : 0u;
  int c_cnt = 0;                       // |S| before the chunk
  // start sum and reservation sum before the chunk: below 4,096 x 2^19, so
  // they (and every partial sum) are exact in 32 bits
  uint32_t c_sum = 0, c_res = 0;
  int min_s = IDLE32, max_s = -1;      // earliest / latest active start
  int nmin = 0, nmax = 0;              // active jobs that started at min_s / max_s
  int pmin = 0, pmax = -1;             // first / last of their start events
  int cnt_last = 0;                    // |S| at the last group end
  int g_nst = 0, gfirst = -1, glast = -1;  // starts of the open group (before this chunk)
  // per lane: E, extent and the two parts of the largest-footprint sums (C and
  // W take c and tau once at the end) in 64 bits; span lengths, busy and
  // unfair steps (the spans of one lane are disjoint, so each sum stays below
  // 2^19) and peak KV in 32 bits; extent and |S| maxima
  uint64_t lE = 0, lX = 0, lSMa = 0, lSMb = 0, lSSMa = 0, lSSMb = 0;
  uint32_t lD = 0, lB = 0, lU = 0, lP = 0;
  int lXm = 0, lAm = 0;
  bool lcap = false, lkv = false, lunf = false;
  // idle steps before the first event
  const int t_first = (int)(EV[0] >> 13);
  const int64_t c0 = a.c * (int64_t)t_first;

  // position of the k-th set bit (k >= 1) of m, which has at least k
  auto kth_bit = [](uint64_t m, int k) -> int {
    int pos = 0;
#pragma unroll
    for (int w = 32; w >= 1; w >>= 1) {
      const uint64_t low = m & ((1ull << w) - 1);
      const int c = __builtin_popcountll(low);
      if (k > c) {
        k -= c;
        m >>= w;
        pos += w;
      } else {
        m = low;
      }
    }
    return pos;
  };
  auto bits_above = [](int d) -> uint64_t {  // lanes > d (d in -1 .. 63)
    return d < 0 ? ~0ull : (d >= 63 ? 0ull : ~((2ull << d) - 1));
  };

  // Span terms of one group end (the span runs to the next event time; the
  // last event has none).  They are added one chunk late, next to the next
  // chunk's scans, which do not depend on them.
  auto span_terms = [&](bool on, int t, int t_next, int cnt_p, uint32_t sum_p, uint32_t res_p,
                        int gmin, int gmax) {
    if (on) {
      // times < 2^19 and |S| <= 4,096: every factor below, and |S| times the
      // span, fit 32 bits, so each product is one 32 x 32 -> 64-bit multiply-add
      const uint32_t D = (uint32_t)(t_next - t);
      lD += D;
      if (cnt_p != 0) {
        const uint32_t s = (uint32_t)cnt_p;
        const uint32_t m0 = (uint32_t)(t - gmin + 1);
        const uint32_t sD = s * D;
        // per step of the span the largest footprint is m0, m0 + 1, ...: its sum
        // is D m0 + D (D - 1) / 2; the halves are taken once at the end
        lSMa += (uint64_t)D * m0;
        lSMb += (uint64_t)D * (D - 1u);
        lSSMa += (uint64_t)sD * m0;
        lSSMb += (uint64_t)sD * (D - 1u);
        // sum of (start - earliest start) over the active jobs: < 4,096 x 2^19
        lE += (uint64_t)D * (sum_p - s * (uint32_t)gmin);
        const int ext = gmax - gmin;
        lX += (uint64_t)D * (uint32_t)ext;
        lB += D;
        if (ext > alpha) {
          lU += D;
          lunf = true;
        }
        lXm = max(lXm, ext);
        lAm = max(lAm, cnt_p);
        lP = max(lP, s * (uint32_t)t_next - sum_p);
        if ((Bcap > 0) & (cnt_p > Bcap)) lcap = true;
        if ((M != 0) & (cnt_p >= 2) & ((int64_t)res_p > M)) lkv = true;
      }
    }
  };
  // the previous chunk's group ends, waiting for their span terms
  bool q_on = false;
  int q_t = 0, q_tn = 0, q_cnt = 0, q_gmin = 0, q_gmax = 0;
  uint32_t q_sum = 0, q_res = 0;
  // keys and lengths are loaded one chunk ahead
  uint32_t nkey = lane < NE ? EV[lane] : 0xFFFFFFFFu;
  int nlen = lane < NE ? (int)LEN[nkey & 0xFFFu] : 0;

  for (int base = 0; base < NE; base += WAVE) {
    const int p = base + lane;
    const bool valid = p < NE;
    const uint32_t key = nkey;
    const int len = nlen;
    const int pn = p + WAVE;
    nkey = pn < NE ? EV[pn] : 0xFFFFFFFFu;
    const int t = (int)(key >> 13);
    const bool is_start = valid & (((key >> 12) & 1u) != 0u);
    const bool is_end = valid & (((key >> 12) & 1u) == 0u);
    const int sj = is_start ? t : t - len;  // the job's start
    const int cnt_p = c_cnt + wave_scan_incl(is_start ? 1 : (is_end ? -1 : 0));
    // within a chunk the deltas sum to less than 64 x 2^20 in magnitude (times
    // < 2^19, lengths < 2^20): 32-bit scans on top of the 64-bit carries
    const uint32_t sum_p = c_sum + (uint32_t)wave_scan_incl(is_start ? sj : (is_end ? -sj : 0));
    const uint32_t res_p = c_res + (uint32_t)wave_scan_incl(is_start ? len : (is_end ? -len : 0));
    span_terms(q_on, q_t, q_tn, q_cnt, q_sum, q_res, q_gmin, q_gmax);
    nlen = pn < NE ? (int)LEN[nkey & 0xFFFu] : 0;
    // the next event's time: the lane above, and for the last lane the first
    // key of the next chunk
    int t_next = dpp<DPP_WAVE_SHL1, 0xf, 0xf, false>(t, t);
    const int t_first_next = (int)((uint32_t)readlane((int)nkey, 0) >> 13);
    if (lane == WAVE - 1) t_next = base + WAVE < NE ? t_first_next : t;
    const bool last = p == NE - 1;
    const bool gend = valid & (last | (t_next > t));
    // lane masks, each from one comparison (combined on the scalar unit)
    const int nv = NE - base;  // valid lanes: 0 .. nv - 1
    const uint64_t vmask = nv >= WAVE ? ~0ull : ((1ull << nv) - 1);
    const uint64_t smask = vmask & ballot((key & 0x1000u) != 0u);
    const uint64_t emask = vmask & ~smask;
    const uint64_t gmask = vmask & (ballot(t_next > t) | (nv <= WAVE ? 1ull << (nv - 1) : 0ull));
    uint64_t emin = emask & ballot(sj == min_s);
    uint64_t emax = emask & ballot(sj == max_s);
    // Common case, with no walk: the active set is never empty at a group end,
    // the earliest start keeps a job through the chunk, and the latest start
    // can only rise: it keeps a job until the chunk's first start (or a group
    // with starts is open from the previous chunk and ends in this one), and no
    // job started in the chunk ends in it while its start is the latest.  Then
    // the earliest start stays, and the latest start at a group end is the
    // later of the one carried in and the latest start time up to it (a prefix
    // max over the chunk; a group's starts come after its ends, so a group end
    // with starts is itself a start and takes its own time).
    int gmin, gmax;
    const int lat = wave_scan_incl_max(is_start ? t : -1);  // latest start time up to the lane
    const int fsl = smask ? __builtin_ctzll(smask) : WAVE;  // first start of the chunk
    const uint64_t pre = fsl >= WAVE ? ~0ull : ((1ull << fsl) - 1);
    const bool open_in = g_nst > 0;  // then the chunk begins with starts of that group
    const bool max_kept =
        open_in ? gmask != 0 : (nmax > 0 && __builtin_popcountll(emax & pre) < nmax);
    const bool fast = min_s != IDLE32 && nmin > 0 && max_kept && !(gmask & ballot(cnt_p == 0)) &&
                      __builtin_popcountll(emin) < nmin && !(emask & ballot(sj == lat));
    if (fast) {
      gmin = min_s;
      gmax = max(max_s, lat);
      nmin -= __builtin_popcountll(emin);
      const uint64_t sg = gmask & smask;  // group ends of groups with starts
      if (sg) {
        // the latest of them: its starts lie after the group end before it,
        // plus those of the previous chunk when it is the open group
        const int gL = 63 - __builtin_clzll(sg);
        const uint64_t below = gmask & ((1ull << gL) - 1);
        const uint64_t rng =
            bits_above(below ? 63 - __builtin_clzll(below) : -1) & (gL == 63 ? ~0ull : ((2ull << gL) - 1));
        max_s = readlane(t, gL);
        nmax = __builtin_popcountll(smask & rng) + (open_in && !below ? g_nst : 0);
        pmax = base + gL;
      } else {
        nmax -= __builtin_popcountll(emax);
      }
      // starts after the chunk's last group end open the next group
      const uint64_t st = smask & bits_above(gmask ? 63 - __builtin_clzll(gmask) : -1);
      g_nst = __builtin_popcountll(st);
      if (st) {
        gfirst = base + __builtin_ctzll(st);
        glast = base + 63 - __builtin_clzll(st);
      }
      if (gmask) cnt_last = readlane(cnt_p, 63 - __builtin_clzll(gmask));
    } else {
      const int min0 = min_s, max0 = max_s;  // in force before the chunk's first visit
      uint64_t chg = 0;                      // visited group ends
      int vmin = 0, vmax = 0;                // values set there
      int done = -1;                         // lanes <= done are accounted for
      bool open = g_nst > 0;                 // the first group of the chunk began earlier
      while (true) {
        const uint64_t after = bits_above(done);
        const uint64_t ge = gmask & after;
        if (!ge) break;
        // the earliest position after `done` at which something can change
        int x = WAVE;
        if (open || (min_s != IDLE32 && nmin <= 0) || (max_s >= 0 && nmax <= 0)) x = 0;
        const uint64_t sa = smask & after;
        if (sa) x = min(x, __builtin_ctzll(sa));
        if (min_s != IDLE32) {
          const uint64_t ea = emin & after;
          if (__builtin_popcountll(ea) >= nmin && nmin > 0) x = min(x, kth_bit(ea, nmin));
        }
        if (max_s >= 0) {
          const uint64_t ea = emax & after;
          if (__builtin_popcountll(ea) >= nmax && nmax > 0) x = min(x, kth_bit(ea, nmax));
        }
        if (x == WAVE) break;
        const uint64_t gx = ge & ~((1ull << x) - 1);
        if (!gx) break;  // the group ends in the next chunk
        const int gL = __builtin_ctzll(gx);
        const uint64_t rng = after & (gL == 63 ? ~0ull : ((2ull << gL) - 1));
        const int tg = readlane(t, gL);
        const int cnt_g = readlane(cnt_p, gL);
        // |S| before this group: at the previous group end
        const uint64_t gprev = gmask & ((1ull << gL) - 1);
        const int cnt_before = gprev ? readlane(cnt_p, 63 - __builtin_clzll(gprev)) : cnt_last;
        nmin -= __builtin_popcountll(emin & rng);
        nmax -= __builtin_popcountll(emax & rng);
        const uint64_t sr = smask & rng;
        const bool with_open = open && !gprev;
        const int nst = __builtin_popcountll(sr) + (with_open ? g_nst : 0);
        if (nst > 0) {
          const int gf = with_open ? gfirst : base + __builtin_ctzll(sr);
          const int gl = sr ? base + 63 - __builtin_clzll(sr) : glast;
          if (cnt_before == 0) {
            min_s = tg;
            nmin = nst;
            pmin = gf;
          }
          max_s = tg;
          nmax = nst;
          pmax = gl;
        }
        open = open && gprev;  // a group end before gL closed the open group
        if (with_open) open = false;
        const int gpos = base + gL;
        if (cnt_g == 0) {
          min_s = IDLE32;
          max_s = -1;
          nmin = nmax = 0;
        } else {
          if (nmin <= 0) {
            // first active start event at or after pmin; then count the active
            // ones at that time
            int q = max(pmin, 0), found = -1, cnt = 0;
            while (q <= gpos) {
              const int ee = q + lane;
              bool ok = false;
              int st_time = 0;
              if (ee >= 0 && ee <= gpos) {
                const uint32_t kk = EV[ee];
                st_time = (int)(kk >> 13);
                ok = ((kk >> 12) & 1u) && st_time + LEN[kk & 0xFFFu] > tg;
              }
              if (found < 0) {
                const uint64_t hm = ballot(ok);
                if (hm) {
                  const int L = __builtin_ctzll(hm);
                  found = q + L;
                  min_s = readlane(st_time, L);
                }
              }
              if (found >= 0) {
                cnt += __builtin_popcountll(ballot(ok & (st_time == min_s)));
                if (ballot((ee >= 0) & (ee <= gpos) & (st_time > min_s))) break;
              }
              q += WAVE;
            }
            pmin = found;
            nmin = cnt;
          }
          if (nmax <= 0) {
            // last active start event at or before pmax; then count the active
            // ones at that time
            int q = pmax, found = -1, cnt = 0;
            while (q >= 0) {
              const int ee = q - lane;
              bool ok = false;
              int st_time = 0;
              if (ee >= 0) {
                const uint32_t kk = EV[ee];
                st_time = (int)(kk >> 13);
                ok = ((kk >> 12) & 1u) && st_time + LEN[kk & 0xFFFu] > tg;
              }
              if (found < 0) {
                const uint64_t hm = ballot(ok);
                if (hm) {
                  const int L = __builtin_ctzll(hm);
                  found = q - L;
                  max_s = readlane(st_time, L);
                }
              }
              if (found >= 0) {
                cnt += __builtin_popcountll(ballot(ok & (st_time == max_s)));
                if (ballot((ee >= 0) & (st_time < max_s))) break;
              }
              q -= WAVE;
            }
            pmax = found;
            nmax = cnt;
          }
        }
        chg |= 1ull << gL;
        if (lane == gL) {
          vmin = min_s;
          vmax = max_s;
        }
        emin = emask & ballot(sj == min_s);
        emax = emask & ballot(sj == max_s);
        done = gL;
      }
      // the rest of the chunk: groups with nothing to change, then the open group
      {
        const uint64_t after = bits_above(done);
        nmin -= __builtin_popcountll(emin & after);
        nmax -= __builtin_popcountll(emax & after);
        const uint64_t glast_m = gmask & after;
        if (glast_m) open = false;
        const uint64_t tail = bits_above(gmask ? 63 - __builtin_clzll(gmask) : -1) & after;
        const uint64_t st = smask & tail;
        if (st) {
          if (!open) {
            g_nst = 0;
            gfirst = base + __builtin_ctzll(st);
          }
          g_nst += __builtin_popcountll(st);
          glast = base + 63 - __builtin_clzll(st);
          open = true;
        }
        if (!open) g_nst = 0;
        if (gmask) cnt_last = readlane(cnt_p, 63 - __builtin_clzll(gmask));
      }
      // earliest / latest start in force at each group end of the chunk
      {
        const uint64_t upto = lane == 63 ? ~0ull : ((2ull << lane) - 1);
        const uint64_t c = chg & upto;
        const int src = c ? 63 - __builtin_clzll(c) : 0;
        const int fmin = __shfl(vmin, src), fmax = __shfl(vmax, src);
        gmin = c ? fmin : min0;
        gmax = c ? fmax : max0;
      }
    }
    q_on = gend & !last;
    q_t = t;
    q_tn = t_next;
    q_cnt = cnt_p;
    q_sum = sum_p;
    q_res = res_p;
    q_gmin = gmin;
    q_gmax = gmax;
    c_cnt = readlane(cnt_p, 63);
    c_sum = (uint32_t)readlane((int)sum_p, 63);
    c_res = (uint32_t)readlane((int)res_p, 63);
  }
  span_terms(q_on, q_t, q_tn, q_cnt, q_sum, q_res, q_gmin, q_gmax);
  const int64_t acc_E = wave_sum64((int64_t)lE);
  const int64_t sD = wave_sum((int)lD);  // the busy and idle steps after the first event
  const int64_t SSM = wave_sum64((int64_t)lSSMa) + wave_sum64((int64_t)lSSMb) / 2;
  const int64_t SM = wave_sum64((int64_t)lSMa) + wave_sum64((int64_t)lSMb) / 2;
  const int64_t acc_C = c0 + a.c * sD + a.tau * SSM;
  const int64_t acc_W = c0 + a.c * sD + a.tau * SM;
  const int64_t acc_ext = wave_sum64((int64_t)lX);
  const int64_t acc_busy = wave_sum((int)lB);
  const int64_t acc_unf = wave_sum((int)lU);
  const int64_t acc_peak = wave_max((int)lP);  // below 4,096 x 2^19
  const int acc_maxext = wave_max(lXm);
  const int acc_maxact = wave_max(lAm);
  if (ballot(lunf)) v |= 8u;
  if (ballot(lcap)) v |= 2u;
  if (ballot(lkv)) v |= 4u;

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

hipError_t launch_decompose(const DecArgs& a, bool narrow, int wpb, size_t lds, hipStream_t s) {
  const int64_t blocks = (a.n_inst + wpb - 1) / wpb;
  if (narrow)
    hipLaunchKernelGGL(decompose_kernel<true>, dim3((unsigned)blocks), dim3((unsigned)(wpb * WAVE)),
                       lds, s, a);
  else
    hipLaunchKernelGGL(decompose_kernel<false>, dim3((unsigned)blocks),
                       dim3((unsigned)(wpb * WAVE)), lds, s, a);
  return hipGetLastError();
}

}  // namespace fs
