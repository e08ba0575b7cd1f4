// Exact alpha-fair optimum makespan for tiny instances (n <= 8): one wavefront
// per instance.
//
// Definition (Appendix A's integer program, with release steps and the KV
// budget added): the least makespan over start vectors with s_i >= r_i, at most
// B jobs active per step, reservations within M_kv unless a job runs alone, and
// |s_i - s_j| <= alpha for every pair active at a common step.
//
// Search.  Schedules are enumerated in start order: after placing a job at
// step sigma, the future depends only on (placed set, sigma clipped to the last
// release, progress of every job still active at sigma), because later jobs
// start at or after sigma and jobs that ended before sigma constrain nothing.
// From such a state the next job k starts after a delay d >= 0, bounded by the
// step at which the machine is empty and every job has been released (waiting
// longer with an empty machine can be removed by shifting the rest earlier).
// Among identical unstarted jobs only the lowest index may start next.
// V(state) = min over (k, d) of d + V(child) is computed by a depth-first
// search (depth <= n) whose memo keeps, per state, either the exact value or a
// lower bound, so a child is explored with the bound "best so far - d" and
// children whose lower bound d + LB(child) cannot beat it are skipped
// (LB = max of: longest remaining active job, latest finish of an unstarted job
// if started at once, total remaining work / B).  The root bound is the ISJL
// makespan of the instance (written into T_opt by a simulation launch just
// before this kernel): the search returns a smaller value only if a better
// schedule exists.
//
// Wave organisation: the state and the DFS control are uniform; the 64 lanes
// evaluate candidate (k, d) pairs in parallel (candidate c: d = c / 8,
// k = c % 8) and pick the next one with a wave minimum over packed keys
// (lb << 16 | d << 3 | k); the memo is an LDS hash table probed 64 slots at a
// time; the DFS stack and the per-frame candidate keys live in LDS.
#include "opt_common.hpp"
#include "wave.hpp"

namespace fs {

namespace {

constexpr int NMAX = 8;
constexpr int MEMO_BYTES = 32768;     // LDS memo bytes per wave (first pass)
constexpr int FRAMES = NMAX + 2;      // DFS depth <= n, plus the root
constexpr int FW = 8;                 // words per frame
constexpr int CACHE = 192;            // cached candidate keys per frame (3 per lane)
constexpr uint32_t NOKEY = 0xFFFFFFFFu;
constexpr int GUARD = 1 << 22;        // DFS pushes per search in the first pass

// frame word offsets
enum { F_S = 0, F_SIG, F_PLO, F_PHI, F_BOUND, F_BEST, F_THR, F_FLAGS };
// flags: bit 0 entered, bit 1 keys cached, bits 8.. dhi

struct Inst {
  int n, B, alpha, rmax;
  int64_t M;
  int len[NMAX], arr[NMAX];
  uint32_t eqprev[NMAX];
  uint32_t compat[NMAX];  // jobs that may run beside job j under the KV budget
  uint32_t full;
  bool compact;           // B <= 3 and every arrival 0: 64-bit memo entries
};

__device__ __forceinline__ int prog_of(uint32_t plo, uint32_t phi, int j) {
  return (int)(((j < 4 ? plo >> (8 * j) : phi >> (8 * (j - 4)))) & 0xFFu);
}

// Key of candidate c from state (S, sig, progress); NOKEY if inadmissible.
__device__ inline uint32_t cand_key(const Inst& I, uint32_t S, int sig, uint32_t plo,
                                    uint32_t phi, int c, int dhi, int sumU) {
  const int d = c >> 3, k = c & 7;
  if (k >= I.n || d > dhi || ((S >> k) & 1u)) return NOKEY;
  int lk = 0, ak = 0;
  uint32_t eq = 0;
#pragma unroll
  for (int j = 0; j < NMAX; ++j)
    if (j == k) {
      lk = I.len[j];
      ak = I.arr[j];
      eq = I.eqprev[j];
    }
  if ((S & eq) != eq) return NOKEY;  // a lower identical job is still unstarted
  if (d < ak - sig) return NOKEY;    // not released yet
  int cnt = 0, maxp = 0, maxrem = lk, sumrem = lk;
  int64_t sumlen = 0;
#pragma unroll
  for (int j = 0; j < NMAX; ++j) {
    const int p = prog_of(plo, phi, j);
    if (p != 0xFF) {
      const int rem = I.len[j] - p;
      if (rem > d) {
        cnt++;
        maxp = max(maxp, p + d);
        sumlen += I.len[j];
        maxrem = max(maxrem, rem - d);
        sumrem += rem - d;
      }
    }
  }
  if (cnt > I.B - 1) return NOKEY;
  if (cnt > 0 && maxp > I.alpha) return NOKEY;
  if (I.M != 0 && cnt > 0 && sumlen + lk > I.M) return NOKEY;
  const int sig2 = sig + d;
  int maxu = 0;
  uint32_t R = 0;  // jobs with work left after the start of k
#pragma unroll
  for (int j = 0; j < NMAX; ++j) {
    if (j < I.n && j != k && !((S >> j) & 1u)) {
      maxu = max(maxu, max(0, I.arr[j] - sig2) + I.len[j]);
      R |= 1u << j;
    }
    const int p = prog_of(plo, phi, j);
    if (p != 0xFF && I.len[j] - p > d) R |= 1u << j;
  }
  R |= 1u << k;
  // A job that fits beside no other remaining job (KV budget, or B = 1) runs
  // alone: its remaining steps are serial with everything else.
  int alone = 0;
#pragma unroll
  for (int j = 0; j < NMAX; ++j) {
    if (((R >> j) & 1u) && (I.compat[j] & R & ~(1u << j)) == 0u) {
      const int p = prog_of(plo, phi, j);
      int rj = I.len[j];
      if (j != k && p != 0xFF) rj = I.len[j] - p - d;
      alone += rj;
    }
  }
  const int work = sumrem + sumU - lk;
  const int lb = max(max(maxrem, maxu), alone + (work - alone + I.B - 1) / I.B);
  return ((uint32_t)(d + lb) << 16) | ((uint32_t)d << 3) | (uint32_t)k;
}

__device__ __forceinline__ uint32_t mix(uint32_t k0, uint32_t k1, uint32_t k2) {
  uint32_t h = k0 * 0x9E3779B1u ^ (k1 + 0x7F4A7C15u) * 0x85EBCA77u ^ (k2 + 0x165667B1u) * 0xC2B2AE3Du;
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  h ^= h >> 12;
  return h;
}

// The memo: a hash table probed 64 slots at a time.  The first pass keeps it in
// LDS; the second pass in its own region of global scratch, read and written
// with agent-scope accesses (they bypass the vector L1, so a lane reads what
// another lane of the wave stored).
struct Memo {
  uint32_t* base;
  bool compact;  // one 64-bit word per entry (LDS only), else 4 words per entry
  bool global;
  int entries;   // power of two

  __device__ uint32_t ld(const uint32_t* p) const {
    if (global) return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return *p;
  }
  __device__ void st(uint32_t* p, uint32_t v) const {
    if (global) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else *p = v;
  }
  // every lane sees the stores of the wave before its next probe
  __device__ void sync() const {
    if (global) __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "agent");
    wave_lds_sync();
  }

  // Compact key: valid | S | up to three active (index, progress) pairs in index order.
  __device__ static uint64_t ckey(uint32_t S, uint32_t plo, uint32_t phi) {
    uint64_t slots = 0;
    int c = 0;
#pragma unroll
    for (int j = 0; j < NMAX; ++j) {
      const int p = prog_of(plo, phi, j);
      if (p != 0xFF && c < 3) {
        slots |= (uint64_t)((j << 8) | p) << (11 * c);
        c++;
      }
    }
    for (int q = c; q < 3; ++q) slots |= (uint64_t)0x7FFu << (11 * q);
    return (1ull << 63) | ((uint64_t)S << 55) | (slots << 16);
  }

  // value | exact << 31, or NOKEY if absent
  __device__ uint32_t get(uint32_t a, uint32_t b, uint32_t c, uint32_t S, int lane) const {
    if (compact) {
      const uint64_t key = ckey(S, b, c);
      const uint64_t* T = (const uint64_t*)base;
      const uint32_t h = mix((uint32_t)(key >> 32), (uint32_t)key, 0u);
      const int slot = (int)((h + (uint32_t)lane) & (uint32_t)(entries - 1));
      const uint64_t x = T[slot];
      const bool hit = (x >> 16) == (key >> 16);
      const bool empty = x == 0ull;
      const uint64_t mh = ballot(hit), me = ballot(empty);
      if (!mh) return NOKEY;
      const int L = __builtin_ctzll(mh);
      if (me && __builtin_ctzll(me) < L) return NOKEY;
      const uint32_t v = (uint32_t)readlane((int)(uint32_t)(x & 0xFFFFu), L);
      return (v & 0x7FFFu) | ((v & 0x8000u) << 16);
    }
    const uint32_t* k0 = base;
    const uint32_t* k1 = base + entries;
    const uint32_t* k2 = base + 2 * (size_t)entries;
    const uint32_t* val = base + 3 * (size_t)entries;
    const uint32_t h = mix(a, b, c);
    const int slot = (int)((h + (uint32_t)lane) & (uint32_t)(entries - 1));
    const uint32_t x = ld(k0 + slot);
    const bool hit = x == a && ld(k1 + slot) == b && ld(k2 + slot) == c;
    const bool empty = x == 0u;
    const uint64_t mh = ballot(hit), me = ballot(empty);
    if (!mh) return NOKEY;
    const int L = __builtin_ctzll(mh);
    if (me && __builtin_ctzll(me) < L) return NOKEY;  // keys sit before any hole
    return (uint32_t)readlane((int)ld(val + slot), L);
  }

  __device__ void put(uint32_t a, uint32_t b, uint32_t c, uint32_t S, uint32_t v, int lane) {
    if (compact) {
      const uint64_t key = ckey(S, b, c);
      uint64_t* T = (uint64_t*)base;
      const uint32_t h = mix((uint32_t)(key >> 32), (uint32_t)key, 0u);
      const int slot = (int)((h + (uint32_t)lane) & (uint32_t)(entries - 1));
      const uint64_t x = T[slot];
      const bool hit = (x >> 16) == (key >> 16);
      const bool empty = x == 0ull;
      const uint64_t mh = ballot(hit), me = ballot(empty);
      const int L = mh ? __builtin_ctzll(mh) : (me ? __builtin_ctzll(me) : 0);
      const uint64_t e = key | (uint64_t)((v & 0x7FFFu) | ((v >> 16) & 0x8000u));
      if (lane == L) T[slot] = e;
      wave_lds_sync();
      return;
    }
    uint32_t* k0 = base;
    uint32_t* k1 = base + entries;
    uint32_t* k2 = base + 2 * (size_t)entries;
    uint32_t* val = base + 3 * (size_t)entries;
    const uint32_t h = mix(a, b, c);
    const int slot = (int)((h + (uint32_t)lane) & (uint32_t)(entries - 1));
    const uint32_t x = ld(k0 + slot);
    const bool hit = x == a && ld(k1 + slot) == b && ld(k2 + slot) == c;
    const bool empty = x == 0u;
    const uint64_t mh = ballot(hit), me = ballot(empty);
    int L;
    if (mh) L = __builtin_ctzll(mh);
    else if (me) L = __builtin_ctzll(me);
    else L = 0;  // probe window full: replace the home slot
    if (lane == L) {
      st(k0 + slot, a);
      st(k1 + slot, b);
      st(k2 + slot, c);
      st(val + slot, v);
    }
    sync();
  }

  __device__ void clear(int lane) {
    const size_t words = compact ? 2 * (size_t)entries : 4 * (size_t)entries;
    for (size_t i = (size_t)lane; i < words; i += WAVE) st(base + i, 0u);
    sync();
  }
};

struct Dfs {
  const Inst& I;
  Memo& memo;
  uint32_t* F;      // FRAMES * FW words
  uint32_t* keys;   // FRAMES * CACHE candidate keys
  int lane;

  __device__ uint32_t frame(int depth, int f) const { return F[depth * FW + f]; }
  __device__ void set(int depth, int f, uint32_t v) {
    if (lane == 0) F[depth * FW + f] = v;
  }

  // state-dependent scalars
  __device__ void state_info(uint32_t S, int sig, uint32_t plo, uint32_t phi, int& dhi,
                             int& sumU) const {
    int maxrem = 0, late = 0;
    sumU = 0;
#pragma unroll
    for (int j = 0; j < NMAX; ++j) {
      const int p = prog_of(plo, phi, j);
      if (p != 0xFF) maxrem = max(maxrem, I.len[j] - p);
      if (j < I.n && !((S >> j) & 1u)) {
        sumU += I.len[j];
        late = max(late, I.arr[j] - sig);
      }
    }
    dhi = max(maxrem, late);
  }

  // smallest candidate key > thr (NOKEY if none)
  __device__ uint32_t pick(int depth, uint32_t S, int sig, uint32_t plo, uint32_t phi,
                           uint32_t flags, uint32_t thr) const {
    const int dhi = (int)(flags >> 8);
    uint32_t best = NOKEY;
    if (flags & 2u) {
      const uint32_t* K = keys + depth * CACHE;
#pragma unroll
      for (int i = 0; i < CACHE / WAVE; ++i) {
        const uint32_t k = K[i * WAVE + lane];
        if (k > thr && k < best) best = k;
      }
    } else {
      int dd, sumU;
      state_info(S, sig, plo, phi, dd, sumU);
      const int nc = (dhi + 1) * 8;
      for (int c0 = 0; c0 < nc; c0 += WAVE) {
        const uint32_t k = cand_key(I, S, sig, plo, phi, c0 + lane, dhi, sumU);
        if (k > thr && k < best) best = k;
      }
    }
    return wave_umin(best);
  }

  // V(root) if it is below `bound`, else a value >= bound; -1 after more than
  // `guard_max` pushes.
  __device__ int run(uint32_t S0, int sig0, uint32_t plo0, uint32_t phi0, int bound0,
                     int guard_max) {
    int depth = 0;
    set(0, F_S, S0);
    set(0, F_SIG, (uint32_t)sig0);
    set(0, F_PLO, plo0);
    set(0, F_PHI, phi0);
    set(0, F_BOUND, (uint32_t)bound0);
    set(0, F_FLAGS, 0u);
    wave_lds_sync();
    int guard = 0;
    while (true) {
      const uint32_t S = frame(depth, F_S);
      const int sig = (int)frame(depth, F_SIG);
      const uint32_t plo = frame(depth, F_PLO), phi = frame(depth, F_PHI);
      const int bound = (int)frame(depth, F_BOUND);
      uint32_t flags = frame(depth, F_FLAGS);
      int ret = -1;
      const uint32_t ka = 1u | (S << 1) | ((uint32_t)min(sig, I.rmax) << 9);
      if (!(flags & 1u)) {
        if (S == I.full) {
          int mr = 0;
#pragma unroll
          for (int j = 0; j < NMAX; ++j) {
            const int p = prog_of(plo, phi, j);
            if (p != 0xFF) mr = max(mr, I.len[j] - p);
          }
          ret = mr;
        } else {
          const uint32_t v = memo.get(ka, plo, phi, S, lane);
          if (v != NOKEY && ((v >> 31) || (int)(v & 0x7FFFFFFFu) >= bound)) {
            ret = (int)(v & 0x7FFFFFFFu);
          } else {
            int dhi, sumU;
            state_info(S, sig, plo, phi, dhi, sumU);
            flags = 1u | ((uint32_t)dhi << 8);
            if ((dhi + 1) * 8 <= CACHE) {
              flags |= 2u;
              uint32_t* K = keys + depth * CACHE;
#pragma unroll
              for (int i = 0; i < CACHE / WAVE; ++i)
                K[i * WAVE + lane] = cand_key(I, S, sig, plo, phi, i * WAVE + lane, dhi, sumU);
            }
            set(depth, F_FLAGS, flags);
            set(depth, F_BEST, (uint32_t)bound);
            set(depth, F_THR, 0u);
            wave_lds_sync();
          }
        }
      }
      if (ret < 0) {
        const int best = (int)frame(depth, F_BEST);
        const uint32_t thr = frame(depth, F_THR);
        const uint32_t key = pick(depth, S, sig, plo, phi, flags, thr);
        if (key != NOKEY && (int)(key >> 16) < best && depth + 1 < FRAMES) {
          const int d = (int)((key >> 3) & 0x1FFFu), k = (int)(key & 7u);
          uint32_t nlo = 0, nhi = 0;
#pragma unroll
          for (int j = 0; j < NMAX; ++j) {
            int p = prog_of(plo, phi, j);
            int q = 0xFF;
            if (j == k) q = 0;
            else if (p != 0xFF && I.len[j] - p > d) q = p + d;
            if (j < 4) nlo |= (uint32_t)q << (8 * j);
            else nhi |= (uint32_t)q << (8 * (j - 4));
          }
          set(depth, F_THR, key);
          set(depth + 1, F_S, S | (1u << k));
          set(depth + 1, F_SIG, (uint32_t)(sig + d));
          set(depth + 1, F_PLO, nlo);
          set(depth + 1, F_PHI, nhi);
          set(depth + 1, F_BOUND, (uint32_t)(best - d));
          set(depth + 1, F_FLAGS, 0u);
          wave_lds_sync();
          depth++;
          if (++guard > guard_max) return -1;
          continue;
        }
        memo.put(ka, plo, phi, S, (uint32_t)best | ((best < bound) ? 0x80000000u : 0u), lane);
        ret = best;
      }
      if (depth == 0) return ret;
      depth--;
      const uint32_t pthr = frame(depth, F_THR);
      const int pd = (int)((pthr >> 3) & 0x1FFFu);
      const int pbest = (int)frame(depth, F_BEST);
      if (ret + pd < pbest) set(depth, F_BEST, (uint32_t)(ret + pd));
      wave_lds_sync();
    }
  }
};

// Read instance `inst` into I.  False (after writing the marker) when a length
// or an arrival is beyond the search's limits.
__device__ bool load_inst(const OptArgs& a, int64_t inst, int lane, Inst& I) {
  const int n = a.n;
  const int64_t row = inst * (int64_t)n;
  int lv = 0, av = 0, bad = 0;
  if (lane < n) {
    lv = a.prompt[row + lane] + a.output[row + lane];
    av = a.arrival[row + lane];
    bad = (lv > OPT_LEN_LIMIT) || (av > OPT_ARR_LIMIT);
  }
  if (ballot(bad != 0)) {
    if (lane == 0) a.T[inst] = FSCHED_T_TOOLARGE;
    return false;
  }
  I.n = n;
  I.B = a.B;
  I.alpha = a.alpha;
  I.M = a.M;
  I.rmax = 0;
#pragma unroll
  for (int j = 0; j < NMAX; ++j) {
    I.len[j] = j < n ? readlane(lv, j) : 0;
    I.arr[j] = j < n ? readlane(av, j) : 0;
    I.rmax = max(I.rmax, I.arr[j]);
  }
#pragma unroll
  for (int k = 0; k < NMAX; ++k) {
    uint32_t e = 0;
#pragma unroll
    for (int j = 0; j < NMAX; ++j)
      if (j < k && k < n && I.len[j] == I.len[k] && I.arr[j] == I.arr[k]) e |= 1u << j;
    I.eqprev[k] = e;
  }
  I.full = (n >= 32) ? 0xFFFFFFFFu : ((1u << n) - 1u);
#pragma unroll
  for (int j = 0; j < NMAX; ++j) {
    uint32_t c = 0;
#pragma unroll
    for (int i = 0; i < NMAX; ++i)
      if (i != j && i < n && j < n && I.B > 1 &&
          (I.M == 0 || (int64_t)I.len[i] + I.len[j] <= I.M))
        c |= 1u << i;
    I.compat[j] = c;
  }
  I.compact = I.B <= 3 && I.rmax == 0;
  return true;
}

// Search instance `inst` below its incumbent (the ISJL makespan in T) and, when
// something better exists, write the optimum and one optimal schedule.  False
// if the search made more than `guard_max` pushes (nothing written then).
__device__ bool solve(const OptArgs& a, int64_t inst, const Inst& I, Memo& memo, uint32_t* frames,
                      uint32_t* keys, int lane, int guard_max) {
  const int64_t row = inst * (int64_t)a.n;
  Dfs dfs{I, memo, frames, keys, lane};
  const uint32_t none = 0xFFFFFFFFu;
  const int bound = (int)a.T[inst];
  const int v = dfs.run(0u, 0, none, none, bound, guard_max);
  if (v < 0) return false;
  if (v >= bound) return true;  // ISJL's schedule (already written) is optimal

  if (lane == 0) a.T[inst] = v;
  if (!a.start) return true;
  // Reconstruct one optimal schedule: from each state take the first candidate
  // (in key order) whose child reaches the state's value.
  uint32_t S = 0u, plo = none, phi = none;
  int sig = 0, val = v;
  int steps = 0;
  while (S != I.full && steps < 2 * NMAX) {
    steps++;
    int dhi, sumU;
    dfs.state_info(S, sig, plo, phi, dhi, sumU);
    const uint32_t flags = 1u | ((uint32_t)dhi << 8);  // no cache: frame 0 is reused below
    uint32_t thr = 0u;
    bool moved = false;
    while (true) {
      const uint32_t key = dfs.pick(FRAMES - 1, S, sig, plo, phi, flags, thr);
      if (key == NOKEY || (int)(key >> 16) > val) break;
      thr = key;
      const int d = (int)((key >> 3) & 0x1FFFu), k = (int)(key & 7u);
      uint32_t nlo = 0, nhi = 0;
#pragma unroll
      for (int j = 0; j < NMAX; ++j) {
        int p = prog_of(plo, phi, j);
        int q = 0xFF;
        if (j == k) q = 0;
        else if (p != 0xFF && I.len[j] - p > d) q = p + d;
        if (j < 4) nlo |= (uint32_t)q << (8 * j);
        else nhi |= (uint32_t)q << (8 * (j - 4));
      }
      const int cv = dfs.run(S | (1u << k), sig + d, nlo, nhi, val - d + 1, guard_max);
      if (cv >= 0 && cv + d == val) {
        if (lane == 0) a.start[row + k] = sig + d;
        S |= 1u << k;
        sig += d;
        plo = nlo;
        phi = nhi;
        val -= d;
        moved = true;
        break;
      }
    }
    if (!moved) break;  // not reachable: some child always attains the value
  }
  return true;
}

}  // namespace

__global__ __launch_bounds__(256) void opt_kernel(OptArgs a) {
  extern __shared__ uint32_t lds_raw[];
  const int wib = threadIdx.x >> 6;
  const int64_t inst = (int64_t)blockIdx.x * (blockDim.x >> 6) + wib;
  if (inst >= a.n_inst) return;
  const int lane = lane_id();
  uint32_t* base = lds_raw + (size_t)wib * (size_t)a.wave_words;
  uint32_t* frames = base + MEMO_BYTES / 4;
  uint32_t* keys = frames + FRAMES * FW;

  if (a.T[inst] < 0) return;  // ISJL's error marker
  Inst I;
  if (!load_inst(a, inst, lane, I)) return;
  Memo memo{base, I.compact, false, I.compact ? MEMO_BYTES / 8 : MEMO_BYTES / 16};
  memo.clear(lane);
  if (!solve(a, inst, I, memo, frames, keys, lane, GUARD)) {
    // the LDS memo was too small for this search: leave it to the second pass
    if (lane == 0) {
      if (a.fb_list) {
        const int slot = atomicAdd(a.fb_count, 1);
        a.fb_list[slot] = (int32_t)inst;
      } else {
        a.T[inst] = FSCHED_T_INTERNAL;
      }
    }
  }
}

// Second pass: OPT_FB_WAVES persistent waves take the listed instances one at a
// time (claimed with an atomic counter) and search them again with a memo of
// OPT_FB_MEMO_ENTRIES entries in their own region of global scratch.  Every
// wave leaves once the list is exhausted.
__global__ __launch_bounds__(64) void opt_fallback_kernel(OptArgs a) {
  extern __shared__ uint32_t lds_raw[];
  const int lane = lane_id();
  uint32_t* frames = lds_raw;
  uint32_t* keys = frames + FRAMES * FW;
  const int nlist = __hip_atomic_load(a.fb_count, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  Memo memo{a.fb_memo + (size_t)blockIdx.x * 4 * (size_t)OPT_FB_MEMO_ENTRIES, false, true,
            OPT_FB_MEMO_ENTRIES};
  while (true) {
    int idx = 0;
    if (lane == 0) idx = atomicAdd(a.fb_count + 1, 1);
    idx = readlane(idx, 0);
    if (idx >= nlist) break;
    const int64_t inst = a.fb_list[idx];
    Inst I;
    if (!load_inst(a, inst, lane, I)) continue;
    memo.clear(lane);
    if (!solve(a, inst, I, memo, frames, keys, lane, OPT_FB_GUARD))
      if (lane == 0) a.T[inst] = FSCHED_T_INTERNAL;
  }
}

hipError_t launch_opt(const OptArgs& a, int wpb, size_t lds, hipStream_t s) {
  const int64_t blocks = (a.n_inst + wpb - 1) / wpb;
  hipLaunchKernelGGL(opt_kernel, dim3((unsigned)blocks), dim3((unsigned)(wpb * WAVE)), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_opt_fallback(const OptArgs& a, size_t lds, hipStream_t s) {
  hipLaunchKernelGGL(opt_fallback_kernel, dim3((unsigned)OPT_FB_WAVES), dim3((unsigned)WAVE), lds,
                     s, a);
  return hipGetLastError();
}

size_t opt_lds_words_per_wave() { return MEMO_BYTES / 4 + FRAMES * FW + FRAMES * CACHE; }

size_t opt_fallback_lds_words_per_wave() { return FRAMES * FW + FRAMES * CACHE; }

}  // namespace fs
