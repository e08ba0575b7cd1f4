// C ABI of libfsched: argument checks, launch configuration, host staging.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <algorithm>
#include <cstring>
#include <mutex>

#include "fsched.h"
#include "sim_common.hpp"
#include "dec_common.hpp"
#include "opt_common.hpp"
#include "abi_internal.hpp"

namespace {

thread_local int g_last_hip = 0;

int hip_fail(hipError_t e) {
  g_last_hip = (int)e;
  return e == hipErrorOutOfMemory ? FSCHED_ENOMEM : FSCHED_EDEVICE;
}

// floor((sqrt(17) - 1) alpha / 4): the largest k >= 0 with (4k + alpha)^2 <= 17 alpha^2.
int32_t beta_sqrt17(int32_t alpha) {
  long double approx = (sqrtl(17.0L) - 1.0L) * (long double)alpha / 4.0L;
  int64_t k = (int64_t)approx;
  if (k < 0) k = 0;
  auto ok = [&](int64_t x) {
    __int128 v = (__int128)(4 * x + alpha);
    return v * v <= (__int128)17 * alpha * alpha;
  };
  while (ok(k + 1)) ++k;
  while (k > 0 && !ok(k)) --k;
  return (int32_t)k;
}

int check_params(const fsched_params* p, bool need_policy) {
  if (!p) return FSCHED_EINVAL;
  if (p->B < 0 || p->alpha < 0 || p->M_kv < 0 || p->cost_c < 0 || p->cost_tau < 0)
    return FSCHED_EINVAL;
  if (need_policy && (p->policy < FSCHED_FCFS || p->policy > FSCHED_SJF)) return FSCHED_EINVAL;
  const uint32_t known =
      FSCHED_F_DEVICE_PTRS | FSCHED_F_SYNC | FSCHED_F_BETA_SQRT17 | FSCHED_F_RESUME_FILL |
      FSCHED_F_PREFILL;
  if (p->flags & ~known) return FSCHED_EINVAL;
  return FSCHED_OK;
}

int next_pow2(int x) {
  int p = 64;
  while (p < x) p <<= 1;
  return p;
}

// Map the per-instance markers of a finished host-mode call to a return code.
int markers_to_code(const fsched_metrics* out, int64_t n_inst) {
  int rc = FSCHED_OK;
  for (int64_t i = 0; i < n_inst; ++i) {
    int64_t T = out[i].T;
    if (T >= 0) continue;
    if (T == FSCHED_T_INVALID) return FSCHED_EINVAL;
    if (T == FSCHED_T_RANGE) rc = FSCHED_ERANGE;
    else if (T == FSCHED_T_TOOLARGE && rc == FSCHED_OK) rc = FSCHED_ETOOLARGE;
    else if (rc == FSCHED_OK) rc = FSCHED_EINTERNAL;
  }
  return rc;
}

// Device copies of the host arrays of one call (host mode).
struct Staging {
  void* ptr[8] = {nullptr};
  int n = 0;
  hipError_t err = hipSuccess;
  void* alloc(size_t bytes) {
    void* d = nullptr;
    if (err == hipSuccess) err = hipMalloc(&d, bytes ? bytes : 1);
    if (err != hipSuccess) return nullptr;
    ptr[n++] = d;
    return d;
  }
  void* upload(const void* h, size_t bytes) {
    void* d = alloc(bytes);
    if (d && bytes) err = hipMemcpy(d, h, bytes, hipMemcpyHostToDevice);
    return err == hipSuccess ? d : nullptr;
  }
  ~Staging() {
    for (int i = 0; i < n; ++i) (void)hipFree(ptr[i]);
  }
};

// Pool of the rank scratch (2 bytes per job) of the current device, created
// once: allocations are stream-ordered, and what a call frees stays in the pool
// (release threshold: never) so that repeated calls allocate nothing new.
// Null when the device cannot make one (or, with create false, has none yet).
hipMemPool_t rank_pool(bool create = true) {
  constexpr int kMaxDev = 64;
  static std::mutex mu;
  static hipMemPool_t pools[kMaxDev] = {};
  static bool tried[kMaxDev] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::lock_guard<std::mutex> g(mu);
  if (!tried[dev] && create) {
    tried[dev] = true;
    hipMemPoolProps props;
    std::memset(&props, 0, sizeof(props));
    props.allocType = hipMemAllocationTypePinned;
    props.location.type = hipMemLocationTypeDevice;
    props.location.id = dev;
    hipMemPool_t pool = nullptr;
    if (hipMemPoolCreate(&pool, &props) == hipSuccess) {
      uint64_t keep = UINT64_MAX;
      (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
      pools[dev] = pool;
    }
    (void)hipGetLastError();
  }
  return pools[dev];
}

size_t round256(size_t b) { return (b + 255) & ~(size_t)255; }

// Launch shape and scratch layout of one simulate call.
struct SimLayout {
  int Beff, K, NW, NP, q_words, stage_words;
  bool q_hbm;
  int32_t rank_stride;
  size_t rank_bytes, qlink_bytes;  // device scratch, each rounded up to 256 bytes
};

int simulate_layout(const fsched_params* p, int64_t n_inst, int32_t n, SimLayout* L) {
  const int Beff = (p->B == 0 || p->B > n) ? n : p->B;
  if (n > fs::MAX_JOBS || Beff > fs::MAX_WORKERS) return FSCHED_ETOOLARGE;
  int K = 1;
  while (K * 64 < Beff) K <<= 1;
  const int NW = n <= 2048 ? 1 : 2;
  const int NP = next_pow2(n);
  const bool isjl = p->policy == FSCHED_ISJL;
  // plan-queue links; with alpha = infinity Phase ONE never plans (no second
  // job is longer than alpha), so the links are not needed
  // (with up to 8 slots per lane, at most 128 VGPRs, 16 waves fit a CU: the
  // links go to HBM scratch when in LDS they would cap a CU below that)
  const bool plans = isjl && p->alpha != FSCHED_ALPHA_INF;
  bool q_hbm = false;
  if (plans && K <= 8) {
    const int w_lds = NP + NP / 2 +
                      std::max((Beff + 1) / 2, 64 * NW);  // words per wave with the links
    const size_t per_wave = (size_t)((w_lds + 3) & ~3) * 4;
    int wpb = 4;
    while (wpb > 1 && per_wave * wpb > 64 * 1024) wpb >>= 1;
    const size_t waves_per_cu = (160 * 1024) / (per_wave * wpb) * wpb;
    q_hbm = waves_per_cu < 16;
  }
  L->Beff = Beff;
  L->K = K;
  L->NW = NW;
  L->NP = NP;
  L->q_hbm = q_hbm;
  L->q_words = (plans && !q_hbm) ? NP / 2 : 0;
  // gather buffer (uint16 per worker), also the release scatter buffer (one
  // word per 32 ranks)
  // FCFS gathers nothing, but with 4 or more slots per lane its sweeps pack up to
  // 64 active slots through this buffer too
  L->stage_words =
      p->policy != FSCHED_FCFS ? std::max((Beff + 1) / 2, 64 * NW) : (K >= 4 ? 64 : 0);
  L->rank_stride = (n + 63) & ~63;
  // the rank table of the release chunks (not FCFS, whose order is the arrival
  // order) and the HBM plan-queue links
  L->rank_bytes =
      p->policy != FSCHED_FCFS ? round256((size_t)n_inst * (size_t)L->rank_stride * 2) : 0;
  L->qlink_bytes = q_hbm ? round256((size_t)n_inst * (size_t)NP * 4) : 0;
  return FSCHED_OK;
}

// Enqueue the simulate kernels.  Scratch comes from `ext` (ext_bytes long, at
// least the layout's rank_bytes + qlink_bytes, 256-byte aligned) when given,
// else from the library's pool.
int launch_simulate(const fsched_params* p, int64_t n_inst, int32_t n, const int32_t* arrival,
                    const int32_t* prompt, const int32_t* output, fsched_metrics* out,
                    int64_t* out_T, int32_t* start, int32_t* finish, hipStream_t s,
                    const int32_t* upper = nullptr, void* ext = nullptr,
                    size_t ext_bytes = 0) {
  SimLayout Lay;
  int lrc = simulate_layout(p, n_inst, n, &Lay);
  if (lrc) return lrc;
  const int Beff = Lay.Beff, K = Lay.K, NW = Lay.NW, NP = Lay.NP;
  const bool q_hbm = Lay.q_hbm;
  const int q_words = Lay.q_words, stage_words = Lay.stage_words;
  if (ext && ext_bytes < Lay.rank_bytes + Lay.qlink_bytes) return FSCHED_ESCRATCH;

  fs::SimArgs a;
  std::memset(&a, 0, sizeof(a));
  a.n_inst = n_inst;
  a.n = n;
  a.Beff = Beff;
  a.alpha = p->alpha;
  a.beta = (p->flags & FSCHED_F_BETA_SQRT17) ? beta_sqrt17(p->alpha) : p->alpha;
  a.resume = (p->flags & FSCHED_F_RESUME_FILL) ? 1 : 0;
  a.M = p->M_kv;
  a.c = p->cost_c;
  a.tau = p->cost_tau;
  a.NP = NP;
  a.arrival = arrival;
  a.prompt = prompt;
  a.output = output;
  a.upper = upper;
  a.out = out;
  a.out_T = out_T;
  a.start = start;
  a.finish = finish;
  // scratch from the caller's buffer, else from the library's pool, else from
  // the device's default pool
  char* ext_next = (char*)ext;
  auto scratch = [&](size_t bytes) -> void* {
    if (ext) {
      void* r = ext_next;
      ext_next += round256(bytes);
      return r;
    }
    hipMemPool_t pool = rank_pool();
    void* r = nullptr;
    hipError_t e = pool ? hipMallocFromPoolAsync(&r, bytes, pool, s) : hipErrorNotSupported;
    if (e != hipSuccess) {
      (void)hipGetLastError();
      r = nullptr;
      e = hipMallocAsync(&r, bytes, s);
    }
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    return r;
  };
  auto release = [&](void* r) {
    if (!ext && r && hipFreeAsync(r, s) != hipSuccess) (void)hipGetLastError();
  };
  a.rank_stride = Lay.rank_stride;
  a.rank = nullptr;
  a.q_stride = NP;
  a.qlink = nullptr;
  if (p->policy != FSCHED_FCFS) {
    a.rank = (uint16_t*)scratch((size_t)n_inst * (size_t)a.rank_stride * 2);
    if (!a.rank) return FSCHED_ENOMEM;
  }
  if (q_hbm) {
    a.qlink = (uint32_t*)scratch((size_t)n_inst * (size_t)a.q_stride * 4);
    if (!a.qlink) {
      release(a.rank);
      return FSCHED_ENOMEM;
    }
  }

  hipError_t err = hipSuccess;
  for (int general = 0; general < 2 && err == hipSuccess; ++general) {
    fs::SimArgs b = a;
    b.off_arr = NP;
    b.off_q = NP + (general ? NP : 0);
    b.off_stage = b.off_q + q_words;
    b.wave_words = b.off_stage + stage_words;
    b.wave_words = (b.wave_words + 3) & ~3;
    size_t per_wave = (size_t)b.wave_words * 4;
    int wpb = 4;
    while (wpb > 1 && per_wave * wpb > 64 * 1024) wpb >>= 1;
    size_t lds = per_wave * wpb;
    hipError_t e;
    const bool pre = (p->flags & FSCHED_F_PREFILL) != 0;
    switch (p->policy) {
      case FSCHED_FCFS:
        e = pre ? fs::launch_sim_fcfs_prefill(b, K, NW, general, wpb, lds, s)
                : fs::launch_sim_fcfs(b, K, NW, general, wpb, lds, s);
        break;
      case FSCHED_LJF:
        e = pre ? fs::launch_sim_ljf_prefill(b, K, NW, general, wpb, lds, s)
                : fs::launch_sim_ljf(b, K, NW, general, wpb, lds, s);
        break;
      case FSCHED_ISJL:
        if (upper)
          e = pre ? fs::launch_sim_isjl_robust_prefill(b, K, NW, general, wpb, lds, s)
                  : fs::launch_sim_isjl_robust(b, K, NW, general, wpb, lds, s);
        else
          e = pre ? fs::launch_sim_isjl_prefill(b, K, NW, general, wpb, lds, s)
                  : fs::launch_sim_isjl(b, K, NW, general, wpb, lds, s);
        break;
      default:
        e = pre ? fs::launch_sim_sjf_prefill(b, K, NW, general, wpb, lds, s)
                : fs::launch_sim_sjf(b, K, NW, general, wpb, lds, s);
        break;
    }
    err = e;
  }
  release(a.rank);
  release(a.qlink);
  if (err != hipSuccess) return hip_fail(err);
  return FSCHED_OK;
}

// fsched_simulate and fsched_simulate_robust (upper non-null).
int simulate_entry(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                   const int32_t* arrival, const int32_t* prompt, const int32_t* output,
                   const int32_t* upper, fsched_metrics* out, int32_t* start, int32_t* finish,
                   void* stream) {
  int rc = check_params(p, true);
  if (rc) return rc;
  if (n_inst < 0 || n_jobs < 1) return FSCHED_EINVAL;
  if (n_inst == 0) return FSCHED_OK;
  if (!arrival || !prompt || !output || !out) return FSCHED_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  if (p->flags & FSCHED_F_DEVICE_PTRS) {
    rc = launch_simulate(p, n_inst, n_jobs, arrival, prompt, output, out, nullptr, start, finish,
                         s, upper);
    if (rc) return rc;
    if (p->flags & FSCHED_F_SYNC) {
      hipError_t e = hipStreamSynchronize(s);
      if (e != hipSuccess) return hip_fail(e);
    }
    return FSCHED_OK;
  }
  const size_t cells = (size_t)n_inst * (size_t)n_jobs;
  const size_t tb = cells * sizeof(int32_t);
  Staging st;
  const int32_t* da = (const int32_t*)st.upload(arrival, tb);
  const int32_t* dp = (const int32_t*)st.upload(prompt, tb);
  const int32_t* dq = (const int32_t*)st.upload(output, tb);
  const int32_t* du = upper ? (const int32_t*)st.upload(upper, tb) : nullptr;
  fsched_metrics* dout = (fsched_metrics*)st.alloc((size_t)n_inst * sizeof(fsched_metrics));
  int32_t* dst = start ? (int32_t*)st.alloc(tb) : nullptr;
  int32_t* dfi = finish ? (int32_t*)st.alloc(tb) : nullptr;
  if (st.err != hipSuccess) return hip_fail(st.err);
  rc = launch_simulate(p, n_inst, n_jobs, da, dp, dq, dout, nullptr, dst, dfi, s, du);
  if (rc) return rc;
  hipError_t e = hipStreamSynchronize(s);
  if (e == hipSuccess)
    e = hipMemcpy(out, dout, (size_t)n_inst * sizeof(fsched_metrics), hipMemcpyDeviceToHost);
  if (e == hipSuccess && start) e = hipMemcpy(start, dst, tb, hipMemcpyDeviceToHost);
  if (e == hipSuccess && finish) e = hipMemcpy(finish, dfi, tb, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e);
  return markers_to_code(out, n_inst);
}

}  // namespace

namespace fs {

int simulate_scratch_need(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                          size_t* bytes) {
  SimLayout L;
  int rc = simulate_layout(p, n_inst, n_jobs, &L);
  if (rc) return rc;
  *bytes = L.rank_bytes + L.qlink_bytes;
  return FSCHED_OK;
}

int simulate_with_scratch(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                          const int32_t* arrival, const int32_t* prompt, const int32_t* output,
                          fsched_metrics* out, int32_t* start, int32_t* finish,
                          hipStream_t stream, void* scratch, size_t scratch_bytes) {
  int rc = launch_simulate(p, n_inst, n_jobs, arrival, prompt, output, out, nullptr, start,
                           finish, stream, nullptr, scratch, scratch_bytes);
  if (rc) return rc;
  if (p->flags & FSCHED_F_SYNC) {
    hipError_t e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(e);
  }
  return FSCHED_OK;
}

int check_simulate_args(const fsched_params* p, int64_t n_inst, int32_t n_jobs) {
  int rc = check_params(p, true);
  if (rc) return rc;
  if (n_inst < 0 || n_jobs < 1) return FSCHED_EINVAL;
  return FSCHED_OK;
}

int record_hip_error(hipError_t e) { return hip_fail(e); }

}  // namespace fs

extern "C" {

const char* fsched_strerror(int code) {
  switch (code) {
    case FSCHED_OK: return "ok";
    case FSCHED_EINVAL: return "invalid argument or job table";
    case FSCHED_ERANGE: return "an int64 accumulator could overflow";
    case FSCHED_ENOMEM: return "out of memory";
    case FSCHED_EDEVICE: return "HIP runtime error";
    case FSCHED_ETOOLARGE: return "instance beyond a kernel limit";
    case FSCHED_ENOTIMPL: return "not implemented";
    case FSCHED_EINTERNAL: return "internal error: no next event";
    case FSCHED_ESCRATCH:
      return "the call needs more scratch than fsched_simulate_noalloc's fixed buffer holds";
    default: return "unknown error code";
  }
}

int fsched_abi_version(void) { return FSCHED_ABI_VERSION; }

int fsched_last_hip_error(void) { return g_last_hip; }

int fsched_release_cache(void) {
  hipMemPool_t pool = rank_pool(false);
  if (!pool) return FSCHED_OK;
  hipError_t e = hipMemPoolTrimTo(pool, 0);
  return e == hipSuccess ? FSCHED_OK : hip_fail(e);
}

int fsched_simulate(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                    const int32_t* arrival, const int32_t* prompt, const int32_t* output,
                    fsched_metrics* out, int32_t* start, int32_t* finish, void* stream) {
  return simulate_entry(p, n_inst, n_jobs, arrival, prompt, output, nullptr, out, start, finish,
                        stream);
}

int fsched_simulate_robust(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                           const int32_t* arrival, const int32_t* prompt, const int32_t* output,
                           const int32_t* upper, fsched_metrics* out, int32_t* start,
                           int32_t* finish, void* stream) {
  if (!p) return FSCHED_EINVAL;
  if (!upper) return FSCHED_EINVAL;
  if (p->policy != FSCHED_ISJL) return FSCHED_ENOTIMPL;
  return simulate_entry(p, n_inst, n_jobs, arrival, prompt, output, upper, out, start, finish,
                        stream);
}

int fsched_cost_decompose(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                          const int32_t* arrival, const int32_t* prompt, const int32_t* output,
                          const int32_t* start, fsched_metrics* out, uint32_t* violation,
                          void* stream) {
  int rc = check_params(p, false);
  if (rc) return rc;
  if (p->flags & FSCHED_F_PREFILL) return FSCHED_ENOTIMPL;  // chunked reading only
  if (n_inst < 0 || n_jobs < 1) return FSCHED_EINVAL;
  if (n_inst == 0) return FSCHED_OK;
  if (!arrival || !prompt || !output || !start || !out || !violation) return FSCHED_EINVAL;
  if (n_jobs > fs::DEC_MAX_JOBS) return FSCHED_ETOOLARGE;
  hipStream_t s = (hipStream_t)stream;
  fs::DecArgs a;
  std::memset(&a, 0, sizeof(a));
  a.n_inst = n_inst;
  a.n = n_jobs;
  a.B = p->B;
  a.alpha = p->alpha;
  a.M = p->M_kv;
  a.c = p->cost_c;
  a.tau = p->cost_tau;
  a.NP2 = next_pow2(2 * n_jobs);
  // Two passes: 16-bit job lengths in LDS, then 32-bit ones for the instances
  // the first pass deferred (a job of 65,536 tokens or more).
  auto launch = [&](const fs::DecArgs& d, hipStream_t st) -> hipError_t {
    for (int narrow = 1; narrow >= 0; --narrow) {
      fs::DecArgs b = d;
      b.deferred_only = narrow ? 0 : 1;
      // sorted events, then the length of each job
      b.wave_words = b.NP2 + (narrow ? (n_jobs + 1) / 2 : n_jobs);
      b.wave_words = (b.wave_words + 3) & ~3;
      const size_t per_wave = (size_t)b.wave_words * 4;
      int wpb = 4;
      while (wpb > 1 && per_wave * wpb > 64 * 1024) wpb >>= 1;
      hipError_t e = fs::launch_decompose(b, narrow != 0, wpb, per_wave * wpb, st);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  };
  if (p->flags & FSCHED_F_DEVICE_PTRS) {
    a.arrival = arrival;
    a.prompt = prompt;
    a.output = output;
    a.start = start;
    a.out = out;
    a.viol = violation;
    hipError_t e = launch(a, s);
    if (e != hipSuccess) return hip_fail(e);
    if (p->flags & FSCHED_F_SYNC) {
      e = hipStreamSynchronize(s);
      if (e != hipSuccess) return hip_fail(e);
    }
    return FSCHED_OK;
  }
  const size_t tb = (size_t)n_inst * (size_t)n_jobs * sizeof(int32_t);
  Staging st;
  a.arrival = (const int32_t*)st.upload(arrival, tb);
  a.prompt = (const int32_t*)st.upload(prompt, tb);
  a.output = (const int32_t*)st.upload(output, tb);
  a.start = (const int32_t*)st.upload(start, tb);
  a.out = (fsched_metrics*)st.alloc((size_t)n_inst * sizeof(fsched_metrics));
  a.viol = (uint32_t*)st.alloc((size_t)n_inst * sizeof(uint32_t));
  if (st.err != hipSuccess) return hip_fail(st.err);
  hipError_t e = launch(a, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e == hipSuccess)
    e = hipMemcpy(out, a.out, (size_t)n_inst * sizeof(fsched_metrics), hipMemcpyDeviceToHost);
  if (e == hipSuccess)
    e = hipMemcpy(violation, a.viol, (size_t)n_inst * sizeof(uint32_t), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e);
  return markers_to_code(out, n_inst);
}

int fsched_bruteforce_opt(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                          const int32_t* arrival, const int32_t* prompt, const int32_t* output,
                          int64_t* T_opt, int32_t* start_opt, void* stream) {
  int rc = check_params(p, false);
  if (rc) return rc;
  if (p->flags & FSCHED_F_PREFILL) return FSCHED_ENOTIMPL;  // chunked reading only
  if (n_inst < 0 || n_jobs < 1) return FSCHED_EINVAL;
  if (n_jobs > fs::OPT_MAX_JOBS) return FSCHED_ETOOLARGE;
  if (n_inst == 0) return FSCHED_OK;
  if (!arrival || !prompt || !output || !T_opt) return FSCHED_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  // The ISJL makespan (and schedule) is the incumbent the exact search has to beat.
  fsched_params sp = *p;
  sp.policy = FSCHED_ISJL;
  sp.flags = 0;
  sp.cost_c = 0;
  sp.cost_tau = 0;
  fs::OptArgs a;
  std::memset(&a, 0, sizeof(a));
  a.n_inst = n_inst;
  a.n = n_jobs;
  a.B = (p->B == 0 || p->B > n_jobs) ? n_jobs : p->B;
  a.alpha = p->alpha;
  a.M = p->M_kv;
  a.wave_words = (int32_t)fs::opt_lds_words_per_wave();
  const int wpb = 1;
  const size_t lds = (size_t)a.wave_words * 4 * wpb;
  // Scratch of the second pass (searches the first pass's LDS memo could not
  // finish): the list of their instances, two counters and a memo region per
  // wave, from the library's pool (else the device's default pool).
  const size_t list_bytes = round256((size_t)n_inst * 4 + 8);
  const size_t memo_bytes = (size_t)fs::OPT_FB_WAVES * fs::OPT_FB_MEMO_ENTRIES * 16;
  void* fb = nullptr;
  {
    hipMemPool_t pool = rank_pool();
    hipError_t e = pool ? hipMallocFromPoolAsync(&fb, list_bytes + memo_bytes, pool, s)
                        : hipErrorNotSupported;
    if (e != hipSuccess) {
      (void)hipGetLastError();
      fb = nullptr;
      if (hipMallocAsync(&fb, list_bytes + memo_bytes, s) != hipSuccess) {
        (void)hipGetLastError();
        fb = nullptr;  // no second pass: a capped search reports FSCHED_T_INTERNAL
      }
    }
  }
  auto run = [&](const int32_t* da, const int32_t* dp, const int32_t* dq, int64_t* dT,
                 int32_t* dS) -> int {
    int r = launch_simulate(&sp, n_inst, n_jobs, da, dp, dq, nullptr, dT, dS, nullptr, s);
    if (r) return r;
    a.arrival = da;
    a.prompt = dp;
    a.output = dq;
    a.T = dT;
    a.start = dS;
    if (fb) {
      a.fb_count = (int32_t*)fb;
      a.fb_list = (int32_t*)fb + 2;
      a.fb_memo = (uint32_t*)((char*)fb + list_bytes);
      hipError_t e = hipMemsetAsync(a.fb_count, 0, 8, s);
      if (e != hipSuccess) return hip_fail(e);
    }
    hipError_t e = fs::launch_opt(a, wpb, lds, s);
    if (e == hipSuccess && fb)
      e = fs::launch_opt_fallback(a, fs::opt_fallback_lds_words_per_wave() * 4, s);
    return e == hipSuccess ? FSCHED_OK : hip_fail(e);
  };
  auto release_fb = [&]() {
    if (fb && hipFreeAsync(fb, s) != hipSuccess) (void)hipGetLastError();
  };
  if (p->flags & FSCHED_F_DEVICE_PTRS) {
    rc = run(arrival, prompt, output, T_opt, start_opt);
    release_fb();
    if (rc) return rc;
    if (p->flags & FSCHED_F_SYNC) {
      hipError_t e = hipStreamSynchronize(s);
      if (e != hipSuccess) return hip_fail(e);
    }
    return FSCHED_OK;
  }
  const size_t tb = (size_t)n_inst * (size_t)n_jobs * sizeof(int32_t);
  Staging st;
  const int32_t* da = (const int32_t*)st.upload(arrival, tb);
  const int32_t* dp = (const int32_t*)st.upload(prompt, tb);
  const int32_t* dq = (const int32_t*)st.upload(output, tb);
  int64_t* dT = (int64_t*)st.alloc((size_t)n_inst * sizeof(int64_t));
  int32_t* dS = start_opt ? (int32_t*)st.alloc(tb) : nullptr;
  if (st.err != hipSuccess) {
    release_fb();
    return hip_fail(st.err);
  }
  rc = run(da, dp, dq, dT, dS);
  release_fb();
  if (rc) return rc;
  hipError_t e = hipStreamSynchronize(s);
  if (e == hipSuccess)
    e = hipMemcpy(T_opt, dT, (size_t)n_inst * sizeof(int64_t), hipMemcpyDeviceToHost);
  if (e == hipSuccess && start_opt) e = hipMemcpy(start_opt, dS, tb, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e);
  for (int64_t i = 0; i < n_inst; ++i) {
    if (T_opt[i] == FSCHED_T_INVALID) return FSCHED_EINVAL;
    if (T_opt[i] == FSCHED_T_INTERNAL) rc = FSCHED_EINTERNAL;
    else if (T_opt[i] < 0) rc = (T_opt[i] == FSCHED_T_RANGE) ? FSCHED_ERANGE : FSCHED_ETOOLARGE;
  }
  return rc;
}

}  // extern "C"
