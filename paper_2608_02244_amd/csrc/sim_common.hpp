// Launch descriptors shared by the host ABI layer and the kernel translation units.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fsched.h"

namespace fs {

// Per-instance markers written into metrics.T (besides the public ones).
constexpr int64_t T_DEFERRED = -100;  // arrivals not sorted: the general kernel finishes it
constexpr int64_t T_INTERNAL = -7;    // the event loop found no next event (internal error)

// Kernel limits.
constexpr int MAX_JOBS = 4096;
constexpr int MAX_WORKERS = 1024;
constexpr int LEN_LIMIT = 1 << 20;    // len < 2^20 (12 bits of job index beside it)
constexpr int ARR_LIMIT = 1 << 20;    // unsorted arrivals must be < 2^20

struct SimArgs {
  int64_t n_inst;
  int32_t n;          // jobs per instance
  int32_t Beff;       // min(B, n), or n when B is unlimited
  int32_t alpha;      // INT32_MAX = infinite
  int32_t beta;       // ISJL pack slack (alpha or floor(beta*))
  int64_t M;          // KV budget, 0 = none
  int64_t c, tau;
  int32_t NP;         // n rounded up to a power of two (>= 64)
  int32_t wave_words; // LDS words per wave
  int32_t off_arr;    // word offset of arrival-by-rank (general kernel)
  int32_t off_q;      // word offset of the plan-queue links (ISJL)
  int32_t off_stage;  // word offset of the gather / release buffer (not FCFS)
  int32_t resume;     // ISJL: Phase TWO resumes once A_max <= alpha (1) or waits
                      // for an empty machine (0)
  const int32_t* arrival;
  const int32_t* prompt;
  const int32_t* output;
  const int32_t* upper;  // predicted upper bounds of the outputs (Robust-ISJL), else null
  fsched_metrics* out;  // per-instance metrics, or
  int64_t* out_T;       // when non-null: only the makespan (or marker) per instance
  int32_t* start;
  int32_t* finish;
  // Scratch: rank of every job in the priority order, written by the
  // sorted-arrival kernel once it has sorted and read back at each release
  // chunk (rows of rank_stride entries, a multiple of 64 so that no 128-byte
  // line is shared by two instances).  Required for every policy but FCFS.
  uint16_t* rank;
  int32_t rank_stride;
  // Scratch: ISJL plan-queue links of the kernels with up to 2 slots per lane
  // (rows of q_stride entries; the other kernels keep them in LDS).  Moving
  // them out of LDS lets 16 waves share a CU.  Null when alpha is infinite
  // (no plans).
  uint32_t* qlink;
  int32_t q_stride;
};

// Chooses and launches the kernel instantiation for one policy.  `general`
// selects the variant for instances whose arrivals are not sorted by index.
hipError_t launch_sim_fcfs(const SimArgs& a, int K, int NW, bool general, int waves_per_block,
                           size_t lds_bytes, hipStream_t s);
hipError_t launch_sim_ljf(const SimArgs& a, int K, int NW, bool general, int waves_per_block,
                          size_t lds_bytes, hipStream_t s);
hipError_t launch_sim_isjl(const SimArgs& a, int K, int NW, bool general, int waves_per_block,
                           size_t lds_bytes, hipStream_t s);
// Robust-ISJL (Section 3.4): ISJL planning on prompt + upper[i].
hipError_t launch_sim_isjl_robust(const SimArgs& a, int K, int NW, bool general,
                                  int waves_per_block, size_t lds_bytes, hipStream_t s);
// The prefill-at-admission variant of each policy (and of Robust-ISJL).
hipError_t launch_sim_fcfs_prefill(const SimArgs& a, int K, int NW, bool general,
                                   int waves_per_block, size_t lds_bytes, hipStream_t s);
hipError_t launch_sim_ljf_prefill(const SimArgs& a, int K, int NW, bool general,
                                  int waves_per_block, size_t lds_bytes, hipStream_t s);
hipError_t launch_sim_isjl_prefill(const SimArgs& a, int K, int NW, bool general,
                                   int waves_per_block, size_t lds_bytes, hipStream_t s);
hipError_t launch_sim_sjf_prefill(const SimArgs& a, int K, int NW, bool general,
                                  int waves_per_block, size_t lds_bytes, hipStream_t s);
hipError_t launch_sim_isjl_robust_prefill(const SimArgs& a, int K, int NW, bool general,
                                          int waves_per_block, size_t lds_bytes, hipStream_t s);
hipError_t launch_sim_sjf(const SimArgs& a, int K, int NW, bool general, int waves_per_block,
                          size_t lds_bytes, hipStream_t s);

}  // namespace fs
