// Launch descriptor of the schedule re-scoring kernel.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fsched.h"

namespace fs {

constexpr int DEC_MAX_JOBS = 4096;
constexpr int64_t DEC_TIME_LIMIT = 1 << 19;  // completion steps < 2^19 (packed event keys)
constexpr int64_t DEC_DEFERRED = -100;       // a job of 65,536 tokens or more: the wide pass scores it

struct DecArgs {
  int64_t n_inst;
  int32_t n;
  int32_t B;          // 0 = no count limit
  int32_t alpha;      // INT32_MAX = infinite
  int32_t NP2;        // 2n rounded up to a power of two (>= 64)
  int64_t M;          // 0 = no KV budget
  int64_t c, tau;
  int32_t wave_words; // LDS words per wave
  int32_t deferred_only;  // wide pass: only the instances the narrow pass deferred
  const int32_t* arrival;
  const int32_t* prompt;
  const int32_t* output;
  const int32_t* start;
  fsched_metrics* out;
  uint32_t* viol;
};

// narrow: 16-bit job lengths in LDS (8 waves per CU at 2,000 jobs), deferring
// instances with a longer job; otherwise the wide pass with 32-bit lengths.
hipError_t launch_decompose(const DecArgs& a, bool narrow, int waves_per_block, size_t lds_bytes,
                            hipStream_t s);

}  // namespace fs
