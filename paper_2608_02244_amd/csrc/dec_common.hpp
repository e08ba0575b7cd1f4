// Launch descriptor of the schedule re-scoring kernel.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fsched.h"

namespace fs {

constexpr int DEC_MAX_JOBS = 4096;
constexpr int64_t DEC_TIME_LIMIT = 1 << 19;  // completion steps < 2^19 (packed event keys)

struct DecArgs {
  int64_t n_inst;
  int32_t n;
  int32_t B;          // 0 = no count limit
  int32_t alpha;      // INT32_MAX = infinite
  int32_t NP2;        // 2n rounded up to a power of two (>= 64)
  int64_t M;          // 0 = no KV budget
  int64_t c, tau;
  int32_t wave_words; // LDS words per wave
  int32_t pad;
  const int32_t* arrival;
  const int32_t* prompt;
  const int32_t* output;
  const int32_t* start;
  fsched_metrics* out;
  uint32_t* viol;
};

hipError_t launch_decompose(const DecArgs& a, int waves_per_block, size_t lds_bytes,
                            hipStream_t s);

}  // namespace fs
