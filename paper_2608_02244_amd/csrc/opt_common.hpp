// Launch descriptor of the exact-optimum search kernel.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fsched.h"

namespace fs {

constexpr int OPT_MAX_JOBS = 8;
constexpr int OPT_LEN_LIMIT = 255;   // every length <= 255 (one byte of progress)
constexpr int OPT_ARR_LIMIT = 4095;  // every arrival <= 4095 (12-bit key field)

struct OptArgs {
  int64_t n_inst;
  int32_t n;
  int32_t B;          // effective capacity (n when unlimited)
  int32_t alpha;      // INT32_MAX = infinite
  int32_t wave_words;
  int64_t M;          // 0 = no KV budget
  const int32_t* arrival;
  const int32_t* prompt;
  const int32_t* output;
  int64_t* T;         // in: ISJL makespan (incumbent) or marker; out: optimum
  int32_t* start;     // in: ISJL schedule; out: an optimal schedule (nullable)
};

hipError_t launch_opt(const OptArgs& a, int waves_per_block, size_t lds_bytes, hipStream_t s);
size_t opt_lds_words_per_wave();

}  // namespace fs
