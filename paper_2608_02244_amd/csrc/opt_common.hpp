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
  // Second pass for the searches that reach the first pass's step cap: the
  // first pass appends their instance indices to fb_list (fb_count[0] of
  // them; fb_count[1] is the claim counter of the second pass, both zero
  // before the first pass) and the second pass solves them again with a large
  // memo in fb_memo (OPT_FB_WAVES regions of OPT_FB_MEMO_ENTRIES 16-byte
  // entries).  Null fb_list: a capped search reports FSCHED_T_INTERNAL.
  int32_t* fb_list;
  int32_t* fb_count;
  uint32_t* fb_memo;
};

constexpr int OPT_FB_WAVES = 16;                // waves of the second pass
constexpr int OPT_FB_MEMO_ENTRIES = 1 << 20;    // memo entries per wave (16 MiB)
constexpr int OPT_FB_GUARD = 1 << 28;           // DFS pushes per search in the second pass

hipError_t launch_opt(const OptArgs& a, int waves_per_block, size_t lds_bytes, hipStream_t s);
hipError_t launch_opt_fallback(const OptArgs& a, size_t lds_bytes, hipStream_t s);
size_t opt_lds_words_per_wave();
size_t opt_fallback_lds_words_per_wave();

}  // namespace fs
