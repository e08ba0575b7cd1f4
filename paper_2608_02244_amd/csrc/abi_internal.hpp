// Entry points of abi.cpp shared with the library's other host translation
// units (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "fsched.h"

namespace fs {

// Bytes of device scratch one fsched_simulate call of this shape needs (the
// rank table and, for ISJL with up to 128 workers, the plan-queue links).
int simulate_scratch_need(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                          size_t* bytes);

// fsched_simulate in device mode with the scratch taken from `scratch`
// (scratch_bytes long, 256-byte aligned) instead of the library's pool.
int simulate_with_scratch(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                          const int32_t* arrival, const int32_t* prompt, const int32_t* output,
                          fsched_metrics* out, int32_t* start, int32_t* finish,
                          hipStream_t stream, void* scratch, size_t scratch_bytes);

// Parameter and size checks of fsched_simulate.
int check_simulate_args(const fsched_params* p, int64_t n_inst, int32_t n_jobs);

// Keep e as the thread's last HIP error and map it to a return code.
int record_hip_error(hipError_t e);

}  // namespace fs
