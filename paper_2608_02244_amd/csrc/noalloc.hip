// fsched_simulate_noalloc: fsched_simulate in device mode with its scratch in a
// fixed device buffer of this translation unit, for callers that cannot
// allocate during a call.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "abi_internal.hpp"
#include "fsched.h"

namespace {

// The buffer itself.  Host code never uses this name as an address: the
// device address is looked up per device with hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[FSCHED_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

// Device address of `scratch` on the current device (looked up once per
// device), or an error code.
int scratch_on_current_device(void** ptr) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fs::record_hip_error(e);
  if (dev < 0 || dev >= kMaxDevices) return FSCHED_EDEVICE;
  std::lock_guard<std::mutex> g(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return fs::record_hip_error(e);
    if (!p) return FSCHED_EDEVICE;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return FSCHED_OK;
}

}  // namespace

extern "C" int fsched_simulate_noalloc(const fsched_params* p, int64_t n_inst, int32_t n_jobs,
                                       const int32_t* arrival, const int32_t* prompt,
                                       const int32_t* output, fsched_metrics* out,
                                       int32_t* start, int32_t* finish, void* stream) {
  int rc = fs::check_simulate_args(p, n_inst, n_jobs);
  if (rc) return rc;
  if (!(p->flags & FSCHED_F_DEVICE_PTRS)) return FSCHED_EINVAL;  // host mode would stage
  if (n_inst == 0) return FSCHED_OK;
  if (!arrival || !prompt || !output || !out) return FSCHED_EINVAL;
  size_t need = 0;
  rc = fs::simulate_scratch_need(p, n_inst, n_jobs, &need);
  if (rc) return rc;
  if (need > FSCHED_NOALLOC_SCRATCH_BYTES) return FSCHED_ESCRATCH;
  void* buf = nullptr;
  rc = scratch_on_current_device(&buf);
  if (rc) return rc;
  return fs::simulate_with_scratch(p, n_inst, n_jobs, arrival, prompt, output, out, start,
                                   finish, (hipStream_t)stream, buf,
                                   FSCHED_NOALLOC_SCRATCH_BYTES);
}
