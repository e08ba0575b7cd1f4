// Kernel instantiations for the ISJL policy, prompt prefilled at admission.
#include "sim_kernel.hpp"

namespace fs {
hipError_t launch_sim_isjl_prefill(const SimArgs& a, int K, int NW, bool general,
                                   int waves_per_block, size_t lds_bytes, hipStream_t s) {
  return launch_sim<POL_ISJL, false, true>(a, K, NW, general, waves_per_block, lds_bytes, s);
}
}  // namespace fs
