// Kernel instantiations for Robust-ISJL: ISJL planned on predicted output sizes.
#include "sim_kernel.hpp"

namespace fs {
hipError_t launch_sim_isjl_robust(const SimArgs& a, int K, int NW, bool general,
                                  int waves_per_block, size_t lds_bytes, hipStream_t s) {
  return launch_sim<POL_ISJL, true>(a, K, NW, general, waves_per_block, lds_bytes, s);
}
}  // namespace fs
