// Kernel instantiations for the SJF policy (one translation unit per policy so
// that they compile in parallel).
#include "sim_kernel.hpp"

namespace fs {
hipError_t launch_sim_sjf(const SimArgs& a, int K, int NW, bool general, int waves_per_block,
                         size_t lds_bytes, hipStream_t s) {
  return launch_sim<POL_SJF>(a, K, NW, general, waves_per_block, lds_bytes, s);
}
}  // namespace fs
