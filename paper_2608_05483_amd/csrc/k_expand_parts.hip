// k_expand_parts.hip -- the expand launch of the two-launch plora_apply (v from the workspace partials).
#include "plora_dev.h"

namespace plora_impl {



void launch_expand_parts(const ApplyArgs& g, unsigned grid, size_t lds, hipStream_t stream) {
  static std::atomic<bool> lds_done{false};
  if (lds > 64 * 1024) allow_lds(reinterpret_cast<const void*>(expand_kernel<true>), lds_done);
  hipLaunchKernelGGL(expand_kernel<true>, dim3(grid), dim3(kNT), lds, stream, g);
}

}  // namespace plora_impl
