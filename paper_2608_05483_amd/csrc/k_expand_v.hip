// k_expand_v.hip -- plora_expand (v from the caller's array).
#include "plora_dev.h"

namespace plora_impl {



void launch_expand_v(const ApplyArgs& g, unsigned grid, size_t lds, hipStream_t stream) {
  static std::atomic<bool> lds_done{false};
  if (lds > 64 * 1024) allow_lds(reinterpret_cast<const void*>(expand_kernel<false>), lds_done);
  hipLaunchKernelGGL(expand_kernel<false>, dim3(grid), dim3(kNT), lds, stream, g);
}

}  // namespace plora_impl
