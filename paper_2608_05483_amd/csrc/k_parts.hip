// k_parts.hip -- the two parts of plora_apply for batches above 256 tokens, in one launch.
// a short segment's adapter (a vector-path tile) is read once per call:
// non-temporal reads; a long segment's is re-read by each of its tiles
#define PLORA_ADAPTER_POLICY 2
#define PLORA_MATRIX_POLICY 0
#include "plora_dev.h"

namespace plora_impl {

// Work group b < n_shrink runs shrink item b, the others expand item
// b - n_shrink (see parts_shrink_item and parts_expand_item).
__global__ __launch_bounds__(kNT, kWGPerCU) void parts_kernel(ApplyArgs g, int32_t n_shrink) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  __shared__ int ok_sh;
  if ((int)blockIdx.x < n_shrink)
    parts_shrink_item(g, blockIdx.x, apply_lds);
  else
    parts_expand_item(g, blockIdx.x - n_shrink, apply_lds, &ok_sh);
}

void launch_parts(const ApplyArgs& g, unsigned n_shrink, unsigned n_expand, size_t lds,
                  hipStream_t stream) {
  static std::atomic<bool> lds_done{false};
  if (lds > 64 * 1024) allow_lds(reinterpret_cast<const void*>(parts_kernel), lds_done);
  hipLaunchKernelGGL(parts_kernel, dim3(n_shrink + n_expand), dim3(kNT), lds, stream, g,
                     (int32_t)n_shrink);
}

}  // namespace plora_impl
