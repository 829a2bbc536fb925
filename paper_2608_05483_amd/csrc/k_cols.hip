// k_cols.hip -- plora_apply as one launch, one h_in slice per tile.
#include "plora_dev.h"

namespace plora_impl {

// plora_apply as one launch, one slice per tile in h_in: item (tile,
// column slice) computes the tile's v over all of h_in, then expands it
// with its slice of B_i (column slices from the tile count, as make_plan
// gives them).  A_i is read by every column slice of its tile; the slices
// of a tile are numbered onto one XCD, so the first read brings A_i into
// that XCD's L2 and the others hit it.
__global__ __launch_bounds__(kNT, kWGPerCU) void apply_cols_kernel(ApplyArgs g) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  const Plan p = make_plan(g, kColSlices);
  Tile t;
  int my_tok, js;
  if ((int)blockIdx.x >= p.n_items) return;
  if (!item_tile(g, p, kColSlices, blockIdx.x, t, my_tok, js)) {
    count_skipped(g, t, js);
    return;
  }
  const Smem sm = tile_prologue(g, my_tok, apply_lds);
  tile_dispatch(g, t, sm, true, true);
}

void launch_apply_cols(const ApplyArgs& g, unsigned grid, size_t lds, hipStream_t stream) {
  static std::atomic<bool> lds_done{false};
  if (lds > 64 * 1024) allow_lds(reinterpret_cast<const void*>(apply_cols_kernel), lds_done);
  hipLaunchKernelGGL(apply_cols_kernel, dim3(grid), dim3(kNT), lds, stream, g);
}

}  // namespace plora_impl
