// k_shrink.hip -- the shrink launch of plora_apply and plora_shrink, and plora_shrink's gather.
#include "plora_dev.h"

namespace plora_impl {

// ---------------------------------------------------------------------------
// kernels
// ---------------------------------------------------------------------------

// Shrink launch (plora_apply, plora_shrink): item (tile, h_in slice) writes
// the slice's partial v of the tile's rows to the workspace.
__global__ __launch_bounds__(kNT, kWGPerCU) void shrink_part_kernel(ApplyArgs g) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  const Plan p = make_plan(g, kRowSlices);
  Tile t;
  int my_tok, ks;
  if ((int)blockIdx.x >= p.n_items) return;
  if (!item_tile(g, p, kRowSlices, blockIdx.x, t, my_tok, ks)) {
    count_skipped(g, t, ks);
    return;
  }
  const Smem sm = tile_prologue(g, my_tok, apply_lds);
  tile_dispatch(g, t, sm, true, false);
  float* dst = g.vpart + ((int64_t)ks * g.T + t.p0) * g.max_rank;
  for (int o = threadIdx.x; o < t.L * t.r; o += kNT) {
    const int l = o / t.r, c = o - l * t.r;
    dst[l * g.max_rank + c] = sm.vs[c * kTT + l];
  }
}

// plora_shrink's second launch: v of each valid token of tile blockIdx.x,
// summed from the partials as the expand launch sums them.
__global__ __launch_bounds__(kNT) void gather_v_kernel(ApplyArgs g) {
  const Plan p = make_plan(g, kRowSlices);
  Tile t;
  int my_tok;
  if ((int)blockIdx.x >= p.n_tiles || !load_tile(g, blockIdx.x, t, my_tok)) return;
  for (int o = threadIdx.x; o < t.L * t.r; o += kNT) {
    const int l = o / t.r, c = o - l * t.r;
    const int tk = g.perm[t.p0 + l];
    if (tk >= 0 && tk < g.T) g.v[(int64_t)tk * g.ldv + c] = sum_parts(g, p, t, l, c);
  }
}

void launch_shrink_part(const ApplyArgs& g, unsigned grid, size_t lds, hipStream_t stream) {
  static std::atomic<bool> lds_done{false};
  if (lds > 64 * 1024) allow_lds(reinterpret_cast<const void*>(shrink_part_kernel), lds_done);
  hipLaunchKernelGGL(shrink_part_kernel, dim3(grid), dim3(kNT), lds, stream, g);
}

void launch_gather_v(const ApplyArgs& g, unsigned grid, hipStream_t stream) {
  hipLaunchKernelGGL(gather_v_kernel, dim3(grid), dim3(kNT), 0, stream, g);
}

}  // namespace plora_impl
