// k_multi.hip -- plora_apply_multi as one launch.
// every adapter byte is read once per call here: non-temporal reads
#define PLORA_ADAPTER_POLICY 2
// decode-sized slices: a prefetch of 4 chunks covers them
#define PLORA_PREFETCH_CHUNKS 4
#define PLORA_X_WINDOW 2048
#include "plora_dev.h"

namespace plora_impl {

// Several projections in one launch, S > 1 slices per tile: tile slot
// p cap8 + u (numbered as exchange_item numbers slots) is tile u of
// projection p, and exchanges through that slot.
__global__ __launch_bounds__(kNT, kWGPerCU) void apply_multi_kernel(MultiArgs m) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  __shared__ ItemStash stash;
  int slot, s;
  exchange_item((int)blockIdx.x, m.g.fixed_slices, slot, s);
  const int p = slot / m.cap8, u = slot - p * m.cap8;
  if (p >= m.n_proj) return;
  ApplyArgs g = m.g;
  const ProjArgs& q = m.proj[p];
  g.A = q.A; g.B = q.B; g.a_len = q.a_len; g.b_len = q.b_len;
  g.A_pool = q.A_pool; g.B_pool = q.B_pool; g.a_pool_len = q.a_pool_len;
  g.b_pool_len = q.b_pool_len;
  g.a_off = q.a_off; g.b_off = q.b_off; g.ranks = q.ranks; g.scales = q.scales;
  g.y = q.y; g.ldy = q.ldy; g.h_out = q.h_out; g.max_rank = q.max_rank;
  const uint64_t ep = xload(g.xep + slot);
  apply_item(g, s, slot, ep, stash, apply_lds,
             [&](Tile& t, int& my_tok) { return load_tile(g, u, t, my_tok); });
}

void launch_apply_multi(const MultiArgs& m, unsigned grid, size_t lds, hipStream_t stream) {
  static std::atomic<bool> lds_done{false};
  if (lds > 64 * 1024) allow_lds(reinterpret_cast<const void*>(apply_multi_kernel), lds_done);
  hipLaunchKernelGGL(apply_multi_kernel, dim3(grid), dim3(kNT), lds, stream, m);
}

}  // namespace plora_impl
