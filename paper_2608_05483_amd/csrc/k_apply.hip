// k_apply.hip -- plora_apply as one launch with the slice exchange.
// every adapter byte is read once per call here: non-temporal reads
#define PLORA_ADAPTER_POLICY 2
// decode-sized slices: a prefetch of 4 chunks covers them
#define PLORA_PREFETCH_CHUNKS 4
#define PLORA_X_WINDOW 2048
#include "plora_dev.h"

namespace plora_impl {

// plora_apply as one launch, tiles in S > 1 slices (S chosen on the host, so
// the item needs no count from the device): work group blockIdx.x is slice
// s of tile u, tile slot u, as exchange_item numbers them, so the work
// groups a tile waits on are dispatched with it.
__global__ __launch_bounds__(kNT, kWGPerCU) void apply_kernel(ApplyArgs g) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  __shared__ ItemStash stash;
  request_adapter_args(g);
  int u, s;
  exchange_item((int)blockIdx.x, g.fixed_slices, u, s);
  // the slot's epoch is requested together with the tile record (the host
  // made sure the slot count is at most kXSlots); apply_item reads it once
  // the tile is loaded
  uint64_t ep = 0;
  apply_item(g, s, u, ep, stash, apply_lds, [&](Tile& t, int& my_tok) {
    // load_tile, with the epoch requested right after the tile record
    t.bad = false;
    if (u >= g.tile_cap) return false;
    int4 ti = g.tiles[u];
    ep = epoch_after(g, u, ti.x);
    if (!tile_from_record(g, ti, t)) return false;
    my_tok = (int)threadIdx.x < t.L ? g.perm[t.p0 + threadIdx.x] : -1;
    return tile_adapter(g, t, my_tok);
  });
}

void launch_apply(const ApplyArgs& g, unsigned grid, size_t lds, hipStream_t stream) {
  static std::atomic<bool> lds_done{false};
  if (lds > 64 * 1024) allow_lds(reinterpret_cast<const void*>(apply_kernel), lds_done);
  hipLaunchKernelGGL(apply_kernel, dim3(grid), dim3(kNT), lds, stream, g);
}

}  // namespace plora_impl
