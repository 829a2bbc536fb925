// k_segapply.hip -- plora_segment_apply as one launch.
// every adapter byte is read once per call here: non-temporal reads
#define PLORA_ADAPTER_POLICY 2
// decode-sized slices: a prefetch of 4 chunks covers them
#define PLORA_PREFETCH_CHUNKS 4
#define PLORA_X_WINDOW 2048
#include "plora_dev.h"

namespace plora_impl {

// plora_segment_apply for T <= kSegApplyMax in the exchange form: above
// kDecodeTokens tokens every work group segments the batch itself (reading
// idx takes the trip the tile record would) and takes its own tile; up to
// kDecodeTokens an item takes its token directly.  Work group 0 also writes
// the segmentation for later calls.  Items are those of apply_kernel.  One
// kernel per form (DIRECT: up to kDecodeTokens tokens), so that each carries
// only its own code (in one kernel, the large decode batch took 48.2 us
// against 47.6).
template <bool DIRECT>
__global__ __launch_bounds__(kNT, kWGPerCU) void segment_apply_kernel(ApplyArgs g,
                                                                      const int32_t* idx,
                                                                      SegOut so) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  __shared__ ItemStash stash;
  __shared__ LocalTile lt;
  request_adapter_args(g);
  int u, s;
  exchange_item((int)blockIdx.x, g.fixed_slices, u, s);
  uint64_t ep = 0;
  static_assert(kDecodeTokens == 64, "wave_segment ranks one wavefront's tokens");
  if constexpr (DIRECT) {
    // Single-token tiles: item (u, s) takes token u itself.  A token's
    // result does not depend on which tile slot carries it (the same slices,
    // summed in the same order), so the items need no ranking: each reads
    // its own id, then its adapter's metadata (decode 11.54 -> 10.74 us
    // against items that took their tiles from every work group's ranking).
    // Work group 0 ranks the batch after its item, to write the
    // segmentation.
    apply_item(g, s, u, ep, stash, apply_lds, [&](Tile& t, int& my_tok) {
      t.bad = false;
      if (u >= g.T) return false;
      int id = idx[u];
      ep = epoch_after(g, u, id);
      id = __builtin_amdgcn_readfirstlane(id);
      if (id < 0 || id >= g.N) return false;
      t.a = id;
      t.p0 = u;
      t.L = 1;
      t.r = g.ranks[id];
      t.s = g.scales[id];
      my_tok = threadIdx.x == 0 ? u : -1;
      return tile_blocks(g, t, my_tok, g.a_off[id], g.b_off[id]);
    });
    if (blockIdx.x == 0 && threadIdx.x < 64) wave_segment(g, idx, so, lt);
    return;
  } else {
    block_segment(g, idx, u, so, blockIdx.x == 0, lt, ep);
    lds_sync();
    apply_item(g, s, u, ep, stash, apply_lds, [&](Tile& t, int& my_tok) {
      // wave-uniform values (from LDS the compiler cannot tell), so that the
      // adapter's metadata and everything derived from it stay scalar
      t.a = __builtin_amdgcn_readfirstlane(lt.a);
      t.p0 = __builtin_amdgcn_readfirstlane(lt.p0);
      t.L = __builtin_amdgcn_readfirstlane(lt.L);
      if (t.L <= 0 || t.a < 0 || t.a >= g.N) return false;
      const int t0 = __builtin_amdgcn_readfirstlane(lt.t0);
      t.r = __builtin_amdgcn_readfirstlane(lt.rank_of[t0]);
      t.s = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(lt.scale_of[t0])));
      const int64_t ao = lt.ao_of[t0], bo = lt.bo_of[t0];
      const int p = t.p0 + (int)threadIdx.x;
      my_tok = (int)threadIdx.x < t.L ? (int)(lt.sorted[p < kSegApplyMax ? p : 0] & lt.tmask)
                                      : -1;
      return tile_blocks(g, t, my_tok, ao, bo);
    });
  }
}

void launch_segment_apply(const ApplyArgs& g, const int32_t* idx, const SegOut& so,
                          unsigned grid, size_t lds, hipStream_t stream) {
  static std::atomic<bool> lds_direct{false}, lds_block{false};
  if (g.T <= kDecodeTokens) {
    if (lds > 64 * 1024)
      allow_lds(reinterpret_cast<const void*>(segment_apply_kernel<true>), lds_direct);
    hipLaunchKernelGGL(segment_apply_kernel<true>, dim3(grid), dim3(kNT), lds, stream, g, idx, so);
  } else {
    if (lds > 64 * 1024)
      allow_lds(reinterpret_cast<const void*>(segment_apply_kernel<false>), lds_block);
    hipLaunchKernelGGL(segment_apply_kernel<false>, dim3(grid), dim3(kNT), lds, stream, g, idx,
                       so);
  }
}

}  // namespace plora_impl
