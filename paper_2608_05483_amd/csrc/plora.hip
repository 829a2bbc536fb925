// plora.hip -- host side and C ABI of the gfx950 batched heterogeneous-
// adapter LoRA apply (declared in include/plora.h).
//
// What runs where:
//   plora_segment  one work group.  Up to 1024 tokens: one thread per token
//                  ranks its (adapter id, token index) key by counting the
//                  keys before it in LDS.  Larger batches: LSD radix sort of
//                  packed keys in LDS with ballot-based stable ranking per
//                  wavefront.  Both then write the segment and tile lists.
//   plora_shrink   one work group per work item: one tile (up to
//   plora_expand   PLORA_TILE_TOKENS tokens of one adapter, section VI-B's
//   plora_apply    per-adapter batch B_i split into tiles) and one slice of
//                  h_in or of the y columns; plora_apply is one launch for
//                  batches of up to kFusedTokens tokens (with the tile's
//                  slices exchanging partial v through the workspace when
//                  the batch has few tiles) and two above; details above the
//                  apply kernels below.
#include "plora_dev.h"

#include <mutex>

namespace plora_impl {
namespace {
// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline int ceil_log2(int64_t v) {
  int b = 0;
  while ((int64_t(1) << b) < v) ++b;
  return b;
}

// Every rank from 0 (a no-op adapter) to max_rank is applied.
inline bool usable_rank(int r, int max_rank) { return r >= 0 && r <= max_rank; }

// Compute units of the current device, queried once per device.
int cu_count() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < 64) {
    const int c = cache[dev].load();
    if (c > 0) return c;
  }
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n <= 0)
    n = 256;
  if (dev < 64) cache[dev].store(n);
  return n;
}

// Apply work groups that one compute unit holds at once, as its LDS allows:
// the dynamic section for this h_in and max_rank plus the largest static one
// (segment_apply_kernel's), with slack for the allocation granularity; at
// most kWGPerCU.  At max_rank 128 (82 KB dynamic) that is one.
int wg_per_cu(int32_t h_in, int32_t max_rank) {
  const size_t per = smem_bytes(h_in, max_rank) + sizeof(LocalTile) + sizeof(ItemStash) + 1024;
  return std::max(1, std::min<int>(kWGPerCU, (int)(kMaxLds / per)));
}

// Resident apply work groups of the device at this h_in and max_rank.
int slots_for_device(int32_t h_in, int32_t max_rank) {
  return std::max(8, cu_count() * wg_per_cu(h_in, max_rank));
}

// One work group per item: the most items make_plan can produce for any tile
// count up to tile_cap with at most s_max slices per tile (see there).
unsigned grid_for(const ApplyArgs& g, int s_max) {
  const int64_t cap8 = (g.tile_cap + 7) & ~7;
  if (g.fixed_slices > 0) return (unsigned)std::max<int64_t>(8, cap8 * g.fixed_slices);
  if (s_max <= 1) return (unsigned)std::max<int64_t>(8, cap8);
  // fit = round(kPlanItems slots / n8) >= 2 needs n8 <= 2/3 kPlanItems slots,
  // so n8 fit <= 4/3 kPlanItems slots
  const int64_t spread = ((int64_t)kPlanItems * g.slots * 4 / 3 + 8 + 7) & ~7;
  return (unsigned)std::max<int64_t>(8, std::min(cap8 * s_max, std::max(cap8, spread)));
}

// Most h_in slices per tile: slices of at least 512 rows, at most 8.
int ks_max_for(int h_in) { return std::max(1, std::min(8, h_in / 512)); }

// plora_apply runs as one launch for batches of up to kFusedTokens tokens.
bool fused_for(int32_t T) { return T <= kFusedTokens; }

// Slices per tile of the one-launch form: the resident work groups (target,
// from slots_for_device, so that every item of the launch is resident at
// once and no exchange partner waits to be dispatched) over the most tiles
// the batch can produce (rounded up to 8), to nearest, within
// [1, min(ks_max, js_max)]; 1 when the tile slots outnumber the exchange
// regions.  The workspace size does not depend on it.  plora_shrink and
// plora_expand take the same slices for such batches, so their results carry
// the very bits of the one-launch apply.
// (For n projections in one launch, plora_apply_multi, the tile slots of
// all of them count: n cap8 of them, and the limit is the smallest
// projection's.)
int fused_slices_for(int slots8, int lim, int target) {
  if (slots8 <= 0 || slots8 > kXSlots) return 1;
  return std::max(1, std::min(lim, (target + slots8 / 2) / slots8));
}

int slice_limit(int32_t h_in, int32_t h_out) {
  return std::min(ks_max_for(h_in), std::max(1, h_out / kMinSlice));
}

int fused_slices(int32_t tile_cap, int32_t h_in, int32_t h_out, int32_t max_rank) {
  return fused_slices_for((tile_cap + 7) & ~7, slice_limit(h_in, h_out),
                          slots_for_device(h_in, max_rank));
}

// Workspace sections, each 256-byte aligned: the epochs of the exchange's
// tile slots (64-bit, kXSlots of them) and the counters; the readiness words
// of the one-launch two-part form (kReadyTiles); the exchange regions of the
// one-launch form (kSlotWords 64-bit words for each of the first
// min(cap8, kXSlots) tile slots); then the partial sums of v of the
// two-part forms and plora_shrink (fp32 [ks_max][T][max_rank]).  The epochs,
// the readiness words and each slot's region sit at the same offsets for
// every batch size, rank and slice count, which their tags rely on (no
// other section ever writes there); only the last section's place and size
// follow the shapes.
struct WsLayout {
  size_t xep, counters, ready, xw, vpart, total;
};

// Workspace bytes of the multi-work-group segmentation (batches above 1024
// tokens over 2048 to 8191 adapters: a table of (ceil(T / 1024) + 1) x
// (N + 2) int32, the groups' counts and the keys' first positions); 0 where
// plora_segment takes a one-work-group kernel (fewer adapters: the counting
// sort of kCountKeys keys; more: the radix sort).
size_t segment_scratch_bytes(int32_t T, int32_t N) {
  if (T <= 1024 || N < 0 || N + 1 <= kCountKeys || N + 1 > 8192) return 0;
  const size_t groups = ((size_t)T + 1023) / 1024;
  return (((groups + 1) * (size_t)(N + 2) * sizeof(int32_t)) + 255) & ~(size_t)255;
}

constexpr int kCounters = 2;   // workspace counters after the epochs (see ApplyArgs)
// Readiness words of the one-launch two-part form (one per tile slot); a
// batch whose tile capacity exceeds it takes two launches.
constexpr int32_t kReadyTiles = 4096;

constexpr size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// n adapter stacks (the projections of plora_apply_multi; n = 1 otherwise)
// sharing the batch: n cap8 tile slots, and the largest partial-sum section.
WsLayout ws_layout(int32_t T, const plora_adapters* ad, int n = 1) {
  WsLayout l{0, 0, 0, 0, 0, 0};
  if (!ad || T <= 0 || n < 1) return l;
  size_t nvp = 0;
  for (int p = 0; p < n; ++p) {
    if (ad[p].h_in <= 0 || ad[p].max_rank <= 0) return l;
    nvp = std::max(nvp, (size_t)ks_max_for(ad[p].h_in) * T * ad[p].max_rank * sizeof(float));
  }
  // the last section also serves plora_segment_apply's segmentation, which
  // runs before the partial sums are written
  nvp = std::max(nvp, segment_scratch_bytes(T, ad->n_adapters));
  const int32_t tcap = plora_tile_capacity(T, ad->n_adapters);
  const size_t slots = (size_t)std::min(kXSlots, std::max(8, n * ((tcap + 7) & ~7)));
  l.xep = 0;
  l.counters = (size_t)kXSlots * sizeof(uint64_t);
  l.ready = align256(l.counters + kCounters * sizeof(uint64_t));
  l.xw = align256(l.ready + kReadyTiles * sizeof(uint64_t));
  l.vpart = align256(l.xw + slots * kSlotWords * sizeof(uint64_t));
  l.total = align256(l.vpart + nvp);
  return l;
}

size_t workspace_bytes(int32_t T, const plora_adapters* ad) { return ws_layout(T, ad).total; }

plora_status check_adapters_host(const plora_adapters* ad) {
  if (!ad) return PLORA_ERR_INVALID_ARG;
  if (ad->n_adapters < 0 || ad->h_in <= 0 || ad->h_out <= 0 || ad->max_rank < 0 ||
      ad->a_len < 0 || ad->b_len < 0 || ad->a_pool_len < 0 || ad->b_pool_len < 0)
    return PLORA_ERR_INVALID_ARG;
  if ((ad->h_in & 7) || (ad->h_out & 7)) return PLORA_ERR_UNSUPPORTED;
  // adapter blocks are read through 32-bit byte offsets
  if ((int64_t)std::max(ad->h_in, ad->h_out) * std::max(ad->max_rank, 0) * 2 >= (INT64_C(1) << 31))
    return PLORA_ERR_UNSUPPORTED;
  if (ad->max_rank == 0 || (ad->max_rank & 7) || ad->max_rank > PLORA_MAX_RANK)
    return PLORA_ERR_UNSUPPORTED;
  if (smem_bytes(ad->h_in, ad->max_rank) > kMaxLds) return PLORA_ERR_UNSUPPORTED;
  if (ad->n_adapters > 0 &&
      ((!ad->A && !ad->A_pool) || (!ad->B && !ad->B_pool) || !ad->a_off || !ad->b_off ||
       !ad->ranks || !ad->scales))
    return PLORA_ERR_INVALID_ARG;
  if (!aligned16(ad->A) || !aligned16(ad->B) || !aligned16(ad->a_off) ||
      !aligned16(ad->b_off) || !aligned16(ad->ranks) || !aligned16(ad->scales) ||
      !aligned16(ad->A_pool) || !aligned16(ad->B_pool))
    return PLORA_ERR_UNSUPPORTED;
  return PLORA_OK;
}

// Host mirror of adapter_block: whether offset o names an n-element block
// inside the device stack (o >= 0) or the pool (o < 0).
bool block_ok(const uint16_t* dev, int64_t dev_len, const uint16_t* pool, int64_t pool_len,
              int64_t o, int64_t n) {
  const bool in_pool = o < 0;
  const int64_t e = in_pool ? -1 - o : o;
  return (in_pool ? pool : dev) && (e & 7) == 0 && e + n <= (in_pool ? pool_len : dev_len);
}

plora_status check_segments_host(const plora_segments* seg, int32_t N) {
  if (!seg) return PLORA_ERR_INVALID_ARG;
  if (seg->T < 0) return PLORA_ERR_INVALID_ARG;
  if (seg->T > PLORA_MAX_TOKENS) return PLORA_ERR_UNSUPPORTED;
  if (seg->cap != std::min(seg->T, N) || seg->tile_cap != plora_tile_capacity(seg->T, N))
    return PLORA_ERR_INVALID_ARG;
  if (seg->T == 0) return PLORA_OK;
  if (!seg->perm || !seg->seg_ptr || !seg->seg_id || !seg->meta || !seg->tiles)
    return PLORA_ERR_INVALID_ARG;
  if (!aligned16(seg->tiles) || !aligned16(seg->perm)) return PLORA_ERR_UNSUPPORTED;
  return PLORA_OK;
}

// The status of a call reports its own launch: an error left pending by
// earlier HIP calls of the caller is cleared before launching.
void clear_stale_error() { (void)hipGetLastError(); }

std::atomic<int32_t> g_last_hip_error{0};
std::atomic<int32_t> g_exchange_polls{kSpinLimit};

plora_status launch_status() {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return PLORA_OK;
  g_last_hip_error.store((int32_t)e);
  return PLORA_ERR_HIP;
}

plora_status prepare(const plora_adapters* ad, const plora_segments* seg, void* ws,
                     size_t ws_bytes, ApplyArgs& g, bool needs_ws) {
  plora_status st = check_adapters_host(ad);
  if (st != PLORA_OK) return st;
  st = check_segments_host(seg, ad->n_adapters);
  if (st != PLORA_OK) return st;
  memset(&g, 0, sizeof g);
  g.A = ad->A; g.B = ad->B; g.a_len = ad->a_len; g.b_len = ad->b_len;
  g.A_pool = ad->A_pool; g.B_pool = ad->B_pool;
  g.a_pool_len = ad->a_pool_len; g.b_pool_len = ad->b_pool_len;
  g.a_off = ad->a_off; g.b_off = ad->b_off; g.ranks = ad->ranks; g.scales = ad->scales;
  g.perm = seg->perm;
  g.tiles = reinterpret_cast<const int4*>(seg->tiles);
  g.meta = seg->meta;
  g.T = seg->T; g.N = ad->n_adapters; g.h_in = ad->h_in; g.h_out = ad->h_out;
  g.max_rank = ad->max_rank; g.tile_cap = seg->tile_cap;
  g.js_max = std::max(1, ad->h_out / kMinSlice);
  g.slots = slots_for_device(ad->h_in, ad->max_rank);
  // one-launch batches take either S > 1 fixed slices per tile (exchange
  // form) or one h_in slice and device-chosen column slices; the split calls
  // take the same slices, so that they reproduce the apply's bits
  const int fs =
      fused_for(seg->T) ? fused_slices(seg->tile_cap, ad->h_in, ad->h_out, ad->max_rank) : 0;
  g.fixed_slices = fs > 1 ? fs : 0;
  g.polls = g_exchange_polls.load();
  g.ks_max = fs == 1 ? 1 : ks_max_for(ad->h_in);
  g.count_skips = 1;
  if (needs_ws && seg->T > 0) {
    const WsLayout l = ws_layout(seg->T, ad);
    if (!ws) return PLORA_ERR_INVALID_ARG;
    if (!aligned16(ws)) return PLORA_ERR_UNSUPPORTED;
    if (ws_bytes < l.total) return PLORA_ERR_WORKSPACE_TOO_SMALL;
    char* base = reinterpret_cast<char*>(ws);
    g.vpart = reinterpret_cast<float*>(base + l.vpart);
    g.xw = reinterpret_cast<uint64_t*>(base + l.xw);
    g.xep = reinterpret_cast<uint64_t*>(base + l.xep);
    g.counters = reinterpret_cast<unsigned long long*>(base + l.counters);
    g.ready = reinterpret_cast<uint64_t*>(base + l.ready);
  } else if (ws && aligned16(ws) && ws_bytes >= ws_layout(1, ad).xw) {
    // a call that needs no workspace still counts into one it is given
    g.counters = reinterpret_cast<unsigned long long*>(reinterpret_cast<char*>(ws) +
                                                       ws_layout(1, ad).counters);
  }
  return PLORA_OK;
}

// plora_segment_apply runs as one launch for batches of up to kSegApplyMax
// tokens in the exchange form (words (key << tbits) | t with key <= N + 1
// and tbits 6 up to 64 tokens, 8 above; tokens without an adapter read
// adapter 0's metadata, so N >= 1).
bool segment_apply_one_launch(int32_t T, const plora_adapters* ad) {
  const int32_t n_limit = T <= 64 ? (1 << 26) - 1 : (1 << 24) - 1;
  return T <= kSegApplyMax && ad->n_adapters > 0 && ad->n_adapters < n_limit &&
         fused_slices(plora_tile_capacity(T, ad->n_adapters), ad->h_in, ad->h_out,
                      ad->max_rank) > 1;
}

typedef void (*ItemLauncher)(const ApplyArgs&, unsigned, size_t, hipStream_t);

plora_status launch_items(ItemLauncher launch, const ApplyArgs& g, int s_max,
                          hipStream_t stream) {
  const size_t lds = smem_bytes(g.h_in, g.max_rank);
  const unsigned grid = grid_for(g, s_max);
  clear_stale_error();
  launch(g, grid, lds, stream);
  return launch_status();
}

// ---------------------------------------------------------------------------
// the allocation-free entry point's scratch
// ---------------------------------------------------------------------------

// Largest batch plora_segment_apply_noalloc takes, and the workspace such a
// batch needs at most: the exchange regions of min(kXSlots, cap8) tile
// slots (cap8 <= kNoAllocTokens) and the partial sums of v for up to 8
// slices of h_in at rank 128, after the epochs, counters and readiness words.
constexpr int32_t kNoAllocTokens = 256;
constexpr size_t kScratchBytes =
    align256(align256(align256(align256((size_t)(kXSlots + kCounters) * sizeof(uint64_t)) +
                               (size_t)kReadyTiles * sizeof(uint64_t)) +
                      (size_t)std::min(kXSlots, kNoAllocTokens) * kSlotWords * sizeof(uint64_t)) +
             (size_t)8 * kNoAllocTokens * PLORA_MAX_RANK * sizeof(float));

// The device address of `scratch` on the current device, looked up once per
// device with that device current (each device holds its own copy of the
// array at its own address); null if the lookup fails.
void* scratch_for_device();

}  // namespace
}  // namespace plora_impl

// The workspace of plora_segment_apply_noalloc: one per device, zero from
// the module's load, then carrying the exchange's epochs from call to call as
// any workspace does.  Host code never uses this name as an address (it is a
// host-side stand-in); it takes the pointer scratch_for_device() returns.
static __device__ __align__(256) unsigned char scratch[plora_impl::kScratchBytes];

namespace plora_impl {
namespace {

std::mutex g_scratch_mu;
void* g_scratch_ptr[64];

void* scratch_for_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace
}  // namespace plora_impl

using namespace plora_impl;

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------

extern "C" {

int32_t plora_tile_capacity(int32_t T, int32_t n_adapters) {
  if (T <= 0) return 0;
  const int32_t cap = std::min(T, std::max(n_adapters, 0));
  return std::min(T, cap + T / tile_tokens(T));
}

size_t plora_workspace_bytes(int32_t T, const plora_adapters* ad) {
  return workspace_bytes(T, ad);
}

plora_status plora_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream) {
  if (ws_bytes == 0) return PLORA_OK;
  if (!ws) return PLORA_ERR_INVALID_ARG;
  if (!aligned16(ws) || (ws_bytes & 15)) return PLORA_ERR_UNSUPPORTED;
  const size_t n16 = ws_bytes / 16;
  const unsigned blocks = (unsigned)std::min<size_t>((n16 + 255) / 256, 4096);
  clear_stale_error();
  launch_zero(reinterpret_cast<uint4*>(ws), n16, blocks, stream);
  return launch_status();
}

size_t plora_segment_workspace_bytes(int32_t T, int32_t n_adapters) {
  return segment_scratch_bytes(T, n_adapters);
}

plora_status plora_segment(const int32_t* idx, const plora_segments* seg, int32_t n_adapters,
                           void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!seg || n_adapters < 0) return PLORA_ERR_INVALID_ARG;
  plora_status st = check_segments_host(seg, n_adapters);
  if (st != PLORA_OK) return st;
  const int32_t T = seg->T;
  if (T == 0) return PLORA_OK;
  if (!idx) return PLORA_ERR_INVALID_ARG;
  const int tbits = ceil_log2(T);
  const int key_bits = n_adapters > 0 ? 32 - __builtin_clz((unsigned)n_adapters) : 0;
  if (tbits + key_bits > 32) return PLORA_ERR_UNSUPPORTED;
  clear_stale_error();
  int4* tiles = reinterpret_cast<int4*>(seg->tiles);
  const size_t scratch = segment_scratch_bytes(T, n_adapters);
  if (scratch > 0 && ws && aligned16(ws) && ws_bytes >= scratch) {
    launch_segment_groups(idx, T, n_adapters, seg->cap, seg->tile_cap, seg->perm, seg->seg_ptr,
                          seg->seg_id, seg->meta, tiles, reinterpret_cast<int32_t*>(ws), stream);
  } else {
    launch_segment(idx, T, n_adapters, seg->cap, seg->tile_cap, tbits, key_bits, seg->perm,
                   seg->seg_ptr, seg->seg_id, seg->meta, tiles, stream);
  }
  return launch_status();
}

plora_status plora_shrink(const uint16_t* x, int64_t ldx, const plora_adapters* ad,
                          const plora_segments* seg, float* v, int64_t ldv, void* ws,
                          size_t ws_bytes, hipStream_t stream) {
  ApplyArgs g;
  plora_status st = prepare(ad, seg, ws, ws_bytes, g, true);
  if (st != PLORA_OK) return st;
  if (seg->T == 0) return PLORA_OK;
  if (!x || !v) return PLORA_ERR_INVALID_ARG;
  if (ldx < ad->h_in || ldv < ad->max_rank) return PLORA_ERR_INVALID_ARG;
  if ((ldx & 7) || (ldv & 3) || !aligned16(x) || !aligned16(v)) return PLORA_ERR_UNSUPPORTED;
  g.x = x; g.ldx = ldx; g.v = v; g.ldv = ldv;
  st = launch_items(launch_shrink_part, g, g.ks_max, stream);
  if (st != PLORA_OK) return st;
  clear_stale_error();
  launch_gather_v(g, (unsigned)g.tile_cap, stream);
  return launch_status();
}

plora_status plora_expand(const float* v, int64_t ldv, const plora_adapters* ad,
                          const plora_segments* seg, uint16_t* y, int64_t ldy, void* ws,
                          size_t ws_bytes, hipStream_t stream) {
  ApplyArgs g;
  plora_status st = prepare(ad, seg, ws, ws_bytes, g, false);
  if (st != PLORA_OK) return st;
  if (seg->T == 0) return PLORA_OK;
  if (!v || !y) return PLORA_ERR_INVALID_ARG;
  if (ldy < ad->h_out || ldv < ad->max_rank) return PLORA_ERR_INVALID_ARG;
  if ((ldy & 7) || (ldv & 3) || !aligned16(y) || !aligned16(v)) return PLORA_ERR_UNSUPPORTED;
  g.v = const_cast<float*>(v); g.ldv = ldv; g.y = y; g.ldy = ldy;
  return launch_items(launch_expand_v, g, g.js_max, stream);
}

plora_status plora_apply(const uint16_t* x, int64_t ldx, const plora_adapters* ad,
                         const plora_segments* seg, uint16_t* y, int64_t ldy, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  ApplyArgs g;
  plora_status st = prepare(ad, seg, ws, ws_bytes, g, true);
  if (st != PLORA_OK) return st;
  if (seg->T == 0) return PLORA_OK;
  if (!x || !y) return PLORA_ERR_INVALID_ARG;
  if (ldx < ad->h_in || ldy < ad->h_out) return PLORA_ERR_INVALID_ARG;
  if ((ldx & 7) || (ldy & 7) || !aligned16(x) || !aligned16(y)) return PLORA_ERR_UNSUPPORTED;
  g.x = x; g.ldx = ldx; g.y = y; g.ldy = ldy;
  if (g.fixed_slices > 1) return launch_items(launch_apply, g, g.js_max, stream);
  if (fused_for(seg->T))
    return launch_items(launch_apply_cols, g, g.js_max, stream);
  if (g.tile_cap <= kReadyTiles) {
    clear_stale_error();
    launch_parts(g, grid_for(g, g.ks_max), grid_for(g, g.js_max),
                 smem_bytes(g.h_in, g.max_rank), stream);
    return launch_status();
  }
  ApplyArgs gs = g;
  gs.count_skips = 0;                 // the expand launch counts the call's skips
  st = launch_items(launch_shrink_part, gs, g.ks_max, stream);
  if (st != PLORA_OK) return st;
  return launch_items(launch_expand_parts, g, g.js_max, stream);
}

plora_status plora_segment_apply_noalloc(const int32_t* idx, const uint16_t* x, int64_t ldx,
                                         const plora_adapters* ad, const plora_segments* seg,
                                         uint16_t* y, int64_t ldy, hipStream_t stream) {
  if (!ad || !seg) return PLORA_ERR_INVALID_ARG;
  plora_status st = check_adapters_host(ad);
  if (st != PLORA_OK) return st;
  st = check_segments_host(seg, ad->n_adapters);
  if (st != PLORA_OK) return st;
  if (seg->T > kNoAllocTokens) return PLORA_ERR_UNSUPPORTED;
  if (seg->T == 0) return PLORA_OK;
  if (!idx || !x || !y) return PLORA_ERR_INVALID_ARG;
  if (ldx < ad->h_in || ldy < ad->h_out) return PLORA_ERR_INVALID_ARG;
  if ((ldx & 7) || (ldy & 7) || !aligned16(x) || !aligned16(y)) return PLORA_ERR_UNSUPPORTED;
  if (ws_layout(seg->T, ad).total > kScratchBytes) return PLORA_ERR_UNSUPPORTED;
  void* ws = scratch_for_device();
  if (!ws) {
    g_last_hip_error.store((int32_t)hipErrorInvalidSymbol);
    return PLORA_ERR_HIP;
  }
  return plora_segment_apply(idx, x, ldx, ad, seg, y, ldy, ws, kScratchBytes, stream);
}

int32_t plora_segment_apply_launches(int32_t T, const plora_adapters* ad) {
  if (T <= 0 || !ad || check_adapters_host(ad) != PLORA_OK) return 0;
  if (segment_apply_one_launch(T, ad)) return 1;
  return fused_for(T) || plora_tile_capacity(T, ad->n_adapters) <= kReadyTiles ? 2 : 3;
}

plora_status plora_segment_apply(const int32_t* idx, const uint16_t* x, int64_t ldx,
                                 const plora_adapters* ad, const plora_segments* seg,
                                 uint16_t* y, int64_t ldy, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  ApplyArgs g;
  plora_status st = prepare(ad, seg, ws, ws_bytes, g, true);
  if (st != PLORA_OK) return st;
  const int32_t T = seg->T;
  if (T == 0) return PLORA_OK;
  if (!idx || !x || !y) return PLORA_ERR_INVALID_ARG;
  if (ldx < ad->h_in || ldy < ad->h_out) return PLORA_ERR_INVALID_ARG;
  if ((ldx & 7) || (ldy & 7) || !aligned16(x) || !aligned16(y)) return PLORA_ERR_UNSUPPORTED;
  if (!segment_apply_one_launch(T, ad)) {
    // the segmentation's scratch is the partial-sum section, free until the
    // apply that follows on the same stream
    const WsLayout l = ws_layout(T, ad);
    st = plora_segment(idx, seg, ad->n_adapters, reinterpret_cast<char*>(ws) + l.vpart,
                       ws_bytes - l.vpart, stream);
    if (st != PLORA_OK) return st;
    return plora_apply(x, ldx, ad, seg, y, ldy, ws, ws_bytes, stream);
  }
  g.x = x; g.ldx = ldx; g.y = y; g.ldy = ldy;
  const SegOut so{seg->perm, seg->seg_ptr, seg->seg_id, seg->meta,
                  reinterpret_cast<int4*>(seg->tiles), seg->cap, seg->tile_cap};
  clear_stale_error();
  launch_segment_apply(g, idx, so, grid_for(g, g.js_max), smem_bytes(g.h_in, g.max_rank), stream);
  return launch_status();
}

size_t plora_workspace_bytes_multi(int32_t T, const plora_adapters* ads, int32_t n_proj) {
  if (!ads || n_proj < 1 || n_proj > PLORA_MAX_PROJECTIONS) return 0;
  return ws_layout(T, ads, n_proj).total;
}

plora_status plora_apply_multi(const uint16_t* x, int64_t ldx, const plora_adapters* ads,
                               int32_t n_proj, const plora_segments* seg,
                               uint16_t* const* ys, const int64_t* ldys, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  if (!ads || !ys || !ldys || n_proj < 1) return PLORA_ERR_INVALID_ARG;
  if (n_proj > PLORA_MAX_PROJECTIONS) return PLORA_ERR_UNSUPPORTED;
  for (int p = 0; p < n_proj; ++p) {
    const plora_status st = check_adapters_host(&ads[p]);
    if (st != PLORA_OK) return st;
    if (ads[p].n_adapters != ads[0].n_adapters || ads[p].h_in != ads[0].h_in)
      return PLORA_ERR_INVALID_ARG;
  }
  plora_status st = check_segments_host(seg, ads[0].n_adapters);
  if (st != PLORA_OK) return st;
  if (seg->T == 0) return PLORA_OK;
  if (!x || ldx < ads[0].h_in) return PLORA_ERR_INVALID_ARG;
  if ((ldx & 7) || !aligned16(x)) return PLORA_ERR_UNSUPPORTED;
  int lim = PLORA_MAX_RANK, max_rank = 0;
  for (int p = 0; p < n_proj; ++p) {
    if (!ys[p] || ldys[p] < ads[p].h_out) return PLORA_ERR_INVALID_ARG;
    if ((ldys[p] & 7) || !aligned16(ys[p])) return PLORA_ERR_UNSUPPORTED;
    lim = std::min(lim, slice_limit(ads[p].h_in, ads[p].h_out));
    max_rank = std::max(max_rank, ads[p].max_rank);
  }
  if (smem_bytes(ads[0].h_in, max_rank) > kMaxLds) return PLORA_ERR_UNSUPPORTED;
  const WsLayout l = ws_layout(seg->T, ads, n_proj);
  if (!ws) return PLORA_ERR_INVALID_ARG;
  if (!aligned16(ws)) return PLORA_ERR_UNSUPPORTED;
  if (ws_bytes < l.total) return PLORA_ERR_WORKSPACE_TOO_SMALL;
  const int cap8 = (seg->tile_cap + 7) & ~7;
  const int S = fused_for(seg->T)
                    ? fused_slices_for(n_proj * cap8, lim, slots_for_device(ads[0].h_in, max_rank))
                    : 1;
  if (S <= 1) {
    // one projection after another (the launch overheads are small next to
    // batches this large)
    for (int p = 0; p < n_proj; ++p) {
      st = plora_apply(x, ldx, &ads[p], seg, ys[p], ldys[p], ws, ws_bytes, stream);
      if (st != PLORA_OK) return st;
    }
    return PLORA_OK;
  }
  MultiArgs m;
  memset(&m, 0, sizeof m);
  st = prepare(&ads[0], seg, ws, ws_bytes, m.g, true);
  if (st != PLORA_OK) return st;
  char* base = reinterpret_cast<char*>(ws);
  m.g.vpart = reinterpret_cast<float*>(base + l.vpart);
  m.g.x = x;
  m.g.ldx = ldx;
  m.g.fixed_slices = S;
  m.n_proj = n_proj;
  m.cap8 = cap8;
  for (int p = 0; p < n_proj; ++p) {
    ProjArgs& q = m.proj[p];
    q.A = ads[p].A; q.B = ads[p].B; q.a_len = ads[p].a_len; q.b_len = ads[p].b_len;
    q.A_pool = ads[p].A_pool; q.B_pool = ads[p].B_pool;
    q.a_pool_len = ads[p].a_pool_len; q.b_pool_len = ads[p].b_pool_len;
    q.a_off = ads[p].a_off; q.b_off = ads[p].b_off; q.ranks = ads[p].ranks;
    q.scales = ads[p].scales; q.y = ys[p]; q.ldy = ldys[p]; q.h_out = ads[p].h_out;
    q.max_rank = ads[p].max_rank;
  }
  clear_stale_error();
  launch_apply_multi(m, (unsigned)(n_proj * cap8 * S), smem_bytes(ads[0].h_in, max_rank), stream);
  return launch_status();
}

plora_status plora_check_adapters(const plora_adapters* ad, int32_t* bad_index,
                                  hipStream_t stream) {
  plora_status st = check_adapters_host(ad);
  if (st != PLORA_OK) return st;
  const int N = ad->n_adapters;
  if (bad_index) *bad_index = -1;
  if (N == 0) return PLORA_OK;
  int32_t* ranks = new int32_t[N];
  int64_t* ao = new int64_t[N];
  int64_t* bo = new int64_t[N];
  plora_status res = PLORA_OK;
  if (hipMemcpyAsync(ranks, ad->ranks, sizeof(int32_t) * N, hipMemcpyDeviceToHost, stream) !=
          hipSuccess ||
      hipMemcpyAsync(ao, ad->a_off, sizeof(int64_t) * N, hipMemcpyDeviceToHost, stream) !=
          hipSuccess ||
      hipMemcpyAsync(bo, ad->b_off, sizeof(int64_t) * N, hipMemcpyDeviceToHost, stream) !=
          hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess) {
    res = PLORA_ERR_HIP;
  } else {
    for (int i = 0; i < N; ++i) {
      const int r = ranks[i];
      bool ok = usable_rank(r, ad->max_rank);
      if (ok && r > 0) {
        ok = block_ok(ad->A, ad->a_len, ad->A_pool, ad->a_pool_len, ao[i],
                      (int64_t)ad->h_in * r) &&
             block_ok(ad->B, ad->b_len, ad->B_pool, ad->b_pool_len, bo[i],
                      (int64_t)ad->h_out * r);
      }
      if (!ok) {
        if (bad_index) *bad_index = i;
        res = PLORA_ERR_INVALID_ARG;
        break;
      }
    }
  }
  delete[] ranks;
  delete[] ao;
  delete[] bo;
  return res;
}

const char* plora_status_string(plora_status status) {
  switch (status) {
    case PLORA_OK: return "PLORA_OK";
    case PLORA_ERR_INVALID_ARG: return "PLORA_ERR_INVALID_ARG";
    case PLORA_ERR_UNSUPPORTED: return "PLORA_ERR_UNSUPPORTED";
    case PLORA_ERR_WORKSPACE_TOO_SMALL: return "PLORA_ERR_WORKSPACE_TOO_SMALL";
    case PLORA_ERR_HIP: return "PLORA_ERR_HIP";
  }
  return "PLORA_ERR_UNKNOWN";
}

plora_status plora_pool_device_pointer(const void* host, const void** device) {
  if (!host || !device) return PLORA_ERR_INVALID_ARG;
  *device = nullptr;
  void* d = nullptr;
  if (hipHostGetDevicePointer(&d, const_cast<void*>(host), 0) != hipSuccess || !d) {
    (void)hipGetLastError();
    return PLORA_ERR_UNSUPPORTED;
  }
  *device = d;
  return PLORA_OK;
}

plora_status plora_workspace_counters(const void* ws, size_t ws_bytes, int64_t* counts,
                                      hipStream_t stream) {
  if (!ws || !counts) return PLORA_ERR_INVALID_ARG;
  const size_t off = (size_t)kXSlots * sizeof(uint64_t);
  if (!aligned16(ws)) return PLORA_ERR_UNSUPPORTED;
  if (ws_bytes < off + kCounters * sizeof(uint64_t)) return PLORA_ERR_WORKSPACE_TOO_SMALL;
  uint64_t host[kCounters];
  if (hipMemcpyAsync(host, reinterpret_cast<const char*>(ws) + off, sizeof host,
                     hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess) {
    g_last_hip_error.store((int32_t)hipGetLastError());
    return PLORA_ERR_HIP;
  }
  for (int i = 0; i < kCounters; ++i) counts[i] = (int64_t)host[i];
  return PLORA_OK;
}

int32_t plora_debug_last_hip_error(void) { return g_last_hip_error.load(); }

void plora_debug_set_exchange_polls(int32_t polls) {
  g_exchange_polls.store(polls < 0 ? kSpinLimit : polls);
}

}  // extern "C"
