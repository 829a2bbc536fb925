// plora_dev.h -- device code shared by the gfx950 kernels of the batched
// heterogeneous-adapter LoRA apply (C ABI in include/plora.h).
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
//
// Each kernel lives in a source file of its own (k_*.hip, compiled in
// parallel), with a host launcher declared at the end of this header;
// plora.hip holds the host side and the C ABI.
#ifndef PLORA_DEV_H
#define PLORA_DEV_H

#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <atomic>

#include "plora.h"

namespace plora_impl {

constexpr int kTT = PLORA_TILE_TOKENS;   // most tokens per tile
static_assert((kTT & (kTT - 1)) == 0, "tile positions are taken modulo kTT with a mask");
constexpr int kFusedTokens = 256;    // largest batch plora_apply runs as one launch
// Tokens per tile by batch size.  Batches of up to kFusedTokens tokens (the
// one-launch forms) are cut into tiles of kSmallTile tokens, which the
// vector path takes at every rank: with tiles of up to kTT tokens, a hot
// adapter's tile of 3 to 14 tokens took the matrix path and finished about
// 3 us after the single-token tiles, setting the launch's length.  A hot
// adapter then has several tiles that read its blocks at the same time (the
// repeats are cache hits).  Batches of up to kDecodeTokens tokens (decode)
// take single-token tiles: every item then has the same chain of loads, and
// the decode workload's launch went from 13.07 to 12.15 us; at 256 tokens
// (rank 64, two slices per tile, each item reading half of A_i) the repeats
// cost more than they save (49.4 -> 52.4 us), so larger one-launch batches
// keep tiles of two.  Batches above kFusedTokens take tiles of kTT tokens.
constexpr int kSmallTile = PLORA_SMALL_BATCH_TILE_TOKENS;
constexpr int kDecodeTile = PLORA_DECODE_TILE_TOKENS;
constexpr int kDecodeTokens = 64;
static_assert(kDecodeTile <= kSmallTile, "the exchange regions hold kSmallTile tokens");
__host__ __device__ constexpr int tile_tokens(int T) {
  return T <= kDecodeTokens ? kDecodeTile : T <= kFusedTokens ? kSmallTile : kTT;
}
constexpr int kSegThreads = 1024;
constexpr int kSegWaves = kSegThreads / 64;
// Groups of 64 words per wave in the radix passes: each wave owns a chunk of
// ceil(T / kSegWaves) words rounded up to 64, at most this many groups.
constexpr int kSegGroups = ((PLORA_MAX_TOKENS + kSegWaves - 1) / kSegWaves + 63) / 64;
// Keys (N + 1: the adapters and "skipped") of the one-launch counting sort,
// which segments batches above kFusedTokens tokens without a workspace; more
// adapters take the radix kernel, or the multi-work-group sort given one.
constexpr int kCountKeys = 2048;
constexpr int kCH = 8;                   // 16-byte chunks per lane per batch
constexpr size_t kMaxLds = 160 * 1024;   // LDS per CU on gfx950

// ---------------------------------------------------------------------------
// small device helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu) != 0u)
    return ((u >> 16) & 0x8000u) | 0x7fc0u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ void unpack8(const uint4& v, float f[8]) {
  f[0] = bf_lo(v.x); f[1] = bf_hi(v.x);
  f[2] = bf_lo(v.y); f[3] = bf_hi(v.y);
  f[4] = bf_lo(v.z); f[5] = bf_hi(v.z);
  f[6] = bf_lo(v.w); f[7] = bf_hi(v.w);
}

__device__ __forceinline__ uint4 ldg16(const uint16_t* p) {
  return *reinterpret_cast<const uint4*>(p);
}

// A 16-byte load of p where ok holds and of safe elsewhere, with zero in
// place of the value there.  The load itself is unconditional: with a branch
// around a load, the compiler waits for every load in flight where the
// branches join instead of for the one it needs, and the vector path's
// prefetching would be serialised.  Used for activation rows (x, y), whose
// lanes read different tokens' rows; callers pick safe inside a line the
// same wavefront reads anyway (the tile's first token row), so masked lanes
// cost no extra traffic.  Adapter blocks go through bld16 below instead.
__device__ __forceinline__ uint4 ldg16z(const uint16_t* p, const uint16_t* safe, bool ok) {
  const uint4 v = ldg16(ok ? p : safe);
  return ok ? v : make_uint4(0, 0, 0, 0);
}

// The 8-byte form of ldg16z.
__device__ __forceinline__ uint2 ldg8z(const uint16_t* p, const uint16_t* safe, bool ok) {
  const uint2 v = *reinterpret_cast<const uint2*>(ok ? p : safe);
  return ok ? v : make_uint2(0, 0);
}

// An adapter block (A_i or B_i: n bf16 values at p) as a raw buffer
// resource.  Loads through it are range-checked by the hardware: a lane
// whose offset lies past the block reads zero and fetches nothing.  That
// makes masked lanes free (no branch, so the compiler keeps its waits
// exact, and no load of a stand-in address) and confines every read to
// the block.  The host keeps blocks below 2^31 bytes (h_in and h_out times
// max_rank), so kPastEnd lies past every one.
typedef __amdgpu_buffer_rsrc_t Rsrc;
typedef int i32x4_t __attribute__((ext_vector_type(4)));
constexpr int kRsrcWord3 = 0x00020000;   // raw buffer, 32-bit data format (gfx9 family)
constexpr int kPastEnd = (int)0x80000000u;   // a byte offset past every block

__device__ __forceinline__ Rsrc block_rsrc(const uint16_t* p, int64_t n) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p), 0, (int)(n * 2),
                                           kRsrcWord3);
}

// Cache policy of adapter reads, set by each kernel's source file before it
// includes this header: PLORA_ADAPTER_POLICY for the vector paths (tiles of
// a few tokens), PLORA_MATRIX_POLICY (by default the same) for the matrix
// and general-rank paths.  The exchange-form kernels read every byte of an
// adapter's blocks once per call, so they read them non-temporally (2): the
// caches then keep what is reused, the kernel's code, the token metadata and
// the exchange words.  The two-part form reads a short segment's adapter
// (one vector-path tile) once too, but re-reads a long segment's A_i and
// B_i once per tile (matrix path), from the caches; the two-launch form
// (shrink and expand launches) keeps the default (0) throughout.
#ifndef PLORA_ADAPTER_POLICY
#define PLORA_ADAPTER_POLICY 0
#endif
#ifndef PLORA_MATRIX_POLICY
#define PLORA_MATRIX_POLICY PLORA_ADAPTER_POLICY
#endif
constexpr int kAdapterPolicy = PLORA_ADAPTER_POLICY;
constexpr int kMatrixPolicy = PLORA_MATRIX_POLICY;

// 16 bytes at element e of the block, zero where !ok (POL: the cache policy).
template <int POL = kAdapterPolicy>
__device__ __forceinline__ uint4 bld16(Rsrc r, int64_t e, bool ok) {
  const i32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, ok ? (int)(e * 2) : kPastEnd, 0,
                                                          POL);
  return make_uint4((uint32_t)v.x, (uint32_t)v.y, (uint32_t)v.z, (uint32_t)v.w);
}

// ---------------------------------------------------------------------------
// apply kernels
// ---------------------------------------------------------------------------
//
// Work items.  An item is one tile and one slice of h_in (KS slices of KR
// rows) or of the y columns (JS slices of W columns), so that each launch
// has about kPlanItems items per resident work group and a batch of a few
// dozen tiles still spreads over the whole chip.  plora_apply takes one of
// three forms, by batch size:
//
//   one launch, S > 1 slices per tile (batches whose tile capacity is at
//   most 2/3 of the resident work groups: decode batches).  S is chosen on
//   the host from the tile capacity; item (tile, s) reduces h_in slice s,
//   trades partial v with the tile's other items through the workspace (see
//   the exchange below) and expands y column slice s.  Each item reads 1/S
//   of A_i and of B_i.
//
//   one launch, one h_in slice (up to kFusedTokens tokens otherwise): item
//   (tile, column slice), JS chosen on the device from the tile count that
//   plora_segment wrote, computes the tile's v over all of h_in, then
//   expands it with its slice of B_i.  A_i is read by every column slice of
//   its tile; the slices of a tile are numbered onto one XCD, so the first
//   read brings A_i into that XCD's L2 and the others hit it.
//
//   two parts (batches above kFusedTokens tokens): item (tile, h_in slice)
//   writes its partial v to the workspace; item (tile, column slice) sums
//   the tile's KS partials in slice order and expands.  Every byte of A_i,
//   B_i and x is then read by one work group only, and a rank-64 tile's
//   stream of A_i is split over KS items (the one-launch form above measured
//   79.5 us on the ragged workload of 512 tokens, against 73 for this one as
//   two launches).  The two parts run as one launch (parts_kernel, the
//   expand items starting on a tile once its partials are stored), or as a
//   shrink launch and an expand launch for a batch with more tile slots than
//   the workspace has readiness words.
//
// Grids are sized on the host for the most items any tile count up to the
// capacity can produce; surplus work groups return after one load.
//
// Two code paths, chosen per tile:
//
// Short tiles (vector ALU, see vector_tokens).  A_i, a contiguous block of h_in
// x r bf16 values, is streamed as 16-byte chunks: thread tid loads chunks
// tid, tid + kNT, ... so it always sees the column octet tid % (r/8) and a
// set of rows, and accumulates x[row] * A_i[row][octet] in registers for
// every token of the tile.  Threads sharing an octet are combined inside the
// wavefront by a butterfly (halving while more than one value remains, then
// all-reducing the remaining row-slot bits) and across wavefronts through
// LDS in wave order.  The expand gives each thread one column octet of the
// slice and all (or a row-slot share of) B_i's r rows.  The first chunks of
// A_i and B_i, x and the y words are all requested before any of them is
// needed, in the order they are consumed (the vector-memory counter retires
// in order).
//
// Longer tiles (matrix cores, v_mfma_f32_16x16x32_bf16).  The shrink
// computes D[token][c] = sum_k x[token][k] A_i[k][c]: each wavefront takes
// every fourth 32-row K step and streams those rows of A_i and the x
// operands straight into a ring of its own LDS stages (global_load_lds), the
// x rows feeding the A operand and A_i read back transposed
// (ds_read_b64_tr_b16) into the B operand; the four wavefronts' partial tiles
// are summed by a fixed pairwise tree.  The expand computes D^T[j][token] =
// sum_c B_i[c][j] v[token][c] with B_i column chunks staged in LDS and read
// transposed into the A operand; v is split into bf16 high and low parts
// (v = hi + lo to about 2^-17 relative) so that no intermediate is rounded
// below fp32 accuracy.  Each lane then owns four consecutive y columns of one
// token.
//
// Every reduction has a fixed order that depends only on the tile and the
// slice widths, so results are bitwise reproducible, and the split calls
// (plora_shrink, which sums the partials in the same order into v, then
// plora_expand, which chooses the same column slices) compute the very same
// values as plora_apply.

constexpr int kNT = 256;             // threads per work group
constexpr int kW = kNT / 64;         // wavefronts per work group
constexpr int kWGPerCU = 2;          // resident work groups per compute unit
// Chunks of A_i and of B_i per thread requested up front by the vector path
// (the rest follow in batches of kCH).  A decode item needs 4 of each, and a
// masked slot still costs address cycles ahead of the real ones: the
// one-launch forms (decode-sized slices) request 4 (decode 14.3 us per
// launch with 16, 13.6 with 8, 13.15 with 4; the large batch 49.7, 50.1,
// 49.5), the two-part forms 8 (ragged 62.9 with 16, 62.1 with 8, 62.8 with
// 4, as two launches; in one launch 60.5 with 8, 60.9 with 4).  A kernel file sets PLORA_PREFETCH_CHUNKS before including this header.
#ifndef PLORA_PREFETCH_CHUNKS
#define PLORA_PREFETCH_CHUNKS 8
#endif
constexpr int kAP = PLORA_PREFETCH_CHUNKS;
constexpr int kBP = PLORA_PREFETCH_CHUNKS;
static_assert(kAP <= kCH || kAP % kCH == 0, "whole batches, or one short one");
// Columns of x staged in LDS per window by the vector path (and shrink_gen).
// A decode slice is 512 columns, which a 2048-column window stages without
// masked slots at one token per tile; a kernel file may set
// PLORA_X_WINDOW before including this header.
#ifndef PLORA_X_WINDOW
#define PLORA_X_WINDOW 4096
#endif
constexpr int kXW = PLORA_X_WINDOW;
constexpr int kChunk = 16384;        // bf16 elements per LDS staging chunk (32 KiB)
constexpr int kWaveRing = 12288;     // bytes of LDS ring per wavefront (matrix shrink)
constexpr int kBufElems = kW * kWaveRing / 2 + 16;   // slack for transposed reads past the end
static_assert(kBufElems >= kChunk, "the LDS buffer also stages B_i chunks and the x window");
constexpr int kRK = 32;              // MFMA K step
constexpr int kMinSlice = 512;       // fewest y columns per work item (but h_out)
// Items per resident work group the device-chosen plans aim at: two, so that
// the work groups that finish early (low-rank tiles) take more items while the
// long ones (rank 64, long segments) run; one per work group measured 73 us on
// the ragged workload, two 67, four 79 (the per-item latency chain then
// outweighs the balance).
constexpr int kPlanItems = 2;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

struct ApplyArgs {
  const uint16_t* x;
  int64_t ldx;
  float* v;            // plora_shrink output / plora_expand input
  int64_t ldv;
  uint16_t* y;
  int64_t ldy;
  const uint16_t* A;
  const uint16_t* B;
  int64_t a_len, b_len;
  const uint16_t* A_pool;   // host-memory pools the device reads directly (may be null)
  const uint16_t* B_pool;
  int64_t a_pool_len, b_pool_len;
  const int64_t* a_off;
  const int64_t* b_off;
  const int32_t* ranks;
  const float* scales;
  const int32_t* perm;
  const int4* tiles;
  const int32_t* meta;
  int32_t T, N, h_in, h_out, max_rank, tile_cap;
  float* vpart;         // workspace: partial v [ks_max][T][max_rank]
  uint64_t* xw;         // workspace: exchange words [S][cap8][kTT][max_rank] (one launch)
  uint64_t* xep;        // workspace: exchange epoch per tile slot [cap8]
  int32_t ks_max;      // most h_in slices per tile
  int32_t js_max;      // most y column slices per tile
  int32_t slots;       // resident work groups the device holds (item target)
  int32_t fixed_slices; // > 0: every tile takes exactly this many h_in and y column slices
  int32_t polls;        // polls of a partner's exchange word before computing v alone
  // workspace counters (null without a workspace): [0] work items that
  // computed v alone, [1] tokens skipped for an unusable adapter entry
  unsigned long long* counters;
  int32_t count_skips;  // this launch counts skipped tokens (one launch per call does)
  // the one-launch two-part form (see parts_kernel): a readiness word per
  // tile slot
  uint64_t* ready;
};

struct Tile {
  int a, p0, L;
  int r;
  bool bad;            // the adapter entry is unusable (see tile_blocks)
  int k0, k1;          // rows of A_i (and columns of x) the shrink covers
  int j0, j1;          // y columns the expand covers
  const uint16_t* Ai;
  const uint16_t* Bi;
  float s;
};

// The slices of one call: n_tiles tiles (as written by plora_segment),
// rounded up to a multiple of 8, times KS slices of KR rows of h_in (a
// multiple of 64, the last one shorter) for the shrink items, or times JS
// slices of W y columns (a multiple of 16, the last one shorter) for the
// expand items.  KS and JS are the slot count over the rounded tile count,
// to nearest, within [1, ks_max] and [1, js_max]; so a launch has at most
// max(4/3 slots, rounded tile count) items and at most ks_max (js_max) times
// the rounded tile count, whichever is less (the host sizes grids by that).
enum SliceKind { kRowSlices, kColSlices };

struct Plan {
  int n_tiles, KS, KR, JS, W, n_items;
};

__device__ __forceinline__ Plan make_plan(const ApplyArgs& g, SliceKind kind) {
  Plan p;
  const int nt = g.meta[4];
  p.n_tiles = nt < 0 ? 0 : (nt > g.tile_cap ? g.tile_cap : nt);
  const int n8 = (p.n_tiles + 7) & ~7;
  int ks = 1, js = 1;
  if (g.fixed_slices > 0) {
    ks = js = g.fixed_slices;
  } else if (n8 > 0) {
    const int fit = (kPlanItems * g.slots + n8 / 2) / n8;
    ks = max(1, min(g.ks_max, fit));
    js = max(1, min(g.js_max, fit));
  }
  p.KR = ((g.h_in + ks - 1) / ks + 63) & ~63;
  p.KS = (g.h_in + p.KR - 1) / p.KR;
  p.W = ((g.h_out + js - 1) / js + 15) & ~15;
  p.JS = (g.h_out + p.W - 1) / p.W;
  p.n_items = n8 * (kind == kRowSlices ? p.KS : p.JS);
  return p;
}

// Start of an adapter's n-element block: offset o >= 0 is element o of the
// device stack, o < 0 element -1 - o of the pool (host memory that the
// device reads directly: the E2 analog, section V-A); null if the block is
// misaligned or runs past its array.
__device__ __forceinline__ const uint16_t* adapter_block(const uint16_t* dev, int64_t dev_len,
                                                         const uint16_t* pool, int64_t pool_len,
                                                         int64_t o, int64_t n) {
  const bool in_pool = o < 0;
  const int64_t e = in_pool ? -1 - o : o;
  const uint16_t* base = in_pool ? pool : dev;
  if (!base || (e & 7) || e + n > (in_pool ? pool_len : dev_len)) return nullptr;
  return base + e;
}

// Adapter t.a's blocks into t, given its element offsets (t.a, t.p0, t.L,
// t.r and t.s already set); false, for the whole work group, for a tile
// with nothing to do: rank 0 (a no-op adapter) or an unusable entry (a rank
// outside [0, max_rank], or a block misaligned or past its array), which
// also sets t.bad so that the call counts the tile's tokens.  Every rank
// from 1 to max_rank is applied.  my_tok (this thread's tile row's token)
// is cleared to -1 if out of range.  tile_adapter below reads the rank,
// scale and offsets first.
__device__ __forceinline__ bool tile_blocks(const ApplyArgs& g, Tile& t, int& my_tok,
                                            int64_t ao, int64_t bo) {
  if (my_tok < 0 || my_tok >= g.T) my_tok = -1;
  if (t.r == 0) return false;
  if (t.r < 0 || t.r > g.max_rank) {
    t.bad = true;
    return false;
  }
  t.Ai = adapter_block(g.A, g.a_len, g.A_pool, g.a_pool_len, ao, (int64_t)g.h_in * t.r);
  t.Bi = adapter_block(g.B, g.b_len, g.B_pool, g.b_pool_len, bo, (int64_t)g.h_out * t.r);
  if (!t.Ai || !t.Bi) {
    t.bad = true;
    return false;
  }
  t.k0 = 0;
  t.k1 = g.h_in;
  t.j0 = 0;
  t.j1 = g.h_out;
  return true;
}

__device__ __forceinline__ bool tile_adapter(const ApplyArgs& g, Tile& t, int& my_tok) {
  t.r = g.ranks[t.a];
  const int64_t ao = g.a_off[t.a], bo = g.b_off[t.a];
  t.s = g.scales[t.a];
  return tile_blocks(g, t, my_tok, ao, bo);
}

// The adapter, first position and length of a tile from its record; false
// for padding entries and records out of range.
__device__ __forceinline__ bool tile_from_record(const ApplyArgs& g, const int4& ti, Tile& t) {
  t.a = ti.x; t.p0 = ti.y; t.L = ti.z;
  return t.a >= 0 && t.a < g.N && t.L > 0 && t.L <= kTT && t.p0 >= 0 && t.p0 + t.L <= g.T;
}

// Read and validate tile u.  Returns false (for the whole work group) for
// padding entries and for adapters the kernels must skip.  Threads below L
// also fetch their tile row's token index (-1 if unusable); it is issued
// together with the adapter metadata so both arrive in one trip.
__device__ __forceinline__ bool load_tile(const ApplyArgs& g, int u, Tile& t, int& my_tok) {
  t.bad = false;
  if (u < 0 || u >= g.tile_cap) return false;
  if (!tile_from_record(g, g.tiles[u], t)) return false;
  my_tok = (int)threadIdx.x < t.L ? g.perm[t.p0 + threadIdx.x] : -1;
  return tile_adapter(g, t, my_tok);
}

// Item i of plan p: items are numbered in groups of eight tiles, slice-major
// inside a group, so that item i is slice (i mod 8S) / 8 of tile
// 8 (i / 8S) + i mod 8, S the slice count; a tile's slices are dispatched
// together, and land on one XCD (work group b runs on XCD b mod 8).  Tiles
// next to each other go to different XCDs: a Zipf-skewed batch's hottest
// adapters (the longest segments, at the lowest ids) are spread over the
// chip; giving each XCD a contiguous range of tiles instead measured 10 us
// slower on the ragged workload.
//
// In the two-part form, an order that sends a long segment's consecutive
// tiles (with one slice) to one XCD, so that its slice of A_i is fetched from
// HBM once and then hit in that XCD's L2, cut the prefill shrink's HBM reads
// by 30% but not its time, and made the ragged workload 1.5 us slower.
__device__ __forceinline__ int item_slot(const Plan& p, SliceKind kind, int i, int& slice) {
  const int per = 8 * (kind == kRowSlices ? p.KS : p.JS);
  const int q = i / per, rem = i - q * per;
  slice = rem >> 3;
  return 8 * q + (rem & 7);
}

__device__ __forceinline__ bool item_tile(const ApplyArgs& g, const Plan& p, SliceKind kind,
                                          int i, Tile& t, int& my_tok, int& slice) {
  const int u = item_slot(p, kind, i, slice);
  t.bad = false;
  if (u >= p.n_tiles) return false;
  if (!load_tile(g, u, t, my_tok)) return false;
  if (kind == kRowSlices) {
    t.k0 = slice * p.KR;
    t.k1 = min(g.h_in, t.k0 + p.KR);
  } else {
    t.j0 = slice * p.W;
    t.j1 = min(g.h_out, t.j0 + p.W);
  }
  return true;
}

// Work-group-uniform counter updates of the workspace (agent scope, so that
// every XCD's additions reach the same word).
__device__ __forceinline__ void bump(const ApplyArgs& g, int which, unsigned long long n) {
  if (g.counters && threadIdx.x == 0 && n)
    __hip_atomic_fetch_add(g.counters + which, n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The tokens of a tile whose adapter entry is unusable are counted once per
// call: by the tile's first slice, in the launch that counts.
__device__ __forceinline__ void count_skipped(const ApplyArgs& g, const Tile& t, int slice) {
  if (t.bad && slice == 0 && g.count_skips) bump(g, 1, (unsigned long long)t.L);
}

// Barrier for LDS traffic only: global loads into registers stay in flight.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// LDS of a tile work group.
//   tok   [kTT]              token index of each tile row, -1 if unusable
//   vs    [max_rank][kTT]    v of the tile, fp32, column-major
//   vhl   [2][kTT][RKmax]    v split into bf16 high and low parts, token-major
//   buf   kBufElems bf16     vector path: x window and the cross-wave partial
//                            sums; matrix path: the A_i ring, B_i chunks and
//                            the wave-tree partial tiles
struct Smem {
  int* tok;
  float* vs;
  uint16_t* vhl;
  uint16_t* buf;
};

// K extent of the matrix-path expand for rank r: r rounded up to whole MFMA
// K steps (rows of B_i and columns of v past r are zero).
__host__ __device__ constexpr int rk_of(int r) {
  return r <= kRK ? kRK : (r + kRK - 1) / kRK * kRK;
}

// Row stride of v's bf16 split in LDS: the K extent of the largest rank.
__host__ __device__ constexpr int rk_max(int max_rank) { return rk_of(max_rank); }

__host__ __device__ constexpr size_t smem_bytes(int h_in, int max_rank) {
  return kTT * sizeof(int) + (size_t)max_rank * kTT * sizeof(float) +
         (size_t)2 * kTT * rk_max(max_rank) * sizeof(uint16_t) +
         (size_t)kBufElems * sizeof(uint16_t) + 0 * h_in;
}

__device__ __forceinline__ Smem carve(void* base, int max_rank) {
  char* p = reinterpret_cast<char*>(base);
  Smem s;
  s.tok = reinterpret_cast<int*>(p);      p += kTT * sizeof(int);
  s.vs = reinterpret_cast<float*>(p);     p += (size_t)max_rank * kTT * sizeof(float);
  s.vhl = reinterpret_cast<uint16_t*>(p); p += (size_t)2 * kTT * rk_max(max_rank) * sizeof(uint16_t);
  s.buf = reinterpret_cast<uint16_t*>(p);
  return s;
}

constexpr int ilog2(int v) { return v <= 1 ? 0 : 1 + ilog2(v / 2); }

// The kernel shape that serves rank r (1..128): the smallest of 8, 16, 32,
// 64, 128 at or above it.  Ranks that are multiples of 8 run that shape with
// their own row stride (the padded columns are masked or dropped); other
// ranks, whose rows of A_i are not 16-byte aligned, take the LDS-staged
// shrink (shrink_gen) and share the expand.
__host__ __device__ constexpr int rank_class(int r) {
  return r <= 8 ? 8 : r <= 16 ? 16 : r <= 32 ? 32 : r <= 64 ? 64 : 128;
}

// ---------------------------------------------------------------------------
// short tiles: vector ALU
// ---------------------------------------------------------------------------

// Longest tile on the vector path: two tokens at ranks up to 16, four at
// ranks of 32 and more.  At the larger ranks a matrix-path stage of A_i fills
// the wavefront's LDS ring in two or three stages, too shallow to stream
// A_i as fast as the vector path's register prefetch does.
__device__ __forceinline__ int vector_tokens(int r) { return r >= 32 ? 4 : 2; }

// A_i and B_i chunks per thread requested up front for TG tokens (the same
// for every token-group width).
template <int TG> constexpr int ap_depth() { return kAP; }
template <int TG> constexpr int bp_depth() { return kBP; }

// Expand lane layout over the slice's n_oct column octets: RSB row slots per
// octet (the largest power of two, at most 64, that still covers every octet
// in one pass when the slice is narrow enough), this thread's first octet
// co0 (relative to the slice) and row slot rb.
struct ExpandMap {
  int RSB, CPW, co0, rb, njb, n_oct;
};

__device__ __forceinline__ ExpandMap expand_map(const Tile& t) {
  ExpandMap m;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  m.n_oct = (t.j1 - t.j0) >> 3;
  int l = 0;
  while (l < 6 && (m.n_oct << (l + 1)) <= kNT) ++l;
  m.RSB = 1 << l;
  m.CPW = 64 / m.RSB;
  m.co0 = w * m.CPW + lane % m.CPW;
  m.rb = lane / m.CPW;
  m.njb = m.rb < t.r ? (t.r - m.rb + m.RSB - 1) / m.RSB : 0;
  return m;
}

// This thread's first BP chunks of B_i (first column batch).
template <int BP>
__device__ __forceinline__ void prefetch_b(const ApplyArgs& g, const Tile& t, uint4 (&bpre)[BP]) {
  const ExpandMap m = expand_map(t);
  const bool col_ok = m.co0 < m.n_oct;
  const Rsrc rb = block_rsrc(t.Bi, (int64_t)g.h_out * t.r);
  const int64_t e0 = (int64_t)m.rb * g.h_out + t.j0 + (int64_t)m.co0 * 8;
  const int64_t bstep = (int64_t)m.RSB * g.h_out;
#pragma unroll
  for (int j = 0; j < BP; ++j) bpre[j] = bld16(rb, e0 + j * bstep, col_ok && j < m.njb);
}

// This thread's y words (first column octet, row slot 0) of the tile's tokens.
template <int TG>
__device__ __forceinline__ void prefetch_y(const ApplyArgs& g, const Tile& t, const int* tok,
                                           uint4 (&ypre)[TG]) {
  const ExpandMap m = expand_map(t);
  const bool ok = m.co0 < m.n_oct && m.rb == 0;
  const uint16_t* safe = g.y + (int64_t)max(tok[0], 0) * g.ldy + t.j0;
#pragma unroll
  for (int tt = 0; tt < TG; ++tt) {
    const int tk = (ok && tt < t.L) ? tok[tt] : -1;
    ypre[tt] = ldg16z(g.y + (int64_t)tk * g.ldy + t.j0 + (int64_t)m.co0 * 8, safe, tk >= 0);
  }
}

// One butterfly step over lane mask M on the first N of V values: the lane
// whose mask bit is set keeps the upper half, the other the lower half, each
// adding the half its partner sends.
template <int V, int N, int M>
__device__ __forceinline__ void halve(float (&val)[V], int lane) {
  const bool up = (lane & M) != 0;
#pragma unroll
  for (int i = 0; i < N / 2; ++i) {
    const float lo = val[i], hi = val[i + N / 2];
    const float send = up ? lo : hi;
    const float keep = up ? hi : lo;
    val[i] = keep + __shfl_xor(send, M, 64);
  }
}

// Butterfly over the row-slot lane bits (masks R_OCT << s, s < S): halve the
// V values while two or more remain, all-reduce over the remaining bits.  On
// return the lane holds V >> H reduced values starting at index base, and
// writer tells whether it is the one lane of its all-reduce group to store.
template <int V, int R_OCT, int S, int s>
__device__ __forceinline__ void butterfly(float (&val)[V], int lane, int& base, bool& writer) {
  if constexpr (s < S) {
    constexpr int H = S < ilog2(V) ? S : ilog2(V);
    constexpr int M = R_OCT << s;
    if constexpr (s < H) {
      constexpr int N = V >> s;
      halve<V, N, M>(val, lane);
      if (lane & M) base += N / 2;
    } else {
      constexpr int VL = V >> H;
#pragma unroll
      for (int j = 0; j < VL; ++j) val[j] += __shfl_xor(val[j], M, 64);
      if (lane & M) writer = false;
    }
    butterfly<V, R_OCT, S, s + 1>(val, lane, base, writer);
  }
}

// The TG bf16 x values of one row of xs (xs[k][TG]), as fp32.
template <int TG>
__device__ __forceinline__ void x_row(const uint16_t* xs, int row, float (&xf)[TG]) {
  if constexpr (TG == 1) {
    xf[0] = __uint_as_float((uint32_t)xs[row] << 16);
  } else if constexpr (TG == 2) {
    const uint32_t v = *reinterpret_cast<const uint32_t*>(xs + row * 2);
    xf[0] = bf_lo(v); xf[1] = bf_hi(v);
  } else {
    const uint2 v = *reinterpret_cast<const uint2*>(xs + row * 4);
    xf[0] = bf_lo(v.x); xf[1] = bf_hi(v.x); xf[2] = bf_lo(v.y); xf[3] = bf_hi(v.y);
  }
}

// acc[tt][e] += x[tt][row] * A[row][oct*8 + e] for chunks jb..jb+kCH-1 of the
// window starting at chunk q0 (rows relative to w0).
template <int R_OCT, int TG, int N = kCH>
__device__ __forceinline__ void fma_a(float (&val)[TG * 8], const uint4* a, const uint16_t* xs,
                                      int q0, int w0, int jb, int nj) {
#pragma unroll
  for (int j = 0; j < N; ++j) {
    if (jb + j < nj) {
      const int row = (q0 + (int)threadIdx.x + (jb + j) * kNT) / R_OCT - w0;
      float xf[TG];
      x_row<TG>(xs, row, xf);
      float af[8];
      unpack8(a[j], af);
#pragma unroll
      for (int tt = 0; tt < TG; ++tt)
#pragma unroll
        for (int e = 0; e < 8; ++e) val[tt * 8 + e] = fmaf(xf[tt], af[e], val[tt * 8 + e]);
    }
  }
}

// v of a tile of L <= TG tokens into sm.vs, for a rank t.r that is a
// multiple of 8 and at most R = 8 R_OCT (R a power of two).  Loads are
// requested in the order they are consumed: x of the window, the first AP
// chunks of A_i and, with prefetch set, this thread's first BP chunks of B_i
// and its y words.
template <int R_OCT, int TG>
__device__ __forceinline__ void shrink_valu(const ApplyArgs& g, const Tile& t, const Smem& sm,
                                            uint4 (&bpre)[bp_depth<TG>()],
                                            uint4 (&ypre)[TG], bool prefetch) {
  constexpr int R = 8 * R_OCT;
  constexpr int V = TG * 8;
  constexpr int S = ilog2(64 / R_OCT);     // row-slot bits inside a wavefront
  constexpr int H = S < ilog2(V) ? S : ilog2(V);
  constexpr int VL = V >> H;               // values a lane keeps
  constexpr int XR = kXW * TG / 8 / kNT;   // x chunks per thread of a full window
  constexpr int AP = ap_depth<TG>();
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int oct = tid % R_OCT;
  // A_i's rows are t.r elements long: a rank below R (a multiple of 8) leaves
  // octets past its last column, whose lanes load nothing
  const bool oct_ok = oct * 8 < t.r;
  const int64_t astep = (int64_t)(kNT / R_OCT) * t.r;   // elements between a thread's chunks
  const int XW = t.k1 - t.k0 < kXW ? t.k1 - t.k0 : kXW;
  uint16_t* xs = sm.buf;                   // [XW][TG]
  float* red = reinterpret_cast<float*>(sm.buf);  // [kW][TG][R], after xs is dead

  const Rsrc ra = block_rsrc(t.Ai, (int64_t)g.h_in * t.r);
  float val[V];
#pragma unroll
  for (int i = 0; i < V; ++i) val[i] = 0.f;
  for (int w0 = t.k0; w0 < t.k1; w0 += XW) {
    const int w1 = min(t.k1, w0 + XW);
    const int q0 = w0 * R_OCT;                         // first chunk of the window
    const int nq = (w1 - w0) * R_OCT;
    const int nj = tid < nq ? (nq - tid + kNT - 1) / kNT : 0;
    const int nj_max = (nq + kNT - 1) / kNT;       // the same for the whole group
    const int n8 = (w1 - w0) >> 3;                     // x chunks per token
    const int64_t ae = (int64_t)(w0 + tid / R_OCT) * t.r + oct * 8;   // this thread's first chunk
    const uint16_t* x_safe = g.x + (int64_t)max(sm.tok[0], 0) * g.ldx + w0;
    uint4 xr[XR], apre[AP];
#pragma unroll
    for (int i = 0; i < XR; ++i) {
      const int c = tid + i * kNT;
      const int tt = c / n8, kc = c - tt * n8;
      const int tk = (tt < t.L && c < TG * n8) ? sm.tok[tt] : -1;
      xr[i] = ldg16z(g.x + (int64_t)tk * g.ldx + w0 + kc * 8, x_safe, tk >= 0);
    }
#pragma unroll
    for (int j = 0; j < AP; ++j)
      apre[j] = bld16(ra, ae + j * astep, oct_ok && j < nj);
    if (prefetch && w0 == t.k0) {
      prefetch_b<bp_depth<TG>()>(g, t, bpre);
      prefetch_y<TG>(g, t, sm.tok, ypre);
    }
#pragma unroll
    for (int i = 0; i < XR; ++i) {
      const int c = tid + i * kNT;
      if (c < TG * n8) {
        const int tt = c / n8, kc = c - tt * n8;
        const uint4 v = xr[i];
        uint16_t* d = xs + (kc * 8) * TG + tt;
        d[0 * TG] = (uint16_t)(v.x & 0xffffu); d[1 * TG] = (uint16_t)(v.x >> 16);
        d[2 * TG] = (uint16_t)(v.y & 0xffffu); d[3 * TG] = (uint16_t)(v.y >> 16);
        d[4 * TG] = (uint16_t)(v.z & 0xffffu); d[5 * TG] = (uint16_t)(v.z >> 16);
        d[6 * TG] = (uint16_t)(v.w & 0xffffu); d[7 * TG] = (uint16_t)(v.w >> 16);
      }
    }
    lds_sync();
    if (nj_max <= AP) {
      // the window's chunks all came with the prefetch (a decode slice):
      // no further batch is requested, not even a masked one (each masked
      // load still takes address cycles ahead of the real ones)
#pragma unroll
      for (int jb = 0; jb < AP; jb += kCH)
        fma_a<R_OCT, TG, (AP < kCH ? AP : kCH)>(val, apre + jb, xs, q0, w0, jb, nj);
    } else {
      // the next batch is requested before the prefetched chunks are
      // consumed, so that two batches are always in flight
      uint4 a0[kCH], a1[kCH];
#pragma unroll
      for (int j = 0; j < kCH; ++j)
        a0[j] = bld16(ra, ae + (AP + j) * astep, oct_ok && AP + j < nj);
#pragma unroll
      for (int jb = 0; jb < AP; jb += kCH)
        fma_a<R_OCT, TG, (AP < kCH ? AP : kCH)>(val, apre + jb, xs, q0, w0, jb, nj);
      for (int jb = AP; jb < nj_max; jb += 2 * kCH) {
#pragma unroll
        for (int j = 0; j < kCH; ++j)
          a1[j] = bld16(ra, ae + (jb + kCH + j) * astep, oct_ok && jb + kCH + j < nj);
        fma_a<R_OCT, TG>(val, a0, xs, q0, w0, jb, nj);
#pragma unroll
        for (int j = 0; j < kCH; ++j)
          a0[j] = bld16(ra, ae + (jb + 2 * kCH + j) * astep, oct_ok && jb + 2 * kCH + j < nj);
        fma_a<R_OCT, TG>(val, a1, xs, q0, w0, jb + kCH, nj);
      }
    }
    lds_sync();                                        // xs free
  }
  int base = 0;
  bool writer = true;
  butterfly<V, R_OCT, S, 0>(val, lane, base, writer);
  if (writer) {
#pragma unroll
    for (int j = 0; j < VL; ++j) {
      const int idx = base + j;
      const int tt = idx >> 3, e = idx & 7;
      red[(w * TG + tt) * R + oct * 8 + e] = val[j];
    }
  }
  lds_sync();
  for (int o = tid; o < TG * R; o += kNT) {
    const int tt = o / R, c = o - tt * R;
    if (tt < t.L && c < t.r) {
      float s = red[tt * R + c];
#pragma unroll
      for (int ww = 1; ww < kW; ++ww) s += red[(ww * TG + tt) * R + c];
      sm.vs[c * kTT + tt] = s;
    }
  }
  lds_sync();
}

// The TG values v[c][0 .. TG) of one row of vs.
template <int TG>
__device__ __forceinline__ void v_row(const float* vs, int c, float (&vf)[TG]) {
  const float* p = vs + c * kTT;
  if constexpr (TG == 1) {
    vf[0] = p[0];
  } else if constexpr (TG == 2) {
    const float2 a = *reinterpret_cast<const float2*>(p);
    vf[0] = a.x; vf[1] = a.y;
  } else {
    const float4 a = *reinterpret_cast<const float4*>(p);
    vf[0] = a.x; vf[1] = a.y; vf[2] = a.z; vf[3] = a.w;
  }
}

// d[tt][e] += v[tt][row] * B_i[row][co*8 + e] for this thread's rows
// jb..jb+kCH-1.
template <int TG, int N = kCH>
__device__ __forceinline__ void fma_b(float (&d)[TG * 8], const uint4* b, const Smem& sm,
                                      const ExpandMap& m, int jb) {
#pragma unroll
  for (int j = 0; j < N; ++j) {
    if (jb + j < m.njb) {
      float vf[TG];
      v_row<TG>(sm.vs, m.rb + (jb + j) * m.RSB, vf);
      float bf[8];
      unpack8(b[j], bf);
#pragma unroll
      for (int tt = 0; tt < TG; ++tt)
#pragma unroll
        for (int e = 0; e < 8; ++e) d[tt * 8 + e] = fmaf(vf[tt], bf[e], d[tt * 8 + e]);
    }
  }
}

// y[tok, cols] = bf16(y + s * v B_i[:, cols]) for a tile of L <= TG tokens.
// The first column batch uses the chunks of B_i and the y words fetched
// before the shrink.
template <int TG>
__device__ __forceinline__ void expand_valu(const ApplyArgs& g, const Tile& t, const Smem& sm,
                                            const uint4 (&bpre)[bp_depth<TG>()],
                                            const uint4 (&ypre)[TG], bool have_y) {
  constexpr int BP = bp_depth<TG>();
  const ExpandMap m = expand_map(t);
  const int n_oct = m.n_oct;
  const Rsrc rb = block_rsrc(t.Bi, (int64_t)g.h_out * t.r);
  const int64_t bstep = (int64_t)m.RSB * g.h_out;
  for (int cb = 0, co = m.co0; cb * kW * m.CPW < n_oct; ++cb, co += kW * m.CPW) {
    const bool col_ok = co < n_oct;
    const int jc = t.j0 + co * 8;                    // first y column of the octet
    const int64_t be = (int64_t)m.rb * g.h_out + jc;   // this thread's first B_i unit
    float d[TG * 8];
#pragma unroll
    for (int i = 0; i < TG * 8; ++i) d[i] = 0.f;
    if (col_ok) {
      int jb0 = 0;
      if (cb == 0) {
#pragma unroll
        for (int jb = 0; jb < BP; jb += kCH) fma_b<TG, (BP < kCH ? BP : kCH)>(d, bpre + jb, sm, m, jb);
        jb0 = BP;
      }
      // the remaining rows in batches of kCH, the next batch always requested
      // before the current one is used (rows past njb load nothing)
      if (jb0 < m.njb) {
        uint4 b0[kCH], b1[kCH];
#pragma unroll
        for (int j = 0; j < kCH; ++j)
          b0[j] = bld16(rb, be + (int64_t)(jb0 + j) * bstep, jb0 + j < m.njb);
        for (int jb = jb0; jb < m.njb; jb += 2 * kCH) {
#pragma unroll
          for (int j = 0; j < kCH; ++j)
            b1[j] = bld16(rb, be + (int64_t)(jb + kCH + j) * bstep, jb + kCH + j < m.njb);
          fma_b<TG>(d, b0, sm, m, jb);
#pragma unroll
          for (int j = 0; j < kCH; ++j)
            b0[j] = bld16(rb, be + (int64_t)(jb + 2 * kCH + j) * bstep,
                          jb + 2 * kCH + j < m.njb);
          fma_b<TG>(d, b1, sm, m, jb + kCH);
        }
      }
    }
    // all-reduce across the row slots of each column octet
    for (int msk = m.CPW; msk < 64; msk <<= 1) {
#pragma unroll
      for (int i = 0; i < TG * 8; ++i) d[i] += __shfl_xor(d[i], msk, 64);
    }
    if (col_ok && m.rb == 0) {
      uint4 yv[TG];
#pragma unroll
      for (int tt = 0; tt < TG; ++tt) {
        const int tk = tt < t.L ? sm.tok[tt] : -1;
        yv[tt] = (have_y && cb == 0) ? ypre[tt]
                 : ldg16z(g.y + (int64_t)tk * g.ldy + jc,
                          g.y + (int64_t)max(sm.tok[0], 0) * g.ldy + jc, tk >= 0);
      }
      // every token's words first, then the stores (as in the matrix path:
      // a y word used after a store would make the compiler wait for it)
      uint4 out[TG];
#pragma unroll
      for (int tt = 0; tt < TG; ++tt) {
        float yf[8];
        unpack8(yv[tt], yf);
        uint32_t ob[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) ob[e] = to_bf16(fmaf(t.s, d[tt * 8 + e], yf[e]));
        out[tt].x = ob[0] | (ob[1] << 16);
        out[tt].y = ob[2] | (ob[3] << 16);
        out[tt].z = ob[4] | (ob[5] << 16);
        out[tt].w = ob[6] | (ob[7] << 16);
      }
#pragma unroll
      for (int tt = 0; tt < TG; ++tt) {
        const int tk = tt < t.L ? sm.tok[tt] : -1;
        if (tk >= 0) *reinterpret_cast<uint4*>(g.y + (int64_t)tk * g.ldy + jc) = out[tt];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// one-launch apply: exchange of a tile's partial v between its slices
// ---------------------------------------------------------------------------
//
// In the one-launch form every tile is split into S items; item s reduces
// rows [s KR, (s+1) KR) of h_in (its partial v) and expands y columns
// [s W, (s+1) W).  Each item needs the full v, the sum of all S partials.
// Items publish their partial as 64-bit words {fp32 bits, tag} in a region
// of the workspace private to the tile slot (slot = tile index), and each
// item polls its partners' words until every one carries this call's tag.
// Tags come from a 64-bit epoch per tile slot, read when the item starts
// and raised (atomic max) to epoch + 1 once its exchange is over: every item of a call
// reads the epoch before any partner can raise it (a partner raises it only
// after it has seen every item's words, or after giving up), so the call's
// tag is new to the slot's region, and stale words from earlier calls, other
// batch sizes or other ranks never match (the tag is the epoch's low 32
// bits: a word would have to lie unused for 2^32 calls of its slot).  The
// state is on the device, so the scheme holds under graph replay too.
// Polling is bounded: if a partner's word has not come after kSpinLimit
// polls (the partner was never scheduled, say because other work holds the
// compute units), the item computes v over all of h_in by itself (plain_v):
// correct to fp32 accuracy, but summed in another order, so such a call's
// bits can differ from the usual result.  No item ever waits without bound.
// The split into slices serves small batches, where a tile's reduction
// spread over S work groups (each reading 1/S of A_i and of B_i) beats one
// work group streaming all of A_i; the exchange costs about one memory
// round trip, which the expand's first loads of B_i and y overlap.

constexpr int kMaxSlices = 8;            // most slices per tile in the one-launch form
constexpr int kXSlots = 336;             // tile slots with an exchange region
constexpr int kSpinLimit = 20000;        // polls of a partner's word before computing v alone
// Words per slot: every entry of a tile of the one-launch form (at most
// kSmallTile tokens, the tile length plora_segment gives batches of up to
// kFusedTokens tokens) at the largest rank, kMaxSlices words each.
constexpr int64_t kSlotWords = (int64_t)kMaxSlices * kSmallTile * PLORA_MAX_RANK;
static_assert((kSmallTile * PLORA_MAX_RANK) % 8 == 0, "the region holds whole groups of 8 entries");

struct Xchg {
  int s, S, kr;          // this item's slice, the tile's slice count, rows of h_in per slice
  uint32_t tag;          // this call's tag for the tile slot
  uint64_t* words;       // the slot's region (see xword)
  int polls;             // polls before giving up on a partner
};

__device__ __forceinline__ uint64_t xload(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Exchange words are written and polled at agent scope (`sc1` on gfx950):
// stores reach memory and polls read past the compute unit's L1 and the
// XCD's L2, so a partner's word is seen wherever the partner ran.  (At
// work-group scope, `sc0`, most partners' words were never seen, even with
// a tile's items on one XCD and the L1 invalidated before each poll.)
__device__ __forceinline__ uint64_t xpoll(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void xpublish(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Item b of an exchange-form launch with S slices per tile slot: slice s
// of slot q, b = q S + s.  A slot's items are neighbours in the grid, so
// they are dispatched together, and (work group b runs on XCD b mod 8) they
// spread over the XCDs.  Numbering a slot's items onto one XCD instead
// measured 1.5 us slower per decode-shaped call: the exchange goes through
// memory either way, and the spread balances the XCDs.
__device__ __forceinline__ void exchange_item(int b, int S, int& q, int& s) {
  q = b / S;
  s = b - q * S;
}

// Word of entry o = l r + c of the tile, slice q, in the slot's region:
// entries in groups of eight, each group a [kMaxSlices][8] block, so that
// the words one item publishes for eight entries fill one 64-byte line of
// their own (whole-line writes; with a line per entry holding all of its
// slices' words, every item wrote 8 bytes into each of its entries' lines:
// 0.19 MB more written per decode launch, and the large decode batch took
// 49.2 us against 47.9), and the words a poll needs for slice q sit at a
// constant offset from slice 0's.
__device__ __forceinline__ int64_t xword(int o, int q) {
  return (int64_t)(o >> 3) * (8 * kMaxSlices) + q * 8 + (o & 7);
}

// Publish this item's partial v (sm.vs) and replace sm.vs by the sum of all
// S partials, in slice order (the order plora_shrink and the two-part form
// sum them in).  A word carrying this call's tag never changes again during
// the call, so a poll simply reloads the entry's S live words (the launch's
// S slices; the words past them are never read).  Returns false, for the
// whole work group, if some partner's word did not arrive in time; sm.vs is
// then undefined.
__device__ __forceinline__ bool exchange_v(const Tile& t, const Smem& sm, const Xchg& xc) {
  const int n = t.L * t.r;
  const uint64_t tagw = (uint64_t)xc.tag << 32;
  for (int o = threadIdx.x; o < n; o += kNT) {
    const int l = o / t.r, c = o - l * t.r;
    xpublish(xc.words + xword(o, xc.s), tagw | __float_as_uint(sm.vs[c * kTT + l]));
  }
  bool late = false;
  for (int o = threadIdx.x; o < n; o += kNT) {
    const uint64_t* e = xc.words + xword(o, 0);
    uint64_t w[kMaxSlices];
    bool ready = false;
    for (int it = 0; !ready && it <= xc.polls; ++it) {
      // the partners publish at about the time this item does: a first poll
      // right away mostly misses and costs a line read (decode: 1.0 KiB per
      // item and poll); after 1024 cycles it reads 0.2 MB less per launch
      if (it > 0) __builtin_amdgcn_s_sleep(2);
      else __builtin_amdgcn_s_sleep(16);
#pragma unroll
      for (int q = 0; q < kMaxSlices; ++q) w[q] = q < xc.S ? xpoll(e + q * 8) : 0;
      ready = true;
#pragma unroll
      for (int q = 0; q < kMaxSlices; ++q)
        ready &= q >= xc.S || (uint32_t)(w[q] >> 32) == xc.tag;
    }
    late |= !ready;
    float v = __uint_as_float((uint32_t)w[0]);
#pragma unroll
    for (int q = 1; q < kMaxSlices; ++q)
      if (q < xc.S) v += __uint_as_float((uint32_t)w[q]);
    const int l = o / t.r, c = o - l * t.r;
    sm.vs[c * kTT + l] = v;
  }
  return __syncthreads_or(late) == 0;
}

// A tile's pass: shrink (v of rows [k0, k1) into sm.vs), expand (columns
// [j0, j1) from sm.vs), or both; with both, the expand's first loads of
// B_i and y are requested with the shrink's.  The hook runs between the
// two (the one-launch form's exchange, which turns the partial v into the
// full one) while those loads travel; only a pass with both takes one.
struct NoHook {
  __device__ void operator()() const {}
};

// Shrink of ranks of 32 and more.  An item's slice of A_i is then long
// enough that B_i and y requested with it delay it, so where a hook follows
// (the exchange) they are requested once the shrink is done, to travel
// during the hook.
template <int R_OCT, int TG>
__device__ __forceinline__ void shrink_late(const ApplyArgs& g, const Tile& t, const Smem& sm,
                                            uint4 (&bpre)[bp_depth<TG>()], uint4 (&ypre)[TG],
                                            bool do_expand, bool hooked) {
  shrink_valu<R_OCT, TG>(g, t, sm, bpre, ypre, do_expand && !hooked);
  if (do_expand && hooked) {
    prefetch_b<bp_depth<TG>()>(g, t, bpre);
    prefetch_y<TG>(g, t, sm.tok, ypre);
  }
}

template <int TG, class H>
__device__ __forceinline__ void valu_tile_tg(const ApplyArgs& g, const Tile& t, const Smem& sm,
                                             bool do_shrink, bool do_expand, bool hooked,
                                             H&& hook) {
  uint4 bpre[bp_depth<TG>()], ypre[TG];
#pragma unroll
  for (int i = 0; i < TG; ++i) ypre[i] = make_uint4(0, 0, 0, 0);
  const bool have_y = do_shrink;
  if (do_shrink) {
    switch (rank_class(t.r)) {
      case 8: shrink_valu<1, TG>(g, t, sm, bpre, ypre, do_expand); break;
      case 16: shrink_valu<2, TG>(g, t, sm, bpre, ypre, do_expand); break;
      case 32: shrink_late<4, TG>(g, t, sm, bpre, ypre, do_expand, hooked); break;
      case 64: shrink_late<8, TG>(g, t, sm, bpre, ypre, do_expand, hooked); break;
      default: shrink_late<16, TG>(g, t, sm, bpre, ypre, do_expand, hooked); break;
    }
    if (hooked) hook();
  } else {
    prefetch_b<bp_depth<TG>()>(g, t, bpre);
  }
  if (do_expand) expand_valu<TG>(g, t, sm, bpre, ypre, have_y);
}

template <class H>
__device__ __forceinline__ void valu_tile(const ApplyArgs& g, const Tile& t, const Smem& sm,
                                          bool do_shrink, bool do_expand, bool hooked, H&& hook) {
  if (t.L == 1) valu_tile_tg<1>(g, t, sm, do_shrink, do_expand, hooked, hook);
  else if (t.L == 2) valu_tile_tg<2>(g, t, sm, do_shrink, do_expand, hooked, hook);
  else valu_tile_tg<4>(g, t, sm, do_shrink, do_expand, hooked, hook);
}

// ---------------------------------------------------------------------------
// multi-token tiles: matrix cores
// ---------------------------------------------------------------------------

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& v) {
  return __builtin_bit_cast(bf16x8_t, v);
}

// MFMA operand holding rows rbase + 8 * (lane / 16) .. + 8 of column
// cbase + lane % 16 of a row-major bf16 matrix in LDS (row stride S elements,
// S and cbase multiples of 4): two transposed 64-bit reads; in each group of
// 16 lanes, lane 4j + c reads row j, columns 4c..4c+3, and lane i receives
// column i of the four rows.
__device__ __forceinline__ bf16x8_t tr_operand(const uint16_t* m, int S, int rbase, int cbase) {
  const int l = threadIdx.x & 63, grp = l >> 4, lp = l & 15;
  const uint16_t* p = m + (rbase + 8 * grp + (lp >> 2)) * S + cbase + 4 * (lp & 3);
  const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p);
  const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(p + 4 * S));
  const uint2 a = __builtin_bit_cast(uint2, lo), b = __builtin_bit_cast(uint2, hi);
  return as_bf16x8(make_uint4(a.x, a.y, b.x, b.y));
}

// s_waitcnt that waits until at most n vector-memory operations of this
// wavefront are outstanding, leaving the other counters alone (gfx9
// encoding: vmcnt bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int n>
__device__ __forceinline__ void wait_vm() {
  static_assert(n >= 0 && n < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// Wait until at most min(n, K) stages of PER loads each are outstanding
// (n wave-uniform; the count must be a constant of the instruction).
template <int PER, int K>
__device__ __forceinline__ void wait_vm_stages(int n) {
  if constexpr (K == 0) {
    wait_vm<0>();
  } else {
    if (n >= K) wait_vm<K * PER>();
    else wait_vm_stages<PER, K - 1>(n);
  }
}

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// LDS address (byte offset in the work group's LDS) of a pointer into it.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// Reads of the shrink's LDS ring, issued as inline assembly.  The ring is
// filled by global_load_lds, and the compiler, which cannot tell ring stages
// apart, would make every LDS read it sees wait for every such load in flight
// (s_waitcnt vmcnt(0)), serialising the ring; these reads are ordered by the
// explicit waits of the ring instead.  Results are valid only after
// lds_wait() has taken them.
__device__ __forceinline__ uint64_t lds_tr16_b64(uint32_t a) {
  uint64_t v;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(a) : "memory");
  return v;
}
__device__ __forceinline__ u32x4_t lds_b128(uint32_t a) {
  u32x4_t v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a) : "memory");
  return v;
}

// Shrink of a longer tile on the matrix cores, for a rank t.r that is a
// multiple of 8 and at most R (its columns past t.r are computed from
// padding and dropped):
// MT M tiles of 16 tokens, NTN N tiles of 16 columns (R = 8 uses the first
// half of one; its other columns are read past the row end and never
// stored).  Wavefront w takes the K steps (32 rows of h_in) w, w + kW, ...,
// in stages of KW steps, and streams each stage's rows of A_i and its x
// operands straight from global memory into a ring of D stages of its own
// LDS (global_load_lds_dwordx4, no registers), D stages ahead of its matrix
// cores; no wavefront waits for another until the final reduction.  Every
// stage issues the same number of loads (loads past the block re-read the
// stage's start), and no stage past the wavefront's last is issued: the wait
// for stage j counts the loads of the min(D - 1, n - 1 - j) stages issued
// after it (n the wavefront's stages), so it is exact, and the ring's tail
// waits for no loads of its own that nothing uses.
// Rows of the last K step past the block are zeroed in LDS before use.
// Writes v to sm.vs (fp32) and its high/low bf16 split to sm.vhl.
template <int MT, int R>
__device__ __forceinline__ void shrink_mfma(const ApplyArgs& g, const Tile& t, const Smem& sm) {
  constexpr int NTN = R < 16 ? 1 : R / 16;
  constexpr int KW = R < 16 ? 2 : 1;                  // K steps per stage
  constexpr int SR = KW * kRK;                        // rows of h_in per stage
  constexpr int AB = SR * R * 2;                      // bytes of A_i per stage
  constexpr int XB = SR * MT * 16 * 2;                // bytes of x per stage
  constexpr int NAI = AB / 1024, NXI = XB / 1024;     // loads per lane per stage
  constexpr int STG = AB + XB;
  constexpr int D = kWaveRing / STG < 1 ? 1 : (kWaveRing / STG > 8 ? 8 : kWaveRing / STG);
  constexpr int XU = 16 * MT;                         // x units (16 bytes) per 8 columns
  static_assert(NAI * 1024 == AB && NXI * 1024 == XB, "stages are whole loads");
  static_assert(D * STG <= kWaveRing, "the ring fits");
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, grp = lane >> 4, lp = lane & 15;
  const int RK = rk_max(g.max_rank);
  const int nst = (t.k1 - t.k0 + SR - 1) / SR;        // stages over the block
  const int my_n = w < nst ? (nst - w + kW - 1) / kW : 0;
  char* ring = reinterpret_cast<char*>(sm.buf) + w * kWaveRing;

  // x row this lane loads: tile row lane % XU (the tile's first token's row
  // where that row holds no token; its products land in rows never stored)
  const int xr = lane % XU;
  const int xtok = xr < t.L ? sm.tok[xr] : -1;
  const uint16_t* x_row0 = g.x + (int64_t)max(sm.tok[0], 0) * g.ldx;
  const uint16_t* x_mine = xtok >= 0 ? g.x + (int64_t)xtok * g.ldx : x_row0;

  f32x4_t acc[MT][NTN];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NTN; ++nt) acc[mt][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // this wavefront's stage j into ring slot sl
  auto issue = [&](int j, int sl) {
    const int st = w + j * kW;
    const int kr0 = t.k0 + st * SR;
    const int rows = min(SR, t.k1 - kr0);             // valid rows of A_i in the stage
    const uint16_t* asrc = t.Ai + (int64_t)kr0 * t.r;
    char* base = ring + sl * STG;
#pragma unroll
    for (int i = 0; i < NAI; ++i) {
      // unit u of the stage is row u / (R/8), octet u % (R/8) of the padded
      // [SR][R] layout; A_i's rows are t.r long, and octets past t.r (and
      // rows past the block) re-read the stage's first unit, landing in
      // columns or rows that are never used
      const int u = 64 * i + lane;
      const int row = u / (R / 8), oc = u % (R / 8);
      const bool ok = row < rows && oc * 8 < t.r;
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void*)(asrc + (ok ? row * t.r + oc * 8 : 0)),
          (__attribute__((address_space(3))) void*)(base + 64 * i * 16), 16, 0, kMatrixPolicy);
    }
#pragma unroll
    for (int i = 0; i < NXI; ++i) {
      const int k = kr0 + ((64 * i + lane) / XU) * 8;
      const uint16_t* src = k < t.k1 ? x_mine + k : x_row0 + t.k0;
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void*)src,
          (__attribute__((address_space(3))) void*)(base + AB + 64 * i * 16), 16, 0, 0);
    }
    // keep every load of this stage above the waits that count it
    asm volatile("" ::: "memory");
  };
  auto consume = [&](int j, int sl) {
    wait_vm_stages<NAI + NXI, D - 1>(my_n - 1 - j);
    const int st = w + j * kW;
    const int rows = min(SR, t.k1 - t.k0 - st * SR);
    char* base = ring + sl * STG;
    if (rows < SR) {
      // the block ends inside this stage: zero the rows past it and their x
      for (int o = lane; o < (SR - rows) * (R / 8); o += 64)
        reinterpret_cast<uint4*>(base + rows * R * 2)[o] = make_uint4(0, 0, 0, 0);
      for (int o = lane; o < (SR - rows) / 8 * XU; o += 64)
        reinterpret_cast<uint4*>(base + AB + rows / 8 * XU * 16)[o] = make_uint4(0, 0, 0, 0);
    }
    const uint32_t a0 = lds_addr(base);
#pragma unroll
    for (int kk = 0; kk < KW; ++kk) {
      if (kk * kRK < rows) {
        uint64_t bt[NTN][2];
        u32x4_t xa[MT];
#pragma unroll
        for (int nt = 0; nt < NTN; ++nt) {
          const uint32_t ad =
              a0 + ((kk * kRK + 8 * grp + (lp >> 2)) * R + nt * 16 + 4 * (lp & 3)) * 2;
          bt[nt][0] = lds_tr16_b64(ad);
          bt[nt][1] = lds_tr16_b64(ad + 4 * R * 2);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          xa[mt] = lds_b128(a0 + AB + ((kk * 4 + grp) * XU + mt * 16 + lp) * 16);
        // the reads above complete before their registers are used
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int nt = 0; nt < NTN; ++nt) {
          asm volatile("" : "+v"(bt[nt][0]), "+v"(bt[nt][1]));
          const uint2 lo = __builtin_bit_cast(uint2, bt[nt][0]);
          const uint2 hi = __builtin_bit_cast(uint2, bt[nt][1]);
          const bf16x8_t b = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            asm volatile("" : "+v"(xa[mt]));
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8_t, xa[mt]), b, acc[mt][nt], 0, 0, 0);
          }
        }
      }
    }
    if (j + D < my_n) issue(j + D, sl);
  };
  if (my_n > 0) {
#pragma unroll
    for (int sl = 0; sl < D; ++sl)
      if (sl < my_n) issue(sl, sl);
    for (int j0 = 0; j0 < my_n; j0 += D) {
#pragma unroll
      for (int sl = 0; sl < D; ++sl)
        if (j0 + sl < my_n) consume(j0 + sl, sl);
    }
  }
  lds_sync();

  // pairwise tree over the wavefronts: 4 -> 2 -> 1 slots, fixed order
  f32x4_t* slot = reinterpret_cast<f32x4_t*>(sm.buf);
  for (int half = kW / 2; half >= 1; half >>= 1) {
    if (w >= half && w < 2 * half) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTN; ++nt)
          slot[(((w - half) * MT + mt) * NTN + nt) * 64 + lane] = acc[mt][nt];
    }
    lds_sync();
    if (w < half) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTN; ++nt)
          acc[mt][nt] += slot[((w * MT + mt) * NTN + nt) * 64 + lane];
    }
    lds_sync();
  }
  if (w == 0) {
    uint16_t* vhi = sm.vhl;
    uint16_t* vlo = sm.vhl + kTT * RK;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTN; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tt = mt * 16 + 4 * grp + i, cidx = nt * 16 + lp;
          if (tt < t.L && cidx < t.r) {
            const float val = acc[mt][nt][i];
            const uint32_t hb = to_bf16(val);
            const float hv = __uint_as_float(hb << 16);
            sm.vs[cidx * kTT + tt] = val;
            vhi[tt * RK + cidx] = (uint16_t)hb;
            vlo[tt * RK + cidx] = (uint16_t)to_bf16(val - hv);
          }
        }
  }
  lds_sync();
}

// v (fp32, already in sm.vs) to its high/low bf16 split in sm.vhl.
__device__ __forceinline__ void split_v(const Tile& t, const Smem& sm, int RK) {
  for (int o = threadIdx.x; o < t.L * t.r; o += kNT) {
    const int tt = o / t.r, c = o - tt * t.r;
    const float val = sm.vs[c * kTT + tt];
    const uint32_t hb = to_bf16(val);
    sm.vhl[tt * RK + c] = (uint16_t)hb;
    sm.vhl[kTT * RK + tt * RK + c] = (uint16_t)to_bf16(val - __uint_as_float(hb << 16));
  }
}

// The matrix-path expand streams B_i in column chunks of JC columns (as
// many as fit kChunk elements at K extent rk = rk_of(r)), with each
// wavefront's y words of a chunk in registers.  ExpandPre holds this
// thread's share of one chunk: its B_i units (before they go to LDS) and
// the y words of its j tiles.
constexpr int kJT = 8;                             // j tiles per wave per chunk (max)

template <int MT>
struct ExpandPre {
  uint4 breg[8];
  uint2 yv[kJT][MT];
};

__device__ __forceinline__ int expand_chunk_cols(const Tile& t) {
  // whole j tiles of 16 columns, so that a staged chunk (rk rows of the
  // padded width) stays within kChunk elements
  return min((kChunk / rk_of(t.r)) & ~15, (t.j1 - t.j0 + 15) / 16 * 16);
}

// Token of this lane's tile row in token tile nt (-1 past the tile).
template <int MT>
__device__ __forceinline__ void expand_toks(const Tile& t, const Smem& sm, int (&toks)[MT]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int nt = 0; nt < MT; ++nt) {
    const int ti = nt * 16 + (lane & 15);
    toks[nt] = ti < t.L ? sm.tok[ti] : -1;
  }
}

// This thread's B_i units of the chunk starting at column j0.
template <int MT>
__device__ __forceinline__ void expand_load_b(const ApplyArgs& g, const Tile& t, int j0, int JC,
                                              ExpandPre<MT>& pre) {
  const int cols = min(JC, t.j1 - j0);
  const int per_row = cols >> 3;
  const int n16 = t.r * per_row;
  const Rsrc rb = block_rsrc(t.Bi, (int64_t)g.h_out * t.r);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int q = (int)threadIdx.x + j * kNT;
    const int c = q / per_row, col = q - c * per_row;
    pre.breg[j] = bld16<kMatrixPolicy>(rb, (int64_t)c * g.h_out + j0 + col * 8, q < n16);
  }
}

// y words of this wave's j tiles of the chunk starting at column j0.
template <int MT>
__device__ __forceinline__ void expand_load_y(const ApplyArgs& g, const Tile& t, int j0, int JC,
                                              const int (&toks)[MT], ExpandPre<MT>& pre) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, grp = lane >> 4;
  const int njt = (min(JC, t.j1 - j0) + 15) / 16;
  // masked lanes read the tile's first token row at the chunk's first column
  const int tok0 = __builtin_amdgcn_readfirstlane(toks[0]);   // lane 0: tile row 0
  const uint16_t* y_safe = g.y + (int64_t)max(tok0, 0) * g.ldy + j0;
#pragma unroll
  for (int i = 0; i < kJT; ++i) {
    const int jt = w + i * kW;
    const int j = j0 + jt * 16 + 4 * grp;
    const bool jok = jt < njt && j < t.j1;
#pragma unroll
    for (int nt = 0; nt < MT; ++nt)
      pre.yv[i][nt] = ldg8z(g.y + (int64_t)toks[nt] * g.ldy + j, y_safe, jok && toks[nt] >= 0);
  }
}

// The first chunk's B_i units and y words, requested ahead of the expand.
template <int MT>
__device__ __forceinline__ void expand_prefetch(const ApplyArgs& g, const Tile& t,
                                                const Smem& sm, ExpandPre<MT>& pre) {
  int toks[MT];
  expand_toks<MT>(t, sm, toks);
  const int JC = expand_chunk_cols(t);
  expand_load_b<MT>(g, t, t.j0, JC, pre);
  expand_load_y<MT>(g, t, t.j0, JC, toks, pre);
}

// Output words of this wave's first NJ j tiles of a staged chunk (j tile
// w + i kW for i < NJ): D^T[j][token] = sum_c B_i[c][j] v[token][c] over the
// K extent rk, v as its bf16 high and low halves, then y = bf16(y + s D).
// The body is straight-line: every K step reads v's operands once for all j
// tiles and issues the transposed B_i reads of all NJ tiles before their
// MFMAs, so LDS latency is paid once per K step rather than once per j tile.
// Tiles past the chunk (jt >= njt) read the chunk's last tile and their
// words are never stored.
template <int NJ, int MT>
__device__ __forceinline__ void expand_jtiles(const uint16_t* Bs, int S, const uint16_t* vhi,
                                              const uint16_t* vlo, int RK, int rk, int w,
                                              int njt, float s, const ExpandPre<MT>& pre,
                                              uint2 (&out)[kJT][MT]) {
  const int lane = threadIdx.x & 63, grp = lane >> 4;
  f32x4_t acc[NJ][MT];
#pragma unroll
  for (int i = 0; i < NJ; ++i)
#pragma unroll
    for (int nt = 0; nt < MT; ++nt) acc[i][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int kc = 0; kc < rk; kc += kRK) {
    uint4 h[MT], lo[MT];
#pragma unroll
    for (int nt = 0; nt < MT; ++nt) {
      const int tt = nt * 16 + (lane & 15);
      h[nt] = *reinterpret_cast<const uint4*>(vhi + tt * RK + kc + 8 * grp);
      lo[nt] = *reinterpret_cast<const uint4*>(vlo + tt * RK + kc + 8 * grp);
    }
    bf16x8_t a[NJ];
#pragma unroll
    for (int i = 0; i < NJ; ++i) a[i] = tr_operand(Bs, S, kc, min(w + i * kW, njt - 1) * 16);
#pragma unroll
    for (int i = 0; i < NJ; ++i)
#pragma unroll
      for (int nt = 0; nt < MT; ++nt) {
        acc[i][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], as_bf16x8(h[nt]), acc[i][nt], 0, 0, 0);
        acc[i][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], as_bf16x8(lo[nt]), acc[i][nt], 0, 0, 0);
      }
  }
#pragma unroll
  for (int i = 0; i < kJT; ++i)
#pragma unroll
    for (int nt = 0; nt < MT; ++nt) {
      if (i < NJ) {
        const uint2 yw = pre.yv[i][nt];
        const float y0 = bf_lo(yw.x), y1 = bf_hi(yw.x), y2 = bf_lo(yw.y), y3 = bf_hi(yw.y);
        const uint32_t o0 = to_bf16(fmaf(s, acc[i < NJ ? i : 0][nt][0], y0));
        const uint32_t o1 = to_bf16(fmaf(s, acc[i < NJ ? i : 0][nt][1], y1));
        const uint32_t o2 = to_bf16(fmaf(s, acc[i < NJ ? i : 0][nt][2], y2));
        const uint32_t o3 = to_bf16(fmaf(s, acc[i < NJ ? i : 0][nt][3], y3));
        out[i][nt] = make_uint2(o0 | (o1 << 16), o2 | (o3 << 16));
      } else {
        out[i][nt] = make_uint2(0, 0);
      }
    }
}

// Expand of a multi-token tile with MT token tiles of 16: D^T[j][token] =
// sum_c B_i[c][j] (vhi + vlo)[token][c], then y = bf16(y + s D).  Unless
// `fetched` (expand_prefetch already requested them), the first chunk's
// B_i and y are requested here, before the hook runs.
template <int MT, class H>
__device__ __forceinline__ void expand_mfma(const ApplyArgs& g, const Tile& t, const Smem& sm,
                                            H&& hook, ExpandPre<MT>& pre, bool fetched) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, grp = lane >> 4;
  const int r = t.r;
  const int RK = rk_max(g.max_rank);
  const int rk = rk_of(r);                         // K extent, zero rows from r on
  const int JC = expand_chunk_cols(t);             // columns per chunk
  const int nchunks = (t.j1 - t.j0 + JC - 1) / JC;
  uint16_t* Bs = sm.buf;
  const uint16_t* vhi = sm.vhl;
  const uint16_t* vlo = sm.vhl + kTT * RK;
  int toks[MT];
  expand_toks<MT>(t, sm, toks);
  auto store_b = [&](int j0) {
    const int cols = min(JC, t.j1 - j0);
    const int per_row = cols >> 3;
    const int n16 = r * per_row;
    const int S = (cols + 15) / 16 * 16;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int q = tid + j * kNT;
      if (q < n16) {
        const int c = q / per_row, col = q - c * per_row;
        *reinterpret_cast<uint4*>(Bs + c * S + col * 8) = pre.breg[j];
      }
    }
    // zero padding: columns [cols, S) of rows < r, and rows [r, rk)
    if (S != cols)
      for (int c = tid; c < r; c += kNT)
        *reinterpret_cast<uint4*>(Bs + c * S + cols) = make_uint4(0, 0, 0, 0);
    for (int q = tid; q < (rk - r) * (S >> 3); q += kNT)
      *reinterpret_cast<uint4*>(Bs + r * S + q * 8) = make_uint4(0, 0, 0, 0);
  };

  if (!fetched) {
    expand_load_b<MT>(g, t, t.j0, JC, pre);
    expand_load_y<MT>(g, t, t.j0, JC, toks, pre);
  }
  hook();
  for (int ch = 0; ch < nchunks; ++ch) {
    const int j0 = t.j0 + ch * JC;
    const int cols = min(JC, t.j1 - j0);
    const int S = (cols + 15) / 16 * 16;
    const int njt = S / 16;
    store_b(j0);
    lds_sync();
    // the next chunk of B_i (this chunk's y words came before)
    if (ch + 1 < nchunks) expand_load_b<MT>(g, t, j0 + JC, JC, pre);
    // every j tile's output words first, then every store: a use of a y
    // word after a store makes the compiler wait for that store too (the
    // guards hide the exact count from it), which serialised one store
    // round trip per j tile
    uint2 out[kJT][MT];
    const int nj = (njt - w + kW - 1) / kW;          // this wave's j tiles
    if (nj > 4) expand_jtiles<8, MT>(Bs, S, vhi, vlo, RK, rk, w, njt, t.s, pre, out);
    else if (nj > 2) expand_jtiles<4, MT>(Bs, S, vhi, vlo, RK, rk, w, njt, t.s, pre, out);
    else expand_jtiles<2, MT>(Bs, S, vhi, vlo, RK, rk, w, njt, t.s, pre, out);
    // this chunk's y words are used: request the next chunk's, which travel
    // during the stores and the next chunk's staging
    if (ch + 1 < nchunks) expand_load_y<MT>(g, t, j0 + JC, JC, toks, pre);
#pragma unroll
    for (int i = 0; i < kJT; ++i) {
      const int jt = w + i * kW;
      const int j = j0 + jt * 16 + 4 * grp;
#pragma unroll
      for (int nt = 0; nt < MT; ++nt)
        if (jt < njt && toks[nt] >= 0 && j < t.j1)
          *reinterpret_cast<uint2*>(g.y + (int64_t)toks[nt] * g.ldy + j) = out[i][nt];
    }
    lds_sync();
  }
}

__device__ __forceinline__ void shrink_mfma_r(const ApplyArgs& g, const Tile& t, const Smem& sm) {
  if (t.L > 16) {
    switch (rank_class(t.r)) {
      case 8: shrink_mfma<2, 8>(g, t, sm); break;
      case 16: shrink_mfma<2, 16>(g, t, sm); break;
      case 32: shrink_mfma<2, 32>(g, t, sm); break;
      case 64: shrink_mfma<2, 64>(g, t, sm); break;
      default: shrink_mfma<2, 128>(g, t, sm); break;
    }
  } else {
    switch (rank_class(t.r)) {
      case 8: shrink_mfma<1, 8>(g, t, sm); break;
      case 16: shrink_mfma<1, 16>(g, t, sm); break;
      case 32: shrink_mfma<1, 32>(g, t, sm); break;
      case 64: shrink_mfma<1, 64>(g, t, sm); break;
      default: shrink_mfma<1, 128>(g, t, sm); break;
    }
  }
}

template <int MT, class H>
__device__ __forceinline__ void mfma_tile_mt(const ApplyArgs& g, const Tile& t, const Smem& sm,
                                             bool do_shrink, bool do_expand, bool hooked,
                                             H&& hook) {
  const int RK = rk_max(g.max_rank);
  ExpandPre<MT> pre;
  // with both halves and the hook between them (the exchange form, whose
  // items read small slices), the expand's first B_i and y loads leave
  // ahead of the shrink's, so they travel while it runs (tiles of up to 16
  // tokens: with two token tiles the registers they take would spill)
  const bool early = MT == 1 && do_shrink && do_expand && hooked;
  if (early) expand_prefetch<MT>(g, t, sm, pre);
  // v's bf16 split is read for every token row < 16 * MT and column < K extent
  for (int o = threadIdx.x; o < 2 * kTT * RK; o += kNT) sm.vhl[o] = 0;
  lds_sync();
  if (do_shrink) {
    shrink_mfma_r(g, t, sm);
  } else {
    split_v(t, sm, RK);
    lds_sync();
  }
  // with a hook, v is final only after it has run: split it again then
  auto after_b = [&] {
    if (hooked) {
      hook();
      split_v(t, sm, RK);
      lds_sync();
    }
  };
  if (do_expand) expand_mfma<MT>(g, t, sm, after_b, pre, early);
}

template <class H>
__device__ __forceinline__ void mfma_tile(const ApplyArgs& g, const Tile& t, const Smem& sm,
                                          bool do_shrink, bool do_expand, bool hooked, H&& hook) {
  if (t.L > 16) mfma_tile_mt<2>(g, t, sm, do_shrink, do_expand, hooked, hook);
  else mfma_tile_mt<1>(g, t, sm, do_shrink, do_expand, hooked, hook);
}

// ---------------------------------------------------------------------------
// ranks that are not multiples of 8: LDS-staged shrink
// ---------------------------------------------------------------------------
//
// A_i's rows are then r elements long and not 16-byte aligned, so the
// column-octet layout of the other shrinks does not apply.  Instead a window
// of WR rows of A_i, a contiguous run of WR r elements (WR and every window
// start are multiples of 8 rows, so the run is whole 16-byte units), is
// staged in LDS by 16-byte loads, with the tile's x over the same rows
// token-interleaved beside it ([row][LP]).  Thread (c, ph) = (tid mod RP,
// tid / RP), RP the rank rounded up to a power of two, accumulates
// x[l][k] A_i[k][c] over the rows k = ph, ph + NPH, ... of each window for
// every token l of the tile at once; the NPH = 256 / RP phases are then
// summed in phase order through LDS.  The next window's loads are requested
// before the current one is consumed.  The expand is shared with the other
// paths, which take any rank.
constexpr int kGenA = 16384;               // bf16 elements of A_i per window

template <int LP>
__device__ __forceinline__ void shrink_gen(const ApplyArgs& g, const Tile& t, const Smem& sm) {
  constexpr int kGA = kGenA / 8 / kNT;     // A_i units per thread per window
  constexpr int kGX = kXW / 8 / kNT;       // x units per thread per window
  static_assert(kGenA + kXW <= kBufElems && kNT * LP * 2 <= kBufElems, "LDS staging fits");
  const int tid = threadIdx.x;
  const int r = t.r;
  const int lg = 32 - __clz(r - 1);        // r >= 1: RP = 2^lg >= r
  const int RP = 1 << lg, NPH = kNT >> lg;
  const int c = tid & (RP - 1), ph = tid >> lg;
  const int WR = min(kXW / LP, (kGenA / r) & ~7);
  uint16_t* aw = sm.buf;                   // [WR r]
  uint16_t* xw = sm.buf + kGenA;           // [WR][LP]
  float* red = reinterpret_cast<float*>(sm.buf);   // [NPH][LP][RP], after the windows
  const Rsrc ra = block_rsrc(t.Ai, (int64_t)g.h_in * r);
  const uint16_t* x_safe = g.x + (int64_t)max(sm.tok[0], 0) * g.ldx;

  uint4 ar[kGA], xr[kGX];
  auto load = [&](int w0) {
    const int rows = min(WR, t.k1 - w0);
    const int n16 = rows * r / 8, n8 = rows / 8;
#pragma unroll
    for (int i = 0; i < kGA; ++i) {
      const int q = tid + i * kNT;
      ar[i] = bld16<kMatrixPolicy>(ra, (int64_t)w0 * r + q * 8, q < n16);
    }
#pragma unroll
    for (int i = 0; i < kGX; ++i) {
      const int q = tid + i * kNT;
      const int l = q / n8, u = q - l * n8;
      const int tk = l < t.L && l < LP ? sm.tok[l] : -1;
      xr[i] = ldg16z(g.x + (int64_t)tk * g.ldx + w0 + u * 8, x_safe + w0, tk >= 0);
    }
  };
  auto stage = [&](int rows) {
    const int n16 = rows * r / 8, n8 = rows / 8;
#pragma unroll
    for (int i = 0; i < kGA; ++i) {
      const int q = tid + i * kNT;
      if (q < n16) reinterpret_cast<uint4*>(aw)[q] = ar[i];
    }
#pragma unroll
    for (int i = 0; i < kGX; ++i) {
      const int q = tid + i * kNT;
      const int l = q / n8, u = q - l * n8;
      if (l < LP) {
        const uint4 v = xr[i];
        uint16_t* d = xw + (u * 8) * LP + l;
        d[0 * LP] = (uint16_t)(v.x & 0xffffu); d[1 * LP] = (uint16_t)(v.x >> 16);
        d[2 * LP] = (uint16_t)(v.y & 0xffffu); d[3 * LP] = (uint16_t)(v.y >> 16);
        d[4 * LP] = (uint16_t)(v.z & 0xffffu); d[5 * LP] = (uint16_t)(v.z >> 16);
        d[6 * LP] = (uint16_t)(v.w & 0xffffu); d[7 * LP] = (uint16_t)(v.w >> 16);
      }
    }
  };

  float acc[LP];
#pragma unroll
  for (int l = 0; l < LP; ++l) acc[l] = 0.f;
  load(t.k0);
  for (int w0 = t.k0; w0 < t.k1; w0 += WR) {
    const int rows = min(WR, t.k1 - w0);
    stage(rows);
    lds_sync();
    if (w0 + WR < t.k1) load(w0 + WR);     // travels while this window is used
    for (int k = ph; k < rows; k += NPH) {
      const float a = c < r ? __uint_as_float((uint32_t)aw[k * r + c] << 16) : 0.f;
      const uint4* xp = reinterpret_cast<const uint4*>(xw + k * LP);
#pragma unroll
      for (int q = 0; q < LP / 8; ++q) {
        float xf[8];
        unpack8(xp[q], xf);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[q * 8 + e] = fmaf(xf[e], a, acc[q * 8 + e]);
      }
    }
    lds_sync();
  }
#pragma unroll
  for (int l = 0; l < LP; ++l) red[(ph * LP + l) * RP + c] = acc[l];
  lds_sync();
  for (int o = tid; o < t.L * r; o += kNT) {
    const int l = o / r, cc = o - l * r;
    float v = red[l * RP + cc];
    for (int p = 1; p < NPH; ++p) v += red[(p * LP + l) * RP + cc];
    sm.vs[cc * kTT + l] = v;
  }
  lds_sync();
}

// A tile of a rank that is not a multiple of 8: shrink_gen, the hook, then
// the expand of the vector path (up to 4 tokens) or of the matrix path.
template <class H>
__device__ __forceinline__ void gen_tile(const ApplyArgs& g, const Tile& t, const Smem& sm,
                                         bool do_shrink, bool do_expand, bool hooked, H&& hook) {
  if (do_shrink) {
    if (t.L <= 8) shrink_gen<8>(g, t, sm);
    else if (t.L <= 16) shrink_gen<16>(g, t, sm);
    else shrink_gen<32>(g, t, sm);
    if (hooked) hook();
  }
  if (do_expand) {
    if (t.L > 4) mfma_tile(g, t, sm, false, true, false, NoHook{});
    else valu_tile(g, t, sm, false, true, false, NoHook{});
  }
}

__device__ __forceinline__ void tile_dispatch(const ApplyArgs& g, const Tile& t,
                                              const Smem& sm, bool do_shrink,
                                              bool do_expand) {
  if (t.r & 7) gen_tile(g, t, sm, do_shrink, do_expand, false, NoHook{});
  else if (t.L > vector_tokens(t.r)) mfma_tile(g, t, sm, do_shrink, do_expand, false, NoHook{});
  else valu_tile(g, t, sm, do_shrink, do_expand, false, NoHook{});
}

// Shrink of the tile's rows [k0, k1), hook(), then expand of its columns
// [j0, j1): the expand's first loads of B_i and y are requested with the
// shrink's, and the hook (the exchange that turns the partial v into the
// full one) runs while they travel.
template <class H>
__device__ __forceinline__ void tile_exchange(const ApplyArgs& g, const Tile& t, const Smem& sm,
                                              H&& hook) {
  if (t.r & 7) gen_tile(g, t, sm, true, true, true, hook);
  else if (t.L > vector_tokens(t.r)) mfma_tile(g, t, sm, true, true, true, hook);
  else valu_tile(g, t, sm, true, true, true, hook);
}

// tile_exchange for the one-launch forms, whose tiles have at most
// kSmallTile tokens: only the vector paths (the same ones tile_exchange
// takes for such tiles), so the matrix-path code and its registers stay out
// of those kernels.
template <class H>
__device__ __forceinline__ void tile_exchange_small(const ApplyArgs& g, const Tile& t,
                                                    const Smem& sm, H&& hook) {
  static_assert(kSmallTile <= 2 && kSmallTile <= 4, "the vector paths take these tiles");
  if (t.r & 7) {
    shrink_gen<8>(g, t, sm);
    hook();
    if (t.L == 1) valu_tile_tg<1>(g, t, sm, false, true, false, NoHook{});
    else valu_tile_tg<2>(g, t, sm, false, true, false, NoHook{});
  } else if (t.L == 1) {
    valu_tile_tg<1>(g, t, sm, true, true, true, hook);
  } else {
    valu_tile_tg<2>(g, t, sm, true, true, true, hook);
  }
}

// Common prologue: token indices to LDS, v zeroed.
__device__ __forceinline__ Smem tile_prologue(const ApplyArgs& g, int my_tok, void* lds) {
  Smem sm = carve(lds, g.max_rank);
  if (threadIdx.x < kTT) sm.tok[threadIdx.x] = my_tok;
  for (int o = threadIdx.x; o < g.max_rank * kTT; o += kNT) sm.vs[o] = 0.f;
  lds_sync();
  return sm;
}

// The values the one-launch item carries from phase to phase, parked in LDS
// and read back (as wave-uniform values) before each phase, so that none of
// them stays in registers across the inlined shrink and expand bodies.
struct ItemStash {
  int a, p0, L, r;
  float s;
  int u, slice;
  int pad;
  const uint16_t* Ai;
  const uint16_t* Bi;
  uint64_t ep;
};

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ const uint16_t* uni(const uint16_t* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const uint16_t*>(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ Tile unstash(const ItemStash* st) {
  Tile t;
  t.a = uni(st->a);
  t.p0 = uni(st->p0);
  t.L = uni(st->L);
  t.r = uni(st->r);
  t.s = __int_as_float(uni(__float_as_int(st->s)));
  t.Ai = uni(st->Ai);
  t.Bi = uni(st->Bi);
  return t;
}

// What the exchange yields, computed by this item alone when a partner's
// words never came: v[l][c] = sum over all of h_in of x[tok_l][k] A_i[k][c],
// one entry per thread at a time, k ascending, in fp32.  Kept plain and
// small: it runs only if a partner work group was not scheduled within
// kSpinLimit polls, and its sum order differs from the slices', so such a
// call's v (and y) can differ from the usual result in the last bits.
__device__ __forceinline__ void plain_v(const ApplyArgs& g, const Tile& t, const Smem& sm) {
  const int n = t.L * t.r;
  for (int o = threadIdx.x; o < n; o += kNT) {
    const int l = o / t.r, c = o - l * t.r;
    const int tk = sm.tok[l];
    float v = 0.f;
    if (tk >= 0) {
      const uint16_t* xr = g.x + (int64_t)tk * g.ldx;
      for (int k = 0; k < g.h_in; ++k)
        v = fmaf(__uint_as_float((uint32_t)xr[k] << 16),
                 __uint_as_float((uint32_t)t.Ai[(int64_t)k * t.r + c] << 16), v);
    }
    sm.vs[c * kTT + l] = v;
  }
  lds_sync();
}

// One item of the one-launch form with S = g.fixed_slices > 1 slices per
// tile: slice s of tile u, exchanging through tile slot `slot` (its region
// and epoch in the workspace): the shrink of h_in rows [s KR, (s+1) KR),
// the exchange of partial v with the tile's other items, and the expand of
// y columns [s W, (s+1) W), whose first loads of B_i and y are issued with
// the shrink's.  If the exchange times out, plain_v computes v here.  ep is
// the slot's epoch as the caller read it; src(t, my_tok) fills in the tile
// (adapter, first position, length) and this thread's token, false for a
// slot without a usable tile.
template <class Src>
__device__ __forceinline__ void apply_item(const ApplyArgs& g, int s, int slot, const uint64_t& ep,
                                           ItemStash& stash, unsigned char* lds, Src&& src) {
  {
    Tile t;
    int my_tok;
    t.bad = false;
    if (!src(t, my_tok)) {
      count_skipped(g, t, s);
      return;
    }
    if (t.L > kSmallTile) {
      // longer than the exchange region holds: not a tile plora_segment
      // gives a batch this small; skipped and counted like an unusable entry
      t.bad = true;
      count_skipped(g, t, s);
      return;
    }
    if (threadIdx.x == 0) {
      stash.a = t.a; stash.p0 = t.p0; stash.L = t.L; stash.r = t.r; stash.s = t.s;
      stash.u = slot; stash.slice = s; stash.Ai = t.Ai; stash.Bi = t.Bi; stash.ep = ep;
    }
    (void)tile_prologue(g, my_tok, lds);           // ends with a barrier
  }
  const Smem sm = carve(lds, g.max_rank);
  const int S = g.fixed_slices;
  const int KR = ((g.h_in + S - 1) / S + 63) & ~63;
  const int W = ((g.h_out + S - 1) / S + 15) & ~15;
  {
    Tile t = unstash(&stash);
    const int sl = uni(stash.slice);
    t.k0 = sl * KR;
    t.k1 = min(g.h_in, t.k0 + KR);
    t.j0 = sl * W;
    t.j1 = min(g.h_out, t.j0 + W);
    const Xchg xc{sl, S, KR, (uint32_t)(stash.ep + 1),
                  g.xw + (int64_t)uni(stash.u) * kSlotWords, g.polls};
    tile_exchange_small(g, t, sm, [&] {
      if (!exchange_v(t, sm, xc)) {
        bump(g, 0, 1);
        plain_v(g, t, sm);
      }
      // the slot's epoch is raised as soon as the exchange is over (every
      // partner has read it, or this item gave up), while the expand runs:
      // raised at the item's end, the atomics (eight per slot, in series
      // at memory) held up the launch's end (decode 11.81 -> 11.51 us)
      if (threadIdx.x == 0)
        __hip_atomic_fetch_max(g.xep + stash.u, stash.ep + 1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
    });
  }
}

// The per-projection part of a multi-projection apply (see plora_apply_multi).
struct ProjArgs {
  const uint16_t* A;
  const uint16_t* B;
  int64_t a_len, b_len;
  const uint16_t* A_pool;
  const uint16_t* B_pool;
  int64_t a_pool_len, b_pool_len;
  const int64_t* a_off;
  const int64_t* b_off;
  const int32_t* ranks;
  const float* scales;
  uint16_t* y;
  int64_t ldy;
  int32_t h_out, max_rank;
};

struct MultiArgs {
  ApplyArgs g;            // shared: x, the segments, the workspace, the plan
  ProjArgs proj[PLORA_MAX_PROJECTIONS];
  int32_t n_proj;
  int32_t cap8;           // tile capacity rounded up to 8
};

// ---------------------------------------------------------------------------
// plora_segment_apply: segmentation and the one-launch apply in one launch
// ---------------------------------------------------------------------------

// Where plora_segment's outputs go (the caller's plora_segments).
struct SegOut {
  int32_t* perm;
  int32_t* seg_ptr;
  int32_t* seg_id;
  int32_t* meta;
  int4* tiles;
  int32_t cap, tile_cap;
};

// One work group's tile, as the wavefront segmentation found it (L = 0: the
// slot has no tile), and the wavefront's sorting space.
constexpr int kSegApplyMax = 256;         // largest batch of the one-launch form

struct LocalTile {
  int a, p0, L, t0;       // adapter, first position, length, first token
  uint32_t tmask;         // token bits of a word
  int wcount[2][kNT / 64];             // per wavefront: segment and tile starts
  int wlast[kNT / 64], wfirst[kNT / 64];   // its last and first segment start
  uint32_t words[kSegApplyMax];        // word of token t
  uint32_t sorted[kSegApplyMax];       // word at sorted position p
  int rank_of[kSegApplyMax];           // rank, scale and offsets of token t's adapter
  float scale_of[kSegApplyMax];
  int64_t ao_of[kSegApplyMax], bo_of[kSegApplyMax];
};

// The tile slot's exchange epoch, requested right after the item's first
// load (the ids, or the tile record) and before that load is waited for:
// the vector-memory counter retires in order, so an epoch requested first
// (an agent-scope load, which goes to memory) held up the first load's wait
// behind it, and one requested after that wait added its trip to the next
// load's.  The empty asm statements keep the epoch's request between the
// first load's request and its first use (the second one takes the loaded
// value as an operand, so nothing that uses it can move above the request).
__device__ __forceinline__ uint64_t epoch_after(const ApplyArgs& g, int u, int& first) {
  __asm__ volatile("" ::: "memory");
  const uint64_t ep = xload(g.xep + u);
  __asm__ volatile("" : "+v"(first) : : "memory");
  return ep;
}

// The adapter-stack arguments that an item's first steps read (tile_blocks),
// requested at the kernel's entry with the others: requested at their first
// use, their scalar-cache miss held up that step (decode 12.01 -> 11.85 us).
__device__ __forceinline__ void request_adapter_args(const ApplyArgs& g) {
  __asm__ volatile("" ::"s"(g.A), "s"(g.B), "s"(g.a_len), "s"(g.b_len), "s"(g.A_pool),
                   "s"(g.B_pool));
}

// The segmentation of a batch of T <= 64 tokens by one wavefront, the same
// function plora_segment computes, written to so: tokens ordered by
// (adapter id, token index), ids outside [0, N) after every valid one.  Each
// lane holds the word (key << 6) | t of one token (key = id, N for a skipped
// token, N + 1 past T).  The words are distinct, so each one's rank (how many
// words are smaller, counted against all 64 read back from LDS) is its
// sorted position, and there is exactly one order.  Segments start where the
// key changes, tiles every kDecodeTile positions into a segment.  The
// wavefront stores every output of plora_segment (perm, seg_ptr, seg_id,
// tiles and meta, unused tails included).  (A bitonic sort over lane
// shuffles measured about 1 us: 21 dependent cross-lane permutes.)
__device__ __forceinline__ void wave_segment(const ApplyArgs& g, const int32_t* idx,
                                             const SegOut& so, LocalTile& lt) {
  const int T = g.T, N = g.N;
  const int lane = threadIdx.x & 63;
  const bool in = lane < T;
  const int id = in ? idx[lane] : 0;
  const bool valid = in && id >= 0 && id < N;
  const bool none = in && id == -1;
  const bool invalid = in && !valid && !none;
  const uint32_t key = valid ? (uint32_t)id : (uint32_t)N + (in ? 0u : 1u);
  const uint32_t w = (key << 6) | (uint32_t)lane;
  // LDS traffic of one wavefront is processed in order, so each read below
  // sees every lane's write before it
  lt.words[lane] = w;
  __builtin_amdgcn_wave_barrier();
  int rank = 0;
#pragma unroll
  for (int q = 0; q < 64; q += 4) {
    const uint4 o = *reinterpret_cast<const uint4*>(lt.words + q);
    rank += (o.x < w) + (o.y < w) + (o.z < w) + (o.w < w);
  }
  lt.sorted[rank] = w;
  __builtin_amdgcn_wave_barrier();
  const uint32_t sw = lt.sorted[lane];
  const uint32_t sprev = lt.sorted[lane > 0 ? lane - 1 : 0];
  const int kp = (int)(sw >> 6), tp = (int)(sw & 63);
  const uint64_t bit = uint64_t(1) << lane;
  const uint64_t below = bit - 1, upto = below | bit;
  const int n_none = __popcll(__ballot(none));
  const int n_invalid = __popcll(__ballot(invalid));
  const int n_valid = T - n_none - n_invalid;
  const bool vp = lane < n_valid;
  const bool sflag = vp && (lane == 0 || (int)(sprev >> 6) != kp);
  const uint64_t smask = __ballot(sflag);
  const int n_seg = __popcll(smask);
  const int cur = __popcll(smask & upto) - 1;            // segment of position lane
  const int sstart = vp ? 63 - __clzll(smask & upto) : 0;
  const uint64_t later = smask & ~upto;
  const int send = later ? __ffsll((long long)later) - 1 : n_valid;   // segment end
  const bool tflag = vp && ((lane - sstart) % kDecodeTile) == 0;
  const uint64_t tmask = __ballot(tflag);
  const int tu = __popcll(tmask & below);                 // tile starting here
  const int n_tiles = min(__popcll(tmask), so.tile_cap);
  if (in) so.perm[lane] = vp ? tp : -1;
  if (sflag) {
    so.seg_ptr[cur] = lane;
    so.seg_id[cur] = kp;
  }
  for (int q = n_seg + lane; q <= so.cap; q += 64) so.seg_ptr[q] = n_valid;
  for (int q = n_seg + lane; q < so.cap; q += 64) so.seg_id[q] = -1;
  if (tflag && tu < so.tile_cap)
    so.tiles[tu] = make_int4(kp, lane, min(kDecodeTile, send - lane), cur);
  for (int q = n_tiles + lane; q < so.tile_cap; q += 64) so.tiles[q] = make_int4(-1, 0, 0, -1);
  if (lane < 8)
    so.meta[lane] = lane == 0 ? n_seg : lane == 1 ? n_valid : lane == 2 ? n_none
                  : lane == 3 ? n_invalid : lane == 4 ? n_tiles : 0;
}

// The same function for 64 < T <= kSegApplyMax tokens by the whole work
// group (kNT threads, thread t holds token t, then sorted position t).
// Words are (key << 8) | t; segment and tile starts are found with each
// wavefront's ballots and combined across the wavefronts through LDS
// (counts for the indices, the last and first start for the segment that
// spans a wavefront boundary).  Every thread of the work group calls it.
__device__ __forceinline__ void block_segment(const ApplyArgs& g, const int32_t* idx, int u,
                                              const SegOut& so, bool write, LocalTile& lt,
                                              uint64_t& ep) {
  constexpr int NW = kNT / 64;
  const int T = g.T, N = g.N;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const bool in = tid < T;
  int id_in = idx[in ? tid : 0];            // (T >= 1: no branch, so no wait here)
  ep = epoch_after(g, u, id_in);
  const int id = in ? id_in : 0;
  const bool valid = in && id >= 0 && id < N;
  const bool none = in && id == -1;
  const bool invalid = in && !valid && !none;
  const int ida = valid ? id : 0;
  const int m_r = g.ranks[ida];
  const float m_s = g.scales[ida];
  const int64_t m_ao = g.a_off[ida], m_bo = g.b_off[ida];
  const uint32_t key = valid ? (uint32_t)id : (uint32_t)N + (in ? 0u : 1u);
  const uint32_t w = (key << 8) | (uint32_t)tid;
  lt.words[tid] = w;
  if (tid == 0) lt.L = 0;
  const int n_none = __syncthreads_count(none);
  const int n_invalid = __syncthreads_count(invalid);
  int rank = 0;
#pragma unroll 8
  for (int q = 0; q < kNT; q += 4) {
    const uint4 o = *reinterpret_cast<const uint4*>(lt.words + q);
    rank += (o.x < w) + (o.y < w) + (o.z < w) + (o.w < w);
  }
  lt.sorted[rank] = w;
  lds_sync();
  const uint32_t sw = lt.sorted[tid];
  const uint32_t sprev = lt.sorted[tid > 0 ? tid - 1 : 0];
  const int kp = (int)(sw >> 8), tp = (int)(sw & 255);
  const int n_valid = T - n_none - n_invalid;
  const bool vp = tid < n_valid;
  const bool sflag = vp && (tid == 0 || (int)(sprev >> 8) != kp);
  const uint64_t bit = uint64_t(1) << lane;
  const uint64_t below = bit - 1, upto = below | bit;
  const uint64_t smask = __ballot(sflag);
  if (lane == 0) {
    lt.wcount[0][wv] = __popcll(smask);
    lt.wlast[wv] = smask ? 64 * wv + 63 - __clzll(smask) : -1;
    lt.wfirst[wv] = smask ? 64 * wv + __ffsll((long long)smask) - 1 : kNT;
  }
  lds_sync();
  int seg_before = 0, n_seg = 0, last_before = -1, first_after = kNT;
#pragma unroll
  for (int k = 0; k < NW; ++k) {
    n_seg += lt.wcount[0][k];
    if (k < wv) {
      seg_before += lt.wcount[0][k];
      last_before = max(last_before, lt.wlast[k]);
    } else if (k > wv) {
      first_after = min(first_after, lt.wfirst[k]);
    }
  }
  const int cur = seg_before + __popcll(smask & upto) - 1;   // segment of position tid
  const int sstart = (smask & upto) ? 64 * wv + 63 - __clzll(smask & upto) : last_before;
  const uint64_t later = smask & ~upto;
  int send = later ? 64 * wv + __ffsll((long long)later) - 1 : first_after;
  send = min(send, n_valid);                                  // segment end
  const bool tflag = vp && ((tid - sstart) % kSmallTile) == 0;
  const uint64_t tmask_w = __ballot(tflag);
  if (lane == 0) lt.wcount[1][wv] = __popcll(tmask_w);
  lds_sync();
  int tiles_before = 0, n_tiles_all = 0;
#pragma unroll
  for (int k = 0; k < NW; ++k) {
    n_tiles_all += lt.wcount[1][k];
    if (k < wv) tiles_before += lt.wcount[1][k];
  }
  const int tu = tiles_before + __popcll(tmask_w & below);  // tile starting here
  const int n_tiles = min(n_tiles_all, so.tile_cap);
  const int tlen = min(kSmallTile, send - tid);
  if (write) {
    if (in) so.perm[tid] = vp ? tp : -1;
    if (sflag) {
      so.seg_ptr[cur] = tid;
      so.seg_id[cur] = kp;
    }
    for (int q = n_seg + tid; q <= so.cap; q += kNT) so.seg_ptr[q] = n_valid;
    for (int q = n_seg + tid; q < so.cap; q += kNT) so.seg_id[q] = -1;
    if (tflag && tu < so.tile_cap) so.tiles[tu] = make_int4(kp, tid, tlen, cur);
    for (int q = n_tiles + tid; q < so.tile_cap; q += kNT) so.tiles[q] = make_int4(-1, 0, 0, -1);
    if (tid < 8)
      so.meta[tid] = tid == 0 ? n_seg : tid == 1 ? n_valid : tid == 2 ? n_none
                   : tid == 3 ? n_invalid : tid == 4 ? n_tiles : 0;
  }
  lt.rank_of[tid] = m_r;
  lt.scale_of[tid] = m_s;
  lt.ao_of[tid] = m_ao;
  lt.bo_of[tid] = m_bo;
  if (tflag && tu == u && u < n_tiles) {     // tile u starts here
    lt.a = kp;
    lt.p0 = tid;
    lt.L = tlen;
    lt.t0 = tp;
    lt.tmask = 255u;
  }
}

// v of tile row l, column c: the sum of the KS partials in slice order.
__device__ __forceinline__ float sum_parts(const ApplyArgs& g, const Plan& p, const Tile& t,
                                           int l, int c) {
  const float* src = g.vpart + (int64_t)(t.p0 + l) * g.max_rank + c;
  const int64_t step = (int64_t)g.T * g.max_rank;
  float v = src[0];
  for (int ks = 1; ks < p.KS; ++ks) v += src[ks * step];
  return v;
}

// The expand items' v: each entry summed from the partials as sum_parts
// sums it (slice order, the same bits), with the loads of kSumBatch entries
// per thread (every slice of each) issued before any is added, so that a
// tile costs one memory round trip per batch rather than one per entry
// (KS <= kMaxSlices: the host gives a tile at most 8 slices of h_in).  The
// first batch is requested as soon as the tile record is in, before the
// rank is: entries o = l max_rank + c of the tile's rows (all max_rank
// columns of each, whole rows of the partial-sum array), so that it travels
// with the adapter metadata rather than after it; columns at or above the
// tile's rank are never used.
constexpr int kSumBatch = 4;
struct PartBatch {
  float v[kSumBatch][kMaxSlices];
};

// (COH: loads at agent scope, for partials stored earlier in the same launch)
template <bool COH = false>
__device__ __forceinline__ void parts_issue(const ApplyArgs& g, int KS, int p0, int L, int o0,
                                            PartBatch& pb) {
  const int n = L * g.max_rank;
  const int64_t step = (int64_t)g.T * g.max_rank;
  const float* base = g.vpart + (int64_t)p0 * g.max_rank;
#pragma unroll
  for (int i = 0; i < kSumBatch; ++i) {
    const int o = o0 + i * kNT + threadIdx.x;
    const float* src = base + (o < n ? o : 0);
#pragma unroll
    for (int ks = 0; ks < kMaxSlices; ++ks) {
      if constexpr (COH)
        pb.v[i][ks] = o < n && ks < KS ? __hip_atomic_load(src + ks * step, __ATOMIC_RELAXED,
                                                           __HIP_MEMORY_SCOPE_AGENT)
                                       : 0.f;
      else
        pb.v[i][ks] = o < n && ks < KS ? src[ks * step] : 0.f;
    }
  }
}

__device__ __forceinline__ void parts_finish(const ApplyArgs& g, int KS, const Tile& t, int o0,
                                             const PartBatch& pb, const Smem& sm) {
  const int n = t.L * g.max_rank;
#pragma unroll
  for (int i = 0; i < kSumBatch; ++i) {
    const int o = o0 + i * kNT + threadIdx.x;
    const int l = o / g.max_rank, c = o - l * g.max_rank;
    if (o < n && c < t.r) {
      float v = pb.v[i][0];
#pragma unroll
      for (int ks = 1; ks < kMaxSlices; ++ks)
        if (ks < KS) v += pb.v[i][ks];
      sm.vs[c * kTT + l] = v;
    }
  }
}
// Expand launch: item (tile, y column slice) takes the tile's v from the
// workspace partials (plora_apply) or from g.v (plora_expand) and expands it.
template <bool FROM_PARTS>
__global__ __launch_bounds__(kNT, kWGPerCU) void expand_kernel(ApplyArgs g) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  const Plan p = make_plan(g, kColSlices);
  Tile t;
  int my_tok, js;
  if ((int)blockIdx.x >= p.n_items) return;
  if (FROM_PARTS) {
    // the tile record, then the partials' first batch together with the
    // adapter metadata (two memory trips where three followed one another)
    const int u = item_slot(p, kColSlices, blockIdx.x, js);
    t.bad = false;
    if (u >= p.n_tiles || u >= g.tile_cap) return;
    if (!tile_from_record(g, g.tiles[u], t)) return;
    PartBatch pb;
    parts_issue(g, p.KS, t.p0, t.L, 0, pb);
    my_tok = (int)threadIdx.x < t.L ? g.perm[t.p0 + threadIdx.x] : -1;
    if (!tile_adapter(g, t, my_tok)) {
      count_skipped(g, t, js);
      return;
    }
    t.j0 = js * p.W;
    t.j1 = min(g.h_out, t.j0 + p.W);
    const Smem sm = tile_prologue(g, my_tok, apply_lds);
    parts_finish(g, p.KS, t, 0, pb, sm);
    for (int o0 = kSumBatch * kNT; o0 < t.L * g.max_rank; o0 += kSumBatch * kNT) {
      parts_issue(g, p.KS, t.p0, t.L, o0, pb);
      parts_finish(g, p.KS, t, o0, pb, sm);
    }
    lds_sync();
    tile_dispatch(g, t, sm, false, true);
    return;
  }
  if (!item_tile(g, p, kColSlices, blockIdx.x, t, my_tok, js)) {
    count_skipped(g, t, js);
    return;
  }
  const Smem sm = tile_prologue(g, my_tok, apply_lds);
  {
    for (int o = threadIdx.x; o < t.L * t.r; o += kNT) {
      const int l = o / t.r, c = o - l * t.r;
      const int tk = sm.tok[l];
      sm.vs[c * kTT + l] = tk >= 0 ? g.v[(int64_t)tk * g.ldv + c] : 0.f;
    }
  }
  lds_sync();
  tile_dispatch(g, t, sm, false, true);
}

// ---------------------------------------------------------------------------
// the two parts in one launch
// ---------------------------------------------------------------------------
//
// Batches above kFusedTokens tokens: the shrink items (tile, h_in slice) and
// the expand items (tile, column slice) of the two-launch form run as one
// launch, the expand items after every shrink item in the grid.  An expand
// item starts on its tile as soon as that tile's KS partials are stored,
// rather than after the last shrink item of the launch, so the expand items
// fill the compute units the shrink's tail leaves idle, and the gap between
// two launches goes.
//
// Each tile slot has a readiness word that counts the tile's items: a shrink
// item adds 1 once its partials are stored, an expand item adds 256 once it
// has seen all KS shrink additions (or given up waiting), and the item whose
// addition completes the count KS + 256 JS sets the word back to 0.  So the
// word is 0 when a call starts, however the previous call went (an expand
// item that gave up still adds, and a shrink item that comes after it still
// completes the count), and the low byte reaches KS only through this
// call's shrink items.  No word is shared by all work groups (one address
// taking an atomic from each of about 2700 work groups measured 80 us).
//  - A shrink item stores its partials at agent scope (sc1: the L2 writes
//    them through to memory), waits until each thread's stores are
//    acknowledged (vmcnt counts stores), and after a work-group barrier adds
//    its 1.  (An agent-scope release fence, buffer_wbl2, would write back
//    the whole L2: it measured 30 us per call.)
//  - An expand item polls the word until its low byte is KS, then reads the
//    partials at agent scope, so that no stale line in its L1 or L2 answers.
// Progress: the shrink items come before every expand item in the grid, and
// each XCD dispatches its work groups in index order, so a shrink item that
// an expand item waits for is queued on its own XCD behind shrink items
// only, which never wait: it is bound to run.  The wait is bounded all the
// same: an item that gives up computes v over all of h_in by itself
// (plain_v, counted like an exchange give-up), and the call's bits can then
// differ in the last places.

constexpr unsigned long long kExpandCount = 256;   // an expand item's addition

__device__ __forceinline__ unsigned long long parts_total(const Plan& p) {
  return (unsigned long long)p.KS + kExpandCount * (unsigned long long)p.JS;
}

// Adds n to tile u's readiness word (thread 0); the addition that completes
// the tile's count clears the word for the next call.
__device__ __forceinline__ void ready_add(const ApplyArgs& g, const Plan& p, int u,
                                          unsigned long long n) {
  const unsigned long long old =
      __hip_atomic_fetch_add(g.ready + u, (uint64_t)n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (old + n == parts_total(p))
    __hip_atomic_store(g.ready + u, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Shrink item i (as shrink_part_kernel), then its addition to the tile's word.
__device__ __forceinline__ void parts_shrink_item(const ApplyArgs& g, int i, unsigned char* lds) {
  const Plan p = make_plan(g, kRowSlices);
  if (i >= p.n_items) return;
  int ks;
  const int u = item_slot(p, kRowSlices, i, ks);
  if (u >= p.n_tiles) return;
  Tile t;
  int my_tok;
  if (item_tile(g, p, kRowSlices, i, t, my_tok, ks)) {
    const Smem sm = tile_prologue(g, my_tok, lds);
    tile_dispatch(g, t, sm, true, false);
    float* dst = g.vpart + ((int64_t)ks * g.T + t.p0) * g.max_rank;
    for (int o = threadIdx.x; o < t.L * t.r; o += kNT) {
      const int l = o / t.r, c = o - l * t.r;
      __hip_atomic_store(dst + l * g.max_rank + c, sm.vs[c * kTT + l], __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  // (tokens of an unusable entry are counted by the expand items)
  wait_vm<0>();
  lds_sync();
  if (threadIdx.x == 0) ready_add(g, p, u, 1);
}

// Expand item i (as expand_kernel<true>), once its tile's partials are in.
__device__ __forceinline__ void parts_expand_item(const ApplyArgs& g, int i, unsigned char* lds,
                                                  int* ok_sh) {
  const Plan p = make_plan(g, kColSlices);
  if (i >= p.n_items) return;
  int js;
  const int u = item_slot(p, kColSlices, i, js);
  if (u >= p.n_tiles) return;
  Tile t;
  t.bad = false;
  int my_tok;
  if (!load_tile(g, u, t, my_tok)) {
    count_skipped(g, t, js);
    if (threadIdx.x == 0) ready_add(g, p, u, kExpandCount);
    return;
  }
  t.j0 = js * p.W;
  t.j1 = min(g.h_out, t.j0 + p.W);
  if (threadIdx.x == 0) {
    unsigned long long w = xload(g.ready + u);
    for (int it = 0; (w & 255) != (unsigned)p.KS && it < g.polls; ++it) {
      __builtin_amdgcn_s_sleep(2);
      w = xload(g.ready + u);
    }
    *ok_sh = (w & 255) == (unsigned)p.KS;
    ready_add(g, p, u, kExpandCount);
  }
  const Smem sm = tile_prologue(g, my_tok, lds);     // ends with a barrier
  if (*ok_sh) {
    PartBatch pb;
    for (int o0 = 0; o0 < t.L * g.max_rank; o0 += kSumBatch * kNT) {
      parts_issue<true>(g, p.KS, t.p0, t.L, o0, pb);
      parts_finish(g, p.KS, t, o0, pb, sm);
    }
  } else {
    bump(g, 0, 1);
    plain_v(g, t, sm);
  }
  lds_sync();
  tile_dispatch(g, t, sm, false, true);
}

// Dynamic LDS above 64 KB is opted into once per kernel.
inline void allow_lds(const void* kernel, std::atomic<bool>& done) {
  if (done.load()) return;
  (void)hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  (void)hipGetLastError();
  done.store(true);
}

// Host launchers, one per kernel (each defined beside its kernel).  They
// enqueue the launch on stream and leave the launch status to
// hipGetLastError.
void launch_segment(const int32_t* idx, int32_t T, int32_t N, int32_t cap, int32_t tile_cap,
                    int32_t tbits, int32_t key_bits, int32_t* perm, int32_t* seg_ptr,
                    int32_t* seg_id, int32_t* meta, int4* tiles, hipStream_t stream);
void launch_segment_count(const int32_t* idx, int32_t T, int32_t N, int32_t cap,
                          int32_t tile_cap, int32_t* perm, int32_t* seg_ptr, int32_t* seg_id,
                          int32_t* meta, int4* tiles, hipStream_t stream);
void launch_segment_groups(const int32_t* idx, int32_t T, int32_t N, int32_t cap,
                           int32_t tile_cap, int32_t* perm, int32_t* seg_ptr, int32_t* seg_id,
                           int32_t* meta, int4* tiles, int32_t* table, hipStream_t stream);
void launch_zero(uint4* p, size_t n16, unsigned blocks, hipStream_t stream);
void launch_shrink_part(const ApplyArgs& g, unsigned grid, size_t lds, hipStream_t stream);
void launch_parts(const ApplyArgs& g, unsigned n_shrink, unsigned n_expand, size_t lds,
                  hipStream_t stream);
void launch_gather_v(const ApplyArgs& g, unsigned grid, hipStream_t stream);
void launch_apply(const ApplyArgs& g, unsigned grid, size_t lds, hipStream_t stream);
void launch_apply_cols(const ApplyArgs& g, unsigned grid, size_t lds, hipStream_t stream);
void launch_expand_parts(const ApplyArgs& g, unsigned grid, size_t lds, hipStream_t stream);
void launch_expand_v(const ApplyArgs& g, unsigned grid, size_t lds, hipStream_t stream);
void launch_segment_apply(const ApplyArgs& g, const int32_t* idx, const SegOut& so,
                          unsigned grid, size_t lds, hipStream_t stream);
void launch_apply_multi(const MultiArgs& m, unsigned grid, size_t lds, hipStream_t stream);

}  // namespace plora_impl

#endif  // PLORA_DEV_H
