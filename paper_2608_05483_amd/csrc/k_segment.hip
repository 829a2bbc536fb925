// k_segment.hip -- plora_segment kernels and the workspace fill.
#include "plora_dev.h"

namespace plora_impl {

// ---------------------------------------------------------------------------
// plora_segment: stable grouping of tokens by adapter id
// ---------------------------------------------------------------------------

// Exclusive scan of one int per thread over a block of NW wavefronts.
template <int NW = kSegWaves>
__device__ int block_exscan(int v, int* total, int* sh /* [NW + 1] */) {
  constexpr int kSegWaves = NW;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[w] = x;
  lds_sync();
  if (w == 0) {
    int s = lane < kSegWaves ? sh[lane] : 0;
    int incl = s;
#pragma unroll
    for (int o = 1; o < kSegWaves; o <<= 1) {
      int y = __shfl_up(incl, o, 64);
      if (lane >= o) incl += y;
    }
    if (lane < kSegWaves) sh[lane] = incl - s;
    if (lane == kSegWaves - 1) sh[kSegWaves] = incl;
  }
  lds_sync();
  int res = x - v + sh[w];
  *total = sh[kSegWaves];
  lds_sync();
  return res;
}

// Batches of T <= NT tokens, one thread per token.  Token t's key is its
// adapter id, N for skipped tokens; its position in the grouping is the
// number of keys below it plus the number of equal keys of earlier tokens
// (a stable sort by key, then token index).  With the distinct words
// (key << tbits) | t (tbits = ceil(log2 T); the host has checked that
// N << tbits fits 32 bits) that is the number of words below the token's
// own, counted four words per LDS read.  Segment and tile starts are then
// flagged per position and numbered by block scans.
template <int NT>
__global__ __launch_bounds__(NT) void segment_small_kernel(
    const int32_t* __restrict__ idx, int32_t T, int32_t N, int32_t cap,
    int32_t tile_cap, int32_t tbits, int32_t* __restrict__ perm, int32_t* __restrict__ seg_ptr,
    int32_t* __restrict__ seg_id, int32_t* __restrict__ meta, int4* __restrict__ tiles) {
  constexpr int NW = NT / 64;
  __shared__ __align__(16) uint32_t word_t[NT];   // word of token t
  __shared__ int32_t key_p[NT];       // key at grouped position p
  __shared__ int32_t start_s[NT + 1]; // segment starts, then n_valid
  __shared__ int32_t scan_sh[NW + 1];
  const int t = threadIdx.x;

  int key = N + 1;                    // threads past T sort after everything
  int none = 0, invalid = 0;
  if (t < T) {
    const int id = idx[t];
    if (id >= 0 && id < N) {
      key = id;
    } else {
      key = N;
      none = id == -1;
      invalid = !none;
    }
  }
  const uint32_t word = ((uint32_t)key << tbits) | (uint32_t)t;   // ranked only for t < T
  word_t[t] = word;
  const int n_none = __syncthreads_count(none);
  const int n_invalid = __syncthreads_count(invalid);
  const int n_valid = T - n_none - n_invalid;

  if (t < T) {
    int rank = 0;
    const int T4 = T & ~3;
#pragma unroll 4
    for (int u = 0; u < T4; u += 4) {
      const uint4 o = *reinterpret_cast<const uint4*>(word_t + u);
      rank += (o.x < word) + (o.y < word) + (o.z < word) + (o.w < word);
    }
    for (int u = T4; u < T; ++u) rank += word_t[u] < word;
    key_p[rank] = key;
    perm[rank] = key < N ? t : -1;
  }
  lds_sync();

  // segments: position p starts one when its key differs from p - 1's
  const int p = t;
  const bool sflag = p < n_valid && (p == 0 || key_p[p - 1] != key_p[p]);
  int n_seg;
  const int sidx = block_exscan<NW>(sflag ? 1 : 0, &n_seg, scan_sh);
  if (sflag) {
    seg_ptr[sidx] = p;
    seg_id[sidx] = key_p[p];
    start_s[sidx] = p;
  }
  if (t == 0) start_s[n_seg] = n_valid;
  lds_sync();
  for (int q = n_seg + t; q <= cap; q += NT) seg_ptr[q] = n_valid;
  for (int q = n_seg + t; q < cap; q += NT) seg_id[q] = -1;

  // tiles: a position starts one when it lies a multiple of the tile length
  // past its segment's start; sidx + sflag - 1 is the segment of position p
  const int cur = sidx + (sflag ? 1 : 0) - 1;
  bool tflag = false;
  int start = 0, end = 0;
  if (p < n_valid) {
    start = start_s[cur];
    end = start_s[cur + 1];
    tflag = ((p - start) % tile_tokens(T)) == 0;
  }
  int n_tiles;
  const int tu = block_exscan<NW>(tflag ? 1 : 0, &n_tiles, scan_sh);
  if (tflag && tu < tile_cap)
    tiles[tu] = make_int4(key_p[p], p, min(tile_tokens(T), end - p), cur);
  n_tiles = min(n_tiles, tile_cap);
  for (int u = n_tiles + t; u < tile_cap; u += NT) tiles[u] = make_int4(-1, 0, 0, -1);
  if (t == 0) {
    meta[0] = n_seg;
    meta[1] = n_valid;
    meta[2] = n_none;
    meta[3] = n_invalid;
    meta[4] = n_tiles;
    meta[5] = 0;
    meta[6] = 0;
    meta[7] = 0;
  }
}

// Words are (key << tbits) | t, key = adapter id or N for skipped tokens.
__global__ __launch_bounds__(kSegThreads) void segment_kernel(
    const int32_t* __restrict__ idx, int32_t T, int32_t N, int32_t cap,
    int32_t tile_cap, int32_t tbits, int32_t key_bits,
    int32_t* __restrict__ perm, int32_t* __restrict__ seg_ptr,
    int32_t* __restrict__ seg_id, int32_t* __restrict__ meta,
    int4* __restrict__ tiles) {
  // Two word buffers of up to PLORA_MAX_TOKENS + 1 entries (128 KB) plus the
  // per-wave digit cursors: static, gfx950 has 160 KB of LDS per CU.
  __shared__ uint32_t seg_lds[2 * (PLORA_MAX_TOKENS + 1)];
  __shared__ int32_t cursor[kSegWaves][256];
  __shared__ int32_t scan_sh[kSegWaves + 1];
  __shared__ int32_t n_none_sh, n_invalid_sh;

  uint32_t* buf0 = seg_lds;
  uint32_t* buf1 = seg_lds + T + 1;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint32_t tmask = (1u << tbits) - 1u;

  if (tid == 0) { n_none_sh = 0; n_invalid_sh = 0; }
  lds_sync();

  // load and pack; count skipped tokens.  Eight loads per thread are issued
  // before any is used (addresses past T re-read idx[0]), so the batch costs
  // one memory round trip per eight, not one per token.
  int my_none = 0, my_invalid = 0;
  constexpr int kLoadBatch = 8;
  for (int t0 = 0; t0 < T; t0 += kLoadBatch * kSegThreads) {
    int ids[kLoadBatch];
#pragma unroll
    for (int j = 0; j < kLoadBatch; ++j) {
      const int t = t0 + j * kSegThreads + tid;
      ids[j] = idx[t < T ? t : 0];
    }
#pragma unroll
    for (int j = 0; j < kLoadBatch; ++j) {
      const int t = t0 + j * kSegThreads + tid;
      if (t < T) {
        const int id = ids[j];
        uint32_t key;
        if (id >= 0 && id < N) {
          key = (uint32_t)id;
        } else {
          key = (uint32_t)N;
          if (id == -1) ++my_none; else ++my_invalid;
        }
        buf0[t] = (key << tbits) | (uint32_t)t;
      }
    }
  }
  if (my_none) atomicAdd(&n_none_sh, my_none);
  if (my_invalid) atomicAdd(&n_invalid_sh, my_invalid);
  lds_sync();

  // LSD radix passes over the key bits; each wave owns a contiguous chunk
  const int chunk = ((T + kSegWaves - 1) / kSegWaves + 63) & ~63;
  const int e_begin = w * chunk;
  const int passes = key_bits > 0 ? (key_bits + 7) / 8 : 0;
  const int dbits = passes ? (key_bits + passes - 1) / passes : 0;
  const int nbuck = 1 << dbits;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

  for (int pass = 0; pass < passes; ++pass) {
    const int shift = tbits + pass * dbits;
    for (int d = lane; d < nbuck; d += 64) cursor[w][d] = 0;
    lds_sync();
    // count digits per wave; each group's words and peer masks stay in
    // registers for the scatter below (a wave has at most kSegGroups groups)
    uint32_t gword[kSegGroups];
    uint64_t gpeers[kSegGroups];
#pragma unroll
    for (int gi = 0; gi < kSegGroups; ++gi) {
      gword[gi] = 0u;
      gpeers[gi] = 0ull;
      if (gi * 64 < chunk) {
        const int e = e_begin + gi * 64 + lane;
        const bool act = e < T;
        const uint32_t word = act ? buf0[e] : 0u;
        const uint32_t dig = (word >> shift) & (uint32_t)(nbuck - 1);
        uint64_t peers = __ballot(act);
        for (int b = 0; b < dbits; ++b) {
          uint64_t m = __ballot((dig >> b) & 1u);
          peers &= ((dig >> b) & 1u) ? m : ~m;
        }
        gword[gi] = word;
        gpeers[gi] = peers;
        if (act && (peers & below) == 0ull) cursor[w][dig] += __popcll(peers);
      }
    }
    lds_sync();
    // exclusive scan in (digit, wave) order
    {
      const int entries = nbuck * kSegWaves;
      const int per = (entries + kSegThreads - 1) / kSegThreads;
      int vals[16];
      int sum = 0;
      for (int i = 0; i < per; ++i) {
        int en = tid * per + i;
        int v = 0;
        if (en < entries) v = cursor[en % kSegWaves][en / kSegWaves];
        vals[i] = v;
        sum += v;
      }
      int tot;
      int base = block_exscan(sum, &tot, scan_sh);
      for (int i = 0; i < per; ++i) {
        int en = tid * per + i;
        if (en < entries) cursor[en % kSegWaves][en / kSegWaves] = base;
        base += vals[i];
      }
    }
    lds_sync();
    // stable scatter: groups of 64 in order, rank by lower peers
#pragma unroll
    for (int gi = 0; gi < kSegGroups; ++gi) {
      if (gi * 64 < chunk) {
        const int e = e_begin + gi * 64 + lane;
        const bool act = e < T;
        const uint32_t word = gword[gi];
        const uint32_t dig = (word >> shift) & (uint32_t)(nbuck - 1);
        const uint64_t peers = gpeers[gi];
        const int base = act ? cursor[w][dig] : 0;
        if (act) buf1[base + __popcll(peers & below)] = word;
        __builtin_amdgcn_wave_barrier();
        if (act && (peers & below) == 0ull) cursor[w][dig] = base + __popcll(peers);
        __builtin_amdgcn_wave_barrier();
      }
    }
    lds_sync();
    uint32_t* tmp = buf0; buf0 = buf1; buf1 = tmp;
  }

  const int n_none = n_none_sh, n_invalid = n_invalid_sh;
  const int n_valid = T - n_none - n_invalid;

  // perm in grouped order, one coalesced pass
  for (int p = tid; p < T; p += kSegThreads)
    perm[p] = p < n_valid ? (int32_t)(buf0[p] & tmask) : -1;

  // blocked positions per thread; the key of the position before this
  // thread's first is read once and then carried along
  const int per = (T + kSegThreads - 1) / kSegThreads;
  const int p_begin = tid * per;
  const uint32_t key_before =
      p_begin > 0 && p_begin - 1 < n_valid ? buf0[p_begin - 1] >> tbits : 0xffffffffu;
  int nflags = 0;
  {
    uint32_t prev = key_before;
    for (int i = 0; i < per; ++i) {
      const int p = p_begin + i;
      if (p < n_valid) {
        const uint32_t k = buf0[p] >> tbits;
        if (p == 0 || prev != k) ++nflags;
        prev = k;
      }
    }
  }
  int n_seg;
  int sbase = block_exscan(nflags, &n_seg, scan_sh);
  // buf1 now holds seg starts (cap + 1 <= T + 1 entries)
  int32_t* seg_lds_ptr = reinterpret_cast<int32_t*>(buf1);
  {
    int s = sbase;
    uint32_t prev = key_before;
    for (int i = 0; i < per; ++i) {
      const int p = p_begin + i;
      if (p < n_valid) {
        const uint32_t k = buf0[p] >> tbits;
        if (p == 0 || prev != k) {
          if (s < cap) {
            seg_ptr[s] = p;
            seg_id[s] = (int32_t)k;
            seg_lds_ptr[s] = p;
          }
          ++s;
        }
        prev = k;
      }
    }
  }
  n_seg = min(n_seg, cap);
  if (tid == 0) seg_lds_ptr[n_seg] = n_valid;
  lds_sync();
  for (int s = n_seg + tid; s <= cap; s += kSegThreads) seg_ptr[s] = n_valid;
  for (int s = n_seg + tid; s < cap; s += kSegThreads) seg_id[s] = -1;

  // tiles: a position starts a tile when it lies a multiple of kTT past its
  // segment's start.  sbase segments start before this thread's first
  // position, so that position belongs to segment sbase - 1 unless it starts
  // segment sbase itself.  Each thread carries its current segment's start
  // and the next segment's start (seg_lds_ptr[n_seg] = n_valid ends the
  // last one) and reads seg_lds_ptr only where a segment begins; cur + 1 <=
  // n_seg throughout, and cur = -1 only until position 0 starts segment 0.
  const int start0 = sbase > 0 ? seg_lds_ptr[sbase - 1] : 0;
  const int next0 = seg_lds_ptr[sbase];
  int ntf = 0;
  {
    int cur = sbase - 1, start = start0, next = next0;
    for (int i = 0; i < per; ++i) {
      const int p = p_begin + i;
      if (p < n_valid) {
        if (p == next) { ++cur; start = next; next = seg_lds_ptr[cur + 1]; }
        if (((p - start) & (kTT - 1)) == 0) ++ntf;
      }
    }
  }
  int n_tiles;
  int tbase = block_exscan(ntf, &n_tiles, scan_sh);
  {
    int tu = tbase;
    int cur = sbase - 1, start = start0, next = next0;
    for (int i = 0; i < per; ++i) {
      const int p = p_begin + i;
      if (p < n_valid) {
        if (p == next) { ++cur; start = next; next = seg_lds_ptr[cur + 1]; }
        if (((p - start) & (kTT - 1)) == 0) {
          const int len = min(kTT, next - p);
          if (tu < tile_cap) tiles[tu] = make_int4((int)(buf0[p] >> tbits), p, len, cur);
          ++tu;
        }
      }
    }
  }
  n_tiles = min(n_tiles, tile_cap);
  for (int u = n_tiles + tid; u < tile_cap; u += kSegThreads)
    tiles[u] = make_int4(-1, 0, 0, -1);
  if (tid == 0) {
    meta[0] = n_seg;
    meta[1] = n_valid;
    meta[2] = n_none;
    meta[3] = n_invalid;
    meta[4] = n_tiles;
    meta[5] = 0;
    meta[6] = 0;
    meta[7] = 0;
  }
}

__global__ void zero_kernel(uint4* p, size_t n16) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n16;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// the multi-work-group segmentation (batches above 1024 tokens)
// ---------------------------------------------------------------------------
//
// The same stable counting sort by adapter id as the kernels above, spread
// over G = ceil(T / 1024) work groups of 1024 tokens each, in three launches:
//   count    group g histograms its tokens' keys in LDS (key = id, N for a
//            skipped token) into row g of a G x (N + 2) table in the
//            workspace; column N + 1 holds the group's tokens with id -1;
//   scan     one work group sums each key's counts over the groups, writes
//            each key's first position in the grouped order (the tokens of
//            smaller keys) into row G of the table, and writes seg_ptr,
//            seg_id, tiles and meta from the key totals;
//   scatter  group g starts key k at that position plus key k's tokens in
//            groups before g, and places each token there plus the number of
//            equal keys before it in the group (token order), which is the
//            stable order; skipped tokens fill the tail with -1.
// The table is only read by the scan, so its loads are all in flight at
// once (rewriting it in place would order each load behind a store).
// Within a wavefront, tokens of equal key are found with ballots over the key
// bits (peer masks): one LDS update per distinct key per wavefront.
constexpr int kGroupTokens = 1024;
constexpr int kGroupWaves = kGroupTokens / 64;
constexpr int kGroupKeys = 8192;         // N + 1 keys must fit one LDS table
constexpr int kMaxGroups = (PLORA_MAX_TOKENS + kGroupTokens - 1) / kGroupTokens;

// sum over groups g < n (n <= kMaxGroups) of table[g][k]: every load issued
// before any is used (from a clamped row, masked), so the sum costs one
// memory round trip rather than one per group
__device__ __forceinline__ int sum_rows(const int32_t* table, int S, int k, int n) {
  int v[kMaxGroups];
#pragma unroll
  for (int g = 0; g < kMaxGroups; ++g) v[g] = table[(int64_t)(g < n ? g : 0) * S + k];
  int s = 0;
#pragma unroll
  for (int g = 0; g < kMaxGroups; ++g) s += g < n ? v[g] : 0;
  return s;
}

// The wavefront's lanes whose key equals this lane's (among lanes with in
// set), from ballots over kbits key bits.
__device__ __forceinline__ uint64_t key_peers(int key, bool in, int kbits) {
  uint64_t peers = __ballot(in);
  for (int b = 0; b < kbits; ++b) {
    const bool bit = (key >> b) & 1;
    const uint64_t m = __ballot(bit);
    peers &= bit ? m : ~m;
  }
  return peers;
}

// key_peers for chunks of few distinct keys (a request's tokens are
// contiguous, so a prefill chunk holds one or two): up to kLeaderRounds times
// the first lane not yet matched takes every lane with its key (a ballot per
// distinct key); lanes left over after that take key_peers' kbits ballots.
// The two agree: every lane of a key matched in a round leaves together, so
// the lanes left over share no key with those that left.
constexpr int kLeaderRounds = 4;
__device__ __forceinline__ uint64_t key_peers_few(int key, bool in, int kbits) {
  uint64_t left = __ballot(in);
  uint64_t peers = 0;
#pragma unroll
  for (int it = 0; it < kLeaderRounds; ++it) {
    if (left == 0) break;                                   // wave-uniform
    const int lead = __builtin_ctzll(left);
    const int lk = __builtin_amdgcn_readlane(key, lead);
    const uint64_t m = __ballot(key == lk) & left;
    if ((m >> (threadIdx.x & 63)) & 1) peers = m;
    left &= ~m;
  }
  if (left != 0) {                                          // wave-uniform
    const uint64_t rest = key_peers(key, in, kbits);
    if ((left >> (threadIdx.x & 63)) & 1) peers = rest;
  }
  return peers;
}

__device__ __forceinline__ int group_key(const int32_t* idx, int t, int T, int N, bool& none) {
  none = false;
  if (t >= T) return N + 1;
  const int id = idx[t];
  if (id >= 0 && id < N) return id;
  none = id == -1;
  return N;
}

// The value of the lane CTRL names (a DPP row shift or row broadcast), 0
// where it names none or ROWS masks the lane's row of 16 lanes off.
template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ int dpp_or_zero(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, 0xf, false);
}

// Inclusive scan over the wavefront's 64 lanes, of four ints at once, with
// DPP moves (no LDS): shifts right by 1, 2, 4 and 8 lanes within each row of
// 16 scan the rows; lane 15's total is then broadcast into rows 1 and 3, and
// lane 31's (rows 0 and 1) into rows 2 and 3.
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += dpp_or_zero<0x111>(x);          // row_shr:1
  x += dpp_or_zero<0x112>(x);          // row_shr:2
  x += dpp_or_zero<0x114>(x);          // row_shr:4
  x += dpp_or_zero<0x118>(x);          // row_shr:8
  x += dpp_or_zero<0x142, 0xa>(x);     // row_bcast:15
  x += dpp_or_zero<0x143, 0xc>(x);     // row_bcast:31
  return x;
}
__device__ __forceinline__ int4 wave_incl_scan4(int4 v) {
  return make_int4(wave_incl_scan(v.x), wave_incl_scan(v.y), wave_incl_scan(v.z),
                   wave_incl_scan(v.w));
}

// Exclusive scan of four ints per thread at once over a block of NW
// wavefronts (one pass of barriers for all four); *total gets the sums.
template <int NW>
__device__ int4 block_exscan4(int4 v, int4* total, int4* sh /* [NW + 1] */) {
  static_assert(NW <= 64, "one wavefront scans the wavefront totals");
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int4 x = wave_incl_scan4(v);
  if (lane == 63) sh[w] = x;
  lds_sync();
  if (w == 0) {
    const int4 s = lane < NW ? sh[lane] : make_int4(0, 0, 0, 0);
    const int4 incl = wave_incl_scan4(s);
    if (lane < NW) sh[lane] = make_int4(incl.x - s.x, incl.y - s.y, incl.z - s.z, incl.w - s.w);
    if (lane == NW - 1) sh[NW] = incl;
  }
  lds_sync();
  const int4 b = sh[w];
  *total = sh[NW];
  return make_int4(x.x - v.x + b.x, x.y - v.y + b.y, x.z - v.z + b.z, x.w - v.w + b.w);
}

__global__ __launch_bounds__(kGroupTokens) void seg_count_kernel(
    const int32_t* __restrict__ idx, int32_t T, int32_t N, int32_t kbits,
    int32_t* __restrict__ table) {
  __shared__ int32_t hist[kGroupKeys];
  const int g = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int nb = N + 1;
  for (int k = tid; k < nb; k += kGroupTokens) hist[k] = 0;
  const int t = g * kGroupTokens + tid;
  bool none;
  const int key = group_key(idx, t, T, N, none);
  const bool in = t < T;
  const int n_none = __syncthreads_count(none);    // also orders the zeroing
  const uint64_t peers = key_peers(key, in, kbits);
  const uint64_t below = (uint64_t(1) << lane) - 1;
  if (in && (peers & below) == 0) atomicAdd(&hist[key], __popcll(peers));
  lds_sync();
  int32_t* row = table + (int64_t)g * (N + 2);
  for (int k = tid; k < nb; k += kGroupTokens) row[k] = hist[k];
  if (tid == 0) row[N + 1] = n_none;
}

__global__ __launch_bounds__(kGroupTokens) void seg_scan_kernel(
    int32_t* __restrict__ table, int32_t G, int32_t T, int32_t N, int32_t cap,
    int32_t tile_cap, int32_t* __restrict__ seg_ptr, int32_t* __restrict__ seg_id,
    int32_t* __restrict__ meta, int4* __restrict__ tiles) {
  constexpr int kPer = kGroupKeys / kGroupTokens;   // keys per thread, at most
  __shared__ int4 scan_sh[kGroupWaves + 1];
  __shared__ int32_t none_sh;
  const int tid = threadIdx.x;
  const int nb = N + 1, S = N + 2;
  const int per = (nb + kGroupTokens - 1) / kGroupTokens;
  const int k0 = tid * per;
  int tot[kPer];
  int mine = 0, mine_valid = 0, flags = 0, ntile = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int k = k0 + i;
    int v = 0;
    if (i < per && k < nb) v = sum_rows(table, S, k, G);
    tot[i] = v;
    mine += v;
    if (k < N) {
      mine_valid += v;
      flags += v > 0;
      ntile += (v + kTT - 1) / kTT;
    }
  }
  if (tid == 0) none_sh = sum_rows(table, S, N + 1, G);
  int4 tot4;
  const int4 ex = block_exscan4<kGroupWaves>(make_int4(mine, mine_valid, flags, ntile), &tot4,
                                             scan_sh);
  int base = ex.x, sidx = ex.z, tu = ex.w;
  const int n_valid = tot4.y, n_seg = tot4.z, n_tiles_all = tot4.w;
  int32_t* starts = table + (int64_t)G * S;          // row G: each key's first position
  const int n_none = none_sh;
  const int n_invalid = T - n_valid - n_none;
  const int n_tiles = min(n_tiles_all, tile_cap);
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int k = k0 + i;
    if (i < per && k < nb) {
      starts[k] = base;
      const int v = tot[i];
      if (k < N && v > 0) {
        seg_ptr[sidx] = base;
        seg_id[sidx] = k;
        for (int j = 0; j * kTT < v; ++j, ++tu)
          if (tu < tile_cap) tiles[tu] = make_int4(k, base + j * kTT, min(kTT, v - j * kTT), sidx);
        ++sidx;
      }
      base += v;
    }
  }
  for (int q = n_seg + tid; q <= cap; q += kGroupTokens) seg_ptr[q] = n_valid;
  for (int q = n_seg + tid; q < cap; q += kGroupTokens) seg_id[q] = -1;
  for (int u = n_tiles + tid; u < tile_cap; u += kGroupTokens) tiles[u] = make_int4(-1, 0, 0, -1);
  if (tid == 0) {
    meta[0] = n_seg;
    meta[1] = n_valid;
    meta[2] = n_none;
    meta[3] = n_invalid;
    meta[4] = n_tiles;
    meta[5] = 0;
    meta[6] = 0;
    meta[7] = 0;
  }
}

__global__ __launch_bounds__(kGroupTokens) void seg_scatter_kernel(
    const int32_t* __restrict__ idx, int32_t T, int32_t N, int32_t kbits,
    const int32_t* __restrict__ table, int32_t* __restrict__ perm) {
  __shared__ int32_t cursor[kGroupKeys];
  const int g = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nb = N + 1, S = N + 2;
  const int32_t* starts = table + (int64_t)gridDim.x * S;
  for (int k = tid; k < nb; k += kGroupTokens) cursor[k] = starts[k] + sum_rows(table, S, k, g);
  const int t = g * kGroupTokens + tid;
  bool none;
  const int key = group_key(idx, t, T, N, none);
  const bool in = t < T;
  const uint64_t peers = key_peers(key, in, kbits);
  const uint64_t below = (uint64_t(1) << lane) - 1;
  lds_sync();
  // wavefronts in token order, each taking its positions from the running
  // cursors and advancing them (one lane per distinct key)
  for (int ww = 0; ww < kGroupWaves; ++ww) {
    if (w == ww && in) {
      const int base = cursor[key];
      perm[base + __popcll(peers & below)] = key < N ? t : -1;
      __builtin_amdgcn_wave_barrier();
      if ((peers & below) == 0) cursor[key] = base + __popcll(peers);
    }
    lds_sync();
  }
}

// ---------------------------------------------------------------------------
// one-launch counting sort (256 < T <= PLORA_MAX_TOKENS, N < kCountKeys)
// ---------------------------------------------------------------------------
//
// One 1024-thread work group; wavefront w owns a contiguous range of
// ceil(T / 16) tokens (rounded up to whole 64-token chunks) and its own row
// of key counts in LDS.
//   count    each wavefront counts its range's keys into its row (the lanes
//            of a chunk with equal key are found with ballots over the key
//            bits; one of them adds the group's size), and keeps each chunk's
//            keys and peer masks in registers;
//   scan     each key's count is summed over the rows and the totals are
//            scanned into segment starts; row w's entry for key k becomes the
//            position of wavefront w's first token of key k (the key's start
//            plus its tokens in earlier wavefronts); seg_ptr, seg_id, tiles
//            and meta are written from the totals;
//   scatter  each wavefront walks its chunks in token order, placing each
//            token at its row's cursor for its key plus the number of equal
//            keys before it in the chunk, then advancing the cursor.
// Every wavefront writes only its own row after the scan, so the scatter needs
// no barrier between wavefronts.  Same output bits as every other form.
constexpr int kCountChunks =
    (PLORA_MAX_TOKENS + kGroupWaves * 64 - 1) / (kGroupWaves * 64);   // chunks per wavefront

__global__ __launch_bounds__(kGroupTokens) void segment_count_kernel(
    const int32_t* __restrict__ idx, int32_t T, int32_t N, int32_t cap, int32_t tile_cap,
    int32_t kbits, int32_t* __restrict__ perm, int32_t* __restrict__ seg_ptr,
    int32_t* __restrict__ seg_id, int32_t* __restrict__ meta, int4* __restrict__ tiles) {
  __shared__ __align__(16) int32_t rows[kGroupWaves][kCountKeys];
  __shared__ int4 scan_sh[kGroupWaves + 1];
  __shared__ int32_t none_sh;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nb = N + 1;
  const int tl = tile_tokens(T);
  const int per_w = ((T + kGroupWaves - 1) / kGroupWaves + 63) & ~63;   // tokens per wavefront
  const int nch = per_w >> 6;                                             // chunks per wavefront
  const uint64_t below = (uint64_t(1) << lane) - 1;
  // the ids of every chunk, requested before anything else (they arrive
  // while the rows are cleared)
  int ids[kCountChunks];
#pragma unroll
  for (int c = 0; c < kCountChunks; ++c) {
    const int t = w * per_w + c * 64 + lane;
    ids[c] = idx[c < nch && t < T ? t : 0];
  }
  for (int k = lane * 4; k < nb; k += 256) *reinterpret_cast<int4*>(&rows[w][k]) = int4{0, 0, 0, 0};
  if (tid == 0) none_sh = 0;
  lds_sync();

  // count
  int keys[kCountChunks];
  uint64_t peers[kCountChunks];
  int my_none = 0;
#pragma unroll
  for (int c = 0; c < kCountChunks; ++c) {
    keys[c] = N + 1;
    peers[c] = 0;
    if (c < nch) {                                  // wave-uniform
      const int t = w * per_w + c * 64 + lane;
      const bool in = t < T;
      const int id = ids[c];
      const bool valid = in && id >= 0 && id < N;
      const int key = !in ? N + 1 : valid ? id : N;
      my_none += in && id == -1;
      const uint64_t pm = key_peers_few(key, in, kbits);
      keys[c] = key;
      peers[c] = pm;
      // one lane per distinct key adds, so no two lanes share an address;
      // an atomic with no return waits for nothing
      if (in && (pm & below) == 0) atomicAdd(&rows[w][key], __popcll(pm));
    }
  }
  if (my_none) atomicAdd(&none_sh, my_none);
  lds_sync();

  // scan: keys k0 .. k0 + per - 1 per thread
  const int per = (nb + kGroupTokens - 1) / kGroupTokens;   // at most 2
  const int k0 = tid * per;
  int tot[2] = {0, 0};
  int mine = 0, mine_valid = 0, flags = 0, ntile = 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int k = k0 + i;
    if (i < per && k < nb) {
      int v = 0;
#pragma unroll
      for (int ww = 0; ww < kGroupWaves; ++ww) v += rows[ww][k];
      tot[i] = v;
      mine += v;
      if (k < N) {
        mine_valid += v;
        flags += v > 0;
        ntile += (v + tl - 1) / tl;
      }
    }
  }
  int4 tot4;
  const int4 ex = block_exscan4<kGroupWaves>(make_int4(mine, mine_valid, flags, ntile), &tot4,
                                             scan_sh);
  int base = ex.x, sidx = ex.z, tu = ex.w;
  const int n_valid = tot4.y, n_seg = tot4.z, n_tiles = min(tot4.w, tile_cap);
  const int n_none = none_sh;
  const int n_invalid = T - n_valid - n_none;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int k = k0 + i;
    if (i < per && k < nb) {
      int run = base;
#pragma unroll
      for (int ww = 0; ww < kGroupWaves; ++ww) {
        const int c = rows[ww][k];
        rows[ww][k] = run;
        run += c;
      }
      const int v = tot[i];
      if (k < N && v > 0) {
        seg_ptr[sidx] = base;
        seg_id[sidx] = k;
        for (int j = 0; j * tl < v; ++j, ++tu)
          if (tu < tile_cap) tiles[tu] = make_int4(k, base + j * tl, min(tl, v - j * tl), sidx);
        ++sidx;
      }
      base += v;
    }
  }
  for (int q = n_seg + tid; q <= cap; q += kGroupTokens) seg_ptr[q] = n_valid;
  for (int q = n_seg + tid; q < cap; q += kGroupTokens) seg_id[q] = -1;
  for (int u = n_tiles + tid; u < tile_cap; u += kGroupTokens) tiles[u] = make_int4(-1, 0, 0, -1);
  if (tid == 0) {
    meta[0] = n_seg;
    meta[1] = n_valid;
    meta[2] = n_none;
    meta[3] = n_invalid;
    meta[4] = n_tiles;
    meta[5] = 0;
    meta[6] = 0;
    meta[7] = 0;
  }
  lds_sync();

  // scatter: each wavefront through its own chunks with its own row of cursors
#pragma unroll
  for (int c = 0; c < kCountChunks; ++c) {
    if (c < nch) {
      const int t = w * per_w + c * 64 + lane;
      const int key = keys[c];
      const uint64_t pm = peers[c];
      if (t < T) {
        const int b = rows[w][key];
        perm[b + __popcll(pm & below)] = key < N ? t : -1;
      }
      __builtin_amdgcn_wave_barrier();
      if (t < T && (pm & below) == 0) rows[w][key] += __popcll(pm);
      __builtin_amdgcn_wave_barrier();
    }
  }
}

void launch_segment_count(const int32_t* idx, int32_t T, int32_t N, int32_t cap,
                          int32_t tile_cap, int32_t* perm, int32_t* seg_ptr, int32_t* seg_id,
                          int32_t* meta, int4* tiles, hipStream_t stream) {
  int kbits = 0;
  while ((1 << kbits) < N + 2) ++kbits;
  hipLaunchKernelGGL(segment_count_kernel, dim3(1), dim3(kGroupTokens), 0, stream, idx, T, N,
                     cap, tile_cap, kbits, perm, seg_ptr, seg_id, meta, tiles);
}

void launch_segment_groups(const int32_t* idx, int32_t T, int32_t N, int32_t cap,
                           int32_t tile_cap, int32_t* perm, int32_t* seg_ptr, int32_t* seg_id,
                           int32_t* meta, int4* tiles, int32_t* table, hipStream_t stream) {
  const int G = (T + kGroupTokens - 1) / kGroupTokens;
  int kbits = 0;
  while ((1 << kbits) < N + 2) ++kbits;
  hipLaunchKernelGGL(seg_count_kernel, dim3(G), dim3(kGroupTokens), 0, stream, idx, T, N, kbits,
                     table);
  hipLaunchKernelGGL(seg_scan_kernel, dim3(1), dim3(kGroupTokens), 0, stream, table, G, T, N,
                     cap, tile_cap, seg_ptr, seg_id, meta, tiles);
  // (seg_scatter_kernel's grid is G: it finds row G, the key starts, by it)
  hipLaunchKernelGGL(seg_scatter_kernel, dim3(G), dim3(kGroupTokens), 0, stream, idx, T, N,
                     kbits, table, perm);
}

void launch_segment(const int32_t* idx, int32_t T, int32_t N, int32_t cap, int32_t tile_cap,
                    int32_t tbits, int32_t key_bits, int32_t* perm, int32_t* seg_ptr,
                    int32_t* seg_id, int32_t* meta, int4* tiles, hipStream_t stream) {
  if (T <= 64)
    hipLaunchKernelGGL(segment_small_kernel<64>, dim3(1), dim3(64), 0, stream, idx, T, N, cap,
                       tile_cap, tbits, perm, seg_ptr, seg_id, meta, tiles);
  else if (T <= 256)
    hipLaunchKernelGGL(segment_small_kernel<256>, dim3(1), dim3(256), 0, stream, idx, T, N, cap,
                       tile_cap, tbits, perm, seg_ptr, seg_id, meta, tiles);
  else if (N + 1 <= kCountKeys)
    launch_segment_count(idx, T, N, cap, tile_cap, perm, seg_ptr, seg_id, meta, tiles, stream);
  else if (T <= 1024)
    hipLaunchKernelGGL(segment_small_kernel<1024>, dim3(1), dim3(1024), 0, stream, idx, T, N,
                       cap, tile_cap, tbits, perm, seg_ptr, seg_id, meta, tiles);
  else
    hipLaunchKernelGGL(segment_kernel, dim3(1), dim3(kSegThreads), 0, stream, idx, T, N, cap,
                       tile_cap, tbits, key_bits, perm, seg_ptr, seg_id, meta, tiles);
}

void launch_zero(uint4* p, size_t n16, unsigned blocks, hipStream_t stream) {
  hipLaunchKernelGGL(zero_kernel, dim3(blocks), dim3(256), 0, stream, p, n16);
}

}  // namespace plora_impl
