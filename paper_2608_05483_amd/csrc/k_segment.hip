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
  __syncthreads();
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
  __syncthreads();
  int res = x - v + sh[w];
  *total = sh[kSegWaves];
  __syncthreads();
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
  __syncthreads();

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
  __syncthreads();
  for (int q = n_seg + t; q <= cap; q += NT) seg_ptr[q] = n_valid;
  for (int q = n_seg + t; q < cap; q += NT) seg_id[q] = -1;

  // tiles: a position starts one when it lies a multiple of kTT past its
  // segment's start; sidx + sflag - 1 is the segment of position p
  const int cur = sidx + (sflag ? 1 : 0) - 1;
  bool tflag = false;
  int start = 0, end = 0;
  if (p < n_valid) {
    start = start_s[cur];
    end = start_s[cur + 1];
    tflag = ((p - start) % kTT) == 0;
  }
  int n_tiles;
  const int tu = block_exscan<NW>(tflag ? 1 : 0, &n_tiles, scan_sh);
  if (tflag && tu < tile_cap) tiles[tu] = make_int4(key_p[p], p, min(kTT, end - p), cur);
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
  __syncthreads();

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
  __syncthreads();

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
    __syncthreads();
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
    __syncthreads();
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
    __syncthreads();
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
    __syncthreads();
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
  __syncthreads();
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

void launch_segment(const int32_t* idx, int32_t T, int32_t N, int32_t cap, int32_t tile_cap,
                    int32_t tbits, int32_t key_bits, int32_t* perm, int32_t* seg_ptr,
                    int32_t* seg_id, int32_t* meta, int4* tiles, hipStream_t stream) {
  if (T <= 64)
    hipLaunchKernelGGL(segment_small_kernel<64>, dim3(1), dim3(64), 0, stream, idx, T, N, cap,
                       tile_cap, tbits, perm, seg_ptr, seg_id, meta, tiles);
  else if (T <= 256)
    hipLaunchKernelGGL(segment_small_kernel<256>, dim3(1), dim3(256), 0, stream, idx, T, N, cap,
                       tile_cap, tbits, perm, seg_ptr, seg_id, meta, tiles);
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
