// plora.hip -- gfx950 kernels and the C ABI of the batched heterogeneous-
// adapter LoRA apply (declared in include/plora.h).
//
// What runs where:
//   plora_segment  one 1024-thread work group: LSD radix sort of packed
//                  (adapter id, token index) words in LDS, ballot-based stable
//                  ranking per wavefront, then segment and tile lists.
//   plora_shrink   one wavefront per (tile, part): split-K over h_in.  Each
//   plora_expand   part streams its rows of A_i (or columns of B_i) once with
//   plora_apply    128-bit loads; partial x A_i sums meet in the workspace.
//
// Work decomposition.  The token batch is grouped into segments (one per
// adapter, section VI-B of the paper: the per-adapter batch B_i) and each
// segment into tiles of at most PLORA_TILE_TOKENS tokens.  A tile is split
// into Q parts: part q owns rows [k0_q, k1_q) of A_i and column octets
// [o0_q, o1_q) of B_i, so every byte of an adapter is read by exactly one
// work group per tile -- the "adapter loads its matrices once per step"
// property of the cost model.  Work group b handles tile u = (b/8/Q)*8 + b%8,
// part q = (b/8) % Q: the Q parts of a tile share b % 8 and hence (with the
// round-robin assignment of work groups to the eight XCDs) one L2, where
// their partial sums meet.
//
// Fused apply.  Every part first computes its partial P_q = x_tile A_i[k0_q:
// k1_q, :], stores it to the workspace and bumps the tile's arrival counter;
// its B_i columns are already in flight.  It then waits for all Q partials,
// sums them in the fixed order q = 0..Q-1 and applies its B_i columns.  The
// wait is bounded: after spin_limit polls the work group recomputes all Q
// partials itself with the same code and order (bitwise the same v), so no
// schedule can deadlock.  The last of the Q parts to finish resets the
// tile's counters, leaving the workspace zeroed for the next call.
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <atomic>

#include "plora.h"

namespace {

constexpr int kTT = PLORA_TILE_TOKENS;   // tokens per tile
constexpr int kSegThreads = 1024;
constexpr int kSegWaves = kSegThreads / 64;
constexpr int kWave = 64;                // apply work group = one wavefront
constexpr int kTG = 4;                   // tokens per register group
constexpr int kCH = 8;                   // 16-byte chunks per lane per batch
constexpr int kMaxQ = 64;
constexpr int kDefaultSpin = 1 << 16;

std::atomic<int32_t> g_spin_limit{kDefaultSpin};

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

// ---------------------------------------------------------------------------
// plora_segment: stable grouping of tokens by adapter id
// ---------------------------------------------------------------------------

// Exclusive scan of one int per thread over the 1024-thread block.
__device__ int block_exscan(int v, int* total, int* sh /* [kSegWaves + 1] */) {
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

  // load and pack; count skipped tokens
  int my_none = 0, my_invalid = 0;
  for (int t = tid; t < T; t += kSegThreads) {
    int id = idx[t];
    uint32_t key;
    if (id >= 0 && id < N) {
      key = (uint32_t)id;
    } else {
      key = (uint32_t)N;
      if (id == -1) ++my_none; else ++my_invalid;
    }
    buf0[t] = (key << tbits) | (uint32_t)t;
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
    // count digits per wave
    for (int g = 0; g < chunk; g += 64) {
      const int e = e_begin + g + lane;
      const bool act = e < T;
      const uint32_t dig = act ? (buf0[e] >> shift) & (uint32_t)(nbuck - 1) : 0u;
      uint64_t peers = __ballot(act);
      for (int b = 0; b < dbits; ++b) {
        uint64_t m = __ballot((dig >> b) & 1u);
        peers &= ((dig >> b) & 1u) ? m : ~m;
      }
      if (act && (peers & below) == 0ull) cursor[w][dig] += __popcll(peers);
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
    for (int g = 0; g < chunk; g += 64) {
      const int e = e_begin + g + lane;
      const bool act = e < T;
      const uint32_t word = act ? buf0[e] : 0u;
      const uint32_t dig = (word >> shift) & (uint32_t)(nbuck - 1);
      uint64_t peers = __ballot(act);
      for (int b = 0; b < dbits; ++b) {
        uint64_t m = __ballot((dig >> b) & 1u);
        peers &= ((dig >> b) & 1u) ? m : ~m;
      }
      const int base = act ? cursor[w][dig] : 0;
      if (act) buf1[base + __popcll(peers & below)] = word;
      __builtin_amdgcn_wave_barrier();
      if (act && (peers & below) == 0ull) cursor[w][dig] = base + __popcll(peers);
      __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    uint32_t* tmp = buf0; buf0 = buf1; buf1 = tmp;
  }

  const int n_none = n_none_sh, n_invalid = n_invalid_sh;
  const int n_valid = T - n_none - n_invalid;

  // blocked positions per thread
  const int per = (T + kSegThreads - 1) / kSegThreads;
  const int p_begin = tid * per;
  int nflags = 0;
  for (int i = 0; i < per; ++i) {
    int p = p_begin + i;
    if (p < n_valid) {
      uint32_t k = buf0[p] >> tbits;
      if (p == 0 || (buf0[p - 1] >> tbits) != k) ++nflags;
    }
  }
  int n_seg;
  int sbase = block_exscan(nflags, &n_seg, scan_sh);
  // buf1 now holds seg starts (cap + 1 <= T + 1 entries)
  int32_t* seg_lds_ptr = reinterpret_cast<int32_t*>(buf1);
  {
    int s = sbase;
    for (int i = 0; i < per; ++i) {
      int p = p_begin + i;
      if (p < T) perm[p] = p < n_valid ? (int32_t)(buf0[p] & tmask) : -1;
      if (p < n_valid) {
        uint32_t k = buf0[p] >> tbits;
        if (p == 0 || (buf0[p - 1] >> tbits) != k) {
          if (s < cap) {
            seg_ptr[s] = p;
            seg_id[s] = (int32_t)k;
            seg_lds_ptr[s] = p;
          }
          ++s;
        }
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
  // segment sbase itself.
  int ntf = 0;
  {
    int cur = sbase - 1;
    for (int i = 0; i < per; ++i) {
      int p = p_begin + i;
      if (p < n_valid) {
        if (cur + 1 < n_seg && seg_lds_ptr[cur + 1] == p) ++cur;
        if (((p - seg_lds_ptr[cur]) % kTT) == 0) ++ntf;
      }
    }
  }
  int cur = sbase - 1;
  int n_tiles;
  int tbase = block_exscan(ntf, &n_tiles, scan_sh);
  {
    int tu = tbase;
    for (int i = 0; i < per; ++i) {
      int p = p_begin + i;
      if (p < n_valid) {
        if (cur + 1 < n_seg && seg_lds_ptr[cur + 1] == p) ++cur;
        const int start = seg_lds_ptr[cur], end = seg_lds_ptr[cur + 1];
        if (((p - start) % kTT) == 0) {
          const int len = min(kTT, end - p);
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

// ---------------------------------------------------------------------------
// apply kernels: shared pieces
// ---------------------------------------------------------------------------

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
  const int64_t* a_off;
  const int64_t* b_off;
  const int32_t* ranks;
  const float* scales;
  const int32_t* perm;
  const int4* tiles;
  int32_t* arrive;     // workspace counters [tile_cap]
  int32_t* consume;
  float* partial;      // workspace [Q][T][max_rank]
  unsigned long long* stats;
  int32_t T, N, h_in, h_out, max_rank, tile_cap, Q, rows_max, spin_limit;
};

struct Tile {
  int a, p0, L, u, q;
  int r;
  const uint16_t* Ai;
  const uint16_t* Bi;
  float s;
};

// Decode work group b into its tile and part and validate the adapter.
// Returns false when the group has nothing to do (padding, skipped adapter);
// the decision is the same for every part of a tile.
__device__ __forceinline__ bool load_tile(const ApplyArgs& g, Tile& t) {
  const int b = blockIdx.x;
  const int i = b >> 3;
  t.u = (i / g.Q) * 8 + (b & 7);
  t.q = i % g.Q;
  if (t.u >= g.tile_cap) return false;
  const int4 ti = g.tiles[t.u];
  t.a = ti.x; t.p0 = ti.y; t.L = ti.z;
  if (t.a < 0 || t.a >= g.N || t.L <= 0 || t.L > kTT || t.p0 < 0 || t.p0 + t.L > g.T)
    return false;
  t.r = g.ranks[t.a];
  if (t.r <= 0 || t.r > g.max_rank || (t.r & 7)) return false;
  const int64_t ao = g.a_off[t.a], bo = g.b_off[t.a];
  if (ao < 0 || (ao & 7) || ao + (int64_t)g.h_in * t.r > g.a_len) return false;
  if (bo < 0 || (bo & 7) || bo + (int64_t)g.h_out * t.r > g.b_len) return false;
  t.Ai = g.A + ao;
  t.Bi = g.B + bo;
  t.s = g.scales[t.a];
  return true;
}

// LDS carve-up of an apply work group.
struct Smem {
  int* tok;        // [kTT]
  uint16_t* xs;    // [rows_max][kTT] bf16, token fastest
  float* red;      // [kTG * 8][kWave]
  float* vs;       // [max_rank][kTT]
  int* flag;       // [4]
};

__device__ __forceinline__ Smem carve(void* base, int rows_max, int max_rank) {
  char* p = reinterpret_cast<char*>(base);
  Smem s;
  s.tok = reinterpret_cast<int*>(p);              p += kTT * sizeof(int);
  s.flag = reinterpret_cast<int*>(p);             p += 4 * sizeof(int);
  s.red = reinterpret_cast<float*>(p);            p += kTG * 8 * kWave * sizeof(float);
  s.vs = reinterpret_cast<float*>(p);             p += (size_t)max_rank * kTT * sizeof(float);
  s.xs = reinterpret_cast<uint16_t*>(p);
  (void)rows_max;
  return s;
}

__host__ __device__ constexpr size_t smem_bytes(int rows_max, int max_rank) {
  return kTT * sizeof(int) + 4 * sizeof(int) + kTG * 8 * kWave * sizeof(float) +
         (size_t)max_rank * kTT * sizeof(float) + (size_t)rows_max * kTT * sizeof(uint16_t);
}

__device__ __forceinline__ void part_rows(int h_in, int Q, int q, int& k0, int& k1) {
  const int n8 = h_in >> 3;
  k0 = 8 * (int)(((int64_t)q * n8) / Q);
  k1 = 8 * (int)(((int64_t)(q + 1) * n8) / Q);
}

__device__ __forceinline__ void part_octs(int h_out, int Q, int q, int& o0, int& o1) {
  const int n8 = h_out >> 3;
  o0 = (int)(((int64_t)q * n8) / Q);
  o1 = (int)(((int64_t)(q + 1) * n8) / Q);
}

// Token rows of the tile into LDS.
__device__ __forceinline__ void load_tokens(const ApplyArgs& g, const Tile& t, int* tok) {
  const int lane = threadIdx.x;
  if (lane < t.L) {
    int tk = g.perm[t.p0 + lane];
    tok[lane] = (tk >= 0 && tk < g.T) ? tk : -1;
  }
  __syncthreads();
}

// Stage x[tok_l, k0:k1) for l < L into xs[row][l], bf16.  Invalid token rows
// (never produced by plora_segment) read as zero.
__device__ void stage_x(const ApplyArgs& g, const Tile& t, const int* tok, int k0,
                        int nrows, uint16_t* xs) {
  const int lane = threadIdx.x;
  const int n8 = nrows >> 3;
  const int total = t.L * n8;
  for (int c = lane; c < total; c += kWave) {
    const int l = c / n8, kc = c - l * n8;
    const int tk = tok[l];
    uint4 v = make_uint4(0, 0, 0, 0);
    if (tk >= 0) v = ldg16(g.x + (int64_t)tk * g.ldx + k0 + kc * 8);
    uint16_t* d = xs + (kc * 8) * kTT + l;
    d[0 * kTT] = (uint16_t)(v.x & 0xffffu); d[1 * kTT] = (uint16_t)(v.x >> 16);
    d[2 * kTT] = (uint16_t)(v.y & 0xffffu); d[3 * kTT] = (uint16_t)(v.y >> 16);
    d[4 * kTT] = (uint16_t)(v.z & 0xffffu); d[5 * kTT] = (uint16_t)(v.z >> 16);
    d[6 * kTT] = (uint16_t)(v.w & 0xffffu); d[7 * kTT] = (uint16_t)(v.w >> 16);
  }
  __syncthreads();
}

// The shrink of one part: for each token group, acc[tt][e] over this lane's
// rows, then a fixed-order reduction across the lanes that share a column
// octet.  Calls sink(l, c, value) for every l < L, c < r.
template <class Sink>
__device__ void shrink_part(const ApplyArgs& g, const Tile& t, int q, const Smem& sm,
                            Sink sink) {
  const int lane = threadIdx.x;
  int k0, k1;
  part_rows(g.h_in, g.Q, q, k0, k1);
  const int nrows = k1 - k0;
  const int r = t.r, r_oct = r >> 3;
  const int RS = kWave / r_oct;
  const int oct = lane % r_oct, rs = lane / r_oct;
  const bool act = rs < RS;
  const int nj = (act && nrows > rs) ? (nrows - rs + RS - 1) / RS : 0;

  stage_x(g, t, sm.tok, k0, nrows, sm.xs);

  const uint16_t* abase = t.Ai + (int64_t)(k0 + rs) * r + oct * 8;
  const int64_t astep = (int64_t)RS * r;

  for (int g0 = 0; g0 < t.L; g0 += kTG) {
    float acc[kTG][8];
#pragma unroll
    for (int tt = 0; tt < kTG; ++tt)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[tt][e] = 0.f;

    for (int jb = 0; jb < nj; jb += kCH) {
      uint4 a[kCH];
#pragma unroll
      for (int j = 0; j < kCH; ++j)
        a[j] = (jb + j < nj) ? ldg16(abase + (jb + j) * astep) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int j = 0; j < kCH; ++j) {
        if (jb + j < nj) {
          const int row = rs + (jb + j) * RS;
          const uint2 xv = *reinterpret_cast<const uint2*>(sm.xs + row * kTT + g0);
          float xf[4] = {bf_lo(xv.x), bf_hi(xv.x), bf_lo(xv.y), bf_hi(xv.y)};
          float af[8];
          unpack8(a[j], af);
#pragma unroll
          for (int tt = 0; tt < kTG; ++tt)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[tt][e] = fmaf(xf[tt], af[e], acc[tt][e]);
        }
      }
    }
    // cross-lane reduction through LDS: red[(tt*8+e)][lane]
#pragma unroll
    for (int tt = 0; tt < kTG; ++tt)
#pragma unroll
      for (int e = 0; e < 8; ++e) sm.red[(tt * 8 + e) * kWave + lane] = acc[tt][e];
    __syncthreads();
    const int gl = min(kTG, t.L - g0);
    const int nout = gl * r;
    for (int o = lane; o < nout; o += kWave) {
      const int tt = o / r, c = o - tt * r;
      const int oc = c >> 3, e = c & 7;
      const float* src = sm.red + (tt * 8 + e) * kWave + oc;
      float s = 0.f;
      for (int k = 0; k < RS; ++k) s += src[k * r_oct];
      sink(g0 + tt, c, s);
    }
    __syncthreads();
  }
}

// The expand of one part for every token of the tile: columns octets
// [o0, o1) of y, d = v B_i[:, cols], y = bf16(y + s d).
__device__ void expand_part(const ApplyArgs& g, const Tile& t, int q, const Smem& sm,
                            const uint4* bpre, int npre) {
  const int lane = threadIdx.x;
  int o0, o1;
  part_octs(g.h_out, g.Q, q, o0, o1);
  const int n_co = o1 - o0;
  const int r = t.r;
  for (int cb = 0; cb * kWave < n_co; ++cb) {
    const int cw = min(kWave, n_co - cb * kWave);
    const int RSB = kWave / cw;
    const int col = lane % cw, rsb = lane / cw;
    const bool act = rsb < RSB;
    const int njb = (act && r > rsb) ? (r - rsb + RSB - 1) / RSB : 0;
    const uint16_t* bbase = t.Bi + (int64_t)rsb * g.h_out + (int64_t)(o0 + cb * kWave + col) * 8;
    const int64_t bstep = (int64_t)RSB * g.h_out;
    for (int g0 = 0; g0 < t.L; g0 += kTG) {
      float d[kTG][8];
#pragma unroll
      for (int tt = 0; tt < kTG; ++tt)
#pragma unroll
        for (int e = 0; e < 8; ++e) d[tt][e] = 0.f;
      for (int jb = 0; jb < njb; jb += kCH) {
        uint4 b[kCH];
        const bool use_pre = (cb == 0 && g0 == 0 && jb == 0);
#pragma unroll
        for (int j = 0; j < kCH; ++j) {
          if (use_pre && j < npre) b[j] = bpre[j];
          else b[j] = (jb + j < njb) ? ldg16(bbase + (jb + j) * bstep) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < kCH; ++j) {
          if (jb + j < njb) {
            const int c = rsb + (jb + j) * RSB;
            const float4 vv = *reinterpret_cast<const float4*>(sm.vs + c * kTT + g0);
            const float vf[4] = {vv.x, vv.y, vv.z, vv.w};
            float bf[8];
            unpack8(b[j], bf);
#pragma unroll
            for (int tt = 0; tt < kTG; ++tt)
#pragma unroll
              for (int e = 0; e < 8; ++e) d[tt][e] = fmaf(vf[tt], bf[e], d[tt][e]);
          }
        }
      }
#pragma unroll
      for (int tt = 0; tt < kTG; ++tt)
#pragma unroll
        for (int e = 0; e < 8; ++e) sm.red[(tt * 8 + e) * kWave + lane] = d[tt][e];
      __syncthreads();
      const int gl = min(kTG, t.L - g0);
      const int nout = gl * cw;
      for (int o = lane; o < nout; o += kWave) {
        const int tt = o / cw, cc = o - tt * cw;
        const int tk = sm.tok[g0 + tt];
        if (tk < 0) continue;
        float acc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float* src = sm.red + (tt * 8 + e) * kWave + cc;
          float s = 0.f;
          for (int k = 0; k < RSB; ++k) s += src[k * cw];
          acc[e] = s;
        }
        uint16_t* yp = g.y + (int64_t)tk * g.ldy + (int64_t)(o0 + cb * kWave + cc) * 8;
        const uint4 yv = ldg16(yp);
        float yf[8];
        unpack8(yv, yf);
        uint32_t ob[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) ob[e] = to_bf16(fmaf(t.s, acc[e], yf[e]));
        uint4 out;
        out.x = ob[0] | (ob[1] << 16);
        out.y = ob[2] | (ob[3] << 16);
        out.z = ob[4] | (ob[5] << 16);
        out.w = ob[6] | (ob[7] << 16);
        *reinterpret_cast<uint4*>(yp) = out;
      }
      __syncthreads();
    }
  }
}

// Issue the first batch of this part's B_i loads (rows of the first column
// batch) so they are in flight during the shrink.
__device__ __forceinline__ int prefetch_b(const ApplyArgs& g, const Tile& t, int q,
                                          uint4* bpre) {
  const int lane = threadIdx.x;
  int o0, o1;
  part_octs(g.h_out, g.Q, q, o0, o1);
  const int n_co = o1 - o0;
  if (n_co <= 0) return 0;
  const int cw = min(kWave, n_co);
  const int RSB = kWave / cw;
  const int col = lane % cw, rsb = lane / cw;
  const bool act = rsb < RSB;
  const int njb = (act && t.r > rsb) ? (t.r - rsb + RSB - 1) / RSB : 0;
  const uint16_t* bbase = t.Bi + (int64_t)rsb * g.h_out + (int64_t)(o0 + col) * 8;
  const int64_t bstep = (int64_t)RSB * g.h_out;
#pragma unroll
  for (int j = 0; j < kCH; ++j)
    bpre[j] = (j < njb) ? ldg16(bbase + j * bstep) : make_uint4(0, 0, 0, 0);
  return kCH;
}

// ---------------------------------------------------------------------------
// kernels
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kWave) void shrink_kernel(ApplyArgs g) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  Tile t;
  if (!load_tile(g, t)) return;
  const Smem sm = carve(apply_lds, g.rows_max, g.max_rank);
  load_tokens(g, t, sm.tok);
  float* part = g.partial + (int64_t)t.q * g.T * g.max_rank;
  shrink_part(g, t, t.q, sm, [&](int l, int c, float val) {
    part[(int64_t)(t.p0 + l) * g.max_rank + c] = val;
  });
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const int old = __hip_atomic_fetch_add(&g.arrive[t.u], 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
    sm.flag[0] = (old == g.Q - 1);
  }
  __syncthreads();
  if (!sm.flag[0]) return;
  // last part to arrive: v = sum of the Q partials in order q = 0..Q-1
  __threadfence();
  const int nout = t.L * t.r;
  for (int o = threadIdx.x; o < nout; o += kWave) {
    const int l = o / t.r, c = o - l * t.r;
    const int64_t row = (int64_t)(t.p0 + l) * g.max_rank + c;
    float s = __hip_atomic_load(&g.partial[row], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (int qq = 1; qq < g.Q; ++qq)
      s += __hip_atomic_load(&g.partial[(int64_t)qq * g.T * g.max_rank + row],
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int tk = sm.tok[l];
    if (tk >= 0) g.v[(int64_t)tk * g.ldv + c] = s;
  }
  if (threadIdx.x == 0)
    __hip_atomic_store(&g.arrive[t.u], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(kWave) void expand_kernel(ApplyArgs g) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  Tile t;
  if (!load_tile(g, t)) return;
  const Smem sm = carve(apply_lds, g.rows_max, g.max_rank);
  load_tokens(g, t, sm.tok);
  uint4 bpre[kCH];
  const int npre = prefetch_b(g, t, t.q, bpre);
  const int nout = t.L * t.r;
  for (int o = threadIdx.x; o < nout; o += kWave) {
    const int l = o / t.r, c = o - l * t.r;
    const int tk = sm.tok[l];
    sm.vs[c * kTT + l] = tk >= 0 ? g.v[(int64_t)tk * g.ldv + c] : 0.f;
  }
  // zero the unused token slots of the last register group
  for (int o = threadIdx.x; o < t.r * kTT; o += kWave) {
    const int l = o % kTT;
    if (l >= t.L) sm.vs[o] = 0.f;
  }
  __syncthreads();
  expand_part(g, t, t.q, sm, bpre, npre);
}

__global__ __launch_bounds__(kWave) void apply_kernel(ApplyArgs g) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  Tile t;
  if (!load_tile(g, t)) return;
  const Smem sm = carve(apply_lds, g.rows_max, g.max_rank);
  load_tokens(g, t, sm.tok);
  uint4 bpre[kCH];
  const int npre = prefetch_b(g, t, t.q, bpre);

  // 1. this part's partial x A_i, published to the workspace
  float* part = g.partial + (int64_t)t.q * g.T * g.max_rank;
  shrink_part(g, t, t.q, sm, [&](int l, int c, float val) {
    part[(int64_t)(t.p0 + l) * g.max_rank + c] = val;
  });
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(&g.arrive[t.u], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // 2. wait for the other parts, bounded
    int polls = 0;
    int seen = __hip_atomic_load(&g.arrive[t.u], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    while (seen < g.Q && polls < g.spin_limit) {
      __builtin_amdgcn_s_sleep(1);
      seen = __hip_atomic_load(&g.arrive[t.u], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      ++polls;
    }
    sm.flag[0] = (seen >= g.Q);
  }
  __syncthreads();
  const bool ready = sm.flag[0] != 0;
  __threadfence();

  // 3. v = sum of the Q partials, q ascending
  for (int o = threadIdx.x; o < t.r * kTT; o += kWave) sm.vs[o] = 0.f;
  __syncthreads();
  if (ready) {
    const int nout = t.L * t.r;
    for (int o = threadIdx.x; o < nout; o += kWave) {
      const int l = o / t.r, c = o - l * t.r;
      const int64_t row = (int64_t)(t.p0 + l) * g.max_rank + c;
      float s = __hip_atomic_load(&g.partial[row], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      for (int qq = 1; qq < g.Q; ++qq)
        s += __hip_atomic_load(&g.partial[(int64_t)qq * g.T * g.max_rank + row],
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      sm.vs[c * kTT + l] = s;
    }
  } else {
    // bounded wait expired: recompute every part locally, same order
    if (threadIdx.x == 0) atomicAdd(g.stats, 1ull);
    for (int qq = 0; qq < g.Q; ++qq) {
      shrink_part(g, t, qq, sm, [&](int l, int c, float val) {
        float* dst = sm.vs + c * kTT + l;
        *dst = (qq == 0) ? val : (*dst + val);
      });
    }
  }
  __syncthreads();

  // 4. this part's columns of y
  expand_part(g, t, t.q, sm, bpre, npre);

  // 5. the last part out resets the tile's counters
  __syncthreads();
  if (threadIdx.x == 0) {
    const int old = __hip_atomic_fetch_add(&g.consume[t.u], 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
    if (old == g.Q - 1) {
      __hip_atomic_store(&g.arrive[t.u], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&g.consume[t.u], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

__global__ void zero_kernel(uint4* p, size_t n16) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n16;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline int ceil_log2(int64_t v) {
  int b = 0;
  while ((int64_t(1) << b) < v) ++b;
  return b;
}

// Parts per tile: split the adapter into pieces of at least ~8 KB, at most
// 32 pieces, each part holding at least one row octet of A_i and one column
// octet of B_i, and at most 512 rows of A_i (the LDS x tile).
int parts_for(int h_in, int h_out, int max_rank) {
  const int64_t bytes = 2LL * (h_in + h_out) * max_rank;
  int q = 1;
  while (q < 32 && bytes / (2 * q) >= 8192) q *= 2;
  while (q < kMaxQ && (h_in / 8 + q - 1) / q > 64) q *= 2;
  q = std::min(q, std::max(1, std::min(h_in / 8, h_out / 8)));
  return q;
}

int rows_max_for(int h_in, int Q) { return 8 * ((h_in / 8 + Q - 1) / Q); }

struct WsLayout {
  size_t stats, arrive, consume, partial, total;
};

inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

WsLayout ws_layout(int32_t T, int32_t N, int h_in, int h_out, int max_rank) {
  WsLayout L;
  const int tile_cap = plora_tile_capacity(T, N);
  const int Q = parts_for(h_in, h_out, max_rank);
  L.stats = 0;
  L.arrive = 256;
  L.consume = align256(L.arrive + sizeof(int32_t) * (size_t)std::max(tile_cap, 1));
  L.partial = align256(L.consume + sizeof(int32_t) * (size_t)std::max(tile_cap, 1));
  L.total = align256(L.partial + sizeof(float) * (size_t)Q * std::max(T, 1) * std::max(max_rank, 8));
  return L;
}

plora_status check_adapters_host(const plora_adapters* ad) {
  if (!ad) return PLORA_ERR_INVALID_ARG;
  if (ad->n_adapters < 0 || ad->h_in <= 0 || ad->h_out <= 0 || ad->max_rank < 0 ||
      ad->a_len < 0 || ad->b_len < 0)
    return PLORA_ERR_INVALID_ARG;
  if ((ad->h_in & 7) || (ad->h_out & 7)) return PLORA_ERR_UNSUPPORTED;
  if (ad->max_rank == 0 || (ad->max_rank & 7) || ad->max_rank > PLORA_MAX_RANK)
    return PLORA_ERR_UNSUPPORTED;
  if (ad->n_adapters > 0 &&
      (!ad->A || !ad->B || !ad->a_off || !ad->b_off || !ad->ranks || !ad->scales))
    return PLORA_ERR_INVALID_ARG;
  if (!aligned16(ad->A) || !aligned16(ad->B) || !aligned16(ad->a_off) ||
      !aligned16(ad->b_off) || !aligned16(ad->ranks) || !aligned16(ad->scales))
    return PLORA_ERR_UNSUPPORTED;
  return PLORA_OK;
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

plora_status launch_status() {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return PLORA_OK;
  g_last_hip_error.store((int32_t)e);
  return PLORA_ERR_HIP;
}

plora_status prepare(const plora_adapters* ad, const plora_segments* seg, void* ws,
                     size_t ws_bytes, bool need_ws, ApplyArgs& g) {
  plora_status st = check_adapters_host(ad);
  if (st != PLORA_OK) return st;
  st = check_segments_host(seg, ad->n_adapters);
  if (st != PLORA_OK) return st;
  memset(&g, 0, sizeof g);
  g.A = ad->A; g.B = ad->B; g.a_len = ad->a_len; g.b_len = ad->b_len;
  g.a_off = ad->a_off; g.b_off = ad->b_off; g.ranks = ad->ranks; g.scales = ad->scales;
  g.perm = seg->perm;
  g.tiles = reinterpret_cast<const int4*>(seg->tiles);
  g.T = seg->T; g.N = ad->n_adapters; g.h_in = ad->h_in; g.h_out = ad->h_out;
  g.max_rank = ad->max_rank; g.tile_cap = seg->tile_cap;
  g.Q = parts_for(ad->h_in, ad->h_out, ad->max_rank);
  g.rows_max = rows_max_for(ad->h_in, g.Q);
  g.spin_limit = g_spin_limit.load();
  if (need_ws) {
    if (!ws) return PLORA_ERR_INVALID_ARG;
    if (!aligned16(ws)) return PLORA_ERR_UNSUPPORTED;
    const WsLayout L = ws_layout(seg->T, ad->n_adapters, ad->h_in, ad->h_out, ad->max_rank);
    if (ws_bytes < L.total) return PLORA_ERR_WORKSPACE_TOO_SMALL;
    char* base = reinterpret_cast<char*>(ws);
    g.stats = reinterpret_cast<unsigned long long*>(base + L.stats);
    g.arrive = reinterpret_cast<int32_t*>(base + L.arrive);
    g.consume = reinterpret_cast<int32_t*>(base + L.consume);
    g.partial = reinterpret_cast<float*>(base + L.partial);
  }
  return PLORA_OK;
}

unsigned grid_for(const ApplyArgs& g) {
  const int groups = (g.tile_cap + 7) / 8;
  return (unsigned)groups * 8u * (unsigned)g.Q;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------

extern "C" {

int32_t plora_tile_capacity(int32_t T, int32_t n_adapters) {
  if (T <= 0) return 0;
  const int32_t cap = std::min(T, std::max(n_adapters, 0));
  return std::min(T, cap + T / PLORA_TILE_TOKENS);
}

size_t plora_workspace_bytes(int32_t T, const plora_adapters* ad) {
  if (!ad || T < 0) return 0;
  return ws_layout(T, ad->n_adapters, std::max(ad->h_in, 8), std::max(ad->h_out, 8),
                   std::max(ad->max_rank, 8)).total;
}

plora_status plora_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!ws) return PLORA_ERR_INVALID_ARG;
  if (!aligned16(ws) || (ws_bytes & 15)) return PLORA_ERR_UNSUPPORTED;
  const size_t n16 = ws_bytes / 16;
  if (n16 == 0) return PLORA_OK;
  const unsigned blocks = (unsigned)std::min<size_t>((n16 + 255) / 256, 4096);
  clear_stale_error();
  hipLaunchKernelGGL(zero_kernel, dim3(blocks), dim3(256), 0, stream,
                     reinterpret_cast<uint4*>(ws), n16);
  return launch_status();
}

plora_status plora_segment(const int32_t* idx, const plora_segments* seg, int32_t n_adapters,
                           void* ws, size_t ws_bytes, hipStream_t stream) {
  (void)ws; (void)ws_bytes;
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
  hipLaunchKernelGGL(segment_kernel, dim3(1), dim3(kSegThreads), 0, stream, idx, T,
                     n_adapters, seg->cap, seg->tile_cap, tbits, key_bits, seg->perm,
                     seg->seg_ptr, seg->seg_id, seg->meta,
                     reinterpret_cast<int4*>(seg->tiles));
  return launch_status();
}

plora_status plora_shrink(const uint16_t* x, int64_t ldx, const plora_adapters* ad,
                          const plora_segments* seg, float* v, int64_t ldv, void* ws,
                          size_t ws_bytes, hipStream_t stream) {
  ApplyArgs g;
  plora_status st = prepare(ad, seg, ws, ws_bytes, true, g);
  if (st != PLORA_OK) return st;
  if (seg->T == 0) return PLORA_OK;
  if (!x || !v) return PLORA_ERR_INVALID_ARG;
  if (ldx < ad->h_in || ldv < ad->max_rank) return PLORA_ERR_INVALID_ARG;
  if ((ldx & 7) || (ldv & 3) || !aligned16(x) || !aligned16(v)) return PLORA_ERR_UNSUPPORTED;
  g.x = x; g.ldx = ldx; g.v = v; g.ldv = ldv;
  clear_stale_error();
  hipLaunchKernelGGL(shrink_kernel, dim3(grid_for(g)), dim3(kWave),
                     smem_bytes(g.rows_max, g.max_rank), stream, g);
  return launch_status();
}

plora_status plora_expand(const float* v, int64_t ldv, const plora_adapters* ad,
                          const plora_segments* seg, uint16_t* y, int64_t ldy, void* ws,
                          size_t ws_bytes, hipStream_t stream) {
  ApplyArgs g;
  plora_status st = prepare(ad, seg, ws, ws_bytes, false, g);
  if (st != PLORA_OK) return st;
  if (seg->T == 0) return PLORA_OK;
  if (!v || !y) return PLORA_ERR_INVALID_ARG;
  if (ldy < ad->h_out || ldv < ad->max_rank) return PLORA_ERR_INVALID_ARG;
  if ((ldy & 7) || (ldv & 3) || !aligned16(y) || !aligned16(v)) return PLORA_ERR_UNSUPPORTED;
  g.v = const_cast<float*>(v); g.ldv = ldv; g.y = y; g.ldy = ldy;
  clear_stale_error();
  hipLaunchKernelGGL(expand_kernel, dim3(grid_for(g)), dim3(kWave),
                     smem_bytes(g.rows_max, g.max_rank), stream, g);
  return launch_status();
}

plora_status plora_apply(const uint16_t* x, int64_t ldx, const plora_adapters* ad,
                         const plora_segments* seg, uint16_t* y, int64_t ldy, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  ApplyArgs g;
  plora_status st = prepare(ad, seg, ws, ws_bytes, true, g);
  if (st != PLORA_OK) return st;
  if (seg->T == 0) return PLORA_OK;
  if (!x || !y) return PLORA_ERR_INVALID_ARG;
  if (ldx < ad->h_in || ldy < ad->h_out) return PLORA_ERR_INVALID_ARG;
  if ((ldx & 7) || (ldy & 7) || !aligned16(x) || !aligned16(y)) return PLORA_ERR_UNSUPPORTED;
  g.x = x; g.ldx = ldx; g.y = y; g.ldy = ldy;
  clear_stale_error();
  hipLaunchKernelGGL(apply_kernel, dim3(grid_for(g)), dim3(kWave),
                     smem_bytes(g.rows_max, g.max_rank), stream, g);
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
      bool ok = r >= 0 && r <= ad->max_rank && (r & 7) == 0;
      if (ok && r > 0) {
        ok = ao[i] >= 0 && (ao[i] & 7) == 0 && ao[i] + (int64_t)ad->h_in * r <= ad->a_len &&
             bo[i] >= 0 && (bo[i] & 7) == 0 && bo[i] + (int64_t)ad->h_out * r <= ad->b_len;
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

void plora_debug_set_spin_limit(int32_t polls) {
  g_spin_limit.store(polls > 0 ? polls : kDefaultSpin);
}

int32_t plora_debug_last_hip_error(void) { return g_last_hip_error.load(); }

int64_t plora_debug_fallbacks(const void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!ws || ws_bytes < 256) return -1;
  unsigned long long v = 0;
  if (hipMemcpyAsync(&v, ws, sizeof v, hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return -1;
  return (int64_t)v;
}

}  // extern "C"
