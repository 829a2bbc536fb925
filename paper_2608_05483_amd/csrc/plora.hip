// plora.hip -- gfx950 kernels and the C ABI of the batched heterogeneous-
// adapter LoRA apply (declared in include/plora.h).
//
// What runs where:
//   plora_segment  one 1024-thread work group: LSD radix sort of packed
//                  (adapter id, token index) words in LDS, ballot-based stable
//                  ranking per wavefront, then segment and tile lists.
//   plora_shrink   one work group per tile (PLORA_TILE_TOKENS tokens of one
//   plora_expand   adapter, section VI-B's per-adapter batch B_i split into
//   plora_apply    tiles), streaming that adapter's A_i and B_i once with
//                  128-bit loads; details above the apply kernels below.
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
constexpr int kTG = 4;                   // tokens per register group
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
// apply kernels: one work group per tile
// ---------------------------------------------------------------------------
//
// A work group of kNT threads owns one tile (<= PLORA_TILE_TOKENS tokens of
// one adapter) and reads every byte of that adapter's A_i and B_i once.
//
// Shrink.  A_i is a contiguous block of h_in x r bf16 values, i.e. h_in * r/8
// 16-byte chunks; thread tid loads chunks tid, tid + kNT, ... so the work
// group streams the block front to back with 128-bit loads.  Because kNT is a
// multiple of r/8, each thread always sees the same column octet
// oct = tid % (r/8) and a set of rows.  For a group of kTG tokens it keeps
// acc[token][8 columns] over its rows, then the partial sums of the threads
// that share a column octet are combined: inside the wavefront by a butterfly
// reduce-scatter over the lane bits that select the row (each step halves the
// values a lane holds), across wavefronts through LDS in wave order.
//
// Expand.  B_i is r x h_out; thread (wave w, lane l) owns column octet
// w * CPW + l % CPW (plus multiples of kW * CPW) and rows l / CPW + j * RSB,
// with RSB row slots per octet chosen so that the whole work group covers
// h_out.  Row-slot partial sums are combined by a butterfly all-reduce inside
// the wavefront and row slot 0 writes y with one 16-byte read-modify-write
// per token and octet.
//
// Every reduction has a fixed order, so results are bitwise reproducible,
// and the split calls (plora_shrink then plora_expand) run the very same
// code on the very same values as the fused call.

constexpr int kNT = 512;             // threads per tile work group
constexpr int kW = kNT / 64;         // wavefronts per work group

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
  int32_t T, N, h_in, h_out, max_rank, tile_cap;
  int32_t rsb_log2;    // expand row slots per column octet (log2)
};

struct Tile {
  int a, p0, L;
  int r;
  const uint16_t* Ai;
  const uint16_t* Bi;
  float s;
};

// Read and validate work group's tile.  Returns false (for the whole work
// group) for padding entries and for adapters the kernels must skip.
__device__ __forceinline__ bool load_tile(const ApplyArgs& g, Tile& t) {
  const int u = blockIdx.x;
  if (u >= g.tile_cap) return false;
  const int4 ti = g.tiles[u];
  t.a = ti.x; t.p0 = ti.y; t.L = ti.z;
  if (t.a < 0 || t.a >= g.N || t.L <= 0 || t.L > kTT || t.p0 < 0 || t.p0 + t.L > g.T)
    return false;
  t.r = g.ranks[t.a];
  // ranks 8, 16, 32, 64, 128 (up to max_rank); anything else is skipped
  if (t.r < 8 || t.r > g.max_rank || (t.r & (t.r - 1))) return false;
  const int64_t ao = g.a_off[t.a], bo = g.b_off[t.a];
  if (ao < 0 || (ao & 7) || ao + (int64_t)g.h_in * t.r > g.a_len) return false;
  if (bo < 0 || (bo & 7) || bo + (int64_t)g.h_out * t.r > g.b_len) return false;
  t.Ai = g.A + ao;
  t.Bi = g.B + bo;
  t.s = g.scales[t.a];
  return true;
}

// LDS of a tile work group.  red (the cross-wavefront partial sums) aliases
// the head of xs: it is only written after every wavefront has finished
// reading xs for the current token group.
struct Smem {
  int* tok;        // [kTT] token index of each tile row, -1 if unusable
  float* vs;       // [max_rank][kTT] v of the tile, column-major
  uint16_t* xs;    // [h_in][kTG] bf16 x of the current token group
  float* red;      // [kW][kTG][max_rank]
};

__host__ __device__ constexpr size_t smem_bytes(int h_in, int max_rank) {
  return kTT * sizeof(int) + (size_t)max_rank * kTT * sizeof(float) +
         ((size_t)h_in * kTG * sizeof(uint16_t) > (size_t)kW * kTG * max_rank * sizeof(float)
              ? (size_t)h_in * kTG * sizeof(uint16_t)
              : (size_t)kW * kTG * max_rank * sizeof(float));
}

__device__ __forceinline__ Smem carve(void* base, int max_rank) {
  char* p = reinterpret_cast<char*>(base);
  Smem s;
  s.tok = reinterpret_cast<int*>(p);    p += kTT * sizeof(int);
  s.vs = reinterpret_cast<float*>(p);   p += (size_t)max_rank * kTT * sizeof(float);
  s.xs = reinterpret_cast<uint16_t*>(p);
  s.red = reinterpret_cast<float*>(p);
  return s;
}

__device__ __forceinline__ void load_tokens(const ApplyArgs& g, const Tile& t, int* tok) {
  if (threadIdx.x < kTT) {
    int tk = -1;
    if ((int)threadIdx.x < t.L) {
      tk = g.perm[t.p0 + threadIdx.x];
      if (tk < 0 || tk >= g.T) tk = -1;
    }
    tok[threadIdx.x] = tk;
  }
}

// x rows of tokens g0..g0+kTG-1 into xs[k][tt], zero for missing tokens.
__device__ void stage_x(const ApplyArgs& g, const int* tok, int g0, int L, uint16_t* xs) {
  const int n8 = g.h_in >> 3;
  const int total = kTG * n8;
  for (int c = threadIdx.x; c < total; c += kNT) {
    const int tt = c / n8, kc = c - tt * n8;
    const int l = g0 + tt;
    const int tk = l < L ? tok[l] : -1;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (tk >= 0) v = ldg16(g.x + (int64_t)tk * g.ldx + kc * 8);
    uint16_t* d = xs + (kc * 8) * kTG + tt;
    d[0 * kTG] = (uint16_t)(v.x & 0xffffu); d[1 * kTG] = (uint16_t)(v.x >> 16);
    d[2 * kTG] = (uint16_t)(v.y & 0xffffu); d[3 * kTG] = (uint16_t)(v.y >> 16);
    d[4 * kTG] = (uint16_t)(v.z & 0xffffu); d[5 * kTG] = (uint16_t)(v.z >> 16);
    d[6 * kTG] = (uint16_t)(v.w & 0xffffu); d[7 * kTG] = (uint16_t)(v.w >> 16);
  }
}

// One butterfly step over lane mask M on N values: the lane whose mask bit is
// set keeps the upper half, the other the lower half, each adding the half
// its partner sends.
template <int N, int M>
__device__ __forceinline__ void halve(float (&val)[kTG * 8], int lane) {
  const bool up = (lane & M) != 0;
#pragma unroll
  for (int i = 0; i < N / 2; ++i) {
    const float lo = val[i], hi = val[i + N / 2];
    const float send = up ? lo : hi;
    const float keep = up ? hi : lo;
    val[i] = keep + __shfl_xor(send, M, 64);
  }
}

// v[l][c] for the whole tile into sm.vs (c < r, l < L; zero elsewhere).
template <int R_OCT>
__device__ void shrink_tile(const ApplyArgs& g, const Tile& t, const Smem& sm) {
  constexpr int R = 8 * R_OCT;
  constexpr int RSW = 64 / R_OCT;          // row slots inside a wavefront
  constexpr int HALV = RSW >= 32 ? 5 : (RSW == 16 ? 4 : (RSW == 8 ? 3 : 2));
  constexpr int VL = (kTG * 8) >> HALV;    // values a lane keeps
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int oct = tid % R_OCT;
  const int n_chunks = g.h_in * R_OCT;     // 16-byte chunks of A_i
  const int nj = tid < n_chunks ? (n_chunks - tid + kNT - 1) / kNT : 0;
  const uint16_t* ap = t.Ai + (int64_t)tid * 8;

  for (int g0 = 0; g0 < t.L; g0 += kTG) {
    stage_x(g, sm.tok, g0, t.L, sm.xs);
    __syncthreads();
    float val[kTG * 8];
#pragma unroll
    for (int i = 0; i < kTG * 8; ++i) val[i] = 0.f;
    for (int jb = 0; jb < nj; jb += kCH) {
      uint4 a[kCH];
#pragma unroll
      for (int j = 0; j < kCH; ++j)
        a[j] = (jb + j < nj) ? ldg16(ap + (int64_t)(jb + j) * kNT * 8) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int j = 0; j < kCH; ++j) {
        if (jb + j < nj) {
          const int row = (tid + (jb + j) * kNT) / R_OCT;
          const uint2 xv = *reinterpret_cast<const uint2*>(sm.xs + row * kTG);
          const float xf[4] = {bf_lo(xv.x), bf_hi(xv.x), bf_lo(xv.y), bf_hi(xv.y)};
          float af[8];
          unpack8(a[j], af);
#pragma unroll
          for (int tt = 0; tt < kTG; ++tt)
#pragma unroll
            for (int e = 0; e < 8; ++e) val[tt * 8 + e] = fmaf(xf[tt], af[e], val[tt * 8 + e]);
        }
      }
    }
    // reduce-scatter across the row slots of the wavefront
    int base = 0;
    if constexpr (HALV >= 1) { halve<32, R_OCT * 1>(val, lane); base += (lane & (R_OCT * 1)) ? 16 : 0; }
    if constexpr (HALV >= 2) { halve<16, R_OCT * 2>(val, lane); base += (lane & (R_OCT * 2)) ? 8 : 0; }
    if constexpr (HALV >= 3) { halve<8, R_OCT * 4>(val, lane); base += (lane & (R_OCT * 4)) ? 4 : 0; }
    if constexpr (HALV >= 4) { halve<4, R_OCT * 8>(val, lane); base += (lane & (R_OCT * 8)) ? 2 : 0; }
    if constexpr (HALV >= 5) { halve<2, R_OCT * 16>(val, lane); base += (lane & (R_OCT * 16)) ? 1 : 0; }
    bool writer = true;
    if constexpr (RSW == 64) {             // r = 8: one more all-reduce step
      val[0] += __shfl_xor(val[0], 32, 64);
      writer = (lane & 32) == 0;
    }
    __syncthreads();                        // xs is dead; red may overwrite it
    if (writer) {
#pragma unroll
      for (int j = 0; j < VL; ++j) {
        const int idx = base + j;
        const int tt = idx >> 3, e = idx & 7;
        sm.red[(w * kTG + tt) * R + oct * 8 + e] = val[j];
      }
    }
    __syncthreads();
    for (int o = tid; o < kTG * R; o += kNT) {
      const int tt = o / R, c = o - tt * R;
      if (g0 + tt < t.L) {
        float s = sm.red[tt * R + c];
#pragma unroll
        for (int ww = 1; ww < kW; ++ww) s += sm.red[(ww * kTG + tt) * R + c];
        sm.vs[c * kTT + g0 + tt] = s;
      }
    }
    __syncthreads();                        // red/xs free for the next group
  }
}

__device__ __forceinline__ void shrink_dispatch(const ApplyArgs& g, const Tile& t,
                                                const Smem& sm) {
  switch (t.r >> 3) {
    case 1: shrink_tile<1>(g, t, sm); break;
    case 2: shrink_tile<2>(g, t, sm); break;
    case 4: shrink_tile<4>(g, t, sm); break;
    case 8: shrink_tile<8>(g, t, sm); break;
    case 16: shrink_tile<16>(g, t, sm); break;
    default: break;  // excluded by load_tile
  }
}

// y[tok, cols] = bf16(y + s * v B_i[:, cols]) for every token of the tile.
__device__ void expand_tile(const ApplyArgs& g, const Tile& t, const Smem& sm) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int RSB = 1 << g.rsb_log2;
  const int CPW = 64 / RSB;                  // column octets per wavefront
  const int n_oct = g.h_out >> 3;
  const int co_l = lane % CPW, rb = lane / CPW;
  const int r = t.r;
  const int njb = rb < r ? (r - rb + RSB - 1) / RSB : 0;
  for (int co = w * CPW + co_l, cb = 0; cb * kW * CPW < n_oct; ++cb, co += kW * CPW) {
    const bool col_ok = co < n_oct;
    const uint16_t* bp = t.Bi + (int64_t)rb * g.h_out + (int64_t)co * 8;
    const int64_t bstep = (int64_t)RSB * g.h_out;
    for (int g0 = 0; g0 < t.L; g0 += kTG) {
      float d[kTG * 8];
#pragma unroll
      for (int i = 0; i < kTG * 8; ++i) d[i] = 0.f;
      if (col_ok) {
        for (int jb = 0; jb < njb; jb += kCH) {
          uint4 b[kCH];
#pragma unroll
          for (int j = 0; j < kCH; ++j)
            b[j] = (jb + j < njb) ? ldg16(bp + (int64_t)(jb + j) * bstep) : make_uint4(0, 0, 0, 0);
#pragma unroll
          for (int j = 0; j < kCH; ++j) {
            if (jb + j < njb) {
              const int c = rb + (jb + j) * RSB;
              const float4 vv = *reinterpret_cast<const float4*>(sm.vs + c * kTT + g0);
              const float vf[4] = {vv.x, vv.y, vv.z, vv.w};
              float bf[8];
              unpack8(b[j], bf);
#pragma unroll
              for (int tt = 0; tt < kTG; ++tt)
#pragma unroll
                for (int e = 0; e < 8; ++e) d[tt * 8 + e] = fmaf(vf[tt], bf[e], d[tt * 8 + e]);
            }
          }
        }
      }
      // all-reduce across the row slots of each column octet
      for (int m = CPW; m < 64; m <<= 1) {
#pragma unroll
        for (int i = 0; i < kTG * 8; ++i) d[i] += __shfl_xor(d[i], m, 64);
      }
      if (col_ok && rb == 0) {
#pragma unroll
        for (int tt = 0; tt < kTG; ++tt) {
          if (g0 + tt < t.L) {
            const int tk = sm.tok[g0 + tt];
            if (tk >= 0) {
              uint16_t* yp = g.y + (int64_t)tk * g.ldy + (int64_t)co * 8;
              const uint4 yv = ldg16(yp);
              float yf[8];
              unpack8(yv, yf);
              uint32_t ob[8];
#pragma unroll
              for (int e = 0; e < 8; ++e) ob[e] = to_bf16(fmaf(t.s, d[tt * 8 + e], yf[e]));
              uint4 out;
              out.x = ob[0] | (ob[1] << 16);
              out.y = ob[2] | (ob[3] << 16);
              out.z = ob[4] | (ob[5] << 16);
              out.w = ob[6] | (ob[7] << 16);
              *reinterpret_cast<uint4*>(yp) = out;
            }
          }
        }
      }
    }
  }
}

// Common prologue: tile, tokens, zeroed v.  Returns false if the work group
// has nothing to do.
__device__ __forceinline__ bool tile_prologue(const ApplyArgs& g, Tile& t, Smem& sm,
                                              void* lds) {
  if (!load_tile(g, t)) return false;
  sm = carve(lds, g.max_rank);
  load_tokens(g, t, sm.tok);
  for (int o = threadIdx.x; o < g.max_rank * kTT; o += kNT) sm.vs[o] = 0.f;
  __syncthreads();
  return true;
}

// ---------------------------------------------------------------------------
// kernels
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kNT) void shrink_kernel(ApplyArgs g) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  Tile t;
  Smem sm;
  if (!tile_prologue(g, t, sm, apply_lds)) return;
  shrink_dispatch(g, t, sm);
  for (int o = threadIdx.x; o < t.L * t.r; o += kNT) {
    const int l = o / t.r, c = o - l * t.r;
    const int tk = sm.tok[l];
    if (tk >= 0) g.v[(int64_t)tk * g.ldv + c] = sm.vs[c * kTT + l];
  }
}

__global__ __launch_bounds__(kNT) void expand_kernel(ApplyArgs g) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  Tile t;
  Smem sm;
  if (!tile_prologue(g, t, sm, apply_lds)) return;
  for (int o = threadIdx.x; o < t.L * t.r; o += kNT) {
    const int l = o / t.r, c = o - l * t.r;
    const int tk = sm.tok[l];
    if (tk >= 0) sm.vs[c * kTT + l] = g.v[(int64_t)tk * g.ldv + c];
  }
  __syncthreads();
  expand_tile(g, t, sm);
}

__global__ __launch_bounds__(kNT) void apply_kernel(ApplyArgs g) {
  extern __shared__ __align__(16) unsigned char apply_lds[];
  Tile t;
  Smem sm;
  if (!tile_prologue(g, t, sm, apply_lds)) return;
  shrink_dispatch(g, t, sm);
  expand_tile(g, t, sm);
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

inline bool usable_rank(int r, int max_rank) {
  return r == 0 || (r >= 8 && r <= max_rank && (r & (r - 1)) == 0);
}

// Expand row slots per column octet: the largest power of two that still
// lets one work group cover every column octet of y in a single pass.
int rsb_log2_for(int h_out) {
  const int n_oct = h_out / 8;
  int l = 0;
  while (l < 6 && (n_oct << (l + 1)) <= kNT) ++l;
  return l;
}

plora_status check_adapters_host(const plora_adapters* ad) {
  if (!ad) return PLORA_ERR_INVALID_ARG;
  if (ad->n_adapters < 0 || ad->h_in <= 0 || ad->h_out <= 0 || ad->max_rank < 0 ||
      ad->a_len < 0 || ad->b_len < 0)
    return PLORA_ERR_INVALID_ARG;
  if ((ad->h_in & 7) || (ad->h_out & 7)) return PLORA_ERR_UNSUPPORTED;
  if (ad->max_rank == 0 || (ad->max_rank & 7) || ad->max_rank > PLORA_MAX_RANK)
    return PLORA_ERR_UNSUPPORTED;
  if (smem_bytes(ad->h_in, ad->max_rank) > kMaxLds) return PLORA_ERR_UNSUPPORTED;
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
                     size_t ws_bytes, ApplyArgs& g) {
  (void)ws; (void)ws_bytes;  // the tile kernels need no workspace
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
  g.rsb_log2 = rsb_log2_for(ad->h_out);
  return PLORA_OK;
}

// Dynamic LDS above 64 KB is opted into once per kernel.
void allow_lds(const void* kernel, std::atomic<bool>& done) {
  if (done.load()) return;
  (void)hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  (void)hipGetLastError();
  done.store(true);
}

std::atomic<bool> g_lds_shrink{false}, g_lds_expand{false}, g_lds_apply{false};

template <class K>
plora_status launch_tiles(K kernel, std::atomic<bool>& lds_done, const ApplyArgs& g,
                          hipStream_t stream) {
  const size_t lds = smem_bytes(g.h_in, g.max_rank);
  if (lds > 64 * 1024) allow_lds(reinterpret_cast<const void*>(kernel), lds_done);
  clear_stale_error();
  hipLaunchKernelGGL(kernel, dim3((unsigned)g.tile_cap), dim3(kNT), lds, stream, g);
  return launch_status();
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
  (void)T; (void)ad;
  return 0;
}

plora_status plora_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream) {
  if (ws_bytes == 0) return PLORA_OK;
  if (!ws) return PLORA_ERR_INVALID_ARG;
  if (!aligned16(ws) || (ws_bytes & 15)) return PLORA_ERR_UNSUPPORTED;
  const size_t n16 = ws_bytes / 16;
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
  plora_status st = prepare(ad, seg, ws, ws_bytes, g);
  if (st != PLORA_OK) return st;
  if (seg->T == 0) return PLORA_OK;
  if (!x || !v) return PLORA_ERR_INVALID_ARG;
  if (ldx < ad->h_in || ldv < ad->max_rank) return PLORA_ERR_INVALID_ARG;
  if ((ldx & 7) || (ldv & 3) || !aligned16(x) || !aligned16(v)) return PLORA_ERR_UNSUPPORTED;
  g.x = x; g.ldx = ldx; g.v = v; g.ldv = ldv;
  return launch_tiles(shrink_kernel, g_lds_shrink, g, stream);
}

plora_status plora_expand(const float* v, int64_t ldv, const plora_adapters* ad,
                          const plora_segments* seg, uint16_t* y, int64_t ldy, void* ws,
                          size_t ws_bytes, hipStream_t stream) {
  ApplyArgs g;
  plora_status st = prepare(ad, seg, ws, ws_bytes, g);
  if (st != PLORA_OK) return st;
  if (seg->T == 0) return PLORA_OK;
  if (!v || !y) return PLORA_ERR_INVALID_ARG;
  if (ldy < ad->h_out || ldv < ad->max_rank) return PLORA_ERR_INVALID_ARG;
  if ((ldy & 7) || (ldv & 3) || !aligned16(y) || !aligned16(v)) return PLORA_ERR_UNSUPPORTED;
  g.v = const_cast<float*>(v); g.ldv = ldv; g.y = y; g.ldy = ldy;
  return launch_tiles(expand_kernel, g_lds_expand, g, stream);
}

plora_status plora_apply(const uint16_t* x, int64_t ldx, const plora_adapters* ad,
                         const plora_segments* seg, uint16_t* y, int64_t ldy, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  ApplyArgs g;
  plora_status st = prepare(ad, seg, ws, ws_bytes, g);
  if (st != PLORA_OK) return st;
  if (seg->T == 0) return PLORA_OK;
  if (!x || !y) return PLORA_ERR_INVALID_ARG;
  if (ldx < ad->h_in || ldy < ad->h_out) return PLORA_ERR_INVALID_ARG;
  if ((ldx & 7) || (ldy & 7) || !aligned16(x) || !aligned16(y)) return PLORA_ERR_UNSUPPORTED;
  g.x = x; g.ldx = ldx; g.y = y; g.ldy = ldy;
  return launch_tiles(apply_kernel, g_lds_apply, g, stream);
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

int32_t plora_debug_last_hip_error(void) { return g_last_hip_error.load(); }

}  // extern "C"
