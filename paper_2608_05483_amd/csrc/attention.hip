// Split-KV decode attention for gfx950 (section V-B): per partition of
// PLORA_ATTN_CHUNK keys an anchor, a sum of shifted exponentials and an
// unnormalised output (plora_attn_partial), then their exact rescaling into
// the output (plora_attn_merge).  The C ABI is declared in
// include/plora_attention.h.
//
// Decode attention is a pair of matrix-vector products per (request, head):
// it reads every key and value once and does two flops per byte, so it is
// HBM-bound and runs on the vector ALUs; the work is spread so that a batch
// of long caches gives tens of thousands of work groups.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstring>

#include "plora_attention.h"

namespace {

constexpr int kD = PLORA_ATTN_HEAD_DIM;   // 128: sixteen 16-byte units per row
constexpr int kC = PLORA_ATTN_CHUNK;      // keys per partition
constexpr int kNT = 256;                  // threads per work group
constexpr int kGroups = kNT / 16;         // keys in flight per pass (16 lanes each)
constexpr int kKeysPerThread = kC / kGroups;

typedef int i32x4_t __attribute__((ext_vector_type(4)));
constexpr int kRsrcWord3 = 0x00020000;    // raw buffer, 32-bit data format (gfx9 family)
constexpr int kPastEnd = (int)0x80000000u;

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

// The len valid rows of one (request, head) cache as a raw buffer resource:
// a load past them reads zero and fetches nothing, so the partition tail
// needs no branch and nothing outside the valid rows is touched.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const uint16_t* p, int len) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p), 0, len * kD * 2,
                                           kRsrcWord3);
}

__device__ __forceinline__ uint4 bld16(__amdgpu_buffer_rsrc_t r, int byte_off) {
  const i32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0);
  return make_uint4((uint32_t)v.x, (uint32_t)v.y, (uint32_t)v.z, (uint32_t)v.w);
}

// Partition blockIdx.x of head blockIdx.y of request blockIdx.z.  Thread
// (g, e) = (tid / 16, tid % 16) takes keys lo + g + 16 j, j < 16, and the
// dimensions 8 e .. 8 e + 7 of each: the sixteen lanes of a key read its row
// as one coalesced 256-byte line, and every thread requests all sixteen of
// its key units and value units before it uses any.
__global__ __launch_bounds__(kNT) void attn_partial_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const int32_t* __restrict__ lens, int32_t heads,
    int64_t max_len, float scale, int32_t P, float* __restrict__ m_out,
    float* __restrict__ l_out, float* __restrict__ o_out) {
  __shared__ float red[kNT / 64][kD];
  __shared__ float wmax[kNT / 64], wsum[kNT / 64];
  const int p = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = tid >> 4, e = tid & 15;
  int n = lens[b];
  n = (n < 0 || n > max_len) ? 0 : n;
  const int lo = p * kC;
  if (lo >= n) return;                            // no key here: nothing written
  const int64_t row0 = ((int64_t)b * heads + h) * max_len;
  const __amdgpu_buffer_rsrc_t kr = rows_rsrc(k + row0 * kD, n);
  const __amdgpu_buffer_rsrc_t vr = rows_rsrc(v + row0 * kD, n);

  uint4 kreg[kKeysPerThread], vreg[kKeysPerThread];
#pragma unroll
  for (int j = 0; j < kKeysPerThread; ++j) {
    const int t = lo + g + kGroups * j;           // < lo + kC; past n reads zero
    kreg[j] = bld16(kr, t < n ? (t * kD + 8 * e) * 2 : kPastEnd);
  }
#pragma unroll
  for (int j = 0; j < kKeysPerThread; ++j) {
    const int t = lo + g + kGroups * j;
    vreg[j] = bld16(vr, t < n ? (t * kD + 8 * e) * 2 : kPastEnd);
  }
  float qf[8];
  unpack8(*reinterpret_cast<const uint4*>(q + ((int64_t)b * heads + h) * kD + 8 * e), qf);
#pragma unroll
  for (int i = 0; i < 8; ++i) qf[i] *= scale;

  // step 1: scores, each summed over the sixteen lanes of its key
  float s[kKeysPerThread];
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < kKeysPerThread; ++j) {
    float kf[8];
    unpack8(kreg[j], kf);
    float d = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) d = fmaf(qf[i], kf[i], d);
#pragma unroll
    for (int msk = 1; msk < 16; msk <<= 1) d += __shfl_xor(d, msk, 64);
    const int t = lo + g + kGroups * j;
    s[j] = t < n ? d : -INFINITY;
    mx = fmaxf(mx, s[j]);
  }
  // the partition's anchor
#pragma unroll
  for (int msk = 16; msk < 64; msk <<= 1) mx = fmaxf(mx, __shfl_xor(mx, msk, 64));
  if (lane == 0) wmax[wv] = mx;
  __syncthreads();
  float m = wmax[0];
#pragma unroll
  for (int w = 1; w < kNT / 64; ++w) m = fmaxf(m, wmax[w]);

  // steps 2 and 3: shifted exponentials, their sum, the weighted values
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < kKeysPerThread; ++j) {
    const float w = expf(s[j] - m);               // 0 for keys past n
    sum += w;
    float vf[8];
    unpack8(vreg[j], vf);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = fmaf(w, vf[i], acc[i]);
  }
  // sum: each key counted once (the sixteen lanes of a key hold the same w)
#pragma unroll
  for (int msk = 16; msk < 64; msk <<= 1) sum += __shfl_xor(sum, msk, 64);
#pragma unroll
  for (int msk = 16; msk < 64; msk <<= 1)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] += __shfl_xor(acc[i], msk, 64);
  if (lane < 16) {
#pragma unroll
    for (int i = 0; i < 8; ++i) red[wv][8 * lane + i] = acc[i];
  }
  if (lane == 0) wsum[wv] = sum;
  __syncthreads();
  const int64_t part = ((int64_t)b * heads + h) * P + p;
  if (tid < kD) {
    float o = red[0][tid];
#pragma unroll
    for (int w = 1; w < kNT / 64; ++w) o += red[w][tid];
    o_out[part * kD + tid] = o;
  }
  if (tid == 0) {
    float l = wsum[0];
#pragma unroll
    for (int w = 1; w < kNT / 64; ++w) l += wsum[w];
    m_out[part] = m;
    l_out[part] = l;
  }
}

// The rescaling: one work group of kD threads per (request, head), thread d
// for output dimension d, partitions in ascending order.
__global__ __launch_bounds__(kD) void attn_merge_kernel(
    const float* __restrict__ m_in, const float* __restrict__ l_in,
    const float* __restrict__ o_in, const int32_t* __restrict__ lens, int32_t heads,
    int64_t max_len, int32_t P, uint16_t* __restrict__ out) {
  const int h = blockIdx.x, b = blockIdx.y, d = threadIdx.x;
  int n = lens[b];
  n = (n < 0 || n > max_len) ? 0 : n;
  const int np = (n + kC - 1) / kC;
  const int64_t base = ((int64_t)b * heads + h) * P;
  float M = -INFINITY;
  for (int p = 0; p < np; ++p) M = fmaxf(M, m_in[base + p]);
  float L = 0.f, o = 0.f;
  for (int p = 0; p < np; ++p) {
    const float w = expf(m_in[base + p] - M);
    L = fmaf(w, l_in[base + p], L);
    o = fmaf(w, o_in[(base + p) * kD + d], o);
  }
  const float r = np > 0 ? o / L : 0.f;
  out[((int64_t)b * heads + h) * kD + d] = (uint16_t)to_bf16(r);
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

std::atomic<int32_t> g_attn_last_error{0};

plora_status launch_status() {
  const hipError_t err = hipGetLastError();
  if (err == hipSuccess) return PLORA_OK;
  g_attn_last_error.store((int32_t)err);
  return PLORA_ERR_HIP;
}

plora_status check_shape(int32_t batch, int32_t heads, int64_t max_len) {
  if (batch < 0 || heads < 0 || max_len < 0) return PLORA_ERR_INVALID_ARG;
  // one (request, head) cache is read through 32-bit byte offsets
  if (max_len * kD * 2 >= (INT64_C(1) << 31)) return PLORA_ERR_UNSUPPORTED;
  return PLORA_OK;
}

}  // namespace

extern "C" {

int32_t plora_attn_partitions(int64_t max_len) {
  return max_len <= 0 ? 0 : (int32_t)((max_len + kC - 1) / kC);
}

size_t plora_attn_workspace_bytes(int32_t batch, int32_t heads, int64_t max_len) {
  if (batch <= 0 || heads <= 0 || max_len <= 0) return 0;
  const size_t parts = (size_t)batch * heads * plora_attn_partitions(max_len);
  return align256(parts * 4) * 2 + align256(parts * kD * 4);
}

plora_status plora_attn_partial(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                const int32_t* lens, int32_t batch, int32_t heads,
                                int64_t max_len, float scale, float* m, float* l, float* o,
                                hipStream_t stream) {
  plora_status st = check_shape(batch, heads, max_len);
  if (st != PLORA_OK) return st;
  if (batch == 0 || heads == 0 || max_len == 0) return PLORA_OK;
  if (!q || !k || !v || !lens || !m || !l || !o) return PLORA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return PLORA_ERR_UNSUPPORTED;
  const int32_t P = plora_attn_partitions(max_len);
  (void)hipGetLastError();
  hipLaunchKernelGGL(attn_partial_kernel, dim3(P, heads, batch), dim3(kNT), 0, stream, q, k,
                     v, lens, heads, max_len, scale, P, m, l, o);
  return launch_status();
}

plora_status plora_attn_merge(const float* m, const float* l, const float* o,
                              const int32_t* lens, int32_t batch, int32_t heads,
                              int64_t max_len, uint16_t* out, hipStream_t stream) {
  plora_status st = check_shape(batch, heads, max_len);
  if (st != PLORA_OK) return st;
  if (batch == 0 || heads == 0 || max_len == 0) return PLORA_OK;
  if (!m || !l || !o || !lens || !out) return PLORA_ERR_INVALID_ARG;
  (void)hipGetLastError();
  hipLaunchKernelGGL(attn_merge_kernel, dim3(heads, batch), dim3(kD), 0, stream, m, l, o,
                     lens, heads, max_len, plora_attn_partitions(max_len), out);
  return launch_status();
}

plora_status plora_attn_decode(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                               const int32_t* lens, int32_t batch, int32_t heads,
                               int64_t max_len, float scale, uint16_t* out, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  plora_status st = check_shape(batch, heads, max_len);
  if (st != PLORA_OK) return st;
  if (batch == 0 || heads == 0 || max_len == 0) return PLORA_OK;
  if (!ws) return PLORA_ERR_INVALID_ARG;
  if (!aligned16(ws)) return PLORA_ERR_UNSUPPORTED;
  if (ws_bytes < plora_attn_workspace_bytes(batch, heads, max_len))
    return PLORA_ERR_WORKSPACE_TOO_SMALL;
  const size_t parts = (size_t)batch * heads * plora_attn_partitions(max_len);
  char* base = reinterpret_cast<char*>(ws);
  float* m = reinterpret_cast<float*>(base);
  float* l = reinterpret_cast<float*>(base + align256(parts * 4));
  float* o = reinterpret_cast<float*>(base + 2 * align256(parts * 4));
  st = plora_attn_partial(q, k, v, lens, batch, heads, max_len, scale, m, l, o, stream);
  if (st != PLORA_OK) return st;
  return plora_attn_merge(m, l, o, lens, batch, heads, max_len, out, stream);
}

}  // extern "C"
