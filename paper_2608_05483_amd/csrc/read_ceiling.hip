// read_ceiling.hip -- a measurement aid, not part of the apply: streams the
// same adapter blocks one plora_apply call must read (A_i and B_i of every
// distinct adapter of a batch) with 128-bit loads and nothing else, giving
// the empirical HBM read ceiling for that exact byte footprint and scatter.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kThreads = 64;
constexpr int kParts = 32;

// Work group b reads part (b % kParts) of adapter ids[b / kParts]: both its
// A_i and B_i blocks split into kParts contiguous pieces.  One 32-bit xor per
// work group is written so the loads cannot be dropped.
__global__ __launch_bounds__(kThreads) void read_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ B,
    const int64_t* __restrict__ a_off, const int64_t* __restrict__ b_off,
    const int32_t* __restrict__ ranks, const int32_t* __restrict__ ids, int32_t n_ids,
    int32_t h_in, int32_t h_out, uint32_t* __restrict__ sink) {
  const int which = blockIdx.x / kParts, part = blockIdx.x % kParts;
  if (which >= n_ids) return;
  const int id = ids[which];
  const int r = ranks[id];
  const int64_t na = (int64_t)h_in * r / 8, nb = (int64_t)h_out * r / 8;  // 16-B chunks
  const uint4* pa = reinterpret_cast<const uint4*>(A + a_off[id]);
  const uint4* pb = reinterpret_cast<const uint4*>(B + b_off[id]);
  const int64_t a0 = na * part / kParts, a1 = na * (part + 1) / kParts;
  const int64_t b0 = nb * part / kParts, b1 = nb * (part + 1) / kParts;
  // eight 16-byte loads in flight per lane before any is consumed
  uint32_t acc = 0;
  constexpr int kU = 8;
  for (int64_t i0 = a0 + threadIdx.x; i0 < a1; i0 += kThreads * kU) {
    uint4 v[kU];
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      const int64_t i = i0 + (int64_t)j * kThreads;
      v[j] = i < a1 ? pa[i] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < kU; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
  }
  for (int64_t i0 = b0 + threadIdx.x; i0 < b1; i0 += kThreads * kU) {
    uint4 v[kU];
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      const int64_t i = i0 + (int64_t)j * kThreads;
      v[j] = i < b1 ? pb[i] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < kU; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
  }
  sink[blockIdx.x * kThreads + threadIdx.x] = acc;
}

}  // namespace

extern "C" int plora_probe_read(const uint16_t* A, const uint16_t* B, const int64_t* a_off,
                                const int64_t* b_off, const int32_t* ranks,
                                const int32_t* ids, int32_t n_ids, int32_t h_in,
                                int32_t h_out, uint32_t* sink, hipStream_t stream) {
  if (n_ids <= 0) return 0;
  hipLaunchKernelGGL(read_kernel, dim3(n_ids * kParts), dim3(kThreads), 0, stream, A, B,
                     a_off, b_off, ranks, ids, n_ids, h_in, h_out, sink);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}

extern "C" int plora_probe_sink_words(int32_t n_ids) { return n_ids * kParts * kThreads; }
