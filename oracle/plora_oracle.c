/*
 * plora_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct CPU reference for the batched
 * heterogeneous-adapter LoRA apply.  Only the test suite, the smoke check and
 * the CPU-baseline leg of the benchmark may load this code; the product path
 * (the HIP library) never does, and this file shares nothing with it.
 *
 * What is computed (paper section II-A, the LoRA layer y = x(W + AB), and
 * section V-A, strategies E1..E4, which all produce the same y):
 *
 *   y[t,j] = y_base[t,j] + s_i * sum_c ( sum_k x[t,k] * A_i[k,c] ) * B_i[c,j],
 *   i = idx[t]
 *
 * where y_base = x W is the base projection, supplied by the caller.  The
 * paper has no scale; s_i = 1 reproduces it exactly.
 *
 * Readings taken where the paper is silent (each also listed in the design doc):
 *  - bf16 storage for x, A, B and y; every accumulation in fp32; the
 *    intermediate m = xA (strategy E4's shipped value, called v here) stays
 *    fp32; one round-to-nearest-even to bf16 at the y store.
 *  - A_i is h_in x r_i row-major at element offset a_off[i] of a flat stack,
 *    B_i is r_i x h_out row-major at b_off[i] (the paper's D1 x R and R x D2).
 *  - idx[t] == -1 means "no adapter"; any other id outside [0, N) is invalid;
 *    both leave y[t] = y_base[t].  r_i == 0 is a no-op adapter.
 *  - Segments (the per-adapter batches B_i of the cost model, section VI-B)
 *    are ordered by ascending adapter id, tokens inside a segment by
 *    ascending token index.
 *
 * Summation order: k ascending for v, c ascending for the expand.  The
 * per-token and the grouped entry points use the same order and therefore
 * give bitwise equal results.  Build with -O2 -ffp-contract=off (no FMA
 * contraction, no fast-math), so every product and every sum is rounded once.
 *
 * Parity pins for every function live in tests/test_oracle_pins.py.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ---- bf16 <-> fp32 (IEEE binary32 truncated to its top 16 bits) -------- */

/* bf16 -> fp32 is exact: the bf16 bits are the high half of the binary32. */
static float oracle_bf16_to_f32(uint16_t h) {
  uint32_t u = ((uint32_t)h) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

/* fp32 -> bf16 with round-to-nearest, ties to even.  NaN stays NaN (quiet,
 * sign kept); values that round past the largest finite bf16 become inf, as
 * IEEE rounding requires. */
static uint16_t oracle_f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu) != 0u) {
    return (uint16_t)(((u >> 16) & 0x8000u) | 0x7fc0u);
  }
  uint32_t lower = u & 0xffffu;
  uint32_t upper = u >> 16;
  if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u))) upper += 1u;
  return (uint16_t)upper;
}

void oracle_bf16_decode(const uint16_t* in, float* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_bf16_to_f32(in[i]);
}

void oracle_bf16_encode(const float* in, uint16_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_f32_to_bf16(in[i]);
}

/* ---- segmentation: counting sort by adapter id ------------------------- */

/*
 * Groups the tokens of a heterogeneous batch by adapter: the per-adapter
 * batch B_i of the cost model (section VI-B) and the request-to-adapter
 * lookup of section VI.  Steps: histogram over [0, N), exclusive prefix sum,
 * scatter in ascending token order (which makes the sort stable), then list
 * the non-empty ids in ascending order.
 *
 * Outputs (cap = min(T, N)):
 *   perm[T]        token indices of valid tokens in segment order; -1 after.
 *   seg_ptr[cap+1] start of each segment in perm; entries after the last
 *                  segment hold n_valid.
 *   seg_id[cap]    adapter id of each segment; -1 after the last.
 *   meta[4]        {n_seg, n_valid, n_none (idx == -1), n_invalid}.
 * Returns 0, or -1 if the scratch histogram cannot be allocated.
 */
int oracle_segment(const int32_t* idx, int32_t T, int32_t n_adapters,
                   int32_t* perm, int32_t* seg_ptr, int32_t* seg_id,
                   int32_t* meta, int32_t* scratch_hist /* [n_adapters+1] */) {
  int32_t cap = T < n_adapters ? T : n_adapters;
  int32_t n_none = 0, n_invalid = 0, n_valid = 0;

  for (int32_t i = 0; i <= n_adapters; ++i) scratch_hist[i] = 0;
  for (int32_t t = 0; t < T; ++t) {
    int32_t id = idx[t];
    if (id == -1) {
      ++n_none;
    } else if (id < 0 || id >= n_adapters) {
      ++n_invalid;
    } else {
      scratch_hist[id] += 1;
      ++n_valid;
    }
  }

  /* exclusive prefix sum: start[id] of each adapter's bucket */
  int32_t running = 0;
  for (int32_t id = 0; id < n_adapters; ++id) {
    int32_t c = scratch_hist[id];
    scratch_hist[id] = running;
    running += c;
  }

  /* stable scatter: tokens visited in ascending t */
  for (int32_t p = 0; p < T; ++p) perm[p] = -1;
  for (int32_t t = 0; t < T; ++t) {
    int32_t id = idx[t];
    if (id >= 0 && id < n_adapters) {
      perm[scratch_hist[id]] = t;
      scratch_hist[id] += 1;
    }
  }

  /* segments: non-empty ids in ascending order */
  int32_t n_seg = 0;
  for (int32_t p = 0; p < n_valid; ++p) {
    int32_t id = idx[perm[p]];
    if (p == 0 || idx[perm[p - 1]] != id) {
      seg_ptr[n_seg] = p;
      seg_id[n_seg] = id;
      ++n_seg;
    }
  }
  for (int32_t s = n_seg; s <= cap; ++s) seg_ptr[s] = n_valid;
  for (int32_t s = n_seg; s < cap; ++s) seg_id[s] = -1;

  meta[0] = n_seg;
  meta[1] = n_valid;
  meta[2] = n_none;
  meta[3] = n_invalid;
  return 0;
}

/* ---- the apply, one token at a time ------------------------------------ */

/* Is token t's adapter a real one with a non-zero rank? */
static int oracle_adapter_of(const int32_t* idx, int32_t t, int32_t n_adapters,
                             const int32_t* ranks) {
  int32_t id = idx[t];
  if (id < 0 || id >= n_adapters) return -1;
  if (ranks[id] <= 0) return -1;
  return id;
}

/* v[c] = sum_{k < h_in} x[k] * A_i[k, c], k ascending, fp32 accumulator.
 * This is the rank-r reduction m = xA of strategy E4 (section V-A). */
static void oracle_shrink_row(const uint16_t* x_row, int32_t h_in,
                              const uint16_t* A_i, int32_t r, float* v) {
  for (int32_t c = 0; c < r; ++c) {
    float acc = 0.0f;
    for (int32_t k = 0; k < h_in; ++k) {
      float xa = oracle_bf16_to_f32(x_row[k]) *
                 oracle_bf16_to_f32(A_i[(int64_t)k * r + c]);
      acc = acc + xa;
    }
    v[c] = acc;
  }
}

/* yref[j] = y[j] + s * sum_{c < r} v[c] * B_i[c, j], c ascending, fp32.
 * This is the expand y = mB of strategy E4 plus the base term. */
static void oracle_expand_row(const float* v, int32_t r, const uint16_t* B_i,
                              int32_t h_out, float s, const uint16_t* y_in,
                              float* yref, uint16_t* y_out) {
  for (int32_t j = 0; j < h_out; ++j) {
    float d = 0.0f;
    for (int32_t c = 0; c < r; ++c) {
      float vb = v[c] * oracle_bf16_to_f32(B_i[(int64_t)c * h_out + j]);
      d = d + vb;
    }
    float sd = s * d;
    float out = oracle_bf16_to_f32(y_in[j]) + sd;
    if (yref) yref[j] = out;
    if (y_out) y_out[j] = oracle_f32_to_bf16(out);
  }
}

static void oracle_copy_row(const uint16_t* y_in, int32_t h_out, float* yref,
                            uint16_t* y_out) {
  for (int32_t j = 0; j < h_out; ++j) {
    if (yref) yref[j] = oracle_bf16_to_f32(y_in[j]);
    if (y_out) y_out[j] = y_in[j];
  }
}

/*
 * v[t, c] for every valid token t and c < r_{idx[t]}; other entries of v are
 * not written.  x is T x h_in (row stride ldx), v is T x ldv fp32.
 */
void oracle_shrink(const uint16_t* x, int64_t ldx, int32_t T,
                   const int32_t* idx, int32_t n_adapters, int32_t h_in,
                   const uint16_t* A, const int64_t* a_off,
                   const int32_t* ranks, float* v, int64_t ldv,
                   int32_t n_threads) {
#ifdef _OPENMP
  if (n_threads < 1) n_threads = 1;
#pragma omp parallel for schedule(static) num_threads(n_threads)
#endif
  for (int32_t t = 0; t < T; ++t) {
    int32_t id = oracle_adapter_of(idx, t, n_adapters, ranks);
    if (id < 0) continue;
    oracle_shrink_row(x + (int64_t)t * ldx, h_in, A + a_off[id], ranks[id],
                      v + (int64_t)t * ldv);
  }
  (void)n_threads;
}

/*
 * Expand from a given v: yref = y_in + s_i * v B_i per valid token, copy of
 * y_in otherwise.  yref (fp32, T x h_out) and y_out (bf16, T x h_out) are
 * both optional (may be NULL).
 */
void oracle_expand(const float* v, int64_t ldv, int32_t T, const int32_t* idx,
                   int32_t n_adapters, int32_t h_out, const uint16_t* B,
                   const int64_t* b_off, const int32_t* ranks,
                   const float* scales, const uint16_t* y_in, int64_t ldy,
                   float* yref, uint16_t* y_out, int32_t n_threads) {
#ifdef _OPENMP
  if (n_threads < 1) n_threads = 1;
#pragma omp parallel for schedule(static) num_threads(n_threads)
#endif
  for (int32_t t = 0; t < T; ++t) {
    const uint16_t* yi = y_in + (int64_t)t * ldy;
    float* yr = yref ? yref + (int64_t)t * h_out : NULL;
    uint16_t* yo = y_out ? y_out + (int64_t)t * h_out : NULL;
    int32_t id = oracle_adapter_of(idx, t, n_adapters, ranks);
    if (id < 0) {
      oracle_copy_row(yi, h_out, yr, yo);
      continue;
    }
    oracle_expand_row(v + (int64_t)t * ldv, ranks[id], B + b_off[id], h_out,
                      scales[id], yi, yr, yo);
  }
  (void)n_threads;
}

/* Largest rank the oracle's per-token stack buffer holds. */
#define ORACLE_MAX_RANK 4096

/*
 * The full apply, one token at a time (ungrouped evaluation):
 *   yref[t] = y_base[t] + s_i * (x[t] A_i) B_i.
 * Returns 0, or -1 if some adapter's rank exceeds ORACLE_MAX_RANK.
 */
int oracle_apply(const uint16_t* x, int64_t ldx, int32_t T, const int32_t* idx,
                 int32_t n_adapters, int32_t h_in, int32_t h_out,
                 const uint16_t* A, const int64_t* a_off, const uint16_t* B,
                 const int64_t* b_off, const int32_t* ranks,
                 const float* scales, const uint16_t* y_base, int64_t ldy,
                 float* yref, uint16_t* y_out, int32_t n_threads) {
  for (int32_t i = 0; i < n_adapters; ++i)
    if (ranks[i] > ORACLE_MAX_RANK) return -1;
#ifdef _OPENMP
  if (n_threads < 1) n_threads = 1;
#pragma omp parallel for schedule(static) num_threads(n_threads)
#endif
  for (int32_t t = 0; t < T; ++t) {
    float v[ORACLE_MAX_RANK];
    const uint16_t* yi = y_base + (int64_t)t * ldy;
    float* yr = yref ? yref + (int64_t)t * h_out : NULL;
    uint16_t* yo = y_out ? y_out + (int64_t)t * h_out : NULL;
    int32_t id = oracle_adapter_of(idx, t, n_adapters, ranks);
    if (id < 0) {
      oracle_copy_row(yi, h_out, yr, yo);
      continue;
    }
    int32_t r = ranks[id];
    oracle_shrink_row(x + (int64_t)t * ldx, h_in, A + a_off[id], r, v);
    oracle_expand_row(v, r, B + b_off[id], h_out, scales[id], yi, yr, yo);
  }
  (void)n_threads;
  return 0;
}

/*
 * The same apply evaluated by segment (grouped evaluation): the tokens of
 * each segment are gathered, the segment's [L, h_in] x [h_in, r] and
 * [L, r] x [r, h_out] products are formed with the same k and c order as the
 * per-token path, and the rows are scattered back.  Takes the output of
 * oracle_segment.  Tokens outside every segment keep y_base.
 * v_scratch holds (longest segment) * max_rank floats, max_rank being at
 * least the largest ranks[i] used.  Returns 0, or -1 on a bad segment id or
 * a rank above max_rank.
 */
int oracle_apply_grouped(const uint16_t* x, int64_t ldx, int32_t T,
                         const int32_t* perm, const int32_t* seg_ptr,
                         const int32_t* seg_id, int32_t n_seg,
                         int32_t n_adapters, int32_t h_in, int32_t h_out,
                         const uint16_t* A, const int64_t* a_off,
                         const uint16_t* B, const int64_t* b_off,
                         const int32_t* ranks, const float* scales,
                         const uint16_t* y_base, int64_t ldy, float* yref,
                         uint16_t* y_out, float* v_scratch, int32_t max_rank) {
  /* every token starts as a copy of y_base; segment rows are overwritten */
  for (int32_t t = 0; t < T; ++t)
    oracle_copy_row(y_base + (int64_t)t * ldy, h_out,
                    yref ? yref + (int64_t)t * h_out : NULL,
                    y_out ? y_out + (int64_t)t * h_out : NULL);

  for (int32_t s = 0; s < n_seg; ++s) {
    int32_t id = seg_id[s];
    if (id < 0 || id >= n_adapters) return -1;
    int32_t r = ranks[id];
    if (r <= 0) continue;
    if (r > max_rank) return -1;
    int32_t p0 = seg_ptr[s], p1 = seg_ptr[s + 1];
    int32_t L = p1 - p0;
    const uint16_t* A_i = A + a_off[id];
    const uint16_t* B_i = B + b_off[id];
    /* V = X_s A_i : [L, r] */
    for (int32_t l = 0; l < L; ++l)
      oracle_shrink_row(x + (int64_t)perm[p0 + l] * ldx, h_in, A_i, r,
                        v_scratch + (int64_t)l * max_rank);
    /* Y_s = Y_base,s + s_i V B_i : [L, h_out] */
    for (int32_t l = 0; l < L; ++l) {
      int32_t t = perm[p0 + l];
      oracle_expand_row(v_scratch + (int64_t)l * max_rank, r, B_i, h_out,
                        scales[id], y_base + (int64_t)t * ldy,
                        yref ? yref + (int64_t)t * h_out : NULL,
                        y_out ? y_out + (int64_t)t * h_out : NULL);
    }
  }
  return 0;
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
