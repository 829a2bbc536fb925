/*
 * Split-KV decode attention on one MI355X: the paper's other reduce-near-data
 * operation (section V-B).  The paper spreads each request's KV cache over
 * memory devices; each device runs the three steps of attention (scores,
 * softmax, weighted sum of values) on its share with a partial softmax that
 * keeps an anchor, and the GPU rescales the partial outputs into the exact
 * global output, whatever order they arrive in.  Here the shares are ranges of
 * PLORA_ATTN_CHUNK keys ("partitions") of one HBM-resident cache:
 *
 *   s_t = scale <q, k_t>                     for t < len_b
 *   m_p = max_{t in p} s_t                   (the partition's anchor)
 *   l_p = sum_{t in p} exp(s_t - m_p)
 *   o_p = sum_{t in p} exp(s_t - m_p) v_t    (unnormalised)
 *   out = sum_p exp(m_p - M) o_p / sum_p exp(m_p - M) l_p,   M = max_p m_p
 *
 * Layouts (row-major, device memory owned by the caller):
 *   q    bf16 [batch][heads][PLORA_ATTN_HEAD_DIM]
 *   k, v bf16 [batch][heads][max_len][PLORA_ATTN_HEAD_DIM]  (keys past len_b unused)
 *   lens int32 [batch], 0 <= len_b <= max_len (checked on the device: a
 *        request with an out-of-range length is treated as empty)
 *   m, l fp32 [batch][heads][P], o fp32 [batch][heads][P][PLORA_ATTN_HEAD_DIM],
 *        P = plora_attn_partitions(max_len); entries of partitions past len_b
 *        are not written
 *   out  bf16 [batch][heads][PLORA_ATTN_HEAD_DIM]; a request with len_b = 0
 *        gets zeros (a softmax over no keys is undefined)
 * Arithmetic: bf16 inputs, fp32 scores, exponentials and sums, one
 * round-to-nearest-even rounding at the output store.  Every call is
 * asynchronous on stream and allocates nothing; the merge is bitwise
 * deterministic (partitions in ascending order).
 * Errors: PLORA_ERR_INVALID_ARG for a null pointer, batch, heads or max_len
 * below 0; PLORA_ERR_UNSUPPORTED for pointers not 16-byte aligned or a
 * per-(request, head) cache of 2^31 bytes or more; PLORA_ERR_WORKSPACE_TOO_SMALL
 * as for plora_apply; PLORA_ERR_HIP for a failed launch.  batch, heads or
 * max_len of 0 is a no-op.
 */
#ifndef PLORA_ATTENTION_H
#define PLORA_ATTENTION_H

#include <stddef.h>
#include <stdint.h>

#include "plora.h"

#ifdef __cplusplus
extern "C" {
#endif

#define PLORA_ATTN_HEAD_DIM 128
#define PLORA_ATTN_CHUNK 256

/* Host.  Partitions per (request, head) for a cache of max_len keys:
 * ceil(max_len / PLORA_ATTN_CHUNK), 0 for max_len <= 0. */
int32_t plora_attn_partitions(int64_t max_len);

/* Host.  Bytes of workspace plora_attn_decode needs: m, l and o as laid out
 * above, each section 256-byte aligned; 0 for an empty shape. */
size_t plora_attn_workspace_bytes(int32_t batch, int32_t heads, int64_t max_len);

/* Steps 1 to 3 on every partition (the devices' share of section V-B): m, l
 * and o of each partition that holds at least one key. */
plora_status plora_attn_partial(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                const int32_t* lens, int32_t batch, int32_t heads,
                                int64_t max_len, float scale, float* m, float* l, float* o,
                                hipStream_t stream);

/* The GPU's rescaling of the partials into out (section V-B). */
plora_status plora_attn_merge(const float* m, const float* l, const float* o,
                              const int32_t* lens, int32_t batch, int32_t heads,
                              int64_t max_len, uint16_t* out, hipStream_t stream);

/* plora_attn_partial then plora_attn_merge through ws (at least
 * plora_attn_workspace_bytes bytes, 16-byte aligned). */
plora_status plora_attn_decode(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                               const int32_t* lens, int32_t batch, int32_t heads,
                               int64_t max_len, float scale, uint16_t* out, void* ws,
                               size_t ws_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PLORA_ATTENTION_H */
