/*
 * plora.h -- C ABI of the MI355X (gfx950) batched heterogeneous-adapter LoRA
 * apply, the hot path of multi-LoRA serving in PLoRA.
 *
 * The operation (paper section II-A: a LoRA layer computes y = x(W + AB) with
 * A: D1 x R and B: R x D2; section II-B: one shared base model serves many
 * adapters, each request using its own; section V-A: strategies E1..E4 all
 * compute y = xAB, E4 by shipping the rank-R intermediate m = xA and forming
 * y = mB afterwards):
 *
 *   y[t, :] = y_base[t, :] + s_i * (x[t, :] A_i) B_i,   i = idx[t]
 *
 * for a batch of T tokens, each naming one of N adapters.  y_base = x W is the
 * base projection, produced by the caller; every call below accumulates into
 * y in place (y holds y_base on entry).  s_i is a per-adapter scale (s_i = 1
 * is the paper's formula).
 *
 * The work is split the way the paper's cost model groups it (section VI-B):
 * tokens are first grouped per adapter (the per-adapter batch B_i), and each
 * adapter's A_i and B_i are then read once per call whatever its batch size.
 *
 *   plora_segment  group tokens by adapter id (stable counting sort)
 *   plora_shrink   v[t, :] = x[t, :] A_i            (E4's m = xA, fp32)
 *   plora_expand   y[t, :] += s_i v[t, :] B_i        (E4's y = mB)
 *   plora_apply    both: one launch for batches of up to 256 tokens, two
 *                  above (per-slice partial sums of v, fp32, pass through the
 *                  workspace; within the one launch too when a tile is
 *                  split among several work groups)
 *
 * Data types and layouts (all row-major, element strides):
 *   x       bf16 [T, ldx], first h_in columns used
 *   y       bf16 [T, ldy], first h_out columns used, read and written
 *   v       fp32 [T, ldv], columns c < r_i of valid tokens defined
 *   A stack bf16, A_i = h_in x r_i at element offset a_off[i]
 *   B stack bf16, B_i = r_i x h_out at element offset b_off[i]
 *   bf16 values are passed as their 16-bit patterns (uint16_t).
 * Arithmetic: bf16 x bf16 products are exact in fp32; all sums are fp32;
 * v is never rounded below fp32; y is rounded once, to nearest even.
 * Reduction orders are fixed, so every call is bitwise deterministic, and
 * plora_apply equals plora_shrink followed by plora_expand bit for bit
 * (one exception, under plora_apply: a work group whose partners were not
 * scheduled in time).
 *
 * Memory and ownership: every pointer below is a DEVICE pointer unless the
 * text says "host"; the caller allocates and owns every buffer, including
 * the workspace (plora_workspace_bytes tells its size).  No call allocates
 * device memory, synchronizes the device or the stream, or keeps a pointer
 * after it returns (plora_check_adapters alone copies to the host and
 * waits).  Every launch goes onto the caller's stream.
 *
 * Errors: a call returns PLORA_OK or an error before launching anything,
 * except PLORA_ERR_HIP, which reports a failed launch.  Rules:
 *   PLORA_ERR_INVALID_ARG      null required pointer, negative size, a leading
 *                              dimension below the row width, or a segments
 *                              struct whose sizes do not match T and N
 *   PLORA_ERR_UNSUPPORTED      h_in or h_out not a multiple of 8; max_rank not
 *                              a multiple of 8 or above PLORA_MAX_RANK; a
 *                              pointer not 16-byte aligned; ldx/ldy not a
 *                              multiple of 8 or ldv not a multiple of 4;
 *                              T above PLORA_MAX_TOKENS; (N+1) * 2^ceil(log2 T)
 *                              beyond 2^32; an adapter block of 2^31 bytes or
 *                              more (max(h_in, h_out) * max_rank * 2)
 *   PLORA_ERR_WORKSPACE_TOO_SMALL  ws_bytes below plora_workspace_bytes()
 *                              where the call needs a workspace (a NULL ws
 *                              there is PLORA_ERR_INVALID_ARG)
 *   PLORA_ERR_HIP              this call's launch failed (hipGetLastError;
 *                              an error left pending by earlier HIP calls
 *                              is cleared before launching)
 * T == 0 launches nothing, writes nothing and returns PLORA_OK.
 * Conditions only the device can see never trap: a token whose idx is -1
 * (no adapter) or outside [0, N) keeps y_base and is counted in meta; an
 * adapter whose rank is 0 is a no-op.  Every rank from 1 to max_rank is
 * applied (the paper's range is 2..128, section V-A).  An adapter entry
 * that breaks the contract -- a rank below 0 or above max_rank, or an
 * A_i/B_i block that is misaligned or runs past a_len/b_len -- cannot be
 * applied: its tokens keep y_base and are counted in the workspace
 * (plora_workspace_counters), and plora_check_adapters reports the first
 * such entry on the host.
 * Calls that share a workspace or a segments struct must not overlap in time
 * (same stream, or externally ordered).
 */
#ifndef PLORA_H
#define PLORA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PLORA_OK = 0,
  PLORA_ERR_INVALID_ARG = 1,
  PLORA_ERR_UNSUPPORTED = 2,
  PLORA_ERR_WORKSPACE_TOO_SMALL = 3,
  PLORA_ERR_HIP = 4
} plora_status;

/* Largest adapter rank (the paper's rank range is 2..128, section V-A). */
#define PLORA_MAX_RANK 128
/* Largest token batch one plora_segment call groups. */
#define PLORA_MAX_TOKENS 16384
/* Tokens per work tile: a segment longer than this is split into tiles.
 * Batches of up to 64 tokens are tiled PLORA_DECODE_TILE_TOKENS tokens at a
 * time, batches of 65 to 256 tokens PLORA_SMALL_BATCH_TILE_TOKENS at a time,
 * larger ones PLORA_TILE_TOKENS at a time. */
#define PLORA_TILE_TOKENS 32
#define PLORA_SMALL_BATCH_TILE_TOKENS 2
#define PLORA_DECODE_TILE_TOKENS 1
/* Most projections one plora_apply_multi call serves. */
#define PLORA_MAX_PROJECTIONS 8
/* Entries of plora_segments.meta. */
#define PLORA_META_WORDS 8

/*
 * The adapter stack.  Host struct; the pointers inside are device pointers
 * (the pools: device-accessible host memory).
 *   n_adapters  N, number of adapters (ids 0..N-1)
 *   h_in, h_out model dimensions D1, D2 (multiples of 8)
 *   max_rank    host upper bound on every ranks[i] (multiple of 8, <= 128);
 *               sizes the workspace and the v stride
 *   A, B        flat bf16 stacks of a_len and b_len elements in device memory
 *   a_off,b_off int64 [N] element offsets of A_i and B_i (multiples of 8);
 *               an offset o < 0 names element -1 - o of the pool instead
 *   ranks       int32 [N], 0 <= r_i <= max_rank (0: a no-op adapter)
 *   scales      fp32  [N], s_i
 *   A_pool, B_pool, a_pool_len, b_pool_len
 *               optional flat bf16 stacks in pinned host memory that the
 *               kernels read directly, element counts (NULL / 0 if unused):
 *               the pooled-memory placement of section V-A, where the GPU
 *               loads A_i and B_i over the link itself (strategy E2); the
 *               Python module paper_2608_05483_amd.placement chooses what
 *               stays in device memory.  A and B may be NULL when every
 *               offset is negative.
 * Appended fields default to zero in C aggregate initialisation, so callers
 * without pools need not set them.
 * Ranks that are multiples of 8 run the vector and matrix-core paths of the
 * next power of two with their own row stride; other ranks (rows of A_i
 * that are not 16-byte aligned) take an LDS-staged shrink, correct but not
 * tuned.  Offsets are multiples of 8 for every rank when h_in and h_out
 * are, as back-to-back blocks give.
 */
typedef struct {
  int32_t n_adapters;
  int32_t h_in;
  int32_t h_out;
  int32_t max_rank;
  const uint16_t* A;
  const uint16_t* B;
  int64_t a_len;
  int64_t b_len;
  const int64_t* a_off;
  const int64_t* b_off;
  const int32_t* ranks;
  const float* scales;
  const uint16_t* A_pool;
  const uint16_t* B_pool;
  int64_t a_pool_len;
  int64_t b_pool_len;
} plora_adapters;

/*
 * The grouping of one token batch, written by plora_segment and read by the
 * other calls.  Host struct; the arrays are device memory owned by the caller.
 *   T          tokens in the batch (host)
 *   cap        min(T, N) (host), the most segments a batch can have
 *   tile_cap   plora_tile_capacity(T, N) (host)
 *   perm       int32 [T]: token indices of valid tokens, grouped by adapter
 *              (ascending id, ascending token index inside a group); -1 after
 *              the n_valid-th entry
 *   seg_ptr    int32 [cap+1]: start of each segment in perm; entries past
 *              the last segment hold n_valid
 *   seg_id     int32 [cap]: adapter id of each segment; -1 past the last
 *   meta       int32 [PLORA_META_WORDS]: {n_seg, n_valid, n_none (idx == -1),
 *              n_invalid (other ids outside [0, N)), n_tiles, 0, 0, 0}
 *   tiles      int32 [tile_cap][4]: the work tiles of the apply kernels,
 *              {adapter id, first perm position, length, segment index};
 *              a segment of L tokens gives ceil(L / K) tiles, K =
 *              PLORA_SMALL_BATCH_TILE_TOKENS for T <= 256, PLORA_TILE_TOKENS
 *              above; unused entries hold {-1, 0, 0, -1}
 * One segmentation serves every projection and layer of a step that shares
 * the token batch.
 */
typedef struct {
  int32_t T;
  int32_t cap;
  int32_t tile_cap;
  int32_t reserved;
  int32_t* perm;
  int32_t* seg_ptr;
  int32_t* seg_id;
  int32_t* meta;
  int32_t* tiles;
} plora_segments;

/* Host.  min(T, cap + T / K) with cap = min(T, N) and K the batch's tile
 * length (see PLORA_TILE_TOKENS): the most tiles a batch of T tokens over N
 * adapters can produce; 0 for T <= 0. */
int32_t plora_tile_capacity(int32_t T, int32_t n_adapters);

/* Host.  Bytes of device workspace plora_apply and plora_shrink need for a
 * batch of up to T tokens over this adapter stack; 0 for T <= 0.  Four
 * sections, each starting on a 256-byte boundary:
 *   1. the epochs of the one-launch apply's tile slots: 336 64-bit words,
 *      then two 64-bit counters (see plora_workspace_counters);
 *   2. the readiness words of the one-launch form above 256 tokens: 4096
 *      64-bit words, one per tile slot;
 *   3. the exchange regions of the one-launch form up to 256 tokens:
 *      8 * PLORA_SMALL_BATCH_TILE_TOKENS * 128 64-bit words (16 KiB) for each
 *      of P = min(336, max(8, cap8)) tile slots, cap8 being
 *      plora_tile_capacity(T, N) rounded up to a multiple of 8;
 *   4. the partial sums of v over up to 8 slices of h_in, fp32,
 *      K * T * max_rank * 4 bytes with K = min(8, max(1, h_in / 512)).
 * Sections 1 to 3 keep their offsets whatever T, the ranks or the slice
 * count, so one workspace serves calls of any batch size up to T and any
 * adapter stack it is large enough for.  Zero it once with
 * plora_workspace_init before its first use; afterwards it carries the
 * epochs and readiness words from call to call (every call leaves the
 * readiness words at zero) and must not be written by the caller.  Calls
 * that share one must not overlap in time.  plora_segment and plora_expand
 * take none (ws may be NULL). */
size_t plora_workspace_bytes(int32_t T, const plora_adapters* ad);

/* Zero a workspace (enqueued on stream; a no-op for ws_bytes == 0), as
 * plora_apply requires once before a workspace's first use. */
plora_status plora_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream);

/* Host.  Bytes of workspace with which plora_segment groups a batch of T
 * tokens over N adapters with many work groups (three launches) instead of
 * one: (ceil(T / 1024) + 1) * (N + 2) int32, rounded up to 256 bytes, for
 * T > 1024 and 2048 <= N < 8192; 0 otherwise (one work group, one launch, no
 * workspace: a counting sort for N < 2048, else a radix sort).
 * plora_workspace_bytes(T, ad) covers it for a stack of N adapters. */
size_t plora_segment_workspace_bytes(int32_t T, int32_t n_adapters);

/*
 * Group the batch: idx is int32 [T] device memory; fills seg->perm, seg_ptr,
 * seg_id, meta and tiles (seg->T, cap and tile_cap must be set).  This is the
 * per-adapter batch of the cost model (section VI-B).  ws may be NULL; given
 * at least plora_segment_workspace_bytes(T, N) bytes (16-byte aligned, no
 * initial contents needed, overwritten), a batch above 1024 tokens over
 * 2048 to 8191 adapters is grouped by many work groups in three launches;
 * every other batch by one work group in one launch.  Every form gives the
 * same output, bitwise deterministic; equal ids keep their token order.
 */
plora_status plora_segment(const int32_t* idx, const plora_segments* seg,
                           int32_t n_adapters, void* ws, size_t ws_bytes,
                           hipStream_t stream);

/*
 * v[t, c] = sum_k x[t, k] * A_i[k, c] for every valid token t and c < r_i
 * (the rank-r reduction m = xA of strategy E4, section V-A).  Entries of v
 * for other tokens and columns are not written.  Two launches: the partial
 * sums over slices of h_in into ws (at least plora_workspace_bytes(T) bytes,
 * 16-byte aligned; one slice for T <= 256 outside the exchange form), then
 * their sum, in slice order, into v.
 */
plora_status plora_shrink(const uint16_t* x, int64_t ldx,
                          const plora_adapters* ad, const plora_segments* seg,
                          float* v, int64_t ldv, void* ws, size_t ws_bytes,
                          hipStream_t stream);

/*
 * y[t, j] = bf16(y[t, j] + s_i * sum_c v[t, c] * B_i[c, j]) for every valid
 * token t (the expand y = mB of strategy E4), in place.  ws may be NULL.
 */
plora_status plora_expand(const float* v, int64_t ldv,
                          const plora_adapters* ad, const plora_segments* seg,
                          uint16_t* y, int64_t ldy, void* ws, size_t ws_bytes,
                          hipStream_t stream);

/*
 * The apply: y[t] = bf16(y[t] + s_i (x[t] A_i) B_i) for every valid token
 * (strategy E1: both matrices resident in GPU memory, section V-A).  One
 * launch: for T <= 256 with each tile split over up to 8 work groups, which
 * trade their partial sums of v through ws; above, with the shrink work
 * groups (one per tile and slice of h_in) storing partial sums of v in ws,
 * and the expand work groups (one per tile and slice of y's columns)
 * starting on a tile once its partial sums are stored.  A batch whose tile
 * capacity exceeds 4096 takes two launches, the shrink's and the expand's.
 * ws must hold plora_workspace_bytes(T) bytes, 16-byte aligned, zeroed once
 * by plora_workspace_init before its first use, in every case.  A work
 * group never waits for another without bound: if a partner does not
 * publish within a bounded number of polls (it was not scheduled), the work
 * group computes v by itself, which is correct to fp32 accuracy but summed
 * in another order.  Apart from that case the result is
 * bit for bit the same as plora_shrink followed by plora_expand, and
 * bitwise deterministic.  x and y must not overlap.
 */
plora_status plora_apply(const uint16_t* x, int64_t ldx,
                         const plora_adapters* ad, const plora_segments* seg,
                         uint16_t* y, int64_t ldy, void* ws, size_t ws_bytes,
                         hipStream_t stream);

/*
 * plora_segment followed by plora_apply on the same batch, as one call: the
 * first projection of a step, which also produces the step's segmentation
 * (seg is filled exactly as plora_segment fills it, so later projections and
 * layers can call plora_apply with it).  Arguments as for the two calls;
 * idx is int32 [T] device memory.  For T <= 256 in plora_apply's split
 * exchange form (and 1 <= N < 2^26 - 1 up to 64 tokens, N < 2^24 - 1 above)
 * this is one launch: above 64 tokens every work group segments the batch
 * itself (the grouping of section VI-B) and applies its own tile; up to 64
 * tokens (single-token tiles) every work group applies its own token
 * directly; one work group also writes seg.
 * Otherwise it makes the two calls.  y gets the bits plora_apply would give
 * after plora_segment (with the same exception for a partner that never
 * publishes).  Errors as for the two calls.
 */
plora_status plora_segment_apply(const int32_t* idx, const uint16_t* x, int64_t ldx,
                                 const plora_adapters* ad, const plora_segments* seg,
                                 uint16_t* y, int64_t ldy, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/*
 * plora_segment_apply for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same call without a workspace argument.  Its workspace is
 * a static device array of the library, 5 MiB on every GPU it runs on, held
 * until the process ends, zero when the library is loaded and then carrying
 * the exchange's epochs from call to call.  Batches of at most 256 tokens;
 * a larger T returns PLORA_ERR_UNSUPPORTED before anything is launched.
 * Allocates nothing and keeps no pointer; results are the bits
 * plora_segment_apply gives with a workspace of its own.  Every call on one
 * GPU shares that GPU's array: calls that overlap in time on one GPU (other
 * streams, other threads) race and must be ordered by the caller.  Other
 * arguments and errors as for plora_segment_apply; PLORA_ERR_HIP also if the
 * array's device address cannot be found.
 */
plora_status plora_segment_apply_noalloc(const int32_t* idx, const uint16_t* x, int64_t ldx,
                                         const plora_adapters* ad, const plora_segments* seg,
                                         uint16_t* y, int64_t ldy, hipStream_t stream);

/* Host.  How many launches plora_segment_apply makes for a batch of T
 * tokens over this stack: 1 (the one-launch form), 2 (plora_segment then
 * a one-launch plora_apply) or 3 (then a two-launch one, for a tile
 * capacity above 4096); 0 for T <= 0 or
 * a stack plora_apply would reject. */
int32_t plora_segment_apply_launches(int32_t T, const plora_adapters* ad);

/*
 * The apply for several projections of one layer that read the same input x
 * and the same token batch (the paper attaches LoRA adapters to the query,
 * key, value and output projections and the FFN, section VII-A; section II-A
 * gives each its own A and B): for p < n_proj,
 *   ys[p][t] = bf16(ys[p][t] + s_i^p (x[t] A_i^p) B_i^p),  i = idx[t],
 * with ads[p] the adapter stack of projection p (host array of n_proj
 * structs; every stack has the same n_adapters and h_in, while h_out and
 * the ranks may differ), ys a host array of n_proj device pointers and ldys
 * a host array of their leading dimensions.  seg, ws and stream as for
 * plora_apply; ws must hold plora_workspace_bytes_multi(T, ads, n_proj)
 * bytes, zeroed once before its first use.  Batches small enough for the
 * split exchange of plora_apply run all projections in one launch (their
 * tiles share the work groups, and each tile gets fewer slices than one
 * projection's alone would, so the bits can differ from separate
 * plora_apply calls while meeting the same bounds); other batches run
 * plora_apply once per projection.  Bitwise deterministic (with the same
 * exception as plora_apply).  Outputs must not overlap x or each other.
 * PLORA_ERR_INVALID_ARG for null arrays, n_proj < 1, stacks whose
 * n_adapters or h_in differ, or a leading dimension below its width;
 * PLORA_ERR_UNSUPPORTED for n_proj > PLORA_MAX_PROJECTIONS and the
 * alignment rules of plora_apply.
 */
plora_status plora_apply_multi(const uint16_t* x, int64_t ldx,
                               const plora_adapters* ads, int32_t n_proj,
                               const plora_segments* seg,
                               uint16_t* const* ys, const int64_t* ldys,
                               void* ws, size_t ws_bytes, hipStream_t stream);

/* Host.  Workspace bytes plora_apply_multi needs for a batch of up to T
 * tokens over these n_proj stacks: the layout of plora_workspace_bytes with
 * n_proj cap8 tile slots (still at most 336) and the largest partial-sum
 * section of the stacks; 0 for bad arguments or T <= 0.  It also serves
 * plora_apply and plora_shrink on any one of the stacks. */
size_t plora_workspace_bytes_multi(int32_t T, const plora_adapters* ads, int32_t n_proj);

/*
 * Host, synchronous (copies ranks and offsets to the host and waits on
 * stream).  Returns PLORA_OK if every adapter entry is usable by the kernels
 * (0 <= rank <= max_rank; offsets multiples of 8; blocks inside a_len /
 * b_len or the pools), else PLORA_ERR_INVALID_ARG with the first bad
 * adapter index in *bad_index (may be NULL).  Not for the hot path.
 */
plora_status plora_check_adapters(const plora_adapters* ad, int32_t* bad_index,
                                  hipStream_t stream);

/* Host.  The device address of pinned host memory (hipHostMalloc'd, as
 * torch's pin_memory gives), for the A_pool / B_pool fields; host is any
 * address inside the allocation.  PLORA_ERR_UNSUPPORTED if the memory is not
 * pinned and mapped for the device (kernels must never be handed it). */
plora_status plora_pool_device_pointer(const void* host, const void** device);

/* Host, synchronous (copies two words and waits on stream).  The counters
 * a workspace keeps since plora_workspace_init zeroed it, summed over every
 * call made with it:
 *   counts[0]  one-launch work items whose partners (the tile's other
 *              slices, or above 256 tokens its shrink work groups) did not
 *              publish in time, so that they computed v alone (their calls' bits can
 *              differ in the last places; see plora_apply);
 *   counts[1]  tokens that kept y_base because their adapter entry breaks
 *              the contract (a rank outside [0, max_rank], or a block
 *              misaligned or outside its array), counted once per call;
 *              plora_expand counts only when it is given a workspace.  A
 *              one-launch call (T <= 256) also skips and counts the tokens
 *              of a tile longer than PLORA_SMALL_BATCH_TILE_TOKENS, which
 *              plora_segment never writes for such a batch.
 * PLORA_ERR_INVALID_ARG for null pointers, PLORA_ERR_WORKSPACE_TOO_SMALL for
 * a buffer that cannot be a workspace, PLORA_ERR_HIP for a failed copy.
 * Not for the hot path. */
plora_status plora_workspace_counters(const void* ws, size_t ws_bytes, int64_t* counts,
                                      hipStream_t stream);

/* Static string naming a status code. */
const char* plora_status_string(plora_status status);

/* Test hook: the hipError_t of the most recent launch that returned
 * PLORA_ERR_HIP in this process, 0 if none did. */
int32_t plora_debug_last_hip_error(void);

/* Test hook: how many times a one-launch plora_apply work item re-reads a
 * partner's partial v before computing v by itself (see plora_apply), for
 * calls made after this one in this process; a negative value restores the
 * default (20000).  0 makes every item whose partners have not yet
 * published take the self-computed path, which tests can then check. */
void plora_debug_set_exchange_polls(int32_t polls);

#ifdef __cplusplus
}
#endif

#endif /* PLORA_H */
