/*
 * paged_attn.h -- C ABI of the MI355X (gfx950) paged decode-attention library.
 *
 * The operation.  An LLM stage of an agentic workflow keeps the prompt
 * context of its calls resident in GPU memory, so successive calls of the
 * stage -- the retries of an SQL error fixer against one schema, the
 * generator calls that all start from that schema -- reuse it instead of
 * rebuilding it (Cortex paper, section 1 "Motivating Example" and section 2
 * "Cortex Benefits", Fig. 2).  That resident context is a paged KV cache: a
 * pool of fixed-size token blocks, reached per sequence through a block
 * table, where shared prompt blocks appear in many tables.  Each decode step
 * of the stage runs, per layer, scaled dot-product softmax attention of one
 * new query row per head over the sequence's whole cached context:
 *
 *     out[b][h] = sum_t softmax_t(scale * <q[b][h], K_g[t]>) V_g[t],
 *     g = h / (Hq / Hkv),  t = 0 .. ctx[b]-1,
 *
 * where token t of sequence b is row t % 16 of physical block
 * block_tables[b][t / 16].  The paper gives no kernel or formula; this is the
 * textbook definition, which the library reaches through an online softmax,
 * optional split-KV partitions and a log-sum-exp merge.
 *
 * Data types and layouts (all row-major, little-endian):
 *   bf16    16-bit brain float, stored as uint16 bit patterns.
 *   K pool  bf16 [num_blocks][num_kv_heads][16][head_dim]   (token-major tiles)
 *   V pool  same shape and layout as the K pool.
 *   q       bf16 [batch][num_q_heads][head_dim]
 *   out     bf16 [batch][num_q_heads][head_dim], rounded to nearest even from
 *           fp32 accumulation.
 *   partial_out  fp32 [batch][num_q_heads][max_partitions][head_dim]
 *   partial_lse  fp32 [batch][num_q_heads][max_partitions]
 *
 * Ownership.  The caller owns every device buffer (pools, q, tables,
 * lengths, outputs, partials).  The library never allocates device memory
 * and never creates streams; a pool handle owns host-side metadata only.
 * Handles are not thread-safe: callers serialise access to one handle.
 *
 * Errors.  Every function returns 0 (PA_OK) or a negative PA_E* code and
 * never aborts; pa_last_error() returns a thread-local description of the
 * last failure.  Host-visible arguments are validated before any HIP call.
 * Device-resident data (table entries, context lengths) is not validated,
 * but kernels stay memory-safe: ids are clamped into [0, num_blocks) and
 * lengths into [0, max_context_len], so bad data gives unspecified values,
 * never an out-of-bounds access.
 *
 * Streams.  `stream` is a hipStream_t passed as void* (NULL = the default
 * stream).  Kernels are enqueued asynchronously; a function returning PA_OK
 * only means the launch was accepted.
 */
#ifndef PAGED_ATTN_H
#define PAGED_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  PA_OK = 0,
  PA_EINVAL = -1,       /* bad argument: null, misaligned, out of range, inconsistent */
  PA_ENOMEM = -2,       /* the block pool has too few free blocks */
  PA_EUNSUPPORTED = -3, /* valid but unsupported geometry (head_dim, group size) */
  PA_EHIP = -4,         /* a HIP runtime call failed (message says which) */
  PA_ESTATE = -5        /* allocator state violation: double release, claim of a used block */
};

#define PA_BLOCK_SIZE 16

typedef struct pa_kv_pool pa_kv_pool;

/* Thread-local description of the last error (never NULL). */
const char *pa_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int32_t pa_version(void);

/* ---------------------------------------------------------------------------
 * KV block pool: layout plus a host-side allocator with reference counts.
 *
 * One pool per stage engine: the paper gives every stage of the workflow its
 * own engine pool, with a queue and a cache of its own (section 2).  A block that
 * holds shared prompt tokens is retained once per extra sequence that maps
 * it and returns to the free list when its count reaches zero.
 * ------------------------------------------------------------------------- */

/* Create a pool handle over caller-owned device buffers.
 *   num_blocks    > 0 physical blocks in each of the K and V pools
 *   block_size    must be 16 (tokens per block)
 *   num_kv_heads  1 .. 64
 *   head_dim      64 or 128 (others: PA_EUNSUPPORTED)
 *   k_pool,v_pool device pointers, 16-byte aligned, each holding
 *                 num_blocks*num_kv_heads*16*head_dim bf16 values
 *   out           receives the handle; *out is untouched on error.
 * All blocks start free. */
int kv_pool_create(int32_t num_blocks, int32_t block_size, int32_t num_kv_heads,
                   int32_t head_dim, void *k_pool, void *v_pool, pa_kv_pool **out);

/* Destroy a handle (the device buffers stay the caller's).  NULL is a no-op. */
int kv_pool_destroy(pa_kv_pool *pool);

/* Take n free blocks (all or nothing), each with reference count 1, and
 * write their ids to ids_out[0..n-1].  PA_ENOMEM if fewer than n are free. */
int kv_pool_alloc(pa_kv_pool *pool, int32_t n, int32_t *ids_out);

/* Take the n listed blocks (all or nothing), each with reference count 1.
 * PA_ESTATE if any is in use or listed twice; PA_EINVAL if out of range.
 * Used when a caller has already chosen the physical placement. */
int kv_pool_claim(pa_kv_pool *pool, int32_t n, const int32_t *ids);

/* Add one reference to each listed block (sharing a prefix with one more
 * sequence).  PA_ESTATE if any listed block is free; nothing changes then. */
int kv_pool_retain(pa_kv_pool *pool, int32_t n, const int32_t *ids);

/* Drop one reference per listing; a block whose count reaches 0 is freed.
 * PA_ESTATE (and nothing changes) if any block would drop below zero. */
int kv_pool_release(pa_kv_pool *pool, int32_t n, const int32_t *ids);

/* Number of free blocks. */
int kv_pool_num_free(const pa_kv_pool *pool, int32_t *n_out);

/* Reference count of one block (0 = free). */
int kv_pool_refcount(const pa_kv_pool *pool, int32_t id, int32_t *count_out);

/* Number of blocks whose reference count is 2 or more (retained for a second
 * table).  While it is 0 the decode kernels load every tile with a streaming
 * cache hint (see paged_attn_decode). */
int kv_pool_num_shared(const pa_kv_pool *pool, int64_t *n_out);

/* Geometry: element strides of the pool [block][kv_head][token][dim], and
 * the bytes of one pool (K or V). */
int kv_pool_layout(const pa_kv_pool *pool, int64_t elem_strides_out[4], int64_t *pool_bytes_out);

/* ---------------------------------------------------------------------------
 * Decode attention.
 * ------------------------------------------------------------------------- */

/* Number of split-KV partitions for a batch whose longest context is
 * max_context_len: ceil(max_context_len / partition_size), at least 1;
 * partition_size 0 means one pass over the whole context (1 partition). */
int paged_attn_num_partitions(int32_t max_context_len, int32_t partition_size, int32_t *p_out);

/* Bytes of partial_out and partial_lse that paged_attn_decode needs when it
 * splits (num_partitions > 1); both are 0 when it does not. */
int paged_attn_workspace_size(int32_t batch, int32_t num_q_heads, int32_t head_dim,
                              int32_t max_context_len, int32_t partition_size,
                              size_t *partial_out_bytes, size_t *partial_lse_bytes);

/* One decode step of attention for a batch over a paged KV pool.
 *   pool             geometry and K/V device pointers (kv_pool_create)
 *   q                device bf16 [batch][num_q_heads][head_dim], 16-byte aligned
 *   block_tables     device int32 [batch][bt_stride]; entries 0..ceil(ctx/16)-1
 *                    of row b are physical ids.  The kernels may load later
 *                    entries of the row (within bt_stride) before the length
 *                    arrives, but never use them: they may hold anything
 *   bt_stride        >= ceil(max_context_len / 16)
 *   context_lens     device int32 [batch]: tokens to attend (the current token
 *                    included); 0 gives a zero output row
 *   batch            >= 0 (0 is a no-op)
 *   num_q_heads      multiple of the pool's num_kv_heads; the group size
 *                    G = num_q_heads / num_kv_heads must be 4 or 8
 *   scale            softmax scale applied to the fp32 dot products
 *   max_context_len  host upper bound of context_lens; sizes the grid
 *   partition_size   split-KV partition in tokens, a multiple of 16; 0 = none
 *   out              device bf16 [batch][num_q_heads][head_dim]; written when
 *                    there is a single partition
 *   partial_out/_lse device fp32 partials (paged_attn_workspace_size), required
 *                    when there is more than one partition; the caller then
 *                    runs paged_attn_reduce on the same stream
 * G = 4 runs on VALU dot products, G = 8 on MFMA tiles.
 * Cache policy: when the pool holds no shared block (kv_pool_num_shared is 0),
 * no tile is read twice in a step and the kernels load the tiles with the
 * non-temporal hint; otherwise with the default policy, so that blocks shared
 * by several tables stay cached.  Tables that share blocks the allocator was
 * not told about give the same results, only possibly slower. */
int paged_attn_decode(const pa_kv_pool *pool, const void *q, const int32_t *block_tables,
                      int32_t bt_stride, const int32_t *context_lens, int32_t batch,
                      int32_t num_q_heads, float scale, int32_t max_context_len,
                      int32_t partition_size, void *out, float *partial_out,
                      float *partial_lse, void *stream);

/* Merge split-KV partials into the bf16 output: for each (b, h) with
 * P_b = ceil(ctx_b / partition_size) partitions, weights w_p = exp(lse_p - max
 * lse) and out = sum_p w_p o_p / sum_p w_p; P_b = 0 gives zeros.  A sequence
 * with one partition reproduces the single-pass output bit for bit.
 *   max_partitions   the P dimension of the partial buffers (>= every P_b)
 * Other arguments as in paged_attn_decode. */
int paged_attn_reduce(const float *partial_out, const float *partial_lse,
                      const int32_t *context_lens, int32_t batch, int32_t num_q_heads,
                      int32_t head_dim, int32_t partition_size, int32_t max_partitions,
                      void *out, void *stream);

/* ---------------------------------------------------------------------------
 * Shared-prefix (cascade) decode.
 *
 * Every sequence of a stage pool's batch starts with the same prompt -- the
 * schema that all SQL-generator calls and all fixer retries share (Cortex
 * paper, section 1; section 2 "Cortex Benefits") -- stored once as the same
 * physical blocks in every block table.  The cascade computes attention over
 * that prefix once per KV head for all B*G query rows together, as dense
 * matrix-core tiles, and over each sequence's remaining tokens with the
 * per-sequence kernels; paged_attn_reduce_cascade merges both kinds of
 * partials by log-sum-exp into the same result as paged_attn_decode.  The
 * per-sequence part loads its tiles (the tokens after everything the batch
 * or a group shares) with the non-temporal cache hint, whatever the pool's
 * reference counts; the shared parts keep the default policy.
 * ------------------------------------------------------------------------- */

/* Partial-buffer sizes of a cascade step and the partition count per
 * (sequence, head) (pass it as max_partitions to the reduce).
 *   partition_size         tokens per partition after the prefix: a positive
 *                          multiple of 16
 *   prefix_len             shared prefix tokens: a multiple of 16, 0 allowed,
 *                          at most max_context_len
 *   prefix_partition_size  tokens per prefix partition: a multiple of 16 in
 *                          [16, 1024] */
int paged_attn_cascade_workspace_size(int32_t batch, int32_t num_q_heads, int32_t head_dim,
                                      int32_t max_context_len, int32_t partition_size,
                                      int32_t prefix_len, int32_t prefix_partition_size,
                                      size_t *partial_out_bytes, size_t *partial_lse_bytes,
                                      int32_t *max_partitions_out);

/* First half of a cascade step: writes the (o, lse) partials of the prefix
 * partitions and of the per-sequence partitions after the prefix into
 * partial_out / partial_lse (sizes from paged_attn_cascade_workspace_size).
 * The caller guarantees that entries 0 .. prefix_len/16 - 1 of every block
 * table row are the same physical blocks (paged_attn_check_tables verifies
 * it on host copies); the prefix pass reads them from row 0.  A sequence shorter than prefix_len attends only to its own
 * context.  The prefix pass needs head_dim 128; other arguments as in
 * paged_attn_decode.  Follow with paged_attn_reduce_cascade on the same
 * stream. */
int paged_attn_decode_cascade(const pa_kv_pool *pool, const void *q, const int32_t *block_tables,
                              int32_t bt_stride, const int32_t *context_lens, int32_t batch,
                              int32_t num_q_heads, float scale, int32_t max_context_len,
                              int32_t partition_size, int32_t prefix_len,
                              int32_t prefix_partition_size, float *partial_out,
                              float *partial_lse, void *stream);

/* Second half of a cascade step: merges, for each (b, h), the prefix
 * partials and the ceil((ctx_b - prefix_len) / partition_size) partials after
 * it into the bf16 output.  Arguments as in paged_attn_decode_cascade and
 * paged_attn_reduce. */
int paged_attn_reduce_cascade(const float *partial_out, const float *partial_lse,
                              const int32_t *context_lens, int32_t batch, int32_t num_q_heads,
                              int32_t head_dim, int32_t partition_size, int32_t prefix_len,
                              int32_t prefix_partition_size, int32_t max_partitions, void *out,
                              void *stream);

/* ---------------------------------------------------------------------------
 * Two-level sharing: the prefix, then per group.
 *
 * The retries of one SQL-error-fixer request repeat the request's prompt --
 * the schema and the failed first attempt -- and differ only in their own
 * tail (Cortex paper, section 1 "Motivating Example"; section 2 "Cortex
 * Benefits").  With the first attempt stored once per request as the same
 * physical blocks in its retries' tables, the grouped cascade computes
 * attention over it once per (request, KV head) for all the request's query
 * rows together, as it does for the batch-wide prefix, instead of once per
 * retry.  The result is again the same as paged_attn_decode.
 * ------------------------------------------------------------------------- */

/* Partial sizes of a grouped cascade step: as
 * paged_attn_cascade_workspace_size, plus one partition per sequence for its
 * group's shared tokens.  group_len: a multiple of 16 in [16, 1024] with
 * prefix_len + group_len <= max_context_len. */
int paged_attn_cascade_groups_workspace_size(int32_t batch, int32_t num_q_heads, int32_t head_dim,
                                             int32_t max_context_len, int32_t partition_size,
                                             int32_t prefix_len, int32_t prefix_partition_size,
                                             int32_t group_len, size_t *partial_out_bytes,
                                             size_t *partial_lse_bytes,
                                             int32_t *max_partitions_out);

/* First half of a grouped cascade step.  Besides paged_attn_decode_cascade's
 * arguments:
 *   group_start     device int32 [num_groups + 1], nondecreasing, from 0 to
 *                   batch: group k is sequences group_start[k] ..
 *                   group_start[k+1]-1; every sequence belongs to a group
 *                   (groups of one are fine)
 *   max_group_size  bound on the sequences of a group; max_group_size * G
 *                   <= 64 (G = num_q_heads / num_kv_heads)
 *   group_len       tokens after the prefix that a group's sequences share:
 *                   table entries prefix_len/16 .. (prefix_len+group_len)/16
 *                   - 1 are the same physical blocks for all of a group's
 *                   sequences, and the group's first sequence holds them all
 *                   (a shorter member attends only to its own context)
 *   items, num_items  a work list of the per-sequence partitions after both
 *                   shared parts (paged_attn_schedule with prefix_len +
 *                   group_len), or items NULL: the full grid
 * Group data on the device is clamped into the batch and the bound; a
 * sequence in no group leaves its group partial unwritten.  head_dim 128.
 * Follow with paged_attn_reduce_cascade_groups. */
int paged_attn_decode_cascade_groups(const pa_kv_pool *pool, const void *q,
                                     const int32_t *block_tables, int32_t bt_stride,
                                     const int32_t *context_lens, int32_t batch,
                                     int32_t num_q_heads, float scale, int32_t max_context_len,
                                     int32_t partition_size, int32_t prefix_len,
                                     int32_t prefix_partition_size, const int32_t *group_start,
                                     int32_t num_groups, int32_t max_group_size, int32_t group_len,
                                     const int32_t *items, int32_t num_items, float *partial_out,
                                     float *partial_lse, void *stream);

/* Second half of a grouped cascade step: merges, for each (b, h), the
 * prefix partials, the group partial and the ceil((ctx_b - prefix_len -
 * group_len) / partition_size) partials after them. */
int paged_attn_reduce_cascade_groups(const float *partial_out, const float *partial_lse,
                                     const int32_t *context_lens, int32_t batch,
                                     int32_t num_q_heads, int32_t head_dim, int32_t partition_size,
                                     int32_t prefix_len, int32_t prefix_partition_size,
                                     int32_t group_len, int32_t max_partitions, void *out,
                                     void *stream);

/* Index-trace variant of paged_attn_decode, for verifying block-table and
 * context-length handling.  It runs the same gather code and, in addition,
 * records for every work item (partition p, sequence b, KV head g) the
 * ordered list of KV tiles it loaded as int32 triples (logical block j,
 * physical id as read from the table, valid rows):
 *   trace[((p * batch + b) * num_kv_heads + g) * trace_tiles + i][3]
 * for the i-th tile, trace_tiles = partition_size / 16 (or
 * ceil(max_context_len / 16) without partitions).  Entries past the last
 * tile are left untouched.  trace_capacity is the number of int32 values
 * the buffer holds; PA_EINVAL if it is too small. */
int paged_attn_decode_trace(const pa_kv_pool *pool, const void *q, const int32_t *block_tables,
                            int32_t bt_stride, const int32_t *context_lens, int32_t batch,
                            int32_t num_q_heads, float scale, int32_t max_context_len,
                            int32_t partition_size, void *out, float *partial_out,
                            float *partial_lse, int32_t *trace, int64_t trace_capacity,
                            void *stream);

/* ---------------------------------------------------------------------------
 * Host-built work lists.
 *
 * A serving scheduler knows each sequence's context length on the host.
 * Given them, the library lists only the work items (partition, sequence)
 * that hold tokens, longest first, so the decode grid carries no empty
 * partitions and the longest items do not start last.  The order of work
 * items does not change any result: the scheduled entry points give the same
 * bits as the unscheduled ones.
 * ------------------------------------------------------------------------- */

/* Work list of a decode or cascade step from HOST context lengths.
 *   context_lens     host int32 [batch] (clamped into [0, max_context_len])
 *   max_context_len, partition_size  as the decode call that will use the list
 *                    (0 = one partition)
 *   prefix_len       0 for paged_attn_decode_scheduled; the cascade's
 *                    prefix_len for paged_attn_decode_cascade_scheduled (its
 *                    per-sequence partitions cover the tokens after it)
 *   items            host int32 [capacity]: item = part * batch + b
 *   num_items        receives the number of items (also when capacity is too
 *                    small, which returns PA_EINVAL)
 * Items with no tokens are left out, except in a single-partition decode
 * without a prefix, where every sequence's item writes its output row.
 * Items are ordered by descending token count; ties keep the order of the
 * unscheduled grid (partition-major, or sequence-major when there are 16 or
 * more partitions). */
int paged_attn_schedule(const int32_t *context_lens, int32_t batch, int32_t max_context_len,
                        int32_t partition_size, int32_t prefix_len, int32_t *items,
                        int32_t capacity, int32_t *num_items);

/* paged_attn_decode over a work list (device int32 [num_items], made by
 * paged_attn_schedule from the same context lengths, copied to the device).
 * The list must hold every item with tokens (and, for a single partition,
 * every sequence); ids are clamped into the grid.  num_items in
 * [0, partitions * batch]. */
int paged_attn_decode_scheduled(const pa_kv_pool *pool, const void *q, const int32_t *block_tables,
                                int32_t bt_stride, const int32_t *context_lens, int32_t batch,
                                int32_t num_q_heads, float scale, int32_t max_context_len,
                                int32_t partition_size, const int32_t *items, int32_t num_items,
                                void *out, float *partial_out, float *partial_lse, void *stream);

/* paged_attn_decode_cascade with the per-sequence partitions taken from a
 * work list (paged_attn_schedule with the same prefix_len); the prefix pass
 * is unchanged.  Follow with paged_attn_reduce_cascade. */
int paged_attn_decode_cascade_scheduled(const pa_kv_pool *pool, const void *q,
                                        const int32_t *block_tables, int32_t bt_stride,
                                        const int32_t *context_lens, int32_t batch,
                                        int32_t num_q_heads, float scale, int32_t max_context_len,
                                        int32_t partition_size, int32_t prefix_len,
                                        int32_t prefix_partition_size, const int32_t *items,
                                        int32_t num_items, float *partial_out,
                                        float *partial_lse, void *stream);

/* ---------------------------------------------------------------------------
 * Index traces of the launches that take a shared prefix, groups or a work
 * list, and a host-side check of the sharing they rely on.
 *
 * Block-table and context-length handling must be exact: every tile a
 * launch reads is named by a table entry and bounded by a context length.
 * The trace variants run the same gather code as their production entry
 * points and also record, for every work item, the ordered list of KV tiles
 * it loaded as int32 triples (logical block j, physical id as read from the
 * table, valid rows).  The stage pools share prompt blocks between
 * sequences (Cortex paper, section 1; section 2, "Cortex Benefits"); the
 * cascade reads those shared entries from one row only, so a caller that
 * holds its tables on the host can verify that they really are shared.
 * ------------------------------------------------------------------------- */

/* paged_attn_decode_scheduled with the index trace of paged_attn_decode_trace
 * (same layout: work item (partition p, sequence b, KV head g) at
 * ((p * batch + b) * num_kv_heads + g) * trace_tiles triples). */
int paged_attn_decode_scheduled_trace(const pa_kv_pool *pool, const void *q,
                                      const int32_t *block_tables, int32_t bt_stride,
                                      const int32_t *context_lens, int32_t batch,
                                      int32_t num_q_heads, float scale, int32_t max_context_len,
                                      int32_t partition_size, const int32_t *items,
                                      int32_t num_items, void *out, float *partial_out,
                                      float *partial_lse, int32_t *trace, int64_t trace_capacity,
                                      void *stream);

/* Layout of a cascade step's index trace, in int32 values (three per tile):
 *   layout_out[0], [1]  offset and tiles per item of the prefix partitions:
 *                       partition p, row group r (64 query rows of one KV
 *                       head, r = 0 .. ceil(batch*G/64)-1), KV head g at
 *                       offset + ((p * row_groups + r) * num_kv_heads + g)
 *                       * tiles * 3; slot i is block i of the partition
 *   layout_out[2], [3]  the same for the groups: group k, KV head g at
 *                       offset + (k * num_kv_heads + g) * tiles * 3
 *   layout_out[4], [5]  the per-sequence partitions after the shared tokens:
 *                       (partition p, sequence b, KV head g) at offset +
 *                       ((p * batch + b) * num_kv_heads + g) * tiles * 3
 *   layout_out[6]       total int32 values
 * Arguments as in paged_attn_decode_cascade_groups (group_len 0: no groups). */
int paged_attn_cascade_trace_layout(const pa_kv_pool *pool, int32_t batch, int32_t num_q_heads,
                                    int32_t max_context_len, int32_t partition_size,
                                    int32_t prefix_len, int32_t prefix_partition_size,
                                    int32_t num_groups, int32_t group_len, int64_t layout_out[7]);

/* The cascade decode (plain: group_len 0 and group_start NULL; grouped:
 * group_len > 0; over a work list: items non-NULL, else the full grid) with
 * its index trace in the layout above; entries of items that load no tile
 * are left untouched.  Every shared-span workgroup records the tiles of its
 * span (all of its row groups read the same ones).  trace_capacity: int32
 * values the buffer holds (PA_EINVAL if fewer than layout_out[6]).  Other
 * arguments and the partials as in paged_attn_decode_cascade_groups. */
int paged_attn_decode_cascade_trace(const pa_kv_pool *pool, const void *q,
                                    const int32_t *block_tables, int32_t bt_stride,
                                    const int32_t *context_lens, int32_t batch,
                                    int32_t num_q_heads, float scale, int32_t max_context_len,
                                    int32_t partition_size, int32_t prefix_len,
                                    int32_t prefix_partition_size, const int32_t *group_start,
                                    int32_t num_groups, int32_t max_group_size, int32_t group_len,
                                    const int32_t *items, int32_t num_items, float *partial_out,
                                    float *partial_lse, int32_t *trace, int64_t trace_capacity,
                                    void *stream);

/* Host-side check of block tables before a launch (HOST pointers; nothing
 * runs on the GPU):
 *   - every context length is in [0, 16 * bt_stride] and every entry that
 *     a sequence's own context uses names a block of the pool;
 *   - prefix_len > 0: for every sequence b, the entries the cascade's
 *     prefix pass reads for it through row 0 (blocks 0 .. ceil(min(ctx_b,
 *     prefix_len) / 16) - 1) equal row b's own;
 *   - group_len > 0: group_start [num_groups + 1] runs nondecreasing from 0
 *     to batch, and every member b of group k has the entries the group pass
 *     reads for it through the group's first row (blocks prefix_len/16 ..
 *     ceil(min(ctx_b, prefix_len + group_len) / 16) - 1) in its own row.
 * Returns PA_OK, or PA_EINVAL with a message naming the sequence, entry and
 * values; *bad_seq_out (may be NULL) receives the failing sequence, or -1. */
int paged_attn_check_tables(const pa_kv_pool *pool, const int32_t *block_tables, int32_t bt_stride,
                            const int32_t *context_lens, int32_t batch, int32_t prefix_len,
                            const int32_t *group_start, int32_t num_groups, int32_t group_len,
                            int32_t *bad_seq_out);

/* ---------------------------------------------------------------------------
 * A decode step that allocates nothing.
 *
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.
 * ------------------------------------------------------------------------- */

/* Bytes of the library's own scratch array per GPU (held from the first call
 * on a GPU until the process ends). */
#define PA_NOALLOC_SCRATCH_BYTES (64u << 20)

/* paged_attn_decode followed, when the batch splits, by paged_attn_reduce,
 * with the split-KV partials in the library's scratch array instead of
 * caller buffers: writes out (bf16 [batch][num_q_heads][head_dim]) for every
 * batch, split or not.  Arguments as in paged_attn_decode.  Calls no
 * hipMalloc, hipFree or allocating routine; the array's device address is
 * looked up on the first call on each GPU (the current device).  Returns
 * PA_EINVAL, before any HIP call, when the partials (paged_attn_workspace_size,
 * the lse part 256-byte aligned after the outputs) exceed
 * PA_NOALLOC_SCRATCH_BYTES.  Every call on a GPU uses the same array: calls
 * that overlap on one GPU (other streams, other threads) race; calls in order
 * on one stream do not. */
int paged_attn_decode_noalloc(const pa_kv_pool *pool, const void *q, const int32_t *block_tables,
                              int32_t bt_stride, const int32_t *context_lens, int32_t batch,
                              int32_t num_q_heads, float scale, int32_t max_context_len,
                              int32_t partition_size, void *out, void *stream);

/* ---------------------------------------------------------------------------
 * KV append.
 *
 * Every decode step adds the key and value rows of the token it produced to
 * the sequence's resident context before the step's attention reads it (the
 * paper keeps a stage's context in its engines' cache across calls: section
 * 2, "Cortex Benefits"; section 3, "Agentic State").
 * ------------------------------------------------------------------------- */

/* Write the new token's K and V rows: for every sequence b with
 * n = context_lens[b] >= 1 and every KV head g,
 *     K pool[block_tables[b][(n-1) / 16]][g][(n-1) % 16][:] = k_new[b][g][:]
 * and likewise for V.  Sequences with n = 0 append nothing; nothing else in
 * the pools changes.
 *   pool          geometry and the K/V device pools (written)
 *   k_new, v_new  device bf16 [batch][num_kv_heads][head_dim], 16-byte aligned
 *   block_tables  device int32 [batch][bt_stride]; entry (n-1)/16 of row b
 *                 must be a block that belongs to sequence b alone: allocate
 *                 one (kv_pool_alloc) whenever n-1 is a multiple of 16, and
 *                 copy a shared block before writing into it
 *   context_lens  device int32 [batch]: lengths including the new token
 *   batch         >= 0 (0 is a no-op)
 * Device data is clamped like the decode's: lengths into [0, 16*bt_stride],
 * ids into [0, num_blocks), so bad data writes a wrong slot inside the pool,
 * never outside it.  Run the step's decode after this call on the same
 * stream. */
int paged_attn_append_kv(const pa_kv_pool *pool, const void *k_new, const void *v_new,
                         const int32_t *block_tables, int32_t bt_stride,
                         const int32_t *context_lens, int32_t batch, void *stream);

/* Append and decode in one launch: the same pools, outputs and partials as
 * paged_attn_append_kv followed by paged_attn_decode (items = NULL) or
 * paged_attn_decode_scheduled (a work list from paged_attn_schedule), bit
 * for bit, with one kernel launch less per decode step.  The work item that
 * holds token n-1 of sequence b (n = context_lens[b] >= 1, clamped into
 * [0, max_context_len] like the decode's lengths) uses k_new[b] / v_new[b]
 * for that token whatever the pool slot holds, and writes them into the slot
 * for later steps.  The slot's block must belong to sequence b alone, as for
 * paged_attn_append_kv.
 *   k_new, v_new  device bf16 [batch][num_kv_heads][head_dim], 16-byte aligned
 * Other arguments as in paged_attn_decode_scheduled. */
int paged_attn_decode_append(const pa_kv_pool *pool, const void *q, const void *k_new,
                             const void *v_new, const int32_t *block_tables, int32_t bt_stride,
                             const int32_t *context_lens, int32_t batch, int32_t num_q_heads,
                             float scale, int32_t max_context_len, int32_t partition_size,
                             const int32_t *items, int32_t num_items, void *out,
                             float *partial_out, float *partial_lse, void *stream);

/* The same for a cascade step: paged_attn_append_kv followed by
 * paged_attn_decode_cascade_groups (group_len > 0), or by
 * paged_attn_decode_cascade / _scheduled (group_len 0: group_start and
 * num_groups are ignored); items may be NULL.  The new token must come after
 * everything the batch or its group shares (n - 1 >= prefix_len + group_len):
 * its row is appended by the per-sequence part of the launch only.  Follow
 * with the matching paged_attn_reduce_cascade* call on the same stream. */
int paged_attn_decode_cascade_append(const pa_kv_pool *pool, const void *q, const void *k_new,
                                     const void *v_new, const int32_t *block_tables,
                                     int32_t bt_stride, const int32_t *context_lens, int32_t batch,
                                     int32_t num_q_heads, float scale, int32_t max_context_len,
                                     int32_t partition_size, int32_t prefix_len,
                                     int32_t prefix_partition_size, const int32_t *group_start,
                                     int32_t num_groups, int32_t max_group_size, int32_t group_len,
                                     const int32_t *items, int32_t num_items, float *partial_out,
                                     float *partial_lse, void *stream);

/* ---------------------------------------------------------------------------
 * Extend (chunked prefill) attention.
 *
 * A retry of the SQL error fixer sends new prompt tokens that attend to the
 * stage's resident context (the shared schema prompt and the first attempt)
 * and, causally, to each other (Cortex paper, section 1, motivating example;
 * section 2, "Cortex Benefits").  With the chunk's K/V already appended to
 * the paged cache, token i of sequence b's chunk sits at position
 * p = n_b - L_b + i and attends to tokens 0 .. p:
 *
 *     out[q_start[b] + i][h] = sum_{t <= p} softmax_t(scale * <q[q_start[b] + i][h], K_g[t]>) V_g[t]
 * ------------------------------------------------------------------------- */

/* Causal attention of each sequence's chunk of new tokens over its paged
 * context, on matrix-core tiles.
 *   pool             geometry and K/V device pools; head_dim must be 128
 *   q                device bf16 [total_q][num_q_heads][128], 16-byte
 *                    aligned; chunk b is rows q_start[b] .. q_start[b+1]-1
 *   q_start          device int32 [batch + 1], nondecreasing, q_start[0] = 0,
 *                    q_start[batch] = total_q
 *   total_q          rows of q and out
 *   block_tables     as in paged_attn_decode, covering each context_lens[b]
 *   context_lens     device int32 [batch]: n_b, the chunk included
 *                    (L_b = q_start[b+1] - q_start[b] <= n_b)
 *   num_q_heads      G = num_q_heads / num_kv_heads must be 4 or 8
 *   max_context_len  host bound of context_lens, at most 8192
 *                    (PA_EUNSUPPORTED above); sizes the stream
 *   max_chunk        host bound of the chunk lengths; sizes the grid
 *   out              device bf16 [total_q][num_q_heads][128], 16-byte aligned
 * Device data is clamped into the buffers' bounds (chunk lengths into
 * [0, min(n_b, max_chunk)] and rows into [0, total_q)), so bad data gives
 * unspecified values, never an out-of-bounds access. */
int paged_attn_extend(const pa_kv_pool *pool, const void *q, const int32_t *q_start,
                      int32_t total_q, const int32_t *block_tables, int32_t bt_stride,
                      const int32_t *context_lens, int32_t batch, int32_t num_q_heads,
                      float scale, int32_t max_context_len, int32_t max_chunk, void *out,
                      void *stream);

/* ---------------------------------------------------------------------------
 * Measurement helpers.
 * ------------------------------------------------------------------------- */

/* Plain device-to-device copy of `bytes` (a multiple of 16; both pointers
 * 16-byte aligned) with a streaming kernel; used to calibrate hardware
 * traffic counters and the achievable HBM bandwidth. */
int pa_stream_copy(const void *src, void *dst, size_t bytes, void *stream);

/* Data-movement reference for a decode: reads the K and V tiles of num_spans
 * token spans for every KV head of the pool, with no arithmetic, in the
 * grid a decode launch uses (one workgroup of four wavefronts per (span,
 * KV head), the head fastest, the span's 16-token blocks dealt round-robin
 * to the wavefronts, tiles_in_flight tiles of K and V in flight per
 * wavefront: 2 suits short spans, 4 long ones), each tile read once, whole
 * token rows per load instruction, with the streaming (non-temporal) cache
 * hint, as the decode kernels read tiles that a step reads once.  The
 * time of one call over the tiles that a decode step reads is what that
 * access pattern costs on the memory system alone, the reference for the
 * decode kernels' own time.  Like pa_stream_copy it is a measurement helper
 * and computes nothing of the method.
 *   block_tables  device int32 [batch][bt_stride]
 *   spans         device int32 [num_spans][3]: sequence b, first token,
 *                 end token; tokens [first, end) of sequence b are read
 *                 through table row b (first rounded down to a block)
 *   sink          device uint32 [num_spans][num_kv_heads][4]: entry
 *                 [s][g][w] = XOR of every 32-bit word of the K and V tiles
 *                 that wavefront w read (blocks w, w+4, ... of the span),
 *                 so the result can be checked exactly on the host
 * Device data is clamped into the buffers (sequence into [0, batch), tokens
 * into [0, 16*bt_stride], ids into [0, num_blocks)): bad data reads other
 * tiles, never out of bounds.  num_spans = 0 is a no-op.  tiles_in_flight
 * other than 2 or 4 is PA_EINVAL. */
int pa_gather_tiles(const pa_kv_pool *pool, const int32_t *block_tables, int32_t bt_stride,
                    int32_t batch, const int32_t *spans, int32_t num_spans,
                    int32_t tiles_in_flight, uint32_t *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PAGED_ATTN_H */
